"""Seeded synthetic inputs for the T-LoopFormer decode/prefill path.

This module is shared by the CPU oracle and the HIP path.  It holds only
input generation (random numbers, storage-dtype rounding, model-shape
presets); none of the method's arithmetic lives here.

Generators (both published methods):
  * SplitMix64 (S. Vigna, public-domain reference ``splitmix64.c``), used in
    counter mode: element ``n`` of stream ``(seed, stream_id)`` is
    ``mix64(key + (n + 1) * 0x9E3779B97F4A7C15)`` with
    ``key = mix64(seed * 0x9E3779B97F4A7C15 ^ stream_id)``.  An element's
    value therefore depends only on its flat index, so any prefix of a tensor
    (e.g. the first rows of the position table) is the same whatever the
    tensor's full size.
  * Box-Muller (1958) for normals: ``n = sqrt(-2 ln u1) * cos(2 pi u2)``,
    with ``u1, u2`` drawn from two consecutive counters.

The paper trains its model on FineWeb-Edu; trained weights and the dataset
are not available, so seeded N(0, 0.02) weights and uniform-random prompts
of the same shapes stand in for them.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import math
import os
from typing import Dict, List, Optional

import numpy as np

SEED = 2609

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# Stream ids: one per tensor so tensors never share random numbers.
STREAM_TOK_EMB = 1
STREAM_POS_EMB = 2
STREAM_ROUTER_W = 3
STREAM_LM_HEAD = 4      # optional untied LM head
STREAM_ROUTER_W1 = 5    # hidden layer of the MLP router
STREAM_LAYER_BASE = 16  # layer j uses 16 + 4j + {0: qkv, 1: o, 2: gate_up, 3: down}
STREAM_COND_BASE = 200  # AdaLN: 200-203 time embedder (w1, b1, w2, b2), 204-207 step embedder,
                        # 210 + 2j / 211 + 2j layer j's modulator weight / bias
FOURIER_DIM = 256       # width of the fixed Fourier features of a conditioning scalar
STREAM_PROMPT = 100
STREAM_CALIB = 101


def _threads() -> int:
    try:
        n = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        n = 0
    return max(1, min(16, n if n > 0 else (os.cpu_count() or 1)))


def _mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function (in place on a fresh uint64 array)."""
    t = np.empty_like(z)
    with np.errstate(over="ignore"):
        np.right_shift(z, np.uint64(30), out=t)
        np.bitwise_xor(z, t, out=z)
        np.multiply(z, _M1, out=z)
        np.right_shift(z, np.uint64(27), out=t)
        np.bitwise_xor(z, t, out=z)
        np.multiply(z, _M2, out=z)
        np.right_shift(z, np.uint64(31), out=t)
        np.bitwise_xor(z, t, out=z)
    return z


def _stream_key(seed: int, stream: int) -> np.uint64:
    with np.errstate(over="ignore"):
        k = np.array([np.uint64(seed) * _GOLDEN ^ np.uint64(stream)], dtype=np.uint64)
    return _mix64(k)[0]


def splitmix64(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Raw 64-bit outputs ``start .. start+count-1`` of stream ``(seed, stream)``."""
    key = _stream_key(seed, stream)
    n = np.arange(start + 1, start + count + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        np.multiply(n, _GOLDEN, out=n)
        np.add(n, key, out=n)
    return _mix64(n)


def uniform01(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Uniforms in (0, 1): top 53 bits of each output, offset by half a step."""
    u = splitmix64(seed, stream, start, count) >> np.uint64(11)
    return (u.astype(np.float64) + 0.5) * (1.0 / 9007199254740992.0)


def normal(seed: int, stream: int, count: int, std: float = 1.0,
           chunk: int = 1 << 22) -> np.ndarray:
    """``count`` N(0, std^2) draws (float64); element n uses counters 2n, 2n+1."""
    out = np.empty(count, dtype=np.float64)

    def fill(s: int) -> None:
        c = min(chunk, count - s)
        u = uniform01(seed, stream, 2 * s, 2 * c)
        u1, u2 = u[0::2], u[1::2]
        out[s:s + c] = np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2) * std

    starts = range(0, count, chunk)
    if count > chunk:
        # numpy ufuncs release the GIL, so chunks fill in parallel; each chunk's
        # values depend only on its counters, so the result is thread-count independent
        with concurrent.futures.ThreadPoolExecutor(max_workers=_threads()) as ex:
            list(ex.map(fill, starts))
    else:
        for s in starts:
            fill(s)
    return out


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even); returns float32 values."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    b = f.view(np.uint32)
    # finite inputs cannot overflow: bits + 0x8000 <= 0xFF807FFF
    r = (b >> np.uint32(16)) & np.uint32(1)
    r += b
    r += np.uint32(0x7FFF)
    r &= np.uint32(0xFFFF0000)
    out = r.view(np.float32)
    nan = np.isnan(f)
    if nan.any():
        out = out.copy()
        out[nan] = np.nan
    return out.reshape(np.shape(x))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are already bf16-representable."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float values once to the storage dtype (returned as float32)."""
    if dtype == "bf16":
        return round_to_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    raise ValueError(f"unknown storage dtype {dtype!r}")


# ---------------------------------------------------------------------------
# Model and workload presets
# ---------------------------------------------------------------------------

# Target routed-depth distribution for the calibrated router bias: long-tailed,
# mean 3.71, with most tokens at depth <= 4, standing in for the paper's
# reported depth mix on FineWeb-Edu (mean 3.69, Figure 1b and Section 4.1).
DEPTH_TARGET_R8 = (0.13, 0.17, 0.20, 0.19, 0.12, 0.09, 0.06, 0.04)


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    dtype: str            # storage dtype of weights / KV cache: "f32" or "bf16"
    vocab: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int             # SwiGLU hidden width
    n_layers: int         # J, layers in the shared block
    max_loops: int        # R = M, router width and loop cap
    batch: int
    prompt_len: int
    steps: int            # decode steps (0 for a prefill-only workload)
    router_bias: str      # "zero" or "calibrated"
    page_tokens: int = 16
    rms_eps: float = 1e-5
    std: float = 0.02
    router_hidden: int = 0  # 0: linear router; else the hidden width of a 2-layer MLP router
    adaln: bool = False     # AdaLN time/step conditioning weights

    @property
    def max_pos(self) -> int:
        return self.prompt_len + self.steps

    def replace(self, **kw) -> "ModelConfig":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, ModelConfig] = {
    # Tiny fp32 model: one-layer shared block, batch 1, 32-token prompt.
    "f32_tiny_b1x32": ModelConfig("f32_tiny_b1x32", "f32", vocab=512, d_model=64, n_heads=4, head_dim=16,
                      d_ff=256, n_layers=1, max_loops=4, batch=1, prompt_len=32,
                      steps=32, router_bias="zero"),
    # 2-layer shared block, d=768, bf16, batch 32 x 512 prompt, 256 steps.
    "bf16_d768_b32x512": ModelConfig("bf16_d768_b32x512", "bf16", vocab=32000, d_model=768, n_heads=12, head_dim=64,
                      d_ff=2048, n_layers=2, max_loops=8, batch=32, prompt_len=512,
                      steps=256, router_bias="calibrated"),
    # Same model, cache-bound regime: batch 256 x 2048 prompt, 128 steps.
    "bf16_d768_b256x2048": ModelConfig("bf16_d768_b256x2048", "bf16", vocab=32000, d_model=768, n_heads=12, head_dim=64,
                      d_ff=2048, n_layers=2, max_loops=8, batch=256, prompt_len=2048,
                      steps=128, router_bias="calibrated"),
    # Larger model: d=2048, 16 heads x 128, batch 64 x 4096 prompt, 128 steps.
    "bf16_d2048_b64x4096": ModelConfig("bf16_d2048_b64x4096", "bf16", vocab=32000, d_model=2048, n_heads=16, head_dim=128,
                      d_ff=5504, n_layers=2, max_loops=8, batch=64, prompt_len=4096,
                      steps=128, router_bias="calibrated"),
    # Prefill-only: d=1024, 16 x 64, batch 8 x 4096.
    "bf16_d1024_prefill_b8x4096": ModelConfig("bf16_d1024_prefill_b8x4096", "bf16", vocab=32000, d_model=1024, n_heads=16, head_dim=64,
                      d_ff=2816, n_layers=2, max_loops=8, batch=8, prompt_len=4096,
                      steps=0, router_bias="calibrated"),
}


def _mat(seed: int, stream: int, rows: int, cols: int, cfg: ModelConfig) -> np.ndarray:
    return to_storage(normal(seed, stream, rows * cols, cfg.std).reshape(rows, cols), cfg.dtype)


# Moments of x * sigmoid(x) for x ~ N(0, 1) (numerical quadrature), used to
# model the MLP router's hidden units as i.i.d. with this mean and variance.
SILU_GAUSS_MEAN = 0.2066209641
SILU_GAUSS_VAR = 0.3130832970


def _fit_bias(mean: np.ndarray, cov: np.ndarray, seed: int, target, samples: int,
              tol: float, max_iter: int) -> np.ndarray:
    """Bias b such that argmax(z + b), z ~ N(mean, cov), has the target histogram
    (Monte Carlo on stream STREAM_CALIB, update b <- b + 0.5 sigma (log q - log p_hat),
    b[0] held at 0)."""
    R = cov.shape[0]
    if len(target) != R:
        raise ValueError("depth target length must equal max_loops")
    L = np.linalg.cholesky(cov + 1e-18 * np.eye(R))
    g = normal(seed, STREAM_CALIB, samples * R).reshape(samples, R)
    z0 = g @ L.T + mean
    sigma = float(np.sqrt(np.mean(np.diag(cov))))
    q = np.asarray(target, dtype=np.float64)
    b = np.zeros(R)
    for _ in range(max_iter):
        hist = np.bincount(np.argmax(z0 + b, axis=1), minlength=R) / samples
        if np.max(np.abs(hist - q)) < tol:
            break
        b = b + 0.5 * sigma * (np.log(q) - np.log(np.maximum(hist, 1.0 / samples)))
        b = b - b[0]
    return b.astype(np.float32)


def calibrate_router_bias(router_w: np.ndarray, cfg: ModelConfig, seed: int = SEED,
                          target=DEPTH_TARGET_R8, samples: int = 1 << 20,
                          tol: float = 2e-3, max_iter: int = 200) -> np.ndarray:
    """Router bias that gives the target depth histogram under a Gaussian input model.

    Linear router: the embedding rows are i.i.d. N(0, std^2), so the router's input
    ``E[x] + P[t]`` has i.i.d. N(0, 2 std^2) elements and the bias-free router
    outputs are jointly Gaussian with covariance ``2 std^2 W W^T``.  MLP router
    (``router_w`` is then the output layer [R][Hr]): its hidden units are modelled
    as i.i.d. with the moments of x * sigmoid(x), x ~ N(0, 1) (the hidden layer is
    scaled so that its pre-activations have unit variance), so the outputs have
    mean ``SILU_GAUSS_MEAN * W 1`` and covariance ``SILU_GAUSS_VAR * W W^T``.
    The realised histogram on the actual tables is measured, not promised.
    """
    w = router_w.astype(np.float64)
    if cfg.router_hidden > 0:
        mean = SILU_GAUSS_MEAN * w.sum(axis=1)
        cov = SILU_GAUSS_VAR * (w @ w.T)
    else:
        mean = np.zeros(w.shape[0])
        cov = 2.0 * cfg.std ** 2 * (w @ w.T)
    return _fit_bias(mean, cov, seed, target, samples, tol, max_iter)


_WEIGHT_CACHE: Dict[tuple, Dict] = {}


def make_weights(cfg: ModelConfig, seed: int = SEED, cache: bool = True) -> Dict:
    """Seeded weights, rounded once to the storage dtype (float32 arrays).

    Layouts (row-major, ``[out][in]`` like a linear layer's weight):
      tok_emb [V][d], pos_emb [max_pos][d], router_w [R][d] (fp32; bf16-rounded
      values for bf16 models), router_b [R] fp32, and per layer j:
      (with router_hidden = Hr > 0: router_w1 [Hr][d] storage dtype, router_b1 [Hr]
      fp32, and router_w [R][Hr] is the output layer)
      w_qkv [3d][d] (rows q | k | v, head-major within each), w_o [d][d],
      w_gate_up [2F][d] (rows gate | up), w_down [d][F].
      With adaln: "cond" = {time_w1 [d][256], time_b1 [d], time_w2 [d][d],
      time_b2 [d], and the same for step_*}, and per layer w_mod [4d][d]
      (rows alpha_msa | alpha_mlp | gamma_msa | gamma_mlp), b_mod [4d]; matrices
      in the storage dtype, biases fp32.  Scales: unit-variance hidden
      pre-activations in the embedders, modulation entries of roughly 0.2.
    """
    key = (cfg, seed)
    if cache and key in _WEIGHT_CACHE:
        return _WEIGHT_CACHE[key]
    d, F, V, R = cfg.d_model, cfg.d_ff, cfg.vocab, cfg.max_loops
    if cfg.n_heads * cfg.head_dim != d:
        raise ValueError("n_heads * head_dim must equal d_model")
    w: Dict = {
        "tok_emb": _mat(seed, STREAM_TOK_EMB, V, d, cfg),
        "pos_emb": _mat(seed, STREAM_POS_EMB, cfg.max_pos, d, cfg),
    }
    Hr = cfg.router_hidden
    if Hr > 0:
        # hidden layer scaled for unit-variance pre-activations on inputs with
        # i.i.d. N(0, 2 std^2) elements; output layer with std 2 / sqrt(Hr)
        w["router_w1"] = to_storage(normal(seed, STREAM_ROUTER_W1, Hr * d,
                                           1.0 / (np.sqrt(2.0 * d) * cfg.std)).reshape(Hr, d), cfg.dtype)
        w["router_b1"] = np.zeros(Hr, dtype=np.float32)
        w["router_w"] = to_storage(normal(seed, STREAM_ROUTER_W, R * Hr, 2.0 / np.sqrt(Hr)).reshape(R, Hr),
                                   cfg.dtype).astype(np.float32)
    else:
        w["router_w"] = _mat(seed, STREAM_ROUTER_W, R, d, cfg).astype(np.float32)
    layers: List[Dict[str, np.ndarray]] = []
    for j in range(cfg.n_layers):
        s = STREAM_LAYER_BASE + 4 * j
        layers.append({
            "w_qkv": _mat(seed, s + 0, 3 * d, d, cfg),
            "w_o": _mat(seed, s + 1, d, d, cfg),
            "w_gate_up": _mat(seed, s + 2, 2 * F, d, cfg),
            "w_down": _mat(seed, s + 3, d, F, cfg),
        })
    w["layers"] = layers
    if cfg.adaln:
        c = STREAM_COND_BASE
        cond = {}
        for k, name in enumerate(("time", "step")):
            base = c + 4 * k
            cond[name + "_w1"] = to_storage(normal(seed, base + 0, d * FOURIER_DIM, 1.0 / np.sqrt(FOURIER_DIM / 2))
                                            .reshape(d, FOURIER_DIM), cfg.dtype)
            cond[name + "_b1"] = normal(seed, base + 1, d, 0.1).astype(np.float32)
            cond[name + "_w2"] = to_storage(normal(seed, base + 2, d * d, 1.0 / np.sqrt(d)).reshape(d, d), cfg.dtype)
            cond[name + "_b2"] = normal(seed, base + 3, d, 0.1).astype(np.float32)
        w["cond"] = cond
        for j, lw in enumerate(layers):
            lw["w_mod"] = to_storage(normal(seed, c + 10 + 2 * j, 4 * d * d, 0.5 / np.sqrt(d)).reshape(4 * d, d),
                                     cfg.dtype)
            lw["b_mod"] = normal(seed, c + 11 + 2 * j, 4 * d, 0.05).astype(np.float32)
    if cfg.router_bias == "zero":
        w["router_b"] = np.zeros(R, dtype=np.float32)
    elif cfg.router_bias == "calibrated":
        target = DEPTH_TARGET_R8 if R == 8 else tuple([1.0 / R] * R)
        w["router_b"] = calibrate_router_bias(w["router_w"], cfg, seed, target)
    else:
        raise ValueError(f"unknown router_bias {cfg.router_bias!r}")
    if cache:
        _WEIGHT_CACHE[key] = w
    return w


def make_lm_head(cfg: ModelConfig, seed: int = SEED) -> np.ndarray:
    """A separate seeded LM head [V][d] (storage dtype), for models whose head
    is not tied to the token embedding."""
    return _mat(seed, STREAM_LM_HEAD, cfg.vocab, cfg.d_model, cfg)


def make_prompts(cfg: ModelConfig, seed: int = SEED, batch: Optional[int] = None,
                 prompt_len: Optional[int] = None) -> np.ndarray:
    """Uniform-random token ids in [0, V), shape [B][T] (int32).

    Row b depends only on (seed, b, T), so a subset of sequences of a large batch
    can be regenerated on its own.
    """
    B = cfg.batch if batch is None else batch
    T = cfg.prompt_len if prompt_len is None else prompt_len
    u = uniform01(seed, STREAM_PROMPT, 0, B * T).reshape(B, T)
    return np.minimum((u * cfg.vocab).astype(np.int64), cfg.vocab - 1).astype(np.int32)


def tiny_config(**kw) -> ModelConfig:
    """A small model for fast CPU tests (defaults: d=32, 2 heads, J=2, R=4)."""
    base = dict(name="tiny", dtype="f32", vocab=97, d_model=32, n_heads=2, head_dim=16,
                d_ff=48, n_layers=2, max_loops=4, batch=2, prompt_len=12, steps=6,
                router_bias="zero")
    base.update(kw)
    return ModelConfig(**base)


STREAM_TRAIN_DEPTH = 102
STREAM_TRAIN_STATE = 103

# Depth mix of the routed decode workload (batch 256 x 2048, argmax router):
# share of tokens at depth 1..8, used as the depth law of the synthetic
# training batches of the gather-scatter operators.
TRAIN_DEPTH_MIX = (0.1315, 0.1791, 0.2033, 0.1950, 0.1180, 0.0901, 0.0638, 0.0192)


def make_train_depths(rows: int, loops: int = 8, seed: int = SEED, mix=TRAIN_DEPTH_MIX) -> np.ndarray:
    """int32 depths in [1, loops] for `rows` tokens, drawn from `mix` (its
    first `loops` entries, renormalised) by inverting the cumulative shares."""
    p = np.asarray(mix[:loops], np.float64)
    cdf = np.cumsum(p / p.sum())
    u = uniform01(seed, STREAM_TRAIN_DEPTH, 0, rows)
    return (np.minimum(np.searchsorted(cdf, u, side="right"), loops - 1) + 1).astype(np.int32)


def make_train_states(rows: int, d: int, seed: int = SEED, stream: int = STREAM_TRAIN_STATE) -> np.ndarray:
    """float32 [rows, d] standard-normal hidden states."""
    return normal(seed, stream, rows * d).reshape(rows, d).astype(np.float32)
