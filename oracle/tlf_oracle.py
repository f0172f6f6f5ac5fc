"""CPU oracle for T-LoopFormer's routed prefill and decode.  TEST INFRASTRUCTURE.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this module.  It shares no code with the HIP library: it reads the
same seeded inputs (``synth``) and nothing else.

Everything is plain numpy in float64.  Weights are the stored values (fp32,
or bf16 values widened) converted to float64; activations, the cache and all
sums are float64.  The only place where floating point decides an integer is
the router: its logits are rounded to float32 (the kernel's precision) before
the depth rule is applied, and the greedy token is the argmax of the float32
rounding of the logits.

Model (T-LoopFormer, Section 3 and Appendix A):
  * h0 = E[x] + P[pos]: token plus learned absolute position embedding, added
    once (Section 3, Section 3.2 definition of h^(0)).
  * One shared block of J pre-norm layers re-applied for every loop:
    x += Attn(RMSNorm(x)) W_o ; x += SwiGLU(RMSNorm(x)).  RMSNorm has no
    learned affine (Appendix A).  The FFN is SwiGLU (the workloads' choice;
    the paper's own model uses a GELU MLP).  No biases, no AdaLN conditioning
    (gamma = 0, unit gate) unless the weights carry it (below), attention
    scale 1/sqrt(D), tied LM head.
  * Optional AdaLN time/step conditioning (Section 3.1, Appendix A): a token
    of depth m at loop i has cumulative time (i - 1) / m and step 1 / m (its
    uniform trajectory, summing to 1 over its m loops); each scalar goes
    through fixed Fourier features (256 wide, max period 10000) and its own
    2-layer SiLU MLP, the two embeddings are summed, and layer j's modulator
    (SiLU, then a linear map to 4d) gives (alpha_msa, alpha_mlp, gamma_msa,
    gamma_mlp): x += (1 + alpha) * F(RMSNorm(x) * (1 + gamma)) for the
    attention and FFN branches (the gate read as 1 + alpha, so that zero
    modulator weights give the unconditioned block).
  * Router: linear map of h0 to R logits (Eq. 2's f_theta); the depth rule is
    argmax (the workloads), the cumulative-probability threshold of Eq. 3-5,
    or a fixed depth.
  * Loop i runs the block on the active set A_i = {t : m_t >= i} only, gathered
    in position order (Eq. 6) and scattered back (Eq. 7); exited tokens keep
    h^(m_t).
  * Recursion-wise KV cache: one cache per (loop i, layer j) (Eq. 8).  A token
    executing loop i writes its k, v there (Eq. 11) and attends to the entries
    of that cache only (Eq. 10): the earlier tokens whose depth is >= i, plus
    itself (the inclusive reading of Eq. 10).

Two cache representations are implemented and must agree:
  * "compact": per (loop, layer) a list of (position, k, v) in position order,
    holding only tokens that executed the loop.
  * "literal": per (loop, layer) a dense array indexed by position, zero for
    tokens that never executed the loop, read with the validity mask
    mu^(i)_t' = [m_t' >= i] (Eq. 10, Appendix B).  ``use_mask=False`` drops
    the mask to show it is required.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

ARGMAX = "argmax"
CUMPROB = "cumprob"
FIXED = "fixed"


def _identity(x: np.ndarray) -> np.ndarray:
    return x


def _round_bf16(x: np.ndarray) -> np.ndarray:
    """bf16 round-to-nearest-even of float64 values via their float32 rounding."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64).reshape(np.shape(x))


class Model:
    """Float64 copy of the model weights plus the routing settings.

    ``weights`` is the dict from ``synth.make_weights``: tok_emb [V][d],
    pos_emb [P][d], router_w [R][d], router_b [R], and per layer w_qkv [3d][d],
    w_o [d][d], w_gate_up [2F][d], w_down [d][F] (linear-layer [out][in] layout,
    so a projection is ``y @ W.T``).  An optional ``lm_head`` [V][d] replaces
    the head tied to the token embedding (the tied head is the default).

    ``round_bf16=True`` rounds q, k, v, the normalised GEMM inputs, the
    attention output and the SwiGLU activation to bf16, which are the points
    where a bf16 implementation stores them.  It is off by default.
    """

    def __init__(self, weights: Dict, n_heads: int, head_dim: int,
                 route_rule: str = ARGMAX, threshold: float = 0.5,
                 fixed_depth: Optional[int] = None, rms_eps: float = 1e-5,
                 round_bf16: bool = False):
        f64 = lambda a: np.asarray(a, dtype=np.float64)
        self.E = f64(weights["tok_emb"])
        self.P = f64(weights["pos_emb"])
        self.Wr = f64(weights["router_w"])
        self.br = f64(weights["router_b"])
        # optional hidden layer of a 2-layer MLP router (Section 3.2)
        self.Wr1 = f64(weights["router_w1"]) if weights.get("router_w1") is not None else None
        self.br1 = f64(weights["router_b1"]) if self.Wr1 is not None else None
        self.V, self.d = self.E.shape
        head = weights.get("lm_head")
        self.head = self.E if head is None else f64(head)
        self.R = self.Wr.shape[0]
        self.H, self.D = n_heads, head_dim
        if self.H * self.D != self.d:
            raise ValueError("n_heads * head_dim must equal d_model")
        self.layers = []
        for lw in weights["layers"]:
            qkv = f64(lw["w_qkv"])
            gu = f64(lw["w_gate_up"])
            F = gu.shape[0] // 2
            self.layers.append(dict(
                Wq=qkv[0:self.d], Wk=qkv[self.d:2 * self.d], Wv=qkv[2 * self.d:3 * self.d],
                Wo=f64(lw["w_o"]), Wg=gu[0:F], Wu=gu[F:2 * F], Wd=f64(lw["w_down"])))
            if weights.get("cond") is not None:
                self.layers[-1].update(Wmod=f64(lw["w_mod"]), bmod=f64(lw["b_mod"]))
        self.J = len(self.layers)
        # AdaLN conditioning: time and step embedders (Appendix A)
        cond = weights.get("cond")
        self.cond = None if cond is None else {k: f64(v) for k, v in cond.items()}
        self._mods: Dict[Tuple[int, int, int], Tuple[np.ndarray, ...]] = {}
        self.route_rule = route_rule
        self.threshold = float(threshold)
        self.fixed_depth = fixed_depth
        self.eps = float(rms_eps)
        self.st = _round_bf16 if round_bf16 else _identity
        if route_rule == FIXED and not (fixed_depth and 1 <= fixed_depth <= self.R):
            raise ValueError("fixed depth must be in [1, R]")
        if route_rule == CUMPROB and not (0.0 < self.threshold < 1.0):
            raise ValueError("threshold must be in (0, 1)")


# ---------------------------------------------------------------------------
# Elementary pieces
# ---------------------------------------------------------------------------

def rms_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm without learned affine (Appendix A): x / sqrt(mean(x^2) + eps)."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax; entries equal to -inf get weight 0."""
    mx = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - mx)
    return e / np.sum(e, axis=-1, keepdims=True)


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """Multi-head scaled dot-product attention.

    q [n][H][D], k/v [m][H][D], allowed [n][m] bool: query a may attend key b.
    Returns [n][H][D]: for each head softmax(q k^T / sqrt(D)) v over allowed keys.
    """
    n, H, D = q.shape
    out = np.empty_like(q)
    scale = 1.0 / math.sqrt(D)
    for h in range(H):
        s = (q[:, h, :] @ k[:, h, :].T) * scale
        s = np.where(allowed, s, -np.inf)
        out[:, h, :] = softmax_rows(s) @ v[:, h, :]
    return out


# ---------------------------------------------------------------------------
# AdaLN time/step conditioning (Section 3.1, Appendix A)
# ---------------------------------------------------------------------------

FOURIER_DIM = 256           # D_f
FOURIER_MAX_PERIOD = 10000.0


def fourier_features(tau: float) -> np.ndarray:
    """[cos(tau w_1), sin(tau w_1), ..., cos(tau w_K), sin(tau w_K)] with
    K = D_f / 2 and w_k = exp(-(k - 1) / K * ln 10000)."""
    K = FOURIER_DIM // 2
    w = np.exp(-np.arange(K, dtype=np.float64) / K * math.log(FOURIER_MAX_PERIOD))
    out = np.empty(FOURIER_DIM)
    out[0::2] = np.cos(tau * w)
    out[1::2] = np.sin(tau * w)
    return out


def trajectory(i: int, m: int) -> Tuple[float, float]:
    """(cumulative time c_{i-1}, step Delta_i) of a token of depth m at loop i
    (1-based) on its uniform trajectory: Delta = 1 / m, c_{i-1} = (i - 1) / m."""
    return (i - 1) / m, 1.0 / m


def scalar_embedding(model: Model, which: str, tau: float) -> np.ndarray:
    """phi(tau) = W_2 silu(W_1 fourier(tau) + b_1) + b_2 for the "time" or "step" embedder."""
    c = model.cond
    h = silu(c[which + "_w1"] @ fourier_features(tau) + c[which + "_b1"])
    return c[which + "_w2"] @ h + c[which + "_b2"]


def modulation(model: Model, j: int, i: int, m: int) -> Tuple[np.ndarray, ...]:
    """(alpha_msa, alpha_mlp, gamma_msa, gamma_mlp) of layer j for a token of
    depth m at loop i: the modulator silu -> linear (4d) of e_t + e_Delta."""
    key = (j, i, m)
    if key not in model._mods:
        t, dt = trajectory(i, m)
        e = scalar_embedding(model, "time", t) + scalar_embedding(model, "step", dt)
        L = model.layers[j]
        v = L["Wmod"] @ silu(e) + L["bmod"]
        d = model.d
        model._mods[key] = (v[0:d], v[d:2 * d], v[2 * d:3 * d], v[3 * d:4 * d])
    return model._mods[key]


def row_modulation(model: Model, j: int, i: int, depths: np.ndarray) -> Optional[Tuple[np.ndarray, ...]]:
    """Per-row (alpha_msa, alpha_mlp, gamma_msa, gamma_mlp) [n][d] for rows of the
    given depths at loop i, or None without conditioning."""
    if model.cond is None:
        return None
    parts = [modulation(model, j, i, int(m)) for m in depths]
    return tuple(np.stack([p[k] for p in parts]) if parts else np.zeros((0, model.d)) for k in range(4))


# ---------------------------------------------------------------------------
# Router: Eq. 2-5
# ---------------------------------------------------------------------------

def router_logits(model: Model, h0: np.ndarray) -> np.ndarray:
    """f_theta(h^(0)): W_r h^(0) + b_r for the linear router, or the two-layer MLP
    W_r silu(W_1 h^(0) + b_1) + b_r; rounded to float32 where it decides depth."""
    h = h0 if model.Wr1 is None else silu(h0 @ model.Wr1.T + model.br1)
    z = h @ model.Wr.T + model.br
    return z.astype(np.float32).astype(np.float64)


def depth_rule(z: np.ndarray, rule: str, threshold: float = 0.5,
               fixed_depth: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Routed depth m (1-based) and decision margin for logits z [..][R].

    ARGMAX: m = 1 + first index of the largest logit; margin = top1 - top2.
    CUMPROB: pi = softmax(z) (Eq. 2); p^(i) = sum_{l >= i} pi_l (Eq. 3), with
      p^(1) = 1 by construction; token active at loop i iff p^(i) > threshold
      (Eq. 4); m = max{i : p^(i) > threshold} (Eq. 5).  margin =
      min(p^(m) - threshold, threshold - p^(m+1)), with p^(R+1) = 0.
    FIXED: m = fixed_depth; margin = +inf.
    """
    z = np.asarray(z, dtype=np.float64)
    R = z.shape[-1]
    if rule == ARGMAX:
        idx = np.argmax(z, axis=-1)
        srt = np.sort(z, axis=-1)
        margin = srt[..., -1] - srt[..., -2] if R > 1 else np.full(z.shape[:-1], np.inf)
        return idx + 1, margin
    if rule == CUMPROB:
        pi = softmax_rows(z)
        p = np.cumsum(pi[..., ::-1], axis=-1)[..., ::-1].copy()
        p[..., 0] = 1.0
        active = p > threshold
        # active sets are nested because p is non-increasing in i
        m = np.sum(active, axis=-1)
        p_ext = np.concatenate([p, np.zeros(z.shape[:-1] + (1,))], axis=-1)
        pm = np.take_along_axis(p_ext, (m - 1)[..., None], axis=-1)[..., 0]
        pn = np.take_along_axis(p_ext, m[..., None], axis=-1)[..., 0]
        margin = np.minimum(pm - threshold, threshold - pn)
        return m, margin
    if rule == FIXED:
        if fixed_depth is None or not 1 <= fixed_depth <= R:
            raise ValueError("fixed depth must be in [1, R]")
        return np.full(z.shape[:-1], fixed_depth, dtype=np.int64), np.full(z.shape[:-1], np.inf)
    raise ValueError(f"unknown route rule {rule!r}")


def route(model: Model, h0: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    z = router_logits(model, h0)
    m, margin = depth_rule(z, model.route_rule, model.threshold, model.fixed_depth)
    return m.astype(np.int64), margin, z


# ---------------------------------------------------------------------------
# Recursion-wise cache of one sequence (Eq. 8, 11)
# ---------------------------------------------------------------------------

class SeqState:
    """Decode state of one sequence.

    compact mode: for loop i (0-based index i-1), ``pos[i][:n[i]]`` are the
    positions that executed loop i, in ascending order, and ``K[i][j]`` /
    ``V[i][j]`` are [H][n][D] arrays of their keys/values for layer j.
    literal mode: ``Klit[i][j]`` is [H][cap][D] indexed by position, zero where
    the token did not execute loop i, and ``valid[i][t]`` = [m_t >= i].
    """

    def __init__(self, model: Model, mode: str = "compact", capacity: int = 0,
                 use_mask: bool = True):
        if mode not in ("compact", "literal"):
            raise ValueError(mode)
        self.mode, self.use_mask = mode, use_mask
        R, J, H, D = model.R, model.J, model.H, model.D
        self.length = 0
        self.depths: List[int] = []
        self.n = np.zeros(R, dtype=np.int64)
        self.pos: List[np.ndarray] = [np.zeros(0, dtype=np.int64) for _ in range(R)]
        self.K = [[np.zeros((H, 0, D)) for _ in range(J)] for _ in range(R)]
        self.V = [[np.zeros((H, 0, D)) for _ in range(J)] for _ in range(R)]
        if mode == "literal":
            cap = max(1, capacity)
            self.cap = cap
            self.Klit = [[np.zeros((H, cap, D)) for _ in range(J)] for _ in range(R)]
            self.Vlit = [[np.zeros((H, cap, D)) for _ in range(J)] for _ in range(R)]
            self.valid = np.zeros((R, cap), dtype=bool)

    def _grow(self, i: int, need: int) -> None:
        cur = self.pos[i].shape[0]
        if need <= cur:
            return
        new = max(need, 2 * cur, 16)
        self.pos[i] = np.concatenate([self.pos[i], np.zeros(new - cur, dtype=np.int64)])
        for j in range(len(self.K[i])):
            H, _, D = self.K[i][j].shape
            pad = np.zeros((H, new - cur, D))
            self.K[i][j] = np.concatenate([self.K[i][j], pad], axis=1)
            self.V[i][j] = np.concatenate([self.V[i][j], pad.copy()], axis=1)

    def write(self, i: int, j: int, positions: np.ndarray, k: np.ndarray, v: np.ndarray) -> None:
        """Eq. 11: store k, v [n][H][D] of the tokens at ``positions`` in cache (i, j).

        In compact mode the entries are appended after the existing ones (the
        new positions are all later than the stored ones); the slot count n[i]
        advances once per loop, when layer 0 writes.
        """
        cnt = len(positions)
        if self.mode == "compact":
            base = self.n[i] if j == 0 else self.n[i] - cnt
            if j == 0:
                self._grow(i, base + cnt)
                self.pos[i][base:base + cnt] = positions
                self.n[i] += cnt
            self.K[i][j][:, base:base + cnt, :] = np.transpose(k, (1, 0, 2))
            self.V[i][j][:, base:base + cnt, :] = np.transpose(v, (1, 0, 2))
        else:
            if positions.size and positions.max() >= self.cap:
                raise ValueError("literal cache capacity exceeded")
            self.Klit[i][j][:, positions, :] = np.transpose(k, (1, 0, 2))
            self.Vlit[i][j][:, positions, :] = np.transpose(v, (1, 0, 2))
            self.valid[i, positions] = True
            if j == 0:
                self.n[i] += cnt

    def keys(self, i: int, j: int, upto: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """Cache (i, j) read for queries at positions <= ``upto``.

        Returns (positions [m], K [m][H][D], V [m][H][D]).  Compact mode returns
        the stored entries (positions <= upto); literal mode returns every slot
        0..upto, with the validity mask applied later.
        """
        if self.mode == "compact":
            p = self.pos[i][:int(self.n[i])]
            c = int(np.searchsorted(p, upto, side="right"))  # positions are ascending
            return (p[:c], np.transpose(self.K[i][j][:, :c, :], (1, 0, 2)),
                    np.transpose(self.V[i][j][:, :c, :], (1, 0, 2)))
        p = np.arange(upto + 1)
        return (p, np.transpose(self.Klit[i][j][:, :upto + 1, :], (1, 0, 2)),
                np.transpose(self.Vlit[i][j][:, :upto + 1, :], (1, 0, 2)))

    def key_mask(self, i: int, key_pos: np.ndarray) -> np.ndarray:
        """Validity of each returned key: mu^(i) in literal mode, all-true in compact mode."""
        if self.mode == "compact" or not self.use_mask:
            return np.ones(len(key_pos), dtype=bool)
        return self.valid[i, key_pos]

    def cache_positions(self, i: int) -> np.ndarray:
        """Ascending positions held in the loop-(i+1) cache."""
        if self.mode == "compact":
            return self.pos[i][:int(self.n[i])].copy()
        return np.flatnonzero(self.valid[i, :self.length])


# ---------------------------------------------------------------------------
# The shared block on a gathered set of rows
# ---------------------------------------------------------------------------

def _layer(model: Model, j: int, X: np.ndarray, attn_fn, mods=None) -> np.ndarray:
    """One pre-norm layer of the shared block on the rows X [n][d]; ``mods`` is
    the rows' AdaLN (alpha_msa, alpha_mlp, gamma_msa, gamma_mlp) or None."""
    L = model.layers[j]
    st = model.st
    n = X.shape[0]
    Y = rms_norm(X, model.eps)
    if mods is not None:
        Y = Y * (1.0 + mods[2])
    Y = st(Y)
    q = st(Y @ L["Wq"].T).reshape(n, model.H, model.D)
    k = st(Y @ L["Wk"].T).reshape(n, model.H, model.D)
    v = st(Y @ L["Wv"].T).reshape(n, model.H, model.D)
    o = st(attn_fn(j, q, k, v).reshape(n, model.d))
    b = o @ L["Wo"].T
    X = X + (b if mods is None else (1.0 + mods[0]) * b)
    Y2 = rms_norm(X, model.eps)
    if mods is not None:
        Y2 = Y2 * (1.0 + mods[3])
    Y2 = st(Y2)
    a = st(silu(Y2 @ L["Wg"].T) * (Y2 @ L["Wu"].T))
    b = a @ L["Wd"].T
    return X + (b if mods is None else (1.0 + mods[1]) * b)


def lm_head(model: Model, h: np.ndarray) -> np.ndarray:
    """Final RMSNorm and LM head: logits = RMSNorm(h) E^T for the tied head."""
    return model.st(rms_norm(h, model.eps)) @ model.head.T


def greedy(logits: np.ndarray) -> np.ndarray:
    """Lowest token id among the float32-rounded maxima."""
    return np.argmax(logits.astype(np.float32), axis=-1)


# ---------------------------------------------------------------------------
# Prefill (Section 3.2 gather-scatter, Section 3.3 batched prefill)
# ---------------------------------------------------------------------------

def prefill(model: Model, tokens: Sequence[int], mode: str = "compact",
            capacity: int = 0, use_mask: bool = True, all_logits: bool = False,
            state: Optional[SeqState] = None
            ) -> Tuple[SeqState, np.ndarray, np.ndarray, np.ndarray]:
    """Prefill of one sequence; returns (state, logits, depths, margins).

    logits are for the last position, or [T][V] with ``all_logits``.

    The T tokens sit at positions t0 .. t0 + T - 1: t0 = 0 and empty caches
    for a new sequence, or t0 = state.length when ``state`` is continued (a
    later chunk of the prompt, or tokens after decode steps; ``mode`` and
    ``use_mask`` are then the state's).

    compact mode: loop i gathers rho = sort(A_i) over the T tokens (Eq. 6),
    writes their k, v after the entries already in cache i (Eq. 11), and runs
    the block on the gathered rows; each row attends over the entries of
    cache i at positions up to its own (Eq. 10): the earlier entries plus
    causal attention among the gathered rows.  The rows are scattered back
    (Eq. 7).
    literal mode: the block runs on all T rows every loop; the cache is written
    only for rows in A_i, attention uses causality plus mu^(i), and only rows in
    A_i take the new state.
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    T = tokens.shape[0]
    if T == 0:
        raise ValueError("empty prompt")
    st = state if state is not None else SeqState(model, mode, max(capacity, T), use_mask)
    t0 = st.length
    if t0 + T > model.P.shape[0]:
        raise ValueError("prompt longer than the position table")
    pos = t0 + np.arange(T)
    Hs = model.E[tokens] + model.P[pos]
    m, margin, _ = route(model, Hs)
    st.depths += [int(x) for x in m]
    for i in range(1, model.R + 1):
        if st.mode == "compact":
            rho = np.flatnonzero(m >= i)
            if rho.size == 0:
                break
            X = Hs[rho]
            qpos = pos[rho]

            def attn_fn(j, q, k, v, i=i, qpos=qpos):
                st.write(i - 1, j, qpos, k, v)
                kp, K, Vv = st.keys(i - 1, j, int(qpos[-1]))
                return attend(q, K, Vv, kp[None, :] <= qpos[:, None])

            Hs[rho] = _layers(model, X, attn_fn, i, m[rho])
        else:
            act = m >= i
            if not act.any():
                break

            def attn_fn(j, q, k, v, i=i, act=act):
                st.write(i - 1, j, pos[act], k[act], v[act])
                kp, K, Vv = st.keys(i - 1, j, int(pos[-1]))
                causal = kp[None, :] <= pos[:, None]
                # rows outside A_i are computed and then discarded; they skip the
                # mask only so that none of them is left without any key
                valid = st.key_mask(i - 1, kp)[None, :] | ~act[:, None]
                return attend(q, K, Vv, causal & valid)

            Xn = _layers(model, Hs.copy(), attn_fn, i, m)
            Hs[act] = Xn[act]
    st.length = t0 + T
    logits = lm_head(model, Hs if all_logits else Hs[-1:])
    return st, (logits if all_logits else logits[0]), m, margin


def _layers(model: Model, X: np.ndarray, attn_fn, i: int, depths: np.ndarray) -> np.ndarray:
    """The shared block at loop i on rows X whose tokens have the given depths."""
    for j in range(model.J):
        X = _layer(model, j, X, attn_fn, row_modulation(model, j, i, depths))
    return X


# ---------------------------------------------------------------------------
# Decode (Section 3.3, Eq. 9-11)
# ---------------------------------------------------------------------------

def decode(model: Model, states: List[SeqState], tokens: Sequence[int]
           ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One decode step for a batch of independent sequences.

    Token b sits at position t_b = states[b].length.  Its depth m_b comes from
    the router on h0.  Loop i runs on the gathered sequences with m_b >= i
    (Eq. 6; for one sequence this is plain early exit).  In each layer every
    active token appends its k, v to cache (i, j) at slot n_{b,i} (Eq. 11) and
    then attends over that cache, its own entry included (Eq. 10).  Returns
    (logits [B][V], depths [B], margins [B]).
    """
    tokens = np.asarray(tokens, dtype=np.int64)
    B = len(states)
    if tokens.shape[0] != B:
        raise ValueError("one token per sequence")
    t = np.array([s.length for s in states], dtype=np.int64)
    if np.any(t >= model.P.shape[0]):
        raise ValueError("position beyond the position table")
    h = model.E[tokens] + model.P[t]
    m, margin, _ = route(model, h)
    for i in range(1, model.R + 1):
        act = np.flatnonzero(m >= i)
        if act.size == 0:
            break

        def attn_fn(j, q, k, v, i=i, act=act):
            out = np.empty_like(q)
            for r, b in enumerate(act):
                s = states[b]
                s.write(i - 1, j, t[b:b + 1], k[r:r + 1], v[r:r + 1])
                kp, K, Vv = s.keys(i - 1, j, int(t[b]))
                allowed = s.key_mask(i - 1, kp)[None, :]
                out[r:r + 1] = attend(q[r:r + 1], K, Vv, allowed)
            return out

        h[act] = _layers(model, h[act], attn_fn, i, m[act])
    for b, s in enumerate(states):
        s.depths.append(int(m[b]))
        s.length += 1
    return lm_head(model, h), m, margin


def prefill_batch(model: Model, tokens: np.ndarray, **kw):
    """Independent prefill of each row of tokens [B][T]."""
    out = [prefill(model, row, **kw) for row in np.asarray(tokens)]
    return ([o[0] for o in out], np.stack([o[1] for o in out]),
            np.stack([o[2] for o in out]), np.stack([o[3] for o in out]))


def cache_index(state: SeqState, R: int) -> List[np.ndarray]:
    """For each loop i = 1..R, the ascending positions stored in its cache."""
    return [state.cache_positions(i) for i in range(R)]
