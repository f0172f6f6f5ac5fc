"""Independent references written with plain PyTorch CPU ops (float64).

They are not the oracle: they restate the model with library attention
(``scaled_dot_product_attention``) on dense tensors so that the oracle can be
checked against something other than itself.
"""
import numpy as np
import torch
import torch.nn.functional as F

f64 = torch.float64


def _t(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def _rms(x, eps):
    return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps)


def _keep(x):
    return x


def bf16_cast(x):
    """torch's own casts: float64 -> float32 -> bfloat16 (round to nearest even),
    widened back to float64."""
    return x.to(torch.float32).to(torch.bfloat16).to(f64)


def _layer(x, lw, H, D, eps, attn_mask=None, is_causal=False, mod=None, rnd=_keep):
    """Pre-norm layer; ``mod`` = per-row AdaLN (shift-free) modulation
    [T][4d] split as (alpha_msa, alpha_mlp, gamma_msa, gamma_mlp), or None.
    ``rnd`` is applied where a bf16 implementation stores a value: the
    normalised inputs of the projections, q, k and v, the attention output
    and the SwiGLU product."""
    T, d = x.shape
    if mod is not None:
        a_msa, a_mlp, g_msa, g_mlp = mod.split(d, dim=-1)
    y = _rms(x, eps)
    if mod is not None:
        y = y * (1 + g_msa)
    qkv = rnd(F.linear(rnd(y), _t(lw["w_qkv"])))
    q, k, v = (t.reshape(T, H, D).transpose(0, 1) for t in qkv.split(d, dim=-1))
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=attn_mask, is_causal=is_causal)
    b = F.linear(rnd(o.transpose(0, 1).reshape(T, d)), _t(lw["w_o"]))
    x = x + (b if mod is None else (1 + a_msa) * b)
    y2 = _rms(x, eps)
    if mod is not None:
        y2 = y2 * (1 + g_mlp)
    g, u = F.linear(rnd(y2), _t(lw["w_gate_up"])).chunk(2, dim=-1)
    b = F.linear(rnd(F.silu(g) * u), _t(lw["w_down"]))
    return x + (b if mod is None else (1 + a_mlp) * b)


def _scalar_embed(cond, which, tau):
    """DiT-style embedder of scalars tau [T]: sinusoidal features (256 wide,
    cos/sin interleaved per frequency, max period 10000), Linear-SiLU-Linear."""
    half = 128
    freqs = torch.exp(-torch.log(torch.tensor(10000.0, dtype=f64)) * torch.arange(half, dtype=f64) / half)
    ang = tau[:, None] * freqs[None, :]
    feats = torch.stack([torch.cos(ang), torch.sin(ang)], dim=-1).reshape(tau.shape[0], 2 * half)
    h = F.silu(F.linear(feats, _t(cond[which + "_w1"]), _t(cond[which + "_b1"])))
    return F.linear(h, _t(cond[which + "_w2"]), _t(cond[which + "_b2"]))


def adaln_modulation(weights, lw, loop, depths):
    """Layer modulation [T][4d] for rows of the given depths at 1-based ``loop``:
    cumulative time (loop - 1) / m and step 1 / m, summed embeddings, SiLU, Linear."""
    m = torch.as_tensor(np.asarray(depths, dtype=np.float64))
    cond = weights["cond"]
    c = _scalar_embed(cond, "time", (loop - 1) / m) + _scalar_embed(cond, "step", 1.0 / m)
    return F.linear(F.silu(c), _t(lw["w_mod"]), _t(lw["b_mod"]))


def tied_gpt_logits(weights, tokens, H, D, loops, eps=1e-5, rnd=_keep):
    """Pre-norm GPT whose layer stack is the J-layer block repeated ``loops``
    times (every token of depth ``loops`` when the weights carry AdaLN)."""
    tokens = torch.as_tensor(np.asarray(tokens, dtype=np.int64))
    E, P = _t(weights["tok_emb"]), _t(weights["pos_emb"])
    x = E[tokens] + P[: tokens.shape[0]]
    T = tokens.shape[0]
    for i in range(1, loops + 1):
        for lw in weights["layers"]:
            mod = adaln_modulation(weights, lw, i, [loops] * T) if weights.get("cond") else None
            x = _layer(x, lw, H, D, eps, is_causal=True, mod=mod, rnd=rnd)
    head = E if weights.get("lm_head") is None else _t(weights["lm_head"])
    return F.linear(rnd(_rms(x, eps)), head).numpy()


def router_logits(weights, h0):
    """Linear router, or Linear -> SiLU -> Linear when router_w1 is given (float64)."""
    h = torch.as_tensor(np.asarray(h0, dtype=np.float64))
    if weights.get("router_w1") is not None:
        h = F.silu(F.linear(h, _t(weights["router_w1"]), _t(weights["router_b1"])))
    return F.linear(h, _t(weights["router_w"]), _t(weights["router_b"]))


def routed_argmax_depths(weights, tokens):
    """1 + argmax of the float32-rounded router logits of h0 = E[x] + P[t]."""
    tokens = np.asarray(tokens, dtype=np.int64)
    h0 = _t(weights["tok_emb"])[tokens] + _t(weights["pos_emb"])[: len(tokens)]
    z = router_logits(weights, h0).to(torch.float32)
    return (torch.argmax(z, dim=-1) + 1).numpy()


def routed_dense_logits(weights, tokens, depths, H, D, eps=1e-5, rnd=_keep):
    """Routed model computed densely: every loop runs on all rows, attention
    is causal and restricted to keys whose depth reaches the loop, and only
    rows whose depth reaches the loop take the new state."""
    tokens = torch.as_tensor(np.asarray(tokens, dtype=np.int64))
    depths = torch.as_tensor(np.asarray(depths, dtype=np.int64))
    T = tokens.shape[0]
    E, P = _t(weights["tok_emb"]), _t(weights["pos_emb"])
    x = E[tokens] + P[:T]
    causal = torch.tril(torch.ones(T, T, dtype=torch.bool))
    R = weights["router_w"].shape[0]
    for i in range(1, R + 1):
        act = depths >= i
        if not bool(act.any()):
            break
        # rows outside the active set keep a causal view so that none is empty;
        # their outputs are discarded below
        mask = causal & (act[None, :] | ~act[:, None])
        xn = x
        for lw in weights["layers"]:
            mod = adaln_modulation(weights, lw, i, depths.numpy()) if weights.get("cond") else None
            xn = _layer(xn, lw, H, D, eps, attn_mask=mask, mod=mod, rnd=rnd)
        x = torch.where(act[:, None], xn, x)
    return F.linear(rnd(_rms(x, eps)), E).numpy()
