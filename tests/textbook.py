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


def _layer(x, lw, H, D, eps, attn_mask=None, is_causal=False):
    T, d = x.shape
    y = _rms(x, eps)
    qkv = F.linear(y, _t(lw["w_qkv"]))
    q, k, v = (t.reshape(T, H, D).transpose(0, 1) for t in qkv.split(d, dim=-1))
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=attn_mask, is_causal=is_causal)
    x = x + F.linear(o.transpose(0, 1).reshape(T, d), _t(lw["w_o"]))
    y2 = _rms(x, eps)
    g, u = F.linear(y2, _t(lw["w_gate_up"])).chunk(2, dim=-1)
    return x + F.linear(F.silu(g) * u, _t(lw["w_down"]))


def tied_gpt_logits(weights, tokens, H, D, loops, eps=1e-5):
    """Pre-norm GPT whose layer stack is the J-layer block repeated ``loops`` times."""
    tokens = torch.as_tensor(np.asarray(tokens, dtype=np.int64))
    E, P = _t(weights["tok_emb"]), _t(weights["pos_emb"])
    x = E[tokens] + P[: tokens.shape[0]]
    for _ in range(loops):
        for lw in weights["layers"]:
            x = _layer(x, lw, H, D, eps, is_causal=True)
    head = E if weights.get("lm_head") is None else _t(weights["lm_head"])
    return F.linear(_rms(x, eps), head).numpy()


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


def routed_dense_logits(weights, tokens, depths, H, D, eps=1e-5):
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
            xn = _layer(xn, lw, H, D, eps, attn_mask=mask)
        x = torch.where(act[:, None], xn, x)
    return F.linear(_rms(x, eps), E).numpy()
