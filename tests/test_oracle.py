"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself: hand-worked
values (tests/golden), closed forms, an independent PyTorch restatement of the
model, brute-force recomputation, or an invariant the paper states.
"""
import json
import math
import os

import numpy as np
import pytest

import synth
from oracle import tlf_oracle as O
from tests import textbook

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _model(cfg, w, **kw):
    return O.Model(w, cfg.n_heads, cfg.head_dim, rms_eps=cfg.rms_eps, **kw)


# ---------------------------------------------------------------------------
# Router rules (Eq. 2-5)
# ---------------------------------------------------------------------------

def test_router_golden_cases():
    cases = json.load(open(os.path.join(GOLDEN, "router_cases.json")))["cases"]
    for c in cases:
        z = np.array(c["z"] if "z" in c else np.log(c["pi"]), dtype=np.float64)[None, :]
        m, margin = O.depth_rule(z, c["rule"], c.get("theta", 0.5), c.get("depth"))
        assert int(m[0]) == c["m"], c
        if c["margin"] is None:
            assert not np.isfinite(margin[0]) or z.shape[1] == 1
        else:
            assert margin[0] == pytest.approx(c["margin"], abs=1e-9), c


def test_cumprob_half_is_lower_median():
    """m = max{i : P(depth >= i) > 1/2} equals min{i : P(depth <= i) >= 1/2}."""
    rng = np.random.default_rng(0)
    z = rng.normal(size=(5000, 8)) * 2.0
    m, _ = O.depth_rule(z, O.CUMPROB, 0.5)
    pi = np.exp(z - z.max(1, keepdims=True))
    pi /= pi.sum(1, keepdims=True)
    cdf = np.cumsum(pi, axis=1)
    med = np.argmax(cdf >= 0.5, axis=1) + 1
    assert np.array_equal(m, med)


def test_cumprob_active_sets_nested_and_threshold_monotone():
    rng = np.random.default_rng(1)
    z = rng.normal(size=(2000, 6))
    prev = None
    for th in (0.2, 0.35, 0.5, 0.65, 0.8):
        m, margin = O.depth_rule(z, O.CUMPROB, th)
        assert m.min() >= 1 and m.max() <= 6
        assert np.all(margin >= 0)
        if prev is not None:
            assert np.all(m <= prev)  # higher threshold never deepens a token
        prev = m


def test_argmax_rule_matches_textbook_argmax_on_model():
    cfg = synth.tiny_config(max_loops=4, prompt_len=40)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    M = _model(cfg, w)
    _, _, m, _ = O.prefill(M, toks)
    assert np.array_equal(m, textbook.routed_argmax_depths(w, toks))


# ---------------------------------------------------------------------------
# Closed forms of the elementary pieces
# ---------------------------------------------------------------------------

def test_rms_norm_closed_form():
    x = np.array([[3.0, 4.0]])
    y = O.rms_norm(x, 0.0)
    assert np.allclose(y, [[3.0 / math.sqrt(12.5), 4.0 / math.sqrt(12.5)]])
    assert np.allclose(O.rms_norm(np.array([[2.0, 2.0, 2.0, 2.0]]), 0.0), 1.0)


def test_attention_closed_forms():
    q = np.array([[[1.0, 0.0]]])                  # [n=1][H=1][D=2]
    k = np.array([[[0.3, 0.7]]])
    v = np.array([[[5.0, -2.0]]])
    # one key: the output is that value
    assert np.allclose(O.attend(q, k, v, np.ones((1, 1), bool)), v)
    # two keys with equal scores: the mean of the values
    k2 = np.array([[[0.0, 1.0]], [[0.0, -1.0]]])
    v2 = np.array([[[1.0, 2.0]], [[3.0, 6.0]]])
    assert np.allclose(O.attend(q, k2, v2, np.ones((1, 2), bool)), [[[2.0, 4.0]]])
    # scores 0 and sqrt(2)*ln 3 / sqrt(2): weights 1/4, 3/4
    k3 = np.array([[[0.0, 0.0]], [[math.sqrt(2) * math.log(3.0), 0.0]]])
    assert np.allclose(O.attend(q, k3, v2, np.ones((1, 2), bool)), [[[2.5, 5.0]]])
    # a masked key gets no weight
    assert np.allclose(O.attend(q, k3, v2, np.array([[True, False]])), [[[1.0, 2.0]]])


def test_silu_closed_form():
    assert O.silu(np.array([0.0]))[0] == 0.0
    assert O.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)))


def _mlp_cfg(**kw):
    base = dict(max_loops=4, prompt_len=24, router_hidden=32, router_bias="calibrated")
    base.update(kw)
    return synth.tiny_config(**base)


def test_mlp_router_matches_library_layers():
    """Two-layer MLP router (Section 3.2) against torch's Linear -> SiLU -> Linear."""
    cfg = _mlp_cfg()
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    M = _model(cfg, w)
    h0 = M.E[toks] + M.P[: len(toks)]
    z = O.router_logits(M, h0)
    ref = textbook.router_logits(w, h0).numpy().astype(np.float32).astype(np.float64)
    assert np.max(np.abs(z - ref)) <= 1e-6 * np.max(np.abs(ref))
    # closed form: with W_1 = 0 every token's hidden layer is silu(b_1)
    w0 = dict(w)
    w0["router_w1"] = np.zeros_like(w["router_w1"])
    w0["router_b1"] = np.linspace(-2.0, 2.0, cfg.router_hidden)
    b1 = w0["router_b1"]
    want = (b1 / (1.0 + np.exp(-b1))) @ np.asarray(w["router_w"], np.float64).T + w["router_b"]
    z0 = O.router_logits(_model(cfg, w0), h0)
    assert np.max(np.abs(z0 - want[None, :])) < 1e-6


def test_mlp_router_depths_and_threshold_monotonicity():
    """Argmax depths equal the library router's; under the cumulative rule a
    higher threshold never deepens a token (p^(i) is non-increasing in i)."""
    cfg = _mlp_cfg(prompt_len=64)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    M = _model(cfg, w)
    h0 = M.E[toks] + M.P[: len(toks)]
    z = O.router_logits(M, h0)
    m, _ = O.depth_rule(z, O.ARGMAX)
    assert np.array_equal(m, textbook.routed_argmax_depths(w, toks))
    prev = None
    for th in (0.1, 0.3, 0.5, 0.7, 0.9):
        d, _ = O.depth_rule(z, O.CUMPROB, th)
        if prev is not None:
            assert np.all(d <= prev)
        prev = d
    assert len(set(O.depth_rule(z, O.CUMPROB, 0.5)[0].tolist())) >= 2


def test_mlp_router_prefill_equals_dense_masked_model():
    """The routed model with an MLP router against the dense masked PyTorch model
    whose depths come from the library router."""
    cfg = _mlp_cfg()
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    _, logits, m, _ = O.prefill(_model(cfg, w), toks, all_logits=True)
    assert np.array_equal(m, textbook.routed_argmax_depths(w, toks))
    assert len(set(m.tolist())) >= 2
    ref = textbook.routed_dense_logits(w, toks, m, cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


# ---------------------------------------------------------------------------
# Block math against an independent dense PyTorch model
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("loops", [1, 3])
def test_fixed_depth_equals_tied_weight_gpt(loops):
    """FIXED(k): the looped model is a pre-norm GPT with k*J weight-tied layers."""
    cfg = synth.tiny_config(max_loops=4, prompt_len=14)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[1]
    M = _model(cfg, w, route_rule=O.FIXED, fixed_depth=loops)
    _, logits, m, _ = O.prefill(M, toks, all_logits=True)
    assert np.all(m == loops)
    ref = textbook.tied_gpt_logits(w, toks, cfg.n_heads, cfg.head_dim, loops, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


def test_fixed_depth_decode_equals_tied_weight_gpt():
    cfg = synth.tiny_config(max_loops=3, prompt_len=9, steps=5)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg, prompt_len=cfg.prompt_len + cfg.steps)[0]
    M = _model(cfg, w, route_rule=O.FIXED, fixed_depth=3)
    st, _, _, _ = O.prefill(M, toks[: cfg.prompt_len])
    ref = textbook.tied_gpt_logits(w, toks, cfg.n_heads, cfg.head_dim, 3, cfg.rms_eps)
    for s in range(cfg.steps):
        t = cfg.prompt_len + s
        lg, _, _ = O.decode(M, [st], [toks[t]])
        assert np.max(np.abs(lg[0] - ref[t])) < 1e-12


def test_untied_head_equals_textbook_gpt():
    """A separate LM head replaces E^T in the last product and nowhere else."""
    cfg = synth.tiny_config(max_loops=3, prompt_len=11)
    w = dict(synth.make_weights(cfg))
    w["lm_head"] = synth.make_lm_head(cfg)
    toks = synth.make_prompts(cfg)[0]
    _, logits, _, _ = O.prefill(_model(cfg, w, route_rule=O.FIXED, fixed_depth=2), toks, all_logits=True)
    ref = textbook.tied_gpt_logits(w, toks, cfg.n_heads, cfg.head_dim, 2, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12
    tied = dict(w)
    del tied["lm_head"]
    _, logits_tied, _, _ = O.prefill(_model(cfg, tied, route_rule=O.FIXED, fixed_depth=2), toks,
                                     all_logits=True)
    assert np.max(np.abs(logits - logits_tied)) > 1e-3


def test_single_loop_model_is_plain_gpt():
    """R = 1: every token takes exactly one pass of the J-layer block."""
    cfg = synth.tiny_config(max_loops=1, n_layers=3, prompt_len=10)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    _, logits, m, _ = O.prefill(_model(cfg, w), toks, all_logits=True)
    assert np.all(m == 1)
    ref = textbook.tied_gpt_logits(w, toks, cfg.n_heads, cfg.head_dim, 1, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


@pytest.mark.parametrize("seed", [3, 4])
def test_routed_prefill_equals_dense_masked_model(seed):
    """Gather-scatter (Eq. 6-7) with compact caches equals the dense formulation
    where each loop sees every row, masks keys by depth (mu, Eq. 10) and only
    updates rows whose depth reaches the loop."""
    cfg = synth.tiny_config(max_loops=4, prompt_len=24)
    w = synth.make_weights(cfg, seed=seed)
    toks = synth.make_prompts(cfg, seed=seed)[0]
    _, logits, m, _ = O.prefill(_model(cfg, w), toks, all_logits=True)
    assert len(set(m.tolist())) >= 3  # several depths present
    ref = textbook.routed_dense_logits(w, toks, m, cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


# ---------------------------------------------------------------------------
# Recursion-wise cache
# ---------------------------------------------------------------------------

def _run(cfg, w, mode="compact", use_mask=True, steps=None, model_kw=None, seed=synth.SEED):
    steps = cfg.steps if steps is None else steps
    M = _model(cfg, w, **(model_kw or {}))
    toks = synth.make_prompts(cfg, seed=seed, prompt_len=cfg.prompt_len + steps)
    states, logits, _, _ = O.prefill_batch(M, toks[:, : cfg.prompt_len], mode=mode,
                                           capacity=cfg.prompt_len + steps, use_mask=use_mask)
    outs = [logits]
    for s in range(steps):
        lg, _, _ = O.decode(M, states, toks[:, cfg.prompt_len + s])
        outs.append(lg)
    return M, states, np.stack(outs, 1), toks


def test_literal_masked_cache_equals_compact_cache():
    cfg = synth.tiny_config(batch=2, prompt_len=10, steps=6)
    w = synth.make_weights(cfg)
    _, _, a, _ = _run(cfg, w, "compact")
    _, _, b, _ = _run(cfg, w, "literal")
    assert np.max(np.abs(a - b)) < 1e-12


def test_dropping_validity_mask_changes_results():
    """Appendix B: without mu the softmax gives weight to exited tokens' zero slots."""
    cfg = synth.tiny_config(batch=2, prompt_len=10, steps=4)
    w = synth.make_weights(cfg)
    _, _, a, _ = _run(cfg, w, "compact")
    _, _, b, _ = _run(cfg, w, "literal", use_mask=False)
    assert np.max(np.abs(a - b)) > 1e-3


def test_cached_decode_equals_full_recompute():
    """Every cached decode step equals the last row of a from-scratch prefill of
    the extended sequence, and of the independent dense masked model."""
    cfg = synth.tiny_config(batch=1, prompt_len=8, steps=7, max_loops=4)
    w = synth.make_weights(cfg, seed=11)
    M, states, logits, toks = _run(cfg, w, seed=11)
    for s in range(cfg.steps + 1):
        T = cfg.prompt_len + s
        _, lg_full, m_full, _ = O.prefill(M, toks[0, :T])
        assert np.max(np.abs(logits[0, s] - lg_full)) < 1e-12
        dense = textbook.routed_dense_logits(w, toks[0, :T], m_full, cfg.n_heads,
                                             cfg.head_dim, cfg.rms_eps)
        assert np.max(np.abs(logits[0, s] - dense[-1])) < 1e-12


# ---------------------------------------------------------------------------
# Chunked prefill: a prompt prefilled in pieces onto the existing caches
# ---------------------------------------------------------------------------

def _prefill_chunks(M, toks, cuts, **kw):
    st, logits, depths = None, [], []
    for a, b in zip((0,) + tuple(cuts), tuple(cuts) + (len(toks),)):
        st, lg, m, _ = O.prefill(M, toks[a:b], all_logits=True, state=st, **kw)
        logits.append(lg)
        depths.append(m)
    return st, np.concatenate(logits), np.concatenate(depths)


@pytest.mark.parametrize("cuts", [(5,), (1, 2, 17), (16, 32), (7, 8, 9, 10)])
def test_chunked_prefill_equals_dense_masked_model(cuts):
    """A prompt prefilled in chunks gives every position the logits of the
    independent dense masked model, the library-argmax depths, and caches that
    hold exactly the positions of depth >= i."""
    cfg = synth.tiny_config(max_loops=4, prompt_len=40)
    w = synth.make_weights(cfg, seed=5)
    toks = synth.make_prompts(cfg, seed=5)[0]
    M = _model(cfg, w)
    st, logits, m = _prefill_chunks(M, toks, cuts)
    assert len(set(m.tolist())) >= 3
    assert np.array_equal(m, textbook.routed_argmax_depths(w, toks))
    ref = textbook.routed_dense_logits(w, toks, m, cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12
    idx = O.cache_index(st, M.R)
    for i in range(M.R):
        assert np.array_equal(idx[i], np.flatnonzero(m >= i + 1))
    assert st.length == len(toks) and st.depths == m.tolist()


def test_one_token_chunk_equals_decode_step():
    """A chunk of one token is a decode step (Eq. 9-11): same depth, logits and cache."""
    cfg = synth.tiny_config(batch=1, prompt_len=12, steps=7, max_loops=4)
    w = synth.make_weights(cfg, seed=6)
    toks = synth.make_prompts(cfg, seed=6, prompt_len=19)[0]
    M = _model(cfg, w)
    sa, _, _, _ = O.prefill(M, toks[:12])
    sb, _, _, _ = O.prefill(M, toks[:12])
    for t in range(12, 19):
        la, ma, _ = O.decode(M, [sa], [toks[t]])
        sb, lb, mb, _ = O.prefill(M, toks[t:t + 1], state=sb)
        assert int(ma[0]) == int(mb[0])
        assert np.max(np.abs(la[0] - lb)) < 1e-12
    for i in range(M.R):
        assert np.array_equal(sa.cache_positions(i), sb.cache_positions(i))
        n = int(sa.n[i])
        for j in range(M.J):
            assert np.max(np.abs(sa.K[i][j][:, :n] - sb.K[i][j][:, :n]), initial=0.0) < 1e-12
            assert np.max(np.abs(sa.V[i][j][:, :n] - sb.V[i][j][:, :n]), initial=0.0) < 1e-12


@pytest.mark.parametrize("mode", ["compact", "literal"])
def test_chunk_after_decode_steps_equals_one_shot_prefill(mode):
    """prefill, decode steps, a further chunk, more decode steps: each output
    equals the matching row of one prefill over the whole token sequence, in
    both cache representations."""
    cfg = synth.tiny_config(batch=1, prompt_len=10, steps=16, max_loops=4)
    w = synth.make_weights(cfg, seed=7)
    toks = synth.make_prompts(cfg, seed=7, prompt_len=26)[0]
    M = _model(cfg, w)
    _, ref, m_ref, _ = O.prefill(M, toks, all_logits=True)
    st, lg, m, _ = O.prefill(M, toks[:10], mode=mode, capacity=26, all_logits=True)
    got, depths = [lg], [m]
    for t in range(10, 13):
        lg, m, _ = O.decode(M, [st], [toks[t]])
        got.append(lg)
        depths.append(m)
    st, lg, m, _ = O.prefill(M, toks[13:22], all_logits=True, state=st)
    got.append(lg)
    depths.append(m)
    for t in range(22, 26):
        lg, m, _ = O.decode(M, [st], [toks[t]])
        got.append(lg)
        depths.append(m)
    assert np.array_equal(np.concatenate(depths), m_ref)
    assert np.max(np.abs(np.concatenate(got) - ref)) < 1e-12


def test_cache_holds_exactly_positions_with_depth_at_least_loop():
    cfg = synth.tiny_config(batch=3, prompt_len=20, steps=10, max_loops=4)
    w = synth.make_weights(cfg)
    M, states, _, _ = _run(cfg, w)
    for st in states:
        depths = np.array(st.depths)
        assert len(depths) == st.length == cfg.prompt_len + cfg.steps
        idx = O.cache_index(st, M.R)
        for i in range(M.R):
            assert np.array_equal(idx[i], np.flatnonzero(depths >= i + 1))
        n = np.array([len(x) for x in idx])
        assert n[0] == st.length                      # A_1 holds every token
        assert np.all(np.diff(n) <= 0)                # nested active sets
        assert n.sum() == depths.sum()                # each token stored once per loop run


def test_batch_composition_does_not_change_a_sequence():
    cfg = synth.tiny_config(batch=3, prompt_len=9, steps=4)
    w = synth.make_weights(cfg)
    _, _, full, toks = _run(cfg, w)
    M = _model(cfg, w)
    for b in (2, 0):
        st, lg, _, _ = O.prefill(M, toks[b, : cfg.prompt_len])
        outs = [lg]
        for s in range(cfg.steps):
            l2, _, _ = O.decode(M, [st], [toks[b, cfg.prompt_len + s]])
            outs.append(l2[0])
        assert np.max(np.abs(np.stack(outs) - full[b])) < 1e-12


def test_single_token_prompt_and_all_deepest():
    cfg = synth.tiny_config(batch=1, prompt_len=1, steps=3, max_loops=3)
    w = synth.make_weights(cfg)
    # bias that routes everything to the deepest loop
    w = dict(w, router_b=np.array([0.0, 0.0, 10.0], dtype=np.float32))
    M, states, logits, toks = _run(cfg, w)
    assert all(d == 3 for d in states[0].depths)
    ref = textbook.tied_gpt_logits(w, toks[0], cfg.n_heads, cfg.head_dim, 3, cfg.rms_eps)
    assert np.max(np.abs(logits[0] - ref[:, :])) < 1e-12


def test_cumprob_rule_end_to_end_with_dense_model():
    cfg = synth.tiny_config(batch=1, prompt_len=16, max_loops=4)
    w = synth.make_weights(cfg)
    w = dict(w, router_w=(w["router_w"] * 200.0).astype(np.float32))  # spread the depths
    M = _model(cfg, w, route_rule=O.CUMPROB, threshold=0.5)
    toks = synth.make_prompts(cfg)[0]
    _, logits, m, _ = O.prefill(M, toks, all_logits=True)
    assert len(set(m.tolist())) >= 2
    ref = textbook.routed_dense_logits(w, toks, m, cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


# ---------------------------------------------------------------------------
# AdaLN time/step conditioning (Section 3.1, Appendix A)
# ---------------------------------------------------------------------------

def test_fourier_features_closed_form():
    f0 = O.fourier_features(0.0)
    assert f0.shape == (256,)
    assert np.array_equal(f0[0::2], np.ones(128)) and np.array_equal(f0[1::2], np.zeros(128))
    f1 = O.fourier_features(1.0)
    assert f1[0] == pytest.approx(math.cos(1.0), abs=1e-15) and f1[1] == pytest.approx(math.sin(1.0), abs=1e-15)
    w_last = 10000.0 ** (-127.0 / 128.0)  # lowest frequency
    assert f1[254] == pytest.approx(math.cos(w_last), abs=1e-15)
    assert f1[255] == pytest.approx(math.sin(w_last), abs=1e-15)


@pytest.mark.parametrize("m", [1, 2, 5])
def test_uniform_trajectory_sums_to_one(m):
    ts = [O.trajectory(i, m) for i in range(1, m + 1)]
    assert ts[0][0] == 0.0
    assert sum(dt for _, dt in ts) == pytest.approx(1.0, abs=1e-15)
    for (c0, dt), (c1, _) in zip(ts, ts[1:]):
        assert c1 == pytest.approx(c0 + dt, abs=1e-15)  # c_i = c_{i-1} + Delta_i


def _adaln_cfg(**kw):
    base = dict(max_loops=4, prompt_len=24, adaln=True)
    base.update(kw)
    return synth.tiny_config(**base)


def test_adaln_zero_modulator_is_unconditioned_model():
    """Zero modulator weights and bias (the paper's initialisation) leave the
    unmodulated backbone, exactly, under the 1 + alpha reading of the gate."""
    cfg = _adaln_cfg()
    w = synth.make_weights(cfg)
    w0 = dict(w, layers=[dict(lw, w_mod=np.zeros_like(lw["w_mod"]), b_mod=np.zeros_like(lw["b_mod"]))
                         for lw in w["layers"]])
    plain = {k: v for k, v in w.items() if k != "cond"}
    plain["layers"] = [{k: v for k, v in lw.items() if k not in ("w_mod", "b_mod")} for lw in w["layers"]]
    toks = synth.make_prompts(cfg)[0]
    _, a, ma, _ = O.prefill(_model(cfg, w0), toks, all_logits=True)
    _, b, mb, _ = O.prefill(_model(cfg, plain), toks, all_logits=True)
    assert np.array_equal(ma, mb) and np.array_equal(a, b)
    _, c, _, _ = O.prefill(_model(cfg, w), toks, all_logits=True)
    assert np.max(np.abs(c - b)) > 1e-3  # the synthetic modulator does act


@pytest.mark.parametrize("seed", [3, 4])
def test_adaln_routed_prefill_equals_dense_masked_model(seed):
    """Per-token conditioning on each token's own trajectory: the oracle's
    gathered prefill equals the independent dense PyTorch model with library
    embedders and the same modulation."""
    cfg = _adaln_cfg()
    w = synth.make_weights(cfg, seed=seed)
    toks = synth.make_prompts(cfg, seed=seed)[0]
    _, logits, m, _ = O.prefill(_model(cfg, w), toks, all_logits=True)
    assert len(set(m.tolist())) >= 3
    ref = textbook.routed_dense_logits(w, toks, m, cfg.n_heads, cfg.head_dim, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


def test_adaln_fixed_depth_equals_conditioned_gpt():
    cfg = _adaln_cfg(max_loops=3)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    M = _model(cfg, w, route_rule=O.FIXED, fixed_depth=3)
    _, logits, _, _ = O.prefill(M, toks, all_logits=True)
    ref = textbook.tied_gpt_logits(w, toks, cfg.n_heads, cfg.head_dim, 3, cfg.rms_eps)
    assert np.max(np.abs(logits - ref)) < 1e-12


def test_adaln_cached_decode_equals_full_recompute():
    cfg = synth.tiny_config(batch=1, prompt_len=8, steps=6, max_loops=4, adaln=True)
    w = synth.make_weights(cfg, seed=12)
    M, states, logits, toks = _run(cfg, w, seed=12)
    for s in range(cfg.steps + 1):
        T = cfg.prompt_len + s
        _, lg_full, m_full, _ = O.prefill(M, toks[0, :T])
        assert np.max(np.abs(logits[0, s] - lg_full)) < 1e-12
        dense = textbook.routed_dense_logits(w, toks[0, :T], m_full, cfg.n_heads, cfg.head_dim, cfg.rms_eps)
        assert np.max(np.abs(logits[0, s] - dense[-1])) < 1e-12


def test_adaln_literal_cache_equals_compact_cache():
    cfg = synth.tiny_config(batch=2, prompt_len=10, steps=5, adaln=True)
    w = synth.make_weights(cfg)
    _, _, a, _ = _run(cfg, w, "compact")
    _, _, b, _ = _run(cfg, w, "literal")
    assert np.max(np.abs(a - b)) < 1e-12


# ---------------------------------------------------------------------------
# bf16 rounding mode of the oracle (the storage points of a bf16 implementation)
# ---------------------------------------------------------------------------

def _f32_from_bits(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def _bf16_by_definition(x32: float) -> float:
    """Nearest bfloat16 to a finite float32 value, ties to the even
    significand, found by comparing exact distances (fractions) to the two
    bfloat16 values that bracket it: the one with the low 16 bits of the
    float32 encoding cleared (toward zero) and the next one away from zero."""
    from fractions import Fraction
    b = int(np.float32(x32).view(np.uint32))
    lo = b & 0xFFFF0000
    if lo == b:
        return float(np.float32(x32))
    hi = lo + 0x10000
    x = Fraction(float(np.float32(x32)))
    vlo = Fraction(float(_f32_from_bits([lo])[0]))
    if (hi & 0x7FFFFFFF) >= 0x7F800000:      # the next one up is infinite
        top = Fraction(2) ** 128              # where the bf16 ladder would put it
        vhi = top if x > 0 else -top
    else:
        vhi = Fraction(float(_f32_from_bits([hi])[0]))
    dlo, dhi = abs(x - vlo), abs(vhi - x)
    if dlo < dhi or (dlo == dhi and ((lo >> 16) & 1) == 0):
        return float(vlo)
    return float(_f32_from_bits([hi])[0])


_BF16_EDGE_BITS = [
    0x3F808000, 0x3F818000, 0xBF808000, 0xBF818000,   # ties: 1 + 2^-8, 1 + 3 * 2^-8 and negatives
    0x3F807FFF, 0x3F808001, 0x3F817FFF, 0x3F818001,   # one float32 step either side of a tie
    0x3F7FFFFF, 0x3FFF8000, 0x3FFF7FFF, 0xBFFF8000,   # carries into the exponent (up to 1.0, 2.0)
    0x00000001, 0x00008000, 0x00018000, 0x00017FFF,   # subnormals: ties at 0 and at the first step
    0x80008000, 0x807FFFFF, 0x00800000, 0x007FFFFF,   # the normal / subnormal boundary
    0x7F7F7FFF, 0x7F7F8000, 0x7F7FFFFF, 0xFF7FFFFF,   # the largest values (the last two overflow)
    0x00000000, 0x80000000, 0x3F800000, 0x42F6E979,   # exact values and one arbitrary value
]


def test_round_bf16_against_definition_and_torch_cast():
    """The oracle's bf16 rounding is round-to-nearest-even: it equals the
    exact nearest-value definition on ties, near-ties, exponent carries,
    subnormals and overflow, and torch's float32 -> bfloat16 cast on those and
    on random float32 encodings."""
    import torch
    x = _f32_from_bits(_BF16_EDGE_BITS)
    got = O._round_bf16(x.astype(np.float64))
    want = np.array([_bf16_by_definition(v) for v in x])
    assert np.array_equal(got, want)
    torch_cast = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(got, torch_cast)
    assert got[0] == 1.0 and got[1] == 1.0 + 2 ** -6 and got[8] == 1.0 and got[9] == 2.0
    assert np.isinf(got[22]) and np.isinf(got[23])
    rng = np.random.default_rng(5)
    bits = rng.integers(0, 2 ** 32, size=200000, dtype=np.uint64).astype(np.uint32)
    bits = bits[(bits & 0x7F800000) != 0x7F800000]          # finite encodings
    r = _f32_from_bits(bits)
    got = O._round_bf16(r.astype(np.float64))
    assert np.array_equal(got, torch.from_numpy(r).to(torch.bfloat16).to(torch.float64).numpy())
    for v, g in zip(r[:300], got[:300]):
        assert g == _bf16_by_definition(v)


def test_round_bf16_of_float64_goes_through_float32():
    """A float64 value is rounded as the float32 value a kernel would hold: to
    float32 first, then to bf16 (1 + 2^-8 + 2^-30 is a float32 tie, so it goes
    to 1.0, where rounding the float64 value directly would give 1 + 2^-7)."""
    import torch
    x = np.array([1.0 + 2 ** -8 + 2 ** -30, -(1.0 + 2 ** -8 + 2 ** -30), 0.1, 1e-40, 3.0e38])
    want = torch.from_numpy(x).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O._round_bf16(x), want)
    assert O._round_bf16(x)[0] == 1.0


@pytest.mark.parametrize("variant", ["fixed3", "routed"])
def test_bf16_rounding_points_equal_library_casts(variant):
    """round_bf16=True rounds exactly where a bf16 implementation stores a
    value (projection inputs, q/k/v, attention output, SwiGLU product, the
    head's normalised input): it equals an independent PyTorch model that
    applies torch's bfloat16 cast at those points, and differs from the
    unrounded model."""
    import torch
    cfg = synth.tiny_config(max_loops=4, prompt_len=14)
    w = synth.make_weights(cfg)
    toks = synth.make_prompts(cfg)[0]
    kw = dict(route_rule=O.FIXED, fixed_depth=3) if variant == "fixed3" else {}
    M = _model(cfg, w, round_bf16=True, **kw)
    st, logits, m, _ = O.prefill(M, toks, all_logits=True)
    if variant == "fixed3":
        ref = textbook.tied_gpt_logits(w, toks, cfg.n_heads, cfg.head_dim, 3, cfg.rms_eps,
                                       rnd=textbook.bf16_cast)
    else:
        assert len(set(m.tolist())) >= 2
        ref = textbook.routed_dense_logits(w, toks, m, cfg.n_heads, cfg.head_dim, cfg.rms_eps,
                                           rnd=textbook.bf16_cast)
    assert np.max(np.abs(logits - ref)) < 1e-12
    _, plain, _, _ = O.prefill(_model(cfg, w, **kw), toks, all_logits=True)
    assert np.max(np.abs(plain - logits)) > 1e-5
    # the cached keys and values are bf16 values
    for i in range(M.R):
        for j in range(M.J):
            for a in (st.K[i][j], st.V[i][j]):
                f = a.astype(np.float32)
                assert np.array_equal(f.astype(np.float64), a)
                assert np.all((f.view(np.uint32) & 0xFFFF) == 0)


def test_bf16_rounding_mode_stays_close():
    cfg = synth.tiny_config(batch=1, prompt_len=12, steps=3)
    w = synth.make_weights(cfg)
    _, _, a, _ = _run(cfg, w)
    _, _, b, _ = _run(cfg, w, model_kw=dict(round_bf16=True))
    err = np.max(np.abs(a - b))
    assert 0 < err < 3e-2


def test_greedy_lowest_id_among_float32_maxima():
    """The greedy token is the lowest id among the maxima of the float32
    rounding of the logits (values equal after that rounding are ties)."""
    import torch
    lg = np.array([[0.1, 0.3, 0.3, -1.0],
                   [1.0, 1.0 + 1e-12, 0.5, 1.0],      # equal in float32: id 0
                   [-2.0, -1.0, -1.0 - 1e-9, -3.0],   # equal in float32: id 1
                   [0.0, 0.0, 0.0, 0.0],
                   [-np.inf, 5.0, np.inf, np.inf]])
    assert O.greedy(lg).tolist() == [1, 0, 1, 0, 2]
    rng = np.random.default_rng(9)
    big = rng.standard_normal((64, 32000))
    big[:, 17] = big[:, 4000] = big.max(axis=1) + 1.0      # two exact maxima per row
    assert np.array_equal(O.greedy(big), np.full(64, 17))
    r = np.round(rng.standard_normal((64, 1000)), 1)        # many ties
    assert np.array_equal(O.greedy(r), torch.argmax(torch.from_numpy(r.astype(np.float32)), -1).numpy())


# ---------------------------------------------------------------------------
# Synthetic inputs
# ---------------------------------------------------------------------------

def test_splitmix64_reference_vector():
    """Sequential SplitMix64 from state 1234567 (Vigna's reference output)."""
    x0 = np.uint64(1234567)
    with np.errstate(over="ignore"):
        states = x0 + np.arange(1, 6, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)
    out = synth._mix64(states.copy())
    assert [int(v) for v in out[:3]] == [6457827717110365317, 3203168211198807973,
                                         9817491932198370423]


def test_generators_are_prefix_stable_and_normal():
    a = synth.normal(7, 3, 10000)
    b = synth.normal(7, 3, 2 * (1 << 22) + 5)[:10000]
    assert np.array_equal(a, b)
    assert abs(b.mean()) < 0.05 and abs(b.std() - 1.0) < 0.05
    assert np.all(synth.round_to_bf16(np.array([1.0 + 2 ** -8], np.float32)) == 1.0)
    assert np.all(synth.round_to_bf16(np.array([1.0 + 3 * 2 ** -8], np.float32)) == 1.0 + 2 ** -6)
