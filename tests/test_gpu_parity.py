"""GPU parity: the HIP path through the C ABI against the oracle.

Bars: fp32 models - depth decisions and cache indices bit-exact, logits
max-abs <= 1e-4.  bf16 models - depth decisions whose router margin exceeds
1e-2 match (flip rate reported), logits max-abs <= 3e-2, cache indices equal
{t : m_t >= i} for the depths the GPU took.
"""
import numpy as np
import pytest

import synth
from tests import parity

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 3e-2
BF16_MARGIN = 1e-2


def _report(tag, **kv):
    print(f"[parity] {tag} " + " ".join(f"{k}={v}" for k, v in kv.items()), flush=True)


def _max_err(g, o):
    return float(np.max(np.abs(np.asarray(g, np.float64) - np.asarray(o, np.float64))))


def _all_depths(g: parity.GpuRun):
    """Depth of every token of every sequence, prompt then decode steps: [B][T+S]."""
    cols = [g.prefill_depths] + [d[:, None] for d in g.step_depths]
    return np.concatenate(cols, axis=1)


def _check_index_matches_depths(g: parity.GpuRun, R: int):
    dep = _all_depths(g)
    for b in range(dep.shape[0]):
        for i in range(R):
            want = np.flatnonzero(dep[b] >= i + 1)
            assert np.array_equal(g.stats["index"][b][i], want), (b, i)


def _f32_small(**kw):
    base = dict(name="f32-small", dtype="f32", vocab=300, d_model=64, n_heads=4, head_dim=16, d_ff=128,
                n_layers=2, max_loops=4, batch=3, prompt_len=37, steps=19, router_bias="zero")
    base.update(kw)
    return synth.ModelConfig(**base)


def _oracle_depths(o: parity.OracleRun):
    """The oracle's depth of every token, prompt then decode steps: [B][T+S]."""
    return np.concatenate([o.prefill_depths] + [d[:, None] for d in o.step_depths], axis=1)


def _oracle_margins(o: parity.OracleRun):
    return np.concatenate([o.prefill_margin] + [mg[:, None] for mg in o.step_margin], axis=1)


def _check_f32(m, w, prompts, g, o, tag):
    assert np.array_equal(g.prefill_depths, o.prefill_depths)
    for s in range(len(g.step_depths)):
        assert np.array_equal(g.step_depths[s], o.step_depths[s]), s
    err = _max_err(g.prefill_logits, o.prefill_logits)
    for s in range(len(g.step_logits)):
        err = max(err, _max_err(g.step_logits[s], o.step_logits[s]))
    for b in range(prompts.shape[0]):
        for i in range(m.max_loops):
            assert np.array_equal(g.stats["index"][b][i], o.index[b][i]), (b, i)
    for s in range(len(g.step_next)):
        assert np.array_equal(g.step_next[s], np.argmax(g.step_logits[s], axis=-1))
    _report(tag, max_abs_logit_err=f"{err:.3g}", steps=len(g.step_logits),
            depth_hist=g.stats["depth_hist"])
    assert err <= F32_TOL
    assert np.all(np.isfinite(g.prefill_logits))


def _check_f32_near_ties(m, w, prompts, g, o, tag, tie_margin=1e-5):
    """For depth rules whose decisions can sit at a near tie (the cumulative
    rule, an MLP router): every decision, prompt and decode steps, that differs
    from the oracle's has an oracle margin <= tie_margin; every sequence whose
    whole depth stream equals the oracle's is checked like _check_f32 (logits,
    cache index), and at least one sequence is.  Greedy ids equal the first
    argmax of the GPU's own logits everywhere."""
    gd, od, om = _all_depths(g), _oracle_depths(o), _oracle_margins(o)
    differ = gd != od
    assert np.all(om[differ] <= tie_margin), om[differ]
    same = [b for b in range(prompts.shape[0]) if not differ[b].any()]
    assert len(same) >= 1, "no sequence with the oracle's depth stream"
    err = 0.0
    for b in same:
        err = max(err, _max_err(g.prefill_logits[b], o.prefill_logits[b]))
        for s in range(len(g.step_logits)):
            err = max(err, _max_err(g.step_logits[s][b], o.step_logits[s][b]))
        for i in range(m.max_loops):
            assert np.array_equal(g.stats["index"][b][i], o.index[b][i]), (b, i)
    _check_index_matches_depths(g, m.max_loops)
    for s in range(len(g.step_next)):
        assert np.array_equal(g.step_next[s], np.argmax(g.step_logits[s], axis=-1))
    _report(tag, compared_sequences=f"{len(same)}/{prompts.shape[0]}", near_tie_flips=int(differ.sum()),
            max_abs_logit_err=f"{err:.3g}", depth_hist=g.stats["depth_hist"])
    assert err <= F32_TOL
    assert np.all(np.isfinite(g.prefill_logits))


def test_f32_tiny_decode_parity():
    m = synth.CONFIGS["f32_tiny_b1x32"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps)
    o = parity.run_oracle(m, w, prompts, g.step_tokens)
    _check_f32(m, w, prompts, g, o, "f32_tiny_b1x32")
    # the oracle's own greedy choice agrees wherever its top-2 gap exceeds the tolerance
    for s in range(m.steps):
        lo = o.step_logits[s]
        srt = np.sort(lo, axis=-1)
        clear = (srt[:, -1] - srt[:, -2]) > 2 * F32_TOL
        assert np.all(g.step_next[s][clear] == np.argmax(lo, axis=-1)[clear])


def test_f32_tiny_prefill_all_positions():
    m = synth.CONFIGS["f32_tiny_b1x32"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, 0, all_logits=True, max_pos=m.max_pos)
    o = parity.run_oracle(m, w, prompts, [], all_logits=True)
    err = _max_err(g.prefill_logits, o.prefill_logits)
    _report("f32_tiny-all-logits", max_abs_logit_err=f"{err:.3g}")
    assert err <= F32_TOL


def test_f32_two_layers_ragged_batch():
    m = _f32_small()
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps)
    o = parity.run_oracle(m, w, prompts, g.step_tokens)
    _check_f32(m, w, prompts, g, o, "f32-small")


def test_f32_batch_over_head_gemm_rows():
    """A decode batch of 130 rows runs the LM head on the 128 x 128 GEMM with
    the norm fused: two row tiles, the second with 2 rows."""
    m = _f32_small(batch=130, prompt_len=9, steps=4, vocab=300)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps)
    o = parity.run_oracle(m, w, prompts, g.step_tokens)
    _check_f32(m, w, prompts, g, o, "f32-b130")


def test_f32_batch_over_planner_threads():
    """1100 sequences: the decode planner's second chunk of sequences (past
    its 1024 threads) reads its cache lengths and page-table entries where it
    uses them.  Every sequence's cache index is checked against its depths;
    four sampled sequences against the oracle."""
    m = _f32_small(batch=1100, prompt_len=6, steps=5, vocab=300)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    sample = [0, 511, 1024, 1099]
    g = parity.run_gpu(m, w, prompts, m.steps, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    assert np.array_equal(g.prefill_depths[sample], o.prefill_depths)
    for s in range(m.steps):
        assert np.array_equal(g.step_depths[s][sample], o.step_depths[s]), s
    _check_index_matches_depths(g, m.max_loops)
    hist = np.bincount(_all_depths(g).ravel(), minlength=m.max_loops + 1)[1:]
    assert np.array_equal(np.asarray(g.stats["depth_hist"]), hist)
    err = _max_err(g.prefill_logits, o.prefill_logits)
    for s in range(m.steps):
        err = max(err, _max_err(g.step_logits[s], o.step_logits[s]))
    _report("f32-b1100", max_abs_logit_err=f"{err:.3g}")
    assert err <= F32_TOL


def test_f32_single_token_prompt_and_deep_tail():
    m = _f32_small(batch=2, prompt_len=1, steps=40)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps)
    o = parity.run_oracle(m, w, prompts, g.step_tokens)
    _check_f32(m, w, prompts, g, o, "f32-T1")


def test_f32_cumprob_rule():
    m = _f32_small(steps=10)
    w = dict(synth.make_weights(m))
    w["router_w"] = (w["router_w"] * 150.0).astype(np.float32)  # spread the routing distribution
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps, route_rule="cumprob", threshold=0.5)
    o = parity.run_oracle(m, w, prompts, g.step_tokens, route_rule="cumprob", threshold=0.5)
    assert len(set(g.prefill_depths.ravel().tolist())) >= 3
    _check_f32_near_ties(m, w, prompts, g, o, "cumprob")


@pytest.mark.parametrize("depth", [1, 4])
def test_f32_fixed_depth(depth):
    m = _f32_small(steps=8)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps, route_rule="fixed", fixed_depth=depth)
    o = parity.run_oracle(m, w, prompts, g.step_tokens, route_rule="fixed", fixed_depth=depth)
    assert np.all(g.prefill_depths == depth)
    _check_f32(m, w, prompts, g, o, f"fixed{depth}")


@pytest.mark.parametrize("head_dim", [64, 128])
def test_f32_wide_heads(head_dim):
    """fp32 kernels at head_dim 64 and 128; the 128 case also uses an untied LM head."""
    m = _f32_small(d_model=2 * head_dim, n_heads=2, head_dim=head_dim, d_ff=192, batch=2, prompt_len=45,
                   steps=10)
    w = dict(synth.make_weights(m))
    if head_dim == 128:
        w["lm_head"] = synth.make_lm_head(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps)
    o = parity.run_oracle(m, w, prompts, g.step_tokens)
    _check_f32(m, w, prompts, g, o, f"f32-D{head_dim}")


@pytest.mark.parametrize("rule", ["argmax", "cumprob", "argmax-B1"])
def test_f32_mlp_router(rule):
    """Two-layer MLP router (hidden 64): decisions differ from the oracle's only
    at near ties; sequences with the oracle's depths match it at the fp32 bar."""
    batch = 1 if rule.endswith("-B1") else 3
    rule = rule.split("-")[0]
    m = _f32_small(router_hidden=64, router_bias="calibrated", steps=10, batch=batch, prompt_len=37 * (4 - batch))
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps, route_rule=rule, threshold=0.5)
    o = parity.run_oracle(m, w, prompts, g.step_tokens, route_rule=rule, threshold=0.5)
    assert len(set(g.prefill_depths.ravel().tolist())) >= 2
    _check_f32_near_ties(m, w, prompts, g, o, f"mlp-router-{rule}")


def test_prefill_in_sequence_groups_is_identical():
    """Groups of two sequences give bitwise the one-group results; a group of
    one sequence (the few-row projections, another summation order) agrees to
    the fp32 bar."""
    m = _f32_small(batch=6, prompt_len=40, steps=3)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    a = parity.run_gpu(m, w, prompts, m.steps)
    b = parity.run_gpu(m, w, prompts, m.steps, max_prefill_tokens=2 * m.prompt_len)
    assert np.array_equal(a.prefill_logits, b.prefill_logits)
    for s in range(m.steps):
        assert np.array_equal(a.step_logits[s], b.step_logits[s])
    c = parity.run_gpu(m, w, prompts, m.steps, max_prefill_tokens=m.prompt_len)
    assert np.array_equal(a.prefill_depths, c.prefill_depths)
    err = max([_max_err(a.prefill_logits, c.prefill_logits)] +
              [_max_err(a.step_logits[s], c.step_logits[s]) for s in range(m.steps)])
    assert err <= F32_TOL


def test_fp32_runs_are_bitwise_deterministic():
    m = synth.CONFIGS["f32_tiny_b1x32"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    a = parity.run_gpu(m, w, prompts, 8)
    b = parity.run_gpu(m, w, prompts, 8)
    for s in range(8):
        assert np.array_equal(a.step_logits[s], b.step_logits[s])


@pytest.mark.parametrize("name", ["f32_tiny_b1x32", "f32-small", "bf16_d768-small"])
def test_graph_replays_match_eager_launches(name):
    """Decode steps replayed from the captured HIP graph equal eager launches,
    every replay, with host reads (eager work and a sync) between replays."""
    if name == "f32_tiny_b1x32":
        m = synth.CONFIGS["f32_tiny_b1x32"]
    elif name == "f32-small":
        m = _f32_small(steps=12)
    else:
        m = synth.CONFIGS["bf16_d768_b32x512"].replace(batch=6, prompt_len=80, steps=12)
    w = synth.make_weights(m if name != "bf16_d768-small" else synth.CONFIGS["bf16_d768_b32x512"])
    prompts = synth.make_prompts(m)
    steps = min(m.steps, 12)
    g = parity.run_gpu(m, w, prompts, steps, max_pos=m.max_pos, decode_graph=True)
    e = parity.run_gpu(m, w, prompts, steps, max_pos=m.max_pos, decode_graph=False)
    for s in range(steps):
        assert np.array_equal(g.step_tokens[s], e.step_tokens[s]), s
        assert np.array_equal(g.step_logits[s], e.step_logits[s]), s
        assert np.array_equal(g.step_depths[s], e.step_depths[s]), s
    for b in range(prompts.shape[0]):
        for i in range(m.max_loops):
            assert np.array_equal(g.stats["index"][b][i], e.stats["index"][b][i])


def test_graph_cache_replays_and_evicts():
    """Greedy decode into two alternating token buffers replays two cached
    graphs; then five distinct logits buffers in turn make every step replace
    the least recently used of the four cached graphs, and a return to an
    earlier buffer set replays it.  Every step equals kernel-by-kernel launches."""
    import torch
    from paper_2609_15160_amd import tlf
    m = _f32_small(steps=24)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    B, V, steps = prompts.shape[0], m.vocab, 24
    # buffer set of each step: ping-pong tokens, then logits buffers 0..4 in turn, then set 1 again
    logit_ids = [0] * 8 + [k % 5 for k in range(12)] + [1, 2, 1, 2]

    def run(graph):
        sess = tlf.Session(m, w, max_batch=B, max_pos=prompts.shape[1] + steps, decode_graph=graph)
        try:
            lg, _ = sess.prefill(torch.from_numpy(prompts.astype(np.int32)).cuda())
            tok = [torch.argmax(lg, -1).to(torch.int32).contiguous(), torch.empty(B, dtype=torch.int32, device="cuda")]
            outs = [torch.empty((B, V), dtype=torch.float32, device="cuda") for _ in range(5)]
            got = []
            for k in range(steps):
                out = outs[logit_ids[k]]
                sess.decode_into(tok[k % 2], out, next_tok=tok[(k + 1) % 2])
                got.append(out.cpu().numpy().copy())  # a host read between replays
            assert sess.stats()["status"] == 0
            return got
        finally:
            sess.close()

    g, e = run(True), run(False)
    for k in range(steps):
        assert np.array_equal(g[k], e[k]), k


def _check_bf16(m, w, prompts, g, o, sample, tag, route_rule="argmax", fixed_depth=None, threshold=0.5):
    """bf16 bar.  Every token's depth (all sequences, prompt and decode steps)
    against the oracle router: decisions with margin > 1e-2 match.  Every
    cache index equals {t : m_t >= i} for the GPU's depths.  On the sampled
    sequences (the oracle's rows): the greedy id is the first argmax of the
    GPU's own logits at every step; each sampled sequence whose depth stream
    equals the oracle's has logits within 3e-2 and the oracle's cache index,
    and at least one sampled sequence is compared."""
    B, T = prompts.shape
    # router decisions of every token against the oracle router
    pos = np.broadcast_to(np.arange(T), (B, T))
    od, om = parity.router_decisions(m, w, prompts.ravel(), pos.ravel(), route_rule, threshold=threshold,
                                     fixed_depth=fixed_depth)
    bad, flips = parity.depth_agreement(g.prefill_depths.ravel(), od, om, BF16_MARGIN)
    nbad, nflips = 0, []
    for s, tok in enumerate(g.step_tokens):
        sd, sm = parity.router_decisions(m, w, tok, np.full(B, T + s), route_rule, threshold=threshold,
                                         fixed_depth=fixed_depth)
        b2, f2 = parity.depth_agreement(g.step_depths[s], sd, sm, BF16_MARGIN)
        nbad += b2
        nflips.append(f2)
    assert bad == 0 and nbad == 0
    _check_index_matches_depths(g, m.max_loops)
    for s in range(len(g.step_next)):
        assert np.array_equal(g.step_next[s][sample], np.argmax(g.step_logits[s], axis=-1)), s
    gd, odep = _all_depths(g), _oracle_depths(o)
    same = [j for j, b in enumerate(sample) if np.array_equal(gd[b], odep[j])]
    assert len(same) >= 1, "no sampled sequence with the oracle's depth stream"
    err = 0.0
    for j in same:
        err = max(err, _max_err(g.prefill_logits[j], o.prefill_logits[j]))
        for s in range(len(g.step_logits)):
            err = max(err, _max_err(g.step_logits[s][j], o.step_logits[s][j]))
        for i in range(m.max_loops):
            assert np.array_equal(g.stats["index"][sample[j]][i], o.index[j][i]), (sample[j], i)
    agree = np.mean([np.mean(g.step_next[s][sample] == np.argmax(o.step_logits[s], -1))
                     for s in range(len(g.step_next))]) if g.step_next else 1.0
    _report(tag, max_abs_logit_err=f"{err:.3g}", compared_sequences=f"{len(same)}/{len(sample)}",
            prefill_flip_rate=flips, decode_flip_rate=float(np.mean(nflips)) if nflips else 0.0,
            greedy_agreement=f"{agree:.3f}", depth_hist=g.stats["depth_hist"])
    assert err <= BF16_TOL
    assert np.all(np.isfinite(g.prefill_logits))


def test_bf16_d768_b32x512_parity_sampled_sequences():
    m = synth.CONFIGS["bf16_d768_b32x512"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    steps = 12
    sample = [0, 13, 31]
    g = parity.run_gpu(m, w, prompts, steps, max_pos=m.max_pos, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16_d768_b32x512")


def test_bf16_fixed_depth_ragged_prompt():
    m = synth.CONFIGS["bf16_d768_b32x512"].replace(batch=4, prompt_len=77, steps=6)
    w = synth.make_weights(synth.CONFIGS["bf16_d768_b32x512"])
    prompts = synth.make_prompts(m)
    sample = [1, 3]
    g = parity.run_gpu(m, w, prompts, m.steps, route_rule="fixed", fixed_depth=8, max_pos=m.max_pos,
                       keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens], route_rule="fixed",
                          fixed_depth=8)
    assert np.all(g.prefill_depths == 8)
    _check_bf16(m, w, prompts, g, o, sample, "bf16-fixed8", route_rule="fixed", fixed_depth=8)


@pytest.mark.parametrize("rule,threshold", [("argmax", 0.5), ("cumprob", 0.6)])
def test_bf16_mlp_router(rule, threshold):
    """The 2x768 model with a 768-wide MLP router on a ragged small batch."""
    full = synth.CONFIGS["bf16_d768_b32x512"].replace(router_hidden=768)
    m = full.replace(batch=6, prompt_len=70, steps=8)
    w = synth.make_weights(full)
    prompts = synth.make_prompts(m)
    sample = [0, 3, 5]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample, route_rule=rule,
                       threshold=threshold)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens], route_rule=rule,
                          threshold=threshold)
    _check_bf16(m, w, prompts, g, o, sample, f"bf16-mlp-router-{rule}", route_rule=rule, threshold=threshold)


@pytest.mark.slow
def test_bf16_d768_b256x2048_sampled_sequences():
    """The benchmark's workload (batch 256 x 2048 prompt) with the oracle on two sequences."""
    m = synth.CONFIGS["bf16_d768_b256x2048"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    steps = 3
    sample = [0, 255]
    g = parity.run_gpu(m, w, prompts, steps, max_pos=m.max_pos, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16_d768_b256x2048")


@pytest.mark.slow
@pytest.mark.timeout(900)
def test_bf16_d1024_prefill_b8x4096_sampled_sequences():
    """The prefill workload's own shape (d 1024, 16 x 64 heads, SwiGLU 2816,
    R 8, J 2) at batch 8 x 4096 in one 32768-row group, with the activations
    entering the prefill's matrix products as one bf16 part, as the benchmark
    runs it (Section 3.3 batched prefill, Eq. 6-7, 10-11): every token's depth,
    every cache index, the last-position logits of two sequences against the
    oracle, then three decode steps."""
    m = synth.CONFIGS["bf16_d1024_prefill_b8x4096"].replace(steps=3)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    sample = [0, 7]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample,
                       max_prefill_tokens=m.batch * m.prompt_len, prefill_act_bf16=True)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens], threads=2)
    _check_bf16(m, w, prompts, g, o, sample, "bf16_d1024_prefill_b8x4096")


def test_bf16_prefill_single_part_activations_d768():
    """The one-part bf16 prefill activations on the 2x768 model: three
    sequences of 300 tokens (the many-row prefill GEMM and attention), all
    positions' logits and eight decode steps against the oracle."""
    full = synth.CONFIGS["bf16_d768_b32x512"]
    m = full.replace(batch=3, prompt_len=300, steps=8)
    w = synth.make_weights(full)
    prompts = synth.make_prompts(m)
    sample = [0, 2]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample, prefill_act_bf16=True)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16-prefill-one-part-d768")


def test_bf16_prefill_single_part_ragged_wide_tiles():
    """One-part bf16 prefill activations on a model whose widths leave ragged
    256-column tiles (d 640 = 5 x 128 heads, QKV 1920 columns, SwiGLU 1664)
    with 4 x 1100 rows, enough for the 256 x 256 GEMM tiles; all sequences'
    last-position logits and four decode steps against the oracle."""
    m = synth.ModelConfig("bf16-d640", "bf16", vocab=5000, d_model=640, n_heads=5, head_dim=128, d_ff=1664,
                          n_layers=2, max_loops=6, batch=4, prompt_len=1100, steps=4, router_bias="calibrated")
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    sample = [0, 1, 2, 3]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample, prefill_act_bf16=True)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens], threads=4)
    _check_bf16(m, w, prompts, g, o, sample, "bf16-prefill-one-part-d640")


def test_bf16_d2048_heads_of_128_small_batch():
    """The d=2048 model (16 heads x 128) on a short ragged prompt: bf16 kernels at head_dim 128."""
    full = synth.CONFIGS["bf16_d2048_b64x4096"]
    m = full.replace(batch=5, prompt_len=70, steps=8)
    w = synth.make_weights(full)
    prompts = synth.make_prompts(m)
    sample = [0, 2, 4]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16_d2048-small")


@pytest.mark.slow
def test_bf16_d2048_b64x4096_sampled_sequences():
    """The d=2048 model at batch 64 x 4096 prompt with the oracle on one sequence."""
    m = synth.CONFIGS["bf16_d2048_b64x4096"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    steps = 3
    sample = [63]
    g = parity.run_gpu(m, w, prompts, steps, max_pos=m.max_pos, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16_d2048_b64x4096")


# ---------------------------------------------------------------------------
# Chunked prefill: prompt chunks appended to the caches, mixed with decode steps
# ---------------------------------------------------------------------------

# chunk sizes off the 16-token pages and the 64-row tiles; a chunk of one token;
# decode steps between chunks (a graph captured before a chunk replays after it)
SCHEDULE = [("prefill", 37), ("prefill", 1), ("prefill", 70), ("prefill", 12), ("decode", 5),
            ("prefill", 9), ("decode", 3)]


def _schedule_len(schedule):
    return sum(n for _, n in schedule)


def _oracle_one_shot(m, w, tokens, **kw):
    return parity.run_oracle(m, w, tokens, [], all_logits=True, **kw)


@pytest.mark.parametrize("head_dim,batch", [(16, 3), (64, 3), (16, 1), (64, 1)])
def test_f32_chunked_prefill_equals_one_shot(head_dim, batch):
    """Every position's logits and depth from a schedule of appended chunks and
    decode steps equal one oracle prefill over the whole token sequence.  A
    single sequence takes the few-row prefill projections."""
    L = _schedule_len(SCHEDULE)
    m = _f32_small(batch=batch, prompt_len=L, steps=0)
    if head_dim == 64:
        m = m.replace(n_heads=2, head_dim=64, d_model=128)
    w = synth.make_weights(m)
    tokens = synth.make_prompts(m, prompt_len=L)
    g = parity.run_gpu_schedule(m, w, tokens, SCHEDULE)
    o = _oracle_one_shot(m, w, tokens)
    assert np.array_equal(g.depths, o.prefill_depths)
    for b in range(tokens.shape[0]):
        for i in range(m.max_loops):
            assert np.array_equal(g.stats["index"][b][i], o.index[b][i]), (b, i)
    err = _max_err(g.logits, o.prefill_logits)
    _report(f"f32-chunked-D{head_dim}-B{batch}", max_abs_logit_err=f"{err:.3g}", depth_hist=g.stats["depth_hist"])
    assert err <= F32_TOL


def test_f32_chunked_prefill_in_sequence_groups():
    """Appended chunks that run in sequence groups (small activation budget)."""
    sched = [("prefill", 40), ("prefill", 23), ("decode", 2), ("prefill", 17)]
    L = _schedule_len(sched)
    m = _f32_small(batch=5, prompt_len=L, steps=0)
    w = synth.make_weights(m)
    tokens = synth.make_prompts(m, prompt_len=L)
    g = parity.run_gpu_schedule(m, w, tokens, sched, max_prefill_tokens=2 * L)
    o = _oracle_one_shot(m, w, tokens)
    assert np.array_equal(g.depths, o.prefill_depths)
    err = _max_err(g.logits, o.prefill_logits)
    _report("f32-chunked-groups", max_abs_logit_err=f"{err:.3g}")
    assert err <= F32_TOL


@pytest.mark.parametrize("batch,one_part", [(3, False), (1, False), (3, True)])
def test_bf16_chunked_prefill_equals_one_shot(batch, one_part):
    """Appended chunks and decode steps against one oracle prefill; with
    one_part the multi-sequence chunks feed their activations as one bf16
    part (queries attending over cache entries of earlier chunks)."""
    m = synth.CONFIGS["bf16_d768_b32x512"].replace(batch=batch)
    w = synth.make_weights(synth.CONFIGS["bf16_d768_b32x512"])
    sched = [("prefill", 100), ("prefill", 29), ("prefill", 200), ("decode", 4), ("prefill", 33)]
    L = _schedule_len(sched)
    tokens = synth.make_prompts(m, prompt_len=L)
    g = parity.run_gpu_schedule(m, w, tokens, sched, prefill_act_bf16=one_part)
    o = _oracle_one_shot(m, w, tokens)
    B = tokens.shape[0]
    pos = np.broadcast_to(np.arange(L), (B, L))
    od, om = parity.router_decisions(m, w, tokens.ravel(), pos.ravel())
    bad, flips = parity.depth_agreement(g.depths.ravel(), od, om, BF16_MARGIN)
    err = _max_err(g.logits, o.prefill_logits)
    _report(f"bf16-chunked-B{batch}{'-one-part' if one_part else ''}", max_abs_logit_err=f"{err:.3g}",
            flip_rate=flips, depth_hist=g.stats["depth_hist"])
    assert bad == 0
    for b in range(B):
        for i in range(m.max_loops):
            assert np.array_equal(g.stats["index"][b][i], np.flatnonzero(g.depths[b] >= i + 1)), (b, i)
    assert err <= BF16_TOL


# ---------------------------------------------------------------------------
# Gather-scatter off (dense decode): every row runs every loop, results discarded
# for exited rows; the outputs are the gathered path's
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("prompt_len", [37, 1])
def test_f32_dense_decode_equals_oracle(prompt_len):
    """A one-token prompt leaves loop caches empty for rows that run a loop
    their token exited: their attention output is discarded."""
    m = _f32_small(prompt_len=prompt_len, steps=16 if prompt_len > 1 else 30)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps, dense_decode=True)
    o = parity.run_oracle(m, w, prompts, g.step_tokens)
    _check_f32(m, w, prompts, g, o, f"f32-dense-T{prompt_len}")
    top = int(g.step_depths[-1].max())
    assert g.stats["last_step_active_rows"] == [m.batch] * top + [0] * (m.max_loops - top)


def test_bf16_dense_decode_sampled_sequences():
    m = synth.CONFIGS["bf16_d768_b32x512"].replace(batch=8, prompt_len=96, steps=10)
    w = synth.make_weights(synth.CONFIGS["bf16_d768_b32x512"])
    prompts = synth.make_prompts(m)
    sample = [0, 5]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample, dense_decode=True)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16-dense")


# ---------------------------------------------------------------------------
# AdaLN time/step conditioning: every row gathers the modulation of its own
# (loop, depth) pair
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("variant", ["routed", "fixed4", "dense", "single-sequence"])
def test_f32_adaln_parity(variant):
    kw = dict(adaln=True, steps=12)
    if variant == "single-sequence":
        kw.update(batch=1, prompt_len=90)
    m = _f32_small(**kw)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    rule = dict(route_rule="fixed", fixed_depth=4) if variant == "fixed4" else {}
    g = parity.run_gpu(m, w, prompts, m.steps, dense_decode=variant == "dense", **rule)
    o = parity.run_oracle(m, w, prompts, g.step_tokens, **rule)
    _check_f32(m, w, prompts, g, o, f"f32-adaln-{variant}")


def test_f32_adaln_chunked_prefill_equals_one_shot():
    L = _schedule_len(SCHEDULE)
    m = _f32_small(batch=2, prompt_len=L, steps=0, adaln=True)
    w = synth.make_weights(m)
    tokens = synth.make_prompts(m, prompt_len=L)
    g = parity.run_gpu_schedule(m, w, tokens, SCHEDULE)
    o = _oracle_one_shot(m, w, tokens)
    assert np.array_equal(g.depths, o.prefill_depths)
    err = _max_err(g.logits, o.prefill_logits)
    _report("f32-adaln-chunked", max_abs_logit_err=f"{err:.3g}")
    assert err <= F32_TOL


def test_bf16_adaln_prefill_single_part():
    """AdaLN with one-part bf16 prefill activations: the QKV and gate/up rows
    carry the (1 + gamma) scale, so they are rounded in LDS from the float
    rows; O and down read bf16 rows and gate with (1 + alpha)."""
    base = synth.CONFIGS["bf16_d768_b32x512"].replace(adaln=True)
    m = base.replace(batch=4, prompt_len=200, steps=6)
    w = synth.make_weights(base)
    prompts = synth.make_prompts(m)
    sample = [0, 3]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample, prefill_act_bf16=True)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, "bf16-adaln-one-part")


@pytest.mark.parametrize("batch", [8, 1])
def test_bf16_adaln_sampled_sequences(batch):
    base = synth.CONFIGS["bf16_d768_b32x512"].replace(adaln=True)
    m = base.replace(batch=batch, prompt_len=96, steps=10)
    w = synth.make_weights(base)
    prompts = synth.make_prompts(m)
    sample = [0, 5] if batch > 1 else [0]
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=m.max_pos, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    _check_bf16(m, w, prompts, g, o, sample, f"bf16-adaln-B{batch}")


# ---------------------------------------------------------------------------
# Maximum sizes
# ---------------------------------------------------------------------------

def test_f32_max_batch():
    """TLF_MAX_BATCH = 4096 sequences: the decode planner's four chunks of
    sequences, the many-row LM head; every sequence's depths and cache index,
    three sampled sequences against the oracle."""
    from paper_2609_15160_amd import tlf
    m = _f32_small(batch=tlf.MAX_BATCH, prompt_len=5, steps=3, vocab=300)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    sample = [0, 2047, tlf.MAX_BATCH - 1]
    g = parity.run_gpu(m, w, prompts, m.steps, keep_logits_rows=sample)
    o = parity.run_oracle(m, w, prompts[sample], [t[sample] for t in g.step_tokens])
    assert np.array_equal(g.prefill_depths[sample], o.prefill_depths)
    for s in range(m.steps):
        assert np.array_equal(g.step_depths[s][sample], o.step_depths[s]), s
        assert np.array_equal(g.step_next[s][sample], np.argmax(g.step_logits[s], axis=-1))
    _check_index_matches_depths(g, m.max_loops)
    err = max([_max_err(g.prefill_logits, o.prefill_logits)] +
              [_max_err(g.step_logits[s], o.step_logits[s]) for s in range(m.steps)])
    _report("f32-max-batch", max_abs_logit_err=f"{err:.3g}")
    assert err <= F32_TOL


def test_f32_max_cache_length_properties():
    """max_pos = 65536, the longest cache whose page list the decode
    attention stages (4096 pages): a 65528-token prompt and 8 decode steps of
    the tiny model.  The oracle cannot replay a prefill this long, so the
    checks are properties that hold at any size: every depth equals the
    oracle router's (fp32: bit-exact), every cache index equals
    {t : m_t >= i}, logits are finite and the greedy id is their first
    argmax."""
    m = synth.CONFIGS["f32_tiny_b1x32"].replace(prompt_len=65528, steps=8)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    g = parity.run_gpu(m, w, prompts, m.steps, max_pos=65536)
    pos = np.arange(m.prompt_len)
    od, _ = parity.router_decisions(m, w, prompts[0], pos)
    assert np.array_equal(g.prefill_depths[0], od)
    for s in range(m.steps):
        sd, _ = parity.router_decisions(m, w, g.step_tokens[s], np.array([m.prompt_len + s]))
        assert np.array_equal(g.step_depths[s], sd), s
        assert np.all(np.isfinite(g.step_logits[s]))
        assert np.array_equal(g.step_next[s], np.argmax(g.step_logits[s], axis=-1))
    _check_index_matches_depths(g, m.max_loops)
    assert np.all(np.isfinite(g.prefill_logits))
    assert g.stats["seq_len"] == 65536
    _report("f32-max-cache", depth_hist=g.stats["depth_hist"])


# ---------------------------------------------------------------------------
# Error handling through the C ABI
# ---------------------------------------------------------------------------

def _session(m, w, **kw):
    from paper_2609_15160_amd import tlf
    return tlf.Session(m, w, **kw)


def test_state_errors():
    import torch
    from paper_2609_15160_amd import tlf
    m = _f32_small(batch=2, prompt_len=5, steps=2)
    w = synth.make_weights(m)
    s = _session(m, w, max_batch=2, max_pos=7)
    try:
        tok = torch.zeros(2, dtype=torch.int32, device="cuda")
        with pytest.raises(tlf.TlfError) as e:
            s.decode(tok)
        assert e.value.status == tlf.E_STATE
        with pytest.raises(tlf.TlfError) as e:
            s.prefill(torch.zeros((3, 5), dtype=torch.int32, device="cuda"))  # batch > max_batch
        assert e.value.status == tlf.E_INVALID_ARG
        s.prefill(torch.zeros((2, 5), dtype=torch.int32, device="cuda"))
        s.decode(tok)
        s.decode(tok)
        with pytest.raises(tlf.TlfError) as e:  # position 7 == max_pos
            s.decode(tok)
        assert e.value.status == tlf.E_STATE
        assert s.stats()["status"] == tlf.OK
    finally:
        s.close()


def test_append_errors():
    import torch
    from paper_2609_15160_amd import tlf
    m = _f32_small(batch=2, prompt_len=5, steps=4)
    w = synth.make_weights(m)
    s = _session(m, w, max_batch=2, max_pos=9)
    try:
        z = lambda b, t: torch.zeros((b, t), dtype=torch.int32, device="cuda")
        with pytest.raises(tlf.TlfError) as e:  # nothing to append to
            s.prefill(z(2, 3), append=True)
        assert e.value.status == tlf.E_STATE
        s.prefill(z(2, 5))
        with pytest.raises(tlf.TlfError) as e:  # another batch size
            s.prefill(z(1, 2), append=True)
        assert e.value.status == tlf.E_INVALID_ARG
        with pytest.raises(tlf.TlfError) as e:  # 5 + 5 > max_pos
            s.prefill(z(2, 5), append=True)
        assert e.value.status == tlf.E_INVALID_ARG
        s.prefill(z(2, 4), append=True)  # exactly max_pos
        assert s.seq_len == 9 and s.stats()["seq_len"] == 9
        with pytest.raises(tlf.TlfError) as e:
            s.decode(torch.zeros(2, dtype=torch.int32, device="cuda"))
        assert e.value.status == tlf.E_STATE
        assert s.stats()["status"] == tlf.OK
    finally:
        s.close()


def test_out_of_pages_detected():
    import torch
    from paper_2609_15160_amd import tlf
    m = _f32_small(batch=1, prompt_len=32, steps=8, max_loops=2)
    w = synth.make_weights(m)
    s = _session(m, w, max_batch=1, max_pos=40, max_pages=1, route_rule="fixed", fixed_depth=2)
    try:
        with pytest.raises(tlf.TlfError) as e:  # 32 tokens fill two pages in loop 1 alone
            s.prefill(torch.zeros((1, 32), dtype=torch.int32, device="cuda"))
        assert e.value.status == tlf.E_OUT_OF_PAGES
    finally:
        s.close()
    # exactly enough pages for the prefill (2 loops x 1 page); the first decode step needs two more
    s = _session(m, w, max_batch=1, max_pos=18, max_pages=2, route_rule="fixed", fixed_depth=2)
    try:
        s.prefill(torch.zeros((1, 16), dtype=torch.int32, device="cuda"))
        assert s.stats()["status"] == tlf.OK
        s.decode(torch.zeros(1, dtype=torch.int32, device="cuda"))
        st = s.stats()
        assert st["status"] == tlf.E_OUT_OF_PAGES
        with pytest.raises(tlf.TlfError) as e:
            s.decode(torch.zeros(1, dtype=torch.int32, device="cuda"))
        assert e.value.status == tlf.E_OUT_OF_PAGES
    finally:
        s.close()


def test_out_of_pages_on_append_detected():
    import torch
    from paper_2609_15160_amd import tlf
    m = _f32_small(batch=1, prompt_len=16, steps=4, max_loops=2)
    w = synth.make_weights(m)
    # the 16-token prompt fills one page per loop; one more token needs two more pages
    s = _session(m, w, max_batch=1, max_pos=20, max_pages=2, route_rule="fixed", fixed_depth=2)
    try:
        s.prefill(torch.zeros((1, 16), dtype=torch.int32, device="cuda"))
        assert s.stats()["status"] == tlf.OK
        s.prefill(torch.zeros((1, 1), dtype=torch.int32, device="cuda"), append=True)
        assert s.stats()["status"] == tlf.E_OUT_OF_PAGES
    finally:
        s.close()


def test_bad_token_reported():
    import torch
    from paper_2609_15160_amd import tlf
    m = _f32_small(batch=1, prompt_len=4, steps=1)
    w = synth.make_weights(m)
    s = _session(m, w, max_batch=1, max_pos=5)
    try:
        s.prefill(torch.zeros((1, 4), dtype=torch.int32, device="cuda"))
        s.decode(torch.full((1,), m.vocab, dtype=torch.int32, device="cuda"))
        assert s.stats()["status"] == tlf.E_DEVICE
    finally:
        s.close()
