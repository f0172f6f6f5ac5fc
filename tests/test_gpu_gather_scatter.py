"""GPU parity of the training-side gather-scatter and the STE through the C
ABI against the oracle (Section 3.2, Eq. 6-7, Appendix B).

Bars: active rows, slots, sequence offsets and counts bit-exact; the gather
bit-exact (it copies); the scatter's fp32 sum within one rounding of the
fp64 oracle (|err| <= 2^-24 |value|, plus 1e-38 for zero sums); gradients
through a float32 block within 1e-4 relative to the oracle's fp64 backward
(the block's own fp32 products set that bar, not the gather-scatter); the
STE's gradient within 1e-6 relative (fp32 exponential and division).
"""
import numpy as np
import pytest

import synth
from oracle import gather_scatter as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _train():
    from paper_2609_15160_amd import train
    return train


def _dev(a, dt=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dt is None else t.to(dt)


def _report(tag, **kv):
    print(f"[gs] {tag} " + " ".join(f"{k}={v}" for k, v in kv.items()), flush=True)


def _check_plan(train, m, batch, seq_len, loop, ws=None):
    p = train.plan(_dev(m), batch, seq_len, loop, workspace=ws)
    want = O.active_rows(m, loop)
    assert p.count == want.shape[0]
    assert np.array_equal(p.index.cpu().numpy(), want)
    if batch * seq_len:
        assert np.array_equal(p.slot.cpu().numpy(), O.compact_slot(m, loop))
    assert np.array_equal(p.offsets.cpu().numpy(), O.sequence_offsets(m, seq_len, loop))
    return p


@pytest.mark.parametrize("planner", ["single", "chunked"])
@pytest.mark.parametrize("batch,seq_len", [(1, 1), (3, 17), (1, 2048), (1, 2049), (5, 7001), (2, 16384),
                                           (1, 16385)])
def test_plan_bit_exact(batch, seq_len, planner):
    """Several passes of the single-workgroup planner, ragged last pass,
    sequence starts anywhere inside a pass; the multi-workgroup planner on
    one chunk, one chunk plus one row, and many chunks with a ragged last."""
    train = _train()
    R = 8
    m = synth.make_train_depths(batch * seq_len, R, seed=batch * 1000 + seq_len)
    ws = train.plan_workspace(batch, seq_len) if planner == "chunked" else None
    _report("plan", planner=planner, batch=batch, seq_len=seq_len)
    for i in range(0, R + 2):
        _check_plan(train, m, batch, seq_len, i, ws)


@pytest.mark.parametrize("planner", ["single", "chunked"])
def test_plan_empty_and_degenerate(planner):
    train = _train()
    for batch, seq_len in [(0, 5), (3, 0), (0, 0)]:
        _report("plan-empty", planner=planner, batch=batch, seq_len=seq_len)
        ws = train.plan_workspace(batch, seq_len) if planner == "chunked" else None
        m = np.zeros(batch * seq_len, np.int32)
        p = train.plan(_dev(m) if m.size else torch.zeros(0, dtype=torch.int32, device="cuda"), batch, seq_len, 1,
                       workspace=ws)
        assert p.count == 0
        assert p.offsets.cpu().numpy().tolist() == [0] * (batch + 1)
    ws = train.plan_workspace(4, 10) if planner == "chunked" else None
    m = np.ones(40, np.int32)
    assert _check_plan(train, m, 4, 10, 2, ws).count == 0     # nobody reaches loop 2
    assert _check_plan(train, m, 4, 10, 1, ws).count == 40    # everybody in loop 1


def test_chunked_plan_equals_single_workgroup_plan():
    """The two planners give bitwise the same plan on the training workload's
    shape (batch 8 x 4096, depths of the decode workload's mix), every loop,
    with the workspace reused from call to call and a stale count left in it
    by a larger call."""
    train = _train()
    B, T = 8, 4096
    m = _dev(synth.make_train_depths(B * T, 8))
    ws = train.plan_workspace(B, T)
    ws.fill_(0x7F)                      # contents need no initialisation
    for i in range(1, 10):
        a = train.plan(m, B, T, i)
        b = train.plan(m, B, T, i, workspace=ws)
        assert a.count == b.count
        for f in ("index", "slot", "offsets"):
            assert torch.equal(getattr(a, f), getattr(b, f)), (i, f)
    small = _dev(synth.make_train_depths(3 * 999, 8, seed=4))
    for i in (1, 3):
        a = train.plan(small, 3, 999, i)
        b = train.plan(small, 3, 999, i, workspace=ws)
        assert a.count == b.count and torch.equal(a.index, b.index) and torch.equal(a.offsets, b.offsets)


def test_chunked_plan_rejects_short_workspace():
    train = _train()
    m = _dev(synth.make_train_depths(5000, 8))
    ws = torch.empty(4, dtype=torch.uint8, device="cuda")   # needs 3 chunk counts
    with pytest.raises(train.tlf.TlfError) as e:
        train.plan(m, 1, 5000, 1, workspace=ws)
    assert e.value.status == train.tlf.E_INVALID_ARG


def _fp32_sum_ok(got, h, y_rows):
    want = np.asarray(h, np.float64) + np.asarray(y_rows, np.float64)
    err = np.abs(np.asarray(got, np.float64) - want)
    assert np.all(err <= np.abs(want) * 2.0 ** -24 + 1e-38), float(err.max())


@pytest.mark.parametrize("batch,seq_len,d", [(2, 37, 4), (3, 300, 64), (1, 5000, 1028)])
def test_gather_scatter_parity(batch, seq_len, d):
    train = _train()
    rows = batch * seq_len
    m = synth.make_train_depths(rows, 8, seed=rows + d)
    H = synth.make_train_states(rows, d, seed=d)
    Hd = _dev(H)
    _report("gather-scatter", batch=batch, seq_len=seq_len, d=d)
    for i in (1, 3, 8, 9):
        p = _check_plan(train, m, batch, seq_len, i)
        idx = O.active_rows(m, i)
        X = train.gather_raw(Hd, p)
        assert np.array_equal(X.cpu().numpy(), O.gather(H, idx).astype(np.float32))
        Y = synth.make_train_states(p.count, d, seed=i, stream=104)
        Yd = _dev(Y)
        out = train.scatter_raw(Hd, Yd, p).cpu().numpy()
        want = O.scatter(H, Y, idx)
        inactive = np.ones(rows, bool)
        inactive[idx] = False
        assert np.array_equal(out[inactive], H[inactive])
        _fp32_sum_ok(out[idx], H[idx], Y)
        # in place: the same values, and rows not in the loop untouched
        Hc = Hd.clone()
        train.scatter_raw(Hc, Yd, p, out=Hc)
        assert np.array_equal(Hc.cpu().numpy(), out)
        assert np.allclose(out, want, rtol=1e-6, atol=1e-6)


def test_full_size_training_batch():
    """Batch 8 x 4096 tokens, d = 1024 (the prefill workload's shape), every
    loop: plan bit-exact, sampled gathered rows bit-exact, sampled scattered
    rows within one rounding."""
    train = _train()
    B, T, d, R = 8, 4096, 1024, 8
    rows = B * T
    m = synth.make_train_depths(rows, R)
    H = synth.make_train_states(rows, d)
    Hd = _dev(H)
    rng = np.random.default_rng(5)
    for i in range(1, R + 1):
        p = _check_plan(train, m, B, T, i)
        idx = O.active_rows(m, i)
        X = train.gather_raw(Hd, p)
        pick = np.unique(np.concatenate([[0, p.count - 1], rng.integers(0, p.count, 64)]))
        assert np.array_equal(X[torch.from_numpy(pick).cuda()].cpu().numpy(), H[idx[pick]])
        Yd = X * 0.5
        out = train.scatter_raw(Hd, Yd, p)
        rows_pick = np.unique(np.concatenate([idx[pick], rng.integers(0, rows, 64)]))
        got = out[torch.from_numpy(rows_pick).cuda()].cpu().numpy()
        slot = O.compact_slot(m, i)[rows_pick]
        for k, r in enumerate(rows_pick):
            if slot[k] < 0:
                assert np.array_equal(got[k], H[r])
            else:
                _fp32_sum_ok(got[k], H[r], np.float32(0.5) * H[r])
        _report("full", loop=i, active=p.count)


def test_autograd_through_loops_matches_oracle_backward():
    """Three loops of gather -> row-wise block -> scatter with torch autograd
    around the HIP operators; dL/dH0 and dL/dA against the oracle's fp64
    forward and backward."""
    train = _train()
    B, T, d, R = 2, 129, 32, 3
    rows = B * T
    m = synth.make_train_depths(rows, R, seed=77)
    H0 = synth.make_train_states(rows, d, seed=78)
    A = synth.make_train_states(d, d, seed=79) * np.float32(0.2)
    W = synth.make_train_states(rows, d, seed=80)
    depth = _dev(m)
    h0 = _dev(H0).requires_grad_(True)
    a = _dev(A).requires_grad_(True)
    h = h0
    for i in range(1, R + 1):
        p = train.plan(depth, B, T, i)
        h = train.scatter(h, torch.tanh(train.gather(h, p) @ a), p)
    loss = (h * _dev(W)).sum()
    loss.backward()
    # the in-place scatter (after an out-of-place first loop) gives the same
    # values and gradients
    h0b = _dev(H0).requires_grad_(True)
    ab = _dev(A).requires_grad_(True)
    hb = h0b
    for i in range(1, R + 1):
        p = train.plan(depth, B, T, i)
        y = torch.tanh(train.gather(hb, p) @ ab)
        hb = train.scatter(hb, y, p) if i == 1 else train.scatter_(hb, y, p)
    (hb * _dev(W)).sum().backward()
    assert torch.equal(hb.detach(), h.detach())
    assert torch.equal(h0b.grad, h0.grad)
    assert torch.equal(ab.grad, a.grad)

    H, saved = H0.astype(np.float64), []
    A64 = A.astype(np.float64)
    for i in range(1, R + 1):
        idx = O.active_rows(m, i)
        X = O.gather(H, idx)
        saved.append((idx, X))
        H = O.scatter(H, np.tanh(X @ A64), idx)
    np.testing.assert_allclose(h.detach().cpu().numpy(), H, rtol=1e-4, atol=1e-5)
    dH, dA = W.astype(np.float64), np.zeros_like(A64)
    for idx, X in reversed(saved):
        dprev, dY = O.scatter_backward(dH, idx)
        dZ = dY * (1.0 - np.tanh(X @ A64) ** 2)
        dA += X.T @ dZ
        dH = dprev + O.gather_backward(dZ @ A64.T, idx, rows)
    np.testing.assert_allclose(h0.grad.cpu().numpy(), dH, rtol=1e-4, atol=1e-4)
    np.testing.assert_allclose(a.grad.cpu().numpy(), dA, rtol=1e-4, atol=1e-3)


def test_ste_parity():
    train = _train()
    n = 10000
    rng = np.random.default_rng(9)
    m = rng.integers(1, 9, n).astype(np.int32)
    s = (rng.standard_normal(n) * 4).astype(np.float32)
    s[:4] = [0.0, 30.0, -30.0, 100.0]
    g = rng.standard_normal(n).astype(np.float32)
    sd = _dev(s).requires_grad_(True)
    v = train.ste(sd, _dev(m))
    assert np.array_equal(v.detach().cpu().numpy(), O.ste_value(m).astype(np.float32))
    v.backward(_dev(g))
    want = O.ste_grad(s, g)
    got = sd.grad.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - want) <= 1e-6 * np.abs(want) + 1e-30), float(np.max(np.abs(got - want)))
