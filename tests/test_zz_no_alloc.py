"""The allocation-free planner tlf_gs_plan_noalloc, called through the C ABI,
against tlf_gs_plan_ws (the entry point it varies) and the oracle: two calls
in a row, the second on a smaller input, so the fixed scratch array carries
the first call's counts into the second.  Active rows, slots, sequence
offsets and counts are integer results: bit-exact."""
import ctypes

import numpy as np
import pytest

import synth
from oracle import gather_scatter as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _plan_outputs(rows, batch):
    dev = "cuda"
    return (torch.full((max(rows, 1),), -7, dtype=torch.int32, device=dev),
            torch.full((max(rows, 1),), -7, dtype=torch.int32, device=dev),
            torch.full((batch + 1,), -7, dtype=torch.int32, device=dev),
            torch.full((1,), -7, dtype=torch.int32, device=dev))


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _run(lib, fn, depth, batch, seq_len, loop, ws=None):
    from paper_2609_15160_amd import tlf
    rows = batch * seq_len
    index, slot, offsets, count = _plan_outputs(rows, batch)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if fn == "ws":
        st = lib.tlf_gs_plan_ws(_p(depth), batch, seq_len, loop, _p(index), _p(slot), _p(offsets), _p(count),
                                _p(ws), ws.numel(), stream)
    else:
        st = lib.tlf_gs_plan_noalloc(_p(depth), batch, seq_len, loop, _p(index), _p(slot), _p(offsets),
                                     _p(count), stream)
    assert st == tlf.OK, st
    torch.cuda.synchronize()
    n = int(count.item())
    return n, index[:n].cpu().numpy(), slot[:rows].cpu().numpy(), offsets.cpu().numpy()


@pytest.mark.parametrize("order", ["large-then-small", "small-then-large-then-small"])
def test_noalloc_plan_equals_workspace_plan(order):
    from paper_2609_15160_amd import tlf
    lib = tlf.load()
    shapes = [(8, 4096, 3), (3, 999, 2)] if order == "large-then-small" else [(2, 1500, 1), (8, 4096, 4), (1, 7, 1)]
    for batch, seq_len, loop in shapes:
        rows = batch * seq_len
        m = synth.make_train_depths(rows, 8, seed=rows + loop)
        depth = torch.from_numpy(m).cuda()
        ws = torch.full((max(tlf.gs_plan_ws_bytes(rows), 4),), 0x55, dtype=torch.uint8, device="cuda")
        a = _run(lib, "ws", depth, batch, seq_len, loop, ws)
        b = _run(lib, "noalloc", depth, batch, seq_len, loop)
        assert a[0] == b[0]
        for x, y in zip(a[1:], b[1:]):
            assert np.array_equal(x, y)
        assert b[0] == O.active_rows(m, loop).shape[0]
        assert np.array_equal(b[1], O.active_rows(m, loop))
        assert np.array_equal(b[2], O.compact_slot(m, loop))
        assert np.array_equal(b[3], O.sequence_offsets(m, seq_len, loop))
        print(f"[noalloc] batch={batch} seq_len={seq_len} loop={loop} active={b[0]}", flush=True)


def test_noalloc_plan_at_its_row_limit():
    """TLF_GS_PLAN_NOALLOC_MAX_ROWS rows (4096 chunks, the whole fixed
    scratch), then a small call: both against tlf_gs_plan_ws and the oracle."""
    from paper_2609_15160_amd import tlf
    lib = tlf.load()
    for batch, seq_len, loop in [(2048, tlf.GS_PLAN_NOALLOC_MAX_ROWS // 2048, 2), (1, 3000, 1)]:
        rows = batch * seq_len
        m = synth.make_train_depths(rows, 8, seed=11 + loop)
        depth = torch.from_numpy(m).cuda()
        ws = torch.empty(tlf.gs_plan_ws_bytes(rows), dtype=torch.uint8, device="cuda")
        a = _run(lib, "ws", depth, batch, seq_len, loop, ws)
        b = _run(lib, "noalloc", depth, batch, seq_len, loop)
        assert a[0] == b[0] == O.active_rows(m, loop).shape[0]
        for x, y in zip(a[1:], b[1:]):
            assert np.array_equal(x, y)
        assert np.array_equal(b[1], O.active_rows(m, loop))
        assert np.array_equal(b[3], O.sequence_offsets(m, seq_len, loop))
        print(f"[noalloc] rows={rows} loop={loop} active={b[0]}", flush=True)


def test_noalloc_plan_empty_and_size_limit():
    from paper_2609_15160_amd import tlf
    lib = tlf.load()
    index, slot, offsets, count = _plan_outputs(0, 3)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    dummy = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert lib.tlf_gs_plan_noalloc(_p(dummy), 3, 0, 1, _p(index), _p(slot), _p(offsets), _p(count), stream) == tlf.OK
    torch.cuda.synchronize()
    assert int(count.item()) == 0 and offsets.cpu().numpy().tolist() == [0, 0, 0, 0]
    big = tlf.GS_PLAN_NOALLOC_MAX_ROWS + 1
    assert lib.tlf_gs_plan_noalloc(_p(dummy), 1, big, 1, _p(index), _p(slot), _p(offsets), _p(count),
                                   stream) == tlf.E_INVALID_ARG
