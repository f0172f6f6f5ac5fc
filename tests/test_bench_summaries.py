"""Host logic of bench.py's profile summaries, on synthetic rocprofv3 kernel
traces whose kernel durations are known: every (loop, layer, kernel) average
and every span must come out exactly."""
import csv
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402

R, J = 3, 2  # loops, layers of the synthetic runs


class Trace:
    """Kernels laid end to end with a fixed gap; timestamps in ns."""

    def __init__(self, gap_ns=1000):
        self.rows, self.t, self.gap = [], 0, gap_ns

    def add(self, name, us):
        start = self.t + self.gap
        end = start + int(round(us * 1e3))
        self.rows.append({"Kernel_Name": name, "Start_Timestamp": str(start), "End_Timestamp": str(end)})
        self.t = end

    def write(self, path):
        rows = list(self.rows)
        rows.reverse()  # the summaries sort by start time themselves
        with open(path, "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
            w.writeheader()
            w.writerows(rows)


PRE = {"qkv": "k_gemm_dual<E_QKV>", "attn": "k_attn_prefill<bf16, 64>", "o": "k_gemm_dual<E_RESID, WM 2>",
       "gate_up": "k_gemm_dual<E_SWIGLU>", "down": "k_gemm_dual<E_RESID, WM 4>"}


def pre_us(p, i, j, kind):
    """Duration of kernel `kind` at loop i, layer j of prefill p."""
    return 10.0 * (1 + list(PRE).index(kind)) + 3.0 * i + 0.5 * j + 0.25 * p


def add_prefill(tr, p):
    tr.add("k_fill_i32", 1.0)
    tr.add("k_embed_route<bf16>", 5.0)
    tr.add("k_plan_prefill", 2.0)
    for i in range(R):
        for j in range(J):
            tr.add(PRE["qkv"], pre_us(p, i, j, "qkv"))
            tr.add(PRE["attn"], pre_us(p, i, j, "attn"))
            tr.add(PRE["o"], pre_us(p, i, j, "o"))
            tr.add("k_resid_norm<1>", 1.0)
            tr.add(PRE["gate_up"], pre_us(p, i, j, "gate_up"))
            tr.add(PRE["down"], pre_us(p, i, j, "down"))
            tr.add("k_resid_norm<1>", 1.0)
    tr.add("k_gemm<E_LOGITS>", 4.0)


def test_prefill_trace_summary(tmp_path):
    tr = Trace()
    for p in range(4):  # a warm-up prefill, then three timed ones
        add_prefill(tr, p)
    for _ in range(3):
        tr.add("__amd_rocclr_copyBuffer", 50.0)  # host copies after the session
    for p in range(4, 6):  # the next session
        add_prefill(tr, p)
    path = tmp_path / "trace.csv"
    tr.write(path)
    out = bench.prefill_trace_summary(str(path), R, J, first=1, count=3)
    assert out["prefills"] == [1, 4]
    for i, row in enumerate(out["per_loop_us"]):
        assert row["loop"] == i + 1
        for kind in PRE:
            want = sum(pre_us(p, i, j, kind) for p in (1, 2, 3) for j in range(J)) / (3 * J)
            assert row[kind] == pytest.approx(want, abs=1e-9), (i, kind)
    for kind in PRE:
        want = sum(pre_us(p, i, j, kind) for p in (1, 2, 3) for i in range(R) for j in range(J)) / 3
        assert out["per_prefill_us"][kind] == pytest.approx(want, abs=1e-9), kind
    # span: the first kernel after the previous prefill's head to this
    # prefill's head, gaps included (one gap per kernel), never the copies
    kernels = 3 + R * J * 7 + 1
    busy = [1.0 + 5.0 + 2.0 + 4.0 + sum(pre_us(p, i, j, k) for i in range(R) for j in range(J) for k in PRE)
            + R * J * 2 * 1.0 for p in (1, 2, 3)]
    want = sum(b + (kernels - 1) * 1.0 for b in busy) / 3
    assert out["span_us"] == pytest.approx(want, abs=1e-6)


DEC = ("qkv", "attn", "o", "gate_up", "down")
DEC_NAME = {"qkv": "k_dgemm<E_QKV>", "attn": "k_attn_decode<bf16, 64, 4>", "o": "k_dgemm<E_RESID>",
            "gate_up": "k_dgemm<E_SWIGLU>", "down": "k_dgemm<E_RESID>"}


def dec_us(st, i, j, kind):
    return 5.0 * (1 + DEC.index(kind)) + 2.0 * i + 0.5 * j + 0.125 * st


def test_decode_trace_summary(tmp_path):
    steps = 6
    tr = Trace()
    for st in range(steps):
        tr.add("k_embed_route<bf16>", 3.0)
        tr.add("k_plan_decode", 2.0)
        for i in range(R):
            for j in range(J):
                for kind in DEC:
                    tr.add(DEC_NAME[kind], dec_us(st, i, j, kind))
        tr.add("k_gemm<E_LOGITS>", 7.0)
        tr.add("k_argmax_finalize", 1.0)
    path = tmp_path / "trace.csv"
    tr.write(path)
    per_step = R * J
    out = bench.trace_summary(str(path), routed_launches=steps * per_step, last_dispatches=2 * per_step,
                              loops=R, layers=J, first_step=1, last_step=4)
    # the attention average over the last two steps' launches
    want = sum(dec_us(st, i, j, "attn") for st in (4, 5) for i in range(R) for j in range(J)) / (2 * per_step)
    assert out["attn_routed_timed_region"]["dispatches"] == 2 * per_step
    assert out["attn_routed_timed_region"]["avg_us"] == pytest.approx(want, abs=1e-9)
    table = {(t["loop"], t["layer"]): t for t in out["decode_steps"]["per_loop_layer_us"]}
    for i in range(R):
        for j in range(J):
            for kind in DEC:
                want = sum(dec_us(st, i, j, kind) for st in (1, 2, 3)) / 3
                assert table[(i + 1, j + 1)][kind] == pytest.approx(want, abs=1e-9), (i, j, kind)
    # a step's span runs from its embedding kernel to the kernel before the
    # next step's embedding kernel; every kernel after the first adds one gap
    kernels = 2 + per_step * 5 + 2
    busy = [3.0 + 2.0 + 7.0 + 1.0 + sum(dec_us(st, i, j, k) for i in range(R) for j in range(J) for k in DEC)
            for st in (1, 2, 3)]
    assert out["decode_steps"]["span_us"] == pytest.approx(sum(busy) / 3 + (kernels - 1) * 1.0, abs=1e-6)
    assert out["decode_steps"]["gaps_us"] == pytest.approx((kernels - 1) * 1.0, abs=1e-6)
