"""CPU checks of the C ABI: the library loads, exports what include/tlf.h
declares, its structs match the binding, and host-side validation rejects bad
arguments before any device work."""
import ctypes
import os
import subprocess
import tempfile

import pytest

import synth
from paper_2609_15160_amd import tlf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return tlf.load()


def test_library_exports_every_declared_symbol(lib):
    declared = tlf.header_exports()
    assert sorted(declared) == sorted(tlf.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_struct_layouts_match_the_header():
    src = r"""
#include <stdio.h>
#include <stddef.h>
#include "tlf.h"
int main(void) {
  printf("%zu %zu %zu %zu\n", sizeof(tlf_config), sizeof(tlf_layer_weights), sizeof(tlf_weights),
         sizeof(tlf_cache_stats_t));
  printf("%zu %zu %zu %zu %zu\n", offsetof(tlf_config, rms_eps), offsetof(tlf_weights, layers),
         offsetof(tlf_cache_stats_t, last_step_active_rows), offsetof(tlf_cache_stats_t, device_error),
         offsetof(tlf_cache_stats_t, attn_ms));
  return 0;
}
"""
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "t.c")
        exe = os.path.join(d, "t")
        open(c, "w").write(src)
        subprocess.check_call(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), c, "-o", exe])
        out = subprocess.check_output([exe]).decode().split()
    sizes = [int(v) for v in out]
    assert sizes[:4] == [ctypes.sizeof(tlf.Config), ctypes.sizeof(tlf.LayerWeights),
                         ctypes.sizeof(tlf.Weights), ctypes.sizeof(tlf.CacheStats)]
    assert sizes[4:] == [tlf.Config.rms_eps.offset, tlf.Weights.layers.offset,
                         tlf.CacheStats.last_step_active_rows.offset, tlf.CacheStats.device_error.offset,
                         tlf.CacheStats.attn_ms.offset]


def _cfg(**kw):
    m = synth.CONFIGS["bf16_d768_b256x2048"]
    c = tlf.make_config(m, max_batch=256, max_pos=m.max_pos,
                        max_pages=tlf.worst_case_pages(256, m.max_pos, m.max_loops))
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_size_query_needs_no_device(lib):
    need = tlf.workspace_bytes(_cfg())
    m = synth.CONFIGS["bf16_d768_b256x2048"]
    page_bytes = m.n_layers * 2 * m.d_model * 16 * 2
    pool = tlf.worst_case_pages(256, m.max_pos, m.max_loops) * page_bytes
    assert pool < need < pool * 1.2


_BAD, _UNS = tlf.E_INVALID_ARG, tlf.E_UNSUPPORTED


@pytest.mark.parametrize("field,value,status", [
    ("abi_version", 4, _BAD), ("abi_version", 6, _BAD), ("dtype", 7, _BAD), ("vocab", 0, _BAD),
    ("d_model", 100, _BAD), ("n_heads", 5, _BAD), ("d_ff", 0, _BAD), ("n_layers", 0, _BAD),
    ("max_loops", 0, _BAD), ("max_pos", 0, _BAD), ("max_batch", 0, _BAD), ("max_pages", 0, _BAD),
    ("max_prefill_tokens", 0, _BAD), ("route_rule", 5, _BAD), ("rms_eps", 0.0, _BAD),
    ("router_hidden", -64, _BAD), ("dense_decode", 2, _BAD), ("adaln", 2, _BAD), ("dense_decode", -1, _BAD),
    ("prefill_act_bf16", 2, _BAD), ("prefill_act_bf16", -1, _BAD),
    # well-formed, outside this build's kernels
    ("d_ff", 1000, _UNS), ("n_layers", 9, _UNS), ("max_loops", 17, _UNS), ("max_batch", 5000, _UNS),
    ("page_tokens", 32, _UNS), ("router_hidden", 96, _UNS), ("router_hidden", 8192, _UNS),
    ("max_pos", 70000, _UNS),
])
def test_invalid_config_rejected(lib, field, value, status):
    c = _cfg(**{field: value})
    need = ctypes.c_size_t(0)
    st = lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None)
    assert st == status


def test_unsupported_head_dim_and_width(lib):
    """A consistent model with 32-wide heads, or a width that is not a multiple
    of the 128-element K tile, is valid but outside the kernels."""
    need = ctypes.c_size_t(0)
    for kw in (dict(head_dim=32, n_heads=24), dict(d_model=704, n_heads=11)):
        c = _cfg(**kw)
        assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == _UNS


def test_route_parameters_validated(lib):
    need = ctypes.c_size_t(0)
    for kw in (dict(route_rule=1, route_threshold=0.0), dict(route_rule=1, route_threshold=1.0),
               dict(route_rule=2, fixed_depth=0), dict(route_rule=2, fixed_depth=9)):
        c = _cfg(**kw)
        assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == tlf.E_INVALID_ARG
    for kw in (dict(route_rule=1, route_threshold=0.5), dict(route_rule=2, fixed_depth=8)):
        c = _cfg(**kw)
        assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == tlf.E_NEED_WORKSPACE


def test_bf16_head_dim_16_rejected_f32_accepted(lib):
    need = ctypes.c_size_t(0)
    c = tlf.make_config(synth.CONFIGS["f32_tiny_b1x32"], 1, 64, 64)
    assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == tlf.E_NEED_WORKSPACE
    c.dtype = tlf.DTYPE_BF16
    assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == tlf.E_UNSUPPORTED


def test_missing_weights_rejected_before_device_work(lib):
    c = _cfg()
    need = ctypes.c_size_t(0)
    w = tlf.Weights()  # all NULL
    fake_ws = ctypes.c_void_p(1 << 20)  # never dereferenced: validation fails first
    ctx = ctypes.c_void_p()
    st = lib.tlf_init(ctypes.byref(c), ctypes.byref(w), fake_ws, 1 << 62, ctypes.byref(need), None,
                      ctypes.byref(ctx))
    assert st == tlf.E_INVALID_ARG and not ctx.value


def test_mlp_router_weights_must_match_the_config(lib):
    """router_hidden > 0 needs router_w1/router_b1 and a linear router must not get them;
    the hidden layer takes workspace."""
    need = ctypes.c_size_t(0)
    c0 = _cfg()
    assert lib.tlf_init(ctypes.byref(c0), None, None, 0, ctypes.byref(need), None, None) == tlf.E_NEED_WORKSPACE
    lin = need.value
    c = _cfg(router_hidden=768)
    assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == tlf.E_NEED_WORKSPACE
    assert need.value > lin
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: validation fails first
    lw = (tlf.LayerWeights * c.n_layers)(*[tlf.LayerWeights(fake, fake, fake, fake) for _ in range(c.n_layers)])
    for hidden, w1 in ((768, None), (0, fake)):
        cc = _cfg(router_hidden=hidden)
        w = tlf.Weights(fake, fake, fake, fake, None, cc.n_layers, lw, w1, w1)
        ctx = ctypes.c_void_p()
        st = lib.tlf_init(ctypes.byref(cc), ctypes.byref(w), fake, 1 << 62, ctypes.byref(need), None,
                          ctypes.byref(ctx))
        assert st == tlf.E_INVALID_ARG and not ctx.value


def test_adaln_weights_must_match_the_config(lib):
    """adaln = 1 needs every conditioning pointer (one modulator per layer) and
    takes workspace for its table; adaln = 0 must not get them."""
    need = ctypes.c_size_t(0)
    c0 = _cfg()
    assert lib.tlf_init(ctypes.byref(c0), None, None, 0, ctypes.byref(need), None, None) == tlf.E_NEED_WORKSPACE
    plain = need.value
    c = _cfg(adaln=1)
    assert lib.tlf_init(ctypes.byref(c), None, None, 0, ctypes.byref(need), None, None) == tlf.E_NEED_WORKSPACE
    # table [J][R][R][4d] float32 plus its set-up scratch
    assert need.value >= plain + c.n_layers * c.max_loops ** 2 * 4 * c.d_model * 4
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: validation fails first
    lw = (tlf.LayerWeights * c.n_layers)(*[tlf.LayerWeights(fake, fake, fake, fake) for _ in range(c.n_layers)])
    mods = (ctypes.c_void_p * c.n_layers)(*([fake.value] * c.n_layers))
    holes = (ctypes.c_void_p * c.n_layers)(*([fake.value] * (c.n_layers - 1) + [None]))
    P = ctypes.POINTER(ctypes.c_void_p)
    full = tlf.AdalnWeights(*([fake] * 8), ctypes.cast(mods, P), ctypes.cast(mods, P))
    missing_layer = tlf.AdalnWeights(*([fake] * 8), ctypes.cast(mods, P), ctypes.cast(holes, P))
    missing_bias = tlf.AdalnWeights(*([fake] * 7), None, ctypes.cast(mods, P), ctypes.cast(mods, P))
    for flag, aw in ((1, None), (0, full), (1, missing_layer), (1, missing_bias)):
        cc = _cfg(adaln=flag)
        w = tlf.Weights(fake, fake, fake, fake, None, cc.n_layers, lw, None, None,
                        ctypes.pointer(aw) if aw is not None else None)
        ctx = ctypes.c_void_p()
        st = lib.tlf_init(ctypes.byref(cc), ctypes.byref(w), fake, 1 << 62, ctypes.byref(need), None,
                          ctypes.byref(ctx))
        assert st == tlf.E_INVALID_ARG and not ctx.value, (flag, aw)


def test_null_context_calls(lib):
    out = tlf.CacheStats()
    assert lib.tlf_prefill(None, 1, 1, None, None, None, 0) == tlf.E_INVALID_ARG
    assert lib.tlf_decode_step(None, None, None, None, None, None) == tlf.E_INVALID_ARG
    assert lib.tlf_cache_stats(None, ctypes.byref(out), None, None, 0) == tlf.E_INVALID_ARG
    assert lib.tlf_set_profiling(None, 1) == tlf.E_INVALID_ARG
    lib.tlf_destroy(None)


def test_status_strings(lib):
    assert lib.tlf_status_str(tlf.OK) == b"ok"
    assert b"page" in lib.tlf_status_str(tlf.E_OUT_OF_PAGES)
    assert lib.tlf_status_str(12345) == b"unknown status"


def test_binding_constants_match_the_header():
    import re
    text = open(os.path.join(ROOT, "include", "tlf.h")).read()
    defs = {m.group(1): int(m.group(2)) for m in
            re.finditer(r"^#define TLF_(\w+)\s+\(?(-?\d+)u?\)?", text, re.M)}
    pairs = {"ABI_VERSION": tlf.ABI_VERSION, "OK": tlf.OK, "E_INVALID_ARG": tlf.E_INVALID_ARG,
             "E_NEED_WORKSPACE": tlf.E_NEED_WORKSPACE, "E_OUT_OF_PAGES": tlf.E_OUT_OF_PAGES,
             "E_STATE": tlf.E_STATE, "E_HIP": tlf.E_HIP, "E_DEVICE": tlf.E_DEVICE,
             "E_UNSUPPORTED": tlf.E_UNSUPPORTED,
             "DTYPE_F32": tlf.DTYPE_F32, "DTYPE_BF16": tlf.DTYPE_BF16,
             "ROUTE_ARGMAX": tlf.ROUTE["argmax"], "ROUTE_CUMPROB": tlf.ROUTE["cumprob"],
             "ROUTE_FIXED": tlf.ROUTE["fixed"], "PREFILL_ALL_LOGITS": tlf.PREFILL_ALL_LOGITS,
             "PREFILL_APPEND": tlf.PREFILL_APPEND,
             "PROFILE_OFF": tlf.PROFILE_OFF, "PROFILE_ATTN": tlf.PROFILE_ATTN,
             "PROFILE_BLOCK": tlf.PROFILE_BLOCK, "GS_PLAN_CHUNK_ROWS": tlf.GS_PLAN_CHUNK_ROWS,
             "GS_PLAN_MAX_ROWS": tlf.GS_PLAN_MAX_ROWS, "GS_PLAN_NOALLOC_MAX_ROWS": tlf.GS_PLAN_NOALLOC_MAX_ROWS,
             "PROBE_READ_GRAIN": tlf.PROBE_READ_GRAIN, "MAX_BATCH": tlf.MAX_BATCH, "MAX_LOOPS": tlf.MAX_LOOPS,
             "MAX_LAYERS": tlf.MAX_LAYERS, "PAGE_TOKENS": tlf.PAGE_TOKENS}
    for name, value in pairs.items():
        assert defs[name] == value, name


def test_profiling_mode_validated(lib):
    # an unknown mode is rejected
    assert lib.tlf_set_profiling(None, 3) == tlf.E_INVALID_ARG
    assert lib.tlf_set_profiling(None, -1) == tlf.E_INVALID_ARG


def test_gather_scatter_argument_errors_need_no_device():
    """Shape errors of the gather-scatter calls are caught on the host, before
    any HIP call, so they can be checked without a GPU."""
    lib = tlf.load()
    bad = tlf.E_INVALID_ARG
    dummy = ctypes.c_void_p(16)
    assert lib.tlf_gs_plan(dummy, -1, 4, 1, dummy, None, None, dummy, None) == bad
    assert lib.tlf_gs_plan(dummy, 2, 4, 1, dummy, None, None, None, None) == bad
    assert lib.tlf_gs_plan(None, 2, 4, 1, dummy, None, None, dummy, None) == bad
    # the multi-workgroup planner: workspace size, presence and alignment, row cap
    need = tlf.gs_plan_ws_bytes(5000)
    assert need == 12
    assert lib.tlf_gs_plan_ws(dummy, 1, 5000, 1, dummy, None, None, dummy, None, 0, None) == bad
    assert lib.tlf_gs_plan_ws(dummy, 1, 5000, 1, dummy, None, None, dummy, dummy, need - 4, None) == bad
    assert lib.tlf_gs_plan_ws(dummy, 1, 5000, 1, dummy, None, None, dummy, ctypes.c_void_p(18), need, None) == bad
    assert lib.tlf_gs_plan_ws(dummy, 1, tlf.GS_PLAN_MAX_ROWS + 1, 1, dummy, None, None, dummy, dummy,
                              1 << 30, None) == bad
    assert lib.tlf_gs_plan_ws(dummy, 2, 4, 1, dummy, None, None, None, dummy, need, None) == bad
    assert lib.tlf_gs_plan_ws(dummy, -1, 4, 1, dummy, None, None, dummy, dummy, need, None) == bad
    # the allocation-free planner rejects sizes beyond its fixed scratch before any HIP call
    assert lib.tlf_gs_plan_noalloc(dummy, 1, tlf.GS_PLAN_NOALLOC_MAX_ROWS + 1, 1, dummy, None, None, dummy,
                                   None) == bad
    assert lib.tlf_gs_plan_noalloc(dummy, 2, 4, 1, dummy, None, None, None, None) == bad
    assert lib.tlf_gs_gather(dummy, dummy, dummy, 8, 6, dummy, None) == bad     # d % 4
    assert lib.tlf_gs_gather(dummy, dummy, dummy, -1, 8, dummy, None) == bad
    assert lib.tlf_gs_gather(ctypes.c_void_p(20), dummy, dummy, 8, 8, dummy, None) == bad  # alignment
    assert lib.tlf_gs_gather(dummy, dummy, dummy, 0, 8, dummy, None) == tlf.OK   # nothing to do
    assert lib.tlf_gs_scatter(dummy, dummy, dummy, 8, 0, dummy, None) == bad
    assert lib.tlf_gs_scatter(dummy, None, dummy, 8, 8, dummy, None) == bad
    assert lib.tlf_gs_scatter(dummy, dummy, dummy, 0, 8, dummy, None) == tlf.OK
    assert lib.tlf_ste(dummy, dummy, dummy, -1, dummy, dummy, None) == bad
    assert lib.tlf_ste(None, dummy, dummy, 4, dummy, None, None) == bad
    assert lib.tlf_ste(dummy, None, dummy, 4, None, dummy, None) == bad
    assert lib.tlf_ste(dummy, dummy, dummy, 4, None, None, None) == tlf.OK
    # the read probe takes whole grains of a 16-byte aligned buffer
    g = tlf.PROBE_READ_GRAIN
    assert lib.tlf_probe_read(dummy, g + 16, dummy, None) == bad
    assert lib.tlf_probe_read(dummy, 0, dummy, None) == bad
    assert lib.tlf_probe_read(ctypes.c_void_p(24), g, dummy, None) == bad
    assert lib.tlf_probe_read(dummy, g, None, None) == bad
