"""ctypes binding of libtlf (argument marshalling only).

Every step of prefill and decode runs in libtlf's HIP kernels; PyTorch only
allocates device memory and supplies the stream.  Loading fails loudly when
the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Dict, Optional

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libtlf.so")
HEADER = os.path.join(os.path.dirname(PKG_DIR), "include", "tlf.h")

ABI_VERSION = 5
MAX_LOOPS = 16
MAX_LAYERS = 8
MAX_BATCH = 4096
PAGE_TOKENS = 16

OK = 0
E_INVALID_ARG = -1
E_NEED_WORKSPACE = -2
E_OUT_OF_PAGES = -3
E_STATE = -4
E_HIP = -5
E_DEVICE = -6
E_UNSUPPORTED = -7

DTYPE_F32 = 0
DTYPE_BF16 = 1
ROUTE = {"argmax": 0, "cumprob": 1, "fixed": 2}
PREFILL_ALL_LOGITS = 1
PREFILL_APPEND = 2
PROFILE_OFF = 0
PROFILE_ATTN = 1
PROFILE_BLOCK = 2


class Config(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_int32), ("dtype", ctypes.c_int32), ("vocab", ctypes.c_int32),
        ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("d_ff", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("max_loops", ctypes.c_int32),
        ("max_pos", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("page_tokens", ctypes.c_int32),
        ("max_pages", ctypes.c_int32), ("max_prefill_tokens", ctypes.c_int32),
        ("route_rule", ctypes.c_int32), ("route_threshold", ctypes.c_float),
        ("fixed_depth", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("decode_graph", ctypes.c_int32),
        ("router_hidden", ctypes.c_int32), ("dense_decode", ctypes.c_int32), ("adaln", ctypes.c_int32),
        ("prefill_act_bf16", ctypes.c_int32),
    ]


class LayerWeights(ctypes.Structure):
    _fields_ = [("w_qkv", ctypes.c_void_p), ("w_o", ctypes.c_void_p),
                ("w_gate_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p)]


class AdalnWeights(ctypes.Structure):
    _fields_ = [
        ("time_w1", ctypes.c_void_p), ("time_b1", ctypes.c_void_p), ("time_w2", ctypes.c_void_p),
        ("time_b2", ctypes.c_void_p), ("step_w1", ctypes.c_void_p), ("step_b1", ctypes.c_void_p),
        ("step_w2", ctypes.c_void_p), ("step_b2", ctypes.c_void_p),
        ("mod_w", ctypes.POINTER(ctypes.c_void_p)), ("mod_b", ctypes.POINTER(ctypes.c_void_p)),
    ]


class Weights(ctypes.Structure):
    _fields_ = [
        ("tok_emb", ctypes.c_void_p), ("pos_emb", ctypes.c_void_p), ("router_w", ctypes.c_void_p),
        ("router_b", ctypes.c_void_p), ("lm_head", ctypes.c_void_p), ("n_layers", ctypes.c_int32),
        ("layers", ctypes.POINTER(LayerWeights)), ("router_w1", ctypes.c_void_p), ("router_b1", ctypes.c_void_p),
        ("adaln", ctypes.POINTER(AdalnWeights)),
    ]


class CacheStats(ctypes.Structure):
    _fields_ = [
        ("slots_per_loop", ctypes.c_int64 * MAX_LOOPS), ("pages_per_loop", ctypes.c_int64 * MAX_LOOPS),
        ("depth_hist", ctypes.c_int64 * MAX_LOOPS), ("pages_used", ctypes.c_int64),
        ("pages_total", ctypes.c_int64), ("kv_bytes_resident", ctypes.c_int64), ("batch", ctypes.c_int64),
        ("seq_len", ctypes.c_int64), ("last_step_kv_read_bytes", ctypes.c_int64),
        ("last_step_kv_write_bytes", ctypes.c_int64), ("last_step_weight_bytes", ctypes.c_int64),
        ("last_step_loops_executed", ctypes.c_int64), ("last_step_active_rows", ctypes.c_int64 * MAX_LOOPS),
        ("decode_steps", ctypes.c_int64), ("attn_launches", ctypes.c_int64), ("attn_algo_bytes", ctypes.c_int64),
        ("attn_ms", ctypes.c_double), ("kv_write_bytes_total", ctypes.c_int64),
        ("loops_executed_total", ctypes.c_int64), ("block_ms", ctypes.c_double),
        ("device_error", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


EXPORTS = ("tlf_init", "tlf_prefill", "tlf_decode_step", "tlf_cache_stats", "tlf_set_profiling", "tlf_destroy",
           "tlf_status_str", "tlf_gs_plan", "tlf_gs_plan_ws", "tlf_gs_plan_noalloc", "tlf_gs_gather",
           "tlf_gs_scatter", "tlf_ste", "tlf_probe_read")

PROBE_READ_GRAIN = 32768

GS_PLAN_CHUNK_ROWS = 2048
GS_PLAN_MAX_ROWS = 8388608
GS_PLAN_NOALLOC_MAX_ROWS = 8388608


def gs_plan_ws_bytes(rows: int) -> int:
    """Workspace bytes of tlf_gs_plan_ws for `rows` rows (tlf_gs_plan_ws_bytes in tlf.h)."""
    return 0 if rows <= 0 else 4 * ((rows + GS_PLAN_CHUNK_ROWS - 1) // GS_PLAN_CHUNK_ROWS)


def header_exports(path: str = HEADER):
    """Function names declared in include/tlf.h."""
    text = open(path).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\*)\s+(tlf_\w+)\s*\(", text, re.M)))


class TlfError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} ({status})")


_lib = None


def load(path: str = LIB_PATH):
    """Loads libtlf.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (__graft_entry__.build())")
    lib = ctypes.CDLL(path)
    vp, i32, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32
    lib.tlf_init.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Weights), vp, ctypes.c_size_t,
                             ctypes.POINTER(ctypes.c_size_t), vp, ctypes.POINTER(vp)]
    lib.tlf_init.restype = ctypes.c_int
    lib.tlf_prefill.argtypes = [vp, i32, i32, vp, vp, vp, u32]
    lib.tlf_prefill.restype = ctypes.c_int
    lib.tlf_decode_step.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.tlf_decode_step.restype = ctypes.c_int
    lib.tlf_cache_stats.argtypes = [vp, ctypes.POINTER(CacheStats), vp, vp, ctypes.c_size_t]
    lib.tlf_cache_stats.restype = ctypes.c_int
    lib.tlf_set_profiling.argtypes = [vp, ctypes.c_int]
    lib.tlf_set_profiling.restype = ctypes.c_int
    lib.tlf_destroy.argtypes = [vp]
    lib.tlf_destroy.restype = None
    lib.tlf_status_str.argtypes = [ctypes.c_int]
    lib.tlf_status_str.restype = ctypes.c_char_p
    lib.tlf_gs_plan.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, vp]
    lib.tlf_gs_plan.restype = ctypes.c_int
    lib.tlf_gs_plan_ws.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tlf_gs_plan_ws.restype = ctypes.c_int
    lib.tlf_gs_plan_noalloc.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, vp]
    lib.tlf_gs_plan_noalloc.restype = ctypes.c_int
    lib.tlf_probe_read.argtypes = [vp, ctypes.c_size_t, vp, vp]
    lib.tlf_probe_read.restype = ctypes.c_int
    lib.tlf_gs_gather.argtypes = [vp, vp, vp, i32, i32, vp, vp]
    lib.tlf_gs_gather.restype = ctypes.c_int
    lib.tlf_gs_scatter.argtypes = [vp, vp, vp, i32, i32, vp, vp]
    lib.tlf_gs_scatter.restype = ctypes.c_int
    lib.tlf_ste.argtypes = [vp, vp, vp, i32, vp, vp, vp]
    lib.tlf_ste.restype = ctypes.c_int
    _lib = lib
    return lib


def status_str(status: int) -> str:
    try:
        return load().tlf_status_str(status).decode()
    except Exception:  # library missing: still give a readable message
        return f"status {status}"


def make_config(model, max_batch: int, max_pos: int, max_pages: int, route_rule: str = "argmax",
                threshold: float = 0.5, fixed_depth: int = 1, max_prefill_tokens: int = 65536,
                decode_graph: bool = True, dense_decode: bool = False, prefill_act_bf16: bool = False) -> Config:
    """Config from a model description with attributes like ``synth.ModelConfig``."""
    return Config(
        abi_version=ABI_VERSION, dtype=DTYPE_BF16 if model.dtype == "bf16" else DTYPE_F32,
        vocab=model.vocab, d_model=model.d_model, n_heads=model.n_heads, head_dim=model.head_dim,
        d_ff=model.d_ff, n_layers=model.n_layers, max_loops=model.max_loops, max_pos=max_pos,
        max_batch=max_batch, page_tokens=PAGE_TOKENS, max_pages=max_pages,
        max_prefill_tokens=max_prefill_tokens, route_rule=ROUTE[route_rule],
        route_threshold=threshold, fixed_depth=fixed_depth, rms_eps=model.rms_eps,
        decode_graph=1 if decode_graph else 0, router_hidden=getattr(model, "router_hidden", 0),
        dense_decode=1 if dense_decode else 0, adaln=1 if getattr(model, "adaln", False) else 0,
        prefill_act_bf16=1 if prefill_act_bf16 else 0)


def workspace_bytes(cfg: Config) -> int:
    """Size query (no device work)."""
    need = ctypes.c_size_t(0)
    st = load().tlf_init(ctypes.byref(cfg), None, None, 0, ctypes.byref(need), None, None)
    if st != E_NEED_WORKSPACE:
        raise TlfError(st, "tlf_init(size query)")
    return need.value


def worst_case_pages(batch: int, max_pos: int, loops: int) -> int:
    """Pages for every (sequence, loop) holding max_pos tokens (the fixed-depth bound)."""
    return batch * loops * ((max_pos + PAGE_TOKENS - 1) // PAGE_TOKENS)


class Session:
    """One libtlf context with its weights and workspace in device memory."""

    def __init__(self, model, weights: Dict, max_batch: int, max_pos: Optional[int] = None,
                 max_pages: Optional[int] = None, route_rule: str = "argmax", threshold: float = 0.5,
                 fixed_depth: int = 1, max_prefill_tokens: int = 65536, device: str = "cuda",
                 decode_graph: bool = True, dense_decode: bool = False, prefill_act_bf16: bool = False):
        import torch
        self.torch = torch
        self.lib = load()
        self.model = model
        self.device = torch.device(device)
        max_pos = max_pos or model.max_pos
        if max_pages is None:
            max_pages = worst_case_pages(max_batch, max_pos, model.max_loops)
        self.cfg = make_config(model, max_batch, max_pos, max_pages, route_rule, threshold,
                               fixed_depth, max_prefill_tokens, decode_graph, dense_decode, prefill_act_bf16)
        sdt = torch.bfloat16 if model.dtype == "bf16" else torch.float32

        def dev(a, dt):
            return torch.from_numpy(a).to(self.device).to(dt).contiguous()

        self.w = {
            "tok_emb": dev(weights["tok_emb"], sdt),
            "pos_emb": dev(weights["pos_emb"][:max_pos], sdt),
            "router_w": dev(weights["router_w"], torch.float32),
            "router_b": dev(weights["router_b"], torch.float32),
        }
        if weights.get("lm_head") is not None:
            self.w["lm_head"] = dev(weights["lm_head"], sdt)
        if weights.get("router_w1") is not None:
            self.w["router_w1"] = dev(weights["router_w1"], sdt)
            self.w["router_b1"] = dev(weights["router_b1"], torch.float32)
        if self.w["pos_emb"].shape[0] < max_pos:
            raise ValueError("position table shorter than max_pos")
        self.layers = []
        for lw in weights["layers"]:
            self.layers.append({k: dev(lw[k], sdt) for k in ("w_qkv", "w_o", "w_gate_up", "w_down")})
        self._lw = (LayerWeights * len(self.layers))(*[
            LayerWeights(l["w_qkv"].data_ptr(), l["w_o"].data_ptr(), l["w_gate_up"].data_ptr(),
                         l["w_down"].data_ptr()) for l in self.layers])
        adaln = None
        if weights.get("cond") is not None:
            cond = weights["cond"]
            self.cond = {k: dev(cond[k], sdt if k.endswith(("_w1", "_w2")) else torch.float32)
                         for k in ("time_w1", "time_b1", "time_w2", "time_b2",
                                   "step_w1", "step_b1", "step_w2", "step_b2")}
            self.mods = [(dev(lw["w_mod"], sdt), dev(lw["b_mod"], torch.float32)) for lw in weights["layers"]]
            J = len(self.mods)
            self._mod_w = (ctypes.c_void_p * J)(*[m[0].data_ptr() for m in self.mods])
            self._mod_b = (ctypes.c_void_p * J)(*[m[1].data_ptr() for m in self.mods])
            self._adaln = AdalnWeights(*[self.cond[k].data_ptr() for k in (
                "time_w1", "time_b1", "time_w2", "time_b2", "step_w1", "step_b1", "step_w2", "step_b2")],
                ctypes.cast(self._mod_w, ctypes.POINTER(ctypes.c_void_p)),
                ctypes.cast(self._mod_b, ctypes.POINTER(ctypes.c_void_p)))
            adaln = ctypes.pointer(self._adaln)
        self._weights = Weights(self.w["tok_emb"].data_ptr(), self.w["pos_emb"].data_ptr(),
                                self.w["router_w"].data_ptr(), self.w["router_b"].data_ptr(),
                                self.w["lm_head"].data_ptr() if "lm_head" in self.w else None,
                                len(self.layers), self._lw,
                                self.w["router_w1"].data_ptr() if "router_w1" in self.w else None,
                                self.w["router_b1"].data_ptr() if "router_b1" in self.w else None, adaln)
        need = workspace_bytes(self.cfg)
        self.workspace = torch.empty(need, dtype=torch.uint8, device=self.device)
        self.stream = torch.cuda.current_stream(self.device)
        ctx = ctypes.c_void_p()
        st = self.lib.tlf_init(ctypes.byref(self.cfg), ctypes.byref(self._weights),
                               self.workspace.data_ptr(), need, None,
                               ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(ctx))
        if st != OK:
            raise TlfError(st, "tlf_init")
        self.ctx = ctx
        self.batch = 0
        self.seq_len = 0

    # ------------------------------------------------------------------
    def _check(self, st: int, where: str) -> None:
        if st != OK:
            raise TlfError(st, where)

    def prefill(self, tokens, all_logits: bool = False, want_depths: bool = True, append: bool = False):
        """tokens: int32 [B][T] device tensor.  Returns (logits, depths).

        append=True continues the current batch (a later prompt chunk, or
        tokens after decode steps) instead of starting a new one."""
        torch = self.torch
        B, T = tokens.shape
        tokens = tokens.to(self.device, torch.int32).contiguous()
        V = self.model.vocab
        logits = torch.empty((B, T, V) if all_logits else (B, V), dtype=torch.float32, device=self.device)
        depths = torch.empty((B, T), dtype=torch.int32, device=self.device) if want_depths else None
        flags = (PREFILL_ALL_LOGITS if all_logits else 0) | (PREFILL_APPEND if append else 0)
        st = self.lib.tlf_prefill(self.ctx, B, T, tokens.data_ptr(), logits.data_ptr(),
                                  depths.data_ptr() if depths is not None else None, flags)
        self._check(st, "tlf_prefill")
        self.batch, self.seq_len = B, (self.seq_len + T if append else T)
        return logits, depths

    def decode_into(self, tokens, logits, next_tok=None, depths=None, margin=None) -> None:
        """One decode step writing into caller buffers (no allocation)."""
        ptr = lambda t: t.data_ptr() if t is not None else None
        st = self.lib.tlf_decode_step(self.ctx, tokens.data_ptr(), logits.data_ptr(), ptr(next_tok),
                                      ptr(depths), ptr(margin))
        self._check(st, "tlf_decode_step")
        self.seq_len += 1

    def decode(self, tokens):
        """tokens: int32 [B].  Returns (logits [B][V], next [B], depths [B], margin [B])."""
        torch = self.torch
        B = self.batch
        tokens = tokens.to(self.device, torch.int32).contiguous()
        logits = torch.empty((B, self.model.vocab), dtype=torch.float32, device=self.device)
        nxt = torch.empty(B, dtype=torch.int32, device=self.device)
        depths = torch.empty(B, dtype=torch.int32, device=self.device)
        margin = torch.empty(B, dtype=torch.float32, device=self.device)
        self.decode_into(tokens, logits, nxt, depths, margin)
        return logits, nxt, depths, margin

    def stats(self, with_index: bool = False) -> Dict:
        """Synchronizing statistics; with_index adds per-(b, i) lengths and positions."""
        import numpy as np
        out = CacheStats()
        R = self.model.max_loops
        lens = pos = None
        lens_p = pos_p = None
        cap = 0
        if with_index:
            lens = np.zeros((max(self.batch, 1), R), dtype=np.int32)
            cap = max(self.batch, 1) * R * max(self.seq_len, 1)
            pos = np.zeros(cap, dtype=np.int32)
            lens_p, pos_p = lens.ctypes.data, pos.ctypes.data
        st = self.lib.tlf_cache_stats(self.ctx, ctypes.byref(out), lens_p, pos_p, cap)
        res = {f: getattr(out, f) for f, _ in CacheStats._fields_}
        for f in ("slots_per_loop", "pages_per_loop", "depth_hist", "last_step_active_rows"):
            res[f] = list(res[f])[:R]
        res["status"] = st
        if with_index:
            index = []
            o = 0
            for b in range(self.batch):
                row = []
                for i in range(R):
                    n = int(lens[b, i])
                    row.append(pos[o:o + n].copy())
                    o += n
                index.append(row)
            res["lens"] = lens[: self.batch]
            res["index"] = index
        return res

    def set_profiling(self, mode) -> None:
        """mode: False/"off", True/"attn" (events around every attention launch and
        the loop region), or "block" (events around the loop region only)."""
        code = {False: PROFILE_OFF, "off": PROFILE_OFF, True: PROFILE_ATTN, "attn": PROFILE_ATTN,
                "block": PROFILE_BLOCK}[mode]
        self._check(self.lib.tlf_set_profiling(self.ctx, code), "tlf_set_profiling")

    def close(self) -> None:
        if getattr(self, "ctx", None):
            self.lib.tlf_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
