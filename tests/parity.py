"""Runs the HIP path (through the C ABI) and the oracle on the same seeded
inputs and compares them.  The oracle is teacher-forced on the tokens the GPU
emits, so a legitimately different greedy pick in bf16 cannot make the two
sequences diverge."""
from __future__ import annotations

import dataclasses
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

import synth
from oracle import tlf_oracle as O


@dataclasses.dataclass
class GpuRun:
    prefill_logits: np.ndarray          # [B][V] or [B][T][V]
    prefill_depths: np.ndarray          # [B][T]
    step_tokens: List[np.ndarray]       # token fed at each decode step [B]
    step_logits: List[np.ndarray]       # [B][V]
    step_next: List[np.ndarray]
    step_depths: List[np.ndarray]
    step_margin: List[np.ndarray]
    stats: Dict


def run_gpu(model: synth.ModelConfig, weights: Dict, prompts: np.ndarray, steps: int,
            route_rule: str = "argmax", threshold: float = 0.5, fixed_depth: int = 1,
            all_logits: bool = False, max_pos: Optional[int] = None, max_pages: Optional[int] = None,
            max_prefill_tokens: int = 65536, keep_logits_rows: Optional[Sequence[int]] = None,
            decode_graph: bool = True, dense_decode: bool = False, prefill_act_bf16: bool = False) -> GpuRun:
    import torch
    from paper_2609_15160_amd import tlf
    B, T = prompts.shape
    sess = tlf.Session(model, weights, max_batch=B, max_pos=max_pos or (T + steps), max_pages=max_pages,
                       route_rule=route_rule, threshold=threshold, fixed_depth=fixed_depth,
                       max_prefill_tokens=max_prefill_tokens, decode_graph=decode_graph,
                       dense_decode=dense_decode, prefill_act_bf16=prefill_act_bf16)
    rows = slice(None) if keep_logits_rows is None else list(keep_logits_rows)
    try:
        toks = torch.from_numpy(prompts.astype(np.int32)).cuda()
        lg, dep = sess.prefill(toks, all_logits=all_logits)
        run = GpuRun(lg.cpu().numpy()[rows], dep.cpu().numpy(), [], [], [], [], [], {})
        # the first decode token is the greedy pick of the prefill logits
        last = lg[:, -1, :] if all_logits else lg
        cur = torch.argmax(last, dim=-1).to(torch.int32)
        for _ in range(steps):
            logits, nxt, d, mg = sess.decode(cur)
            run.step_tokens.append(cur.cpu().numpy())
            run.step_logits.append(logits.cpu().numpy()[rows])
            run.step_next.append(nxt.cpu().numpy())
            run.step_depths.append(d.cpu().numpy())
            run.step_margin.append(mg.cpu().numpy())
            cur = nxt
        run.stats = sess.stats(with_index=True)
        torch.cuda.synchronize()
        return run
    finally:
        sess.close()


@dataclasses.dataclass
class ScheduleRun:
    logits: np.ndarray      # [B][L][V] logits of every position
    depths: np.ndarray      # [B][L]
    stats: Dict


def run_gpu_schedule(model: synth.ModelConfig, weights: Dict, tokens: np.ndarray, schedule,
                     route_rule: str = "argmax", threshold: float = 0.5, fixed_depth: int = 1,
                     max_prefill_tokens: int = 65536, decode_graph: bool = True,
                     prefill_act_bf16: bool = False) -> ScheduleRun:
    """Feeds the columns of tokens [B][L] left to right as the schedule says:
    ("prefill", n) prefills the next n tokens (the first item starts the batch,
    later ones append chunks to it) and ("decode", n) runs n decode steps, each
    fed the next column (teacher forcing)."""
    import torch
    from paper_2609_15160_amd import tlf
    B, L = tokens.shape
    sess = tlf.Session(model, weights, max_batch=B, max_pos=L, route_rule=route_rule, threshold=threshold,
                       fixed_depth=fixed_depth, max_prefill_tokens=max_prefill_tokens,
                       decode_graph=decode_graph, prefill_act_bf16=prefill_act_bf16)
    try:
        toks = torch.from_numpy(tokens.astype(np.int32)).cuda()
        logits = np.zeros((B, L, model.vocab), np.float32)
        depths = np.zeros((B, L), np.int32)
        t = 0
        for k, (kind, n) in enumerate(schedule):
            if kind == "prefill":
                lg, dep = sess.prefill(toks[:, t:t + n], all_logits=True, append=k > 0)
                logits[:, t:t + n] = lg.cpu().numpy()
                depths[:, t:t + n] = dep.cpu().numpy()
                t += n
            else:
                for _ in range(n):
                    lg, _, dep, _ = sess.decode(toks[:, t])
                    logits[:, t] = lg.cpu().numpy()
                    depths[:, t] = dep.cpu().numpy()
                    t += 1
        if t != L:
            raise ValueError("the schedule does not cover the tokens")
        stats = sess.stats(with_index=True)
        torch.cuda.synchronize()
        return ScheduleRun(logits, depths, stats)
    finally:
        sess.close()


@dataclasses.dataclass
class OracleRun:
    prefill_logits: np.ndarray
    prefill_depths: np.ndarray
    prefill_margin: np.ndarray
    step_logits: List[np.ndarray]
    step_depths: List[np.ndarray]
    step_margin: List[np.ndarray]
    index: List[List[np.ndarray]]       # [b][i] ascending positions
    seconds_prefill: float = 0.0
    seconds_decode: float = 0.0


def run_oracle(model: synth.ModelConfig, weights: Dict, prompts: np.ndarray,
               step_tokens: Sequence[np.ndarray], route_rule: str = "argmax", threshold: float = 0.5,
               fixed_depth: Optional[int] = None, all_logits: bool = False, threads: int = 1) -> OracleRun:
    """The oracle on the same prompts, teacher-forced on ``step_tokens``.
    ``threads`` > 1 prefills the (independent) sequences concurrently."""
    M = O.Model(weights, model.n_heads, model.head_dim, route_rule=route_rule, threshold=threshold,
                fixed_depth=fixed_depth, rms_eps=model.rms_eps)
    t0 = time.perf_counter()
    if threads > 1 and len(prompts) > 1:
        import concurrent.futures
        cap = prompts.shape[1] + len(step_tokens)
        with concurrent.futures.ThreadPoolExecutor(max_workers=threads) as ex:
            outs = list(ex.map(lambda row: O.prefill(M, row, capacity=cap, all_logits=all_logits),
                               np.asarray(prompts)))
        states = [x[0] for x in outs]
        lg, dep, mg = (np.stack([x[k] for x in outs]) for k in (1, 2, 3))
    else:
        states, lg, dep, mg = O.prefill_batch(M, prompts, all_logits=all_logits)
    t1 = time.perf_counter()
    run = OracleRun(lg, dep, mg, [], [], [], [])
    for tok in step_tokens:
        l, d, m = O.decode(M, states, tok)
        run.step_logits.append(l)
        run.step_depths.append(d)
        run.step_margin.append(m)
    run.seconds_prefill = t1 - t0
    run.seconds_decode = time.perf_counter() - t1
    run.index = [O.cache_index(s, M.R) for s in states]
    return run


def router_decisions(model: synth.ModelConfig, weights: Dict, tokens: np.ndarray, positions: np.ndarray,
                     route_rule: str = "argmax", threshold: float = 0.5, fixed_depth: Optional[int] = None):
    """Oracle depth and margin for arbitrary (token, position) pairs (router only)."""
    M = O.Model(weights, model.n_heads, model.head_dim, route_rule=route_rule, threshold=threshold,
                fixed_depth=fixed_depth, rms_eps=model.rms_eps)
    h0 = M.E[tokens] + M.P[positions]
    m, margin, _ = O.route(M, h0)
    return m, margin


def depth_agreement(gpu_depths: np.ndarray, oracle_depths: np.ndarray, oracle_margin: np.ndarray,
                    min_margin: float):
    """(mismatches among decisions with margin > min_margin, overall flip rate)."""
    g = np.asarray(gpu_depths).ravel()
    o = np.asarray(oracle_depths).ravel()
    mg = np.asarray(oracle_margin).ravel()
    strong = mg > min_margin
    return int(np.sum((g != o) & strong)), float(np.mean(g != o)) if g.size else 0.0
