#!/usr/bin/env python3
"""Decode-step benchmark of the routed looped transformer on one MI355X.

Workload (default): the 2-layer d=768 looped block (12 heads x 64, SwiGLU
2048, vocab 32000, R = 8 loops, bf16 storage) decoding a batch of 256
sequences after a 2048-token prompt, KV cache paged in 16-token pages, router
bias calibrated to a long-tailed depth mix with mean ~3.7.  A step is one
decode step of every sequence: embedding + routing, the depth-sorted plan,
every executed loop and layer (QKV + cache append, recursion-wise attention,
O projection, SwiGLU FFN), the LM head and the greedy pick.

Prints one JSON line: decoded tokens/s, the decode attention's achieved HBM
bandwidth against 8 TB/s (HIP events around every attention launch on the
library's stream), the same kernels forced to fixed depth R, the same step
with gather-scatter off, the step with AdaLN conditioning, the batch 32 x 512
and batch 64 x 4096 (d=2048) decode workloads, the tiny fp32 model's
per-step latency, time to first token over prompt lengths, a prefill
measurement, the MLP-router threshold sweep, the per-step latency
distribution, a streaming-read ceiling, and the CPU oracle on a bounded
sample (all host threads) and on one thread for the small workloads.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
METRIC = "decoded tokens/s at batch B; recursion-wise KV attn HBM GB/s (% of peak)"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def decode_run(sess, torch, B, V, warmup, steps, profiled, first_tokens, latency_steps=0):
    """Warmup, `steps` timed decode steps (HIP-graph replays), then two passes of
    `profiled` steps launched kernel by kernel: the first with HIP events around
    each step's loop-and-layer region only, the second with events around every
    attention launch as well; then `latency_steps` graph-replayed steps with an
    event pair around each (the per-step latency distribution).  Greedy
    feedback throughout, no allocation inside any region.  Returns (ms of the
    timed steps, block-pass stats, attention-pass stats, per-step ms list)."""
    dev = sess.device
    tok = [first_tokens.to(torch.int32).contiguous(), torch.empty(B, dtype=torch.int32, device=dev)]
    logits = torch.empty((B, V), dtype=torch.float32, device=dev)
    k = 0
    for _ in range(warmup):
        sess.decode_into(tok[k % 2], logits, next_tok=tok[(k + 1) % 2])
        k += 1
    log(f"warmup: {warmup} steps enqueued")
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        sess.decode_into(tok[k % 2], logits, next_tok=tok[(k + 1) % 2])
        k += 1
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    log(f"timed: {steps} steps in {ms:.1f} ms")
    stats = []
    for mode in ("block", "attn"):
        sess.set_profiling(mode)
        for p in range(profiled):
            sess.decode_into(tok[k % 2], logits, next_tok=tok[(k + 1) % 2])
            k += 1
            if p % 10 == 9:
                log(f"profiled ({mode} events): {p + 1} of {profiled} steps enqueued")
        torch.cuda.synchronize()
        st = sess.stats()
        sess.set_profiling(False)
        if st["status"] != 0:
            raise RuntimeError(f"device error {st['status']}")
        stats.append(st)
    lat = []
    if latency_steps:
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(latency_steps + 1)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for p in range(latency_steps):
            sess.decode_into(tok[k % 2], logits, next_tok=tok[(k + 1) % 2])
            k += 1
            ev[p + 1].record(stream)
        torch.cuda.synchronize()
        lat = [ev[p].elapsed_time(ev[p + 1]) for p in range(latency_steps)]
        log(f"latency pass: {latency_steps} steps, median {sorted(lat)[len(lat) // 2]:.3f} ms")
    if not bool(torch.isfinite(logits).all()):
        raise RuntimeError("non-finite logits")
    return ms, stats[0], stats[1], lat


def hot_path_bytes(st, model, steps, B):
    """Algorithmic HBM bytes of the timed steps' loop-and-layer region."""
    s = 2 if model.dtype == "bf16" else 4
    d, F, J = model.d_model, model.d_ff, model.n_layers
    block_weights = (4 * d * d + 3 * d * F) * s
    weights = st["loops_executed_total"] * J * block_weights
    return st["attn_algo_bytes"] + st["kv_write_bytes_total"] + weights


def run_config(torch, tlf, model, w, prompts, warmup, steps, profiled, route_rule="argmax", fixed_depth=1,
               graph=True, latency_steps=0):
    B, T = prompts.shape
    max_pos = T + warmup + steps + 2 * profiled + latency_steps
    sess = tlf.Session(model, w, max_batch=B, max_pos=max_pos, route_rule=route_rule,
                       fixed_depth=fixed_depth, max_prefill_tokens=65536, decode_graph=graph)
    try:
        toks = torch.from_numpy(prompts).cuda()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        logits, _ = sess.prefill(toks, want_depths=False)
        torch.cuda.synchronize()
        prefill_s = time.perf_counter() - t0
        first = torch.argmax(logits, dim=-1)
        del logits
        ms, st_block, st_attn, lat = decode_run(sess, torch, B, model.vocab, warmup, steps, profiled, first,
                                                latency_steps)
        hist = sess.stats()["depth_hist"]
        if latency_steps:
            return ms, (st_block, st_attn), prefill_s, hist, lat
        return ms, (st_block, st_attn), prefill_s, hist
    finally:
        sess.close()
        torch.cuda.empty_cache()


def stream_read_gbs(torch, tlf, nbytes=4 << 30, reps=10):
    """Read rate of libtlf's streaming probe (the decode attention's 16-byte
    non-temporal loads) over `nbytes` of device memory: bytes read per second,
    the practical ceiling of a streaming kernel on this device."""
    buf = torch.ones(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    lib = tlf.load()
    stream = torch.cuda.current_stream().cuda_stream

    def once():
        st = lib.tlf_probe_read(buf.data_ptr(), nbytes, sink.data_ptr(), stream)
        if st != tlf.OK:
            raise RuntimeError(f"tlf_probe_read: {st}")
    once()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        once()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    del buf, sink
    torch.cuda.empty_cache()
    return nbytes * reps / (ms / 1e3) / 1e9


def _oracle_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        return os.cpu_count() or 1


def _oracle_decode(model, w, prompts, budget_s, max_steps):
    """Oracle prefill of `prompts` (timed), then greedy decode steps until
    `budget_s` is spent or `max_steps` are done (at least 2).  Returns
    (prefill seconds, steps, decode seconds)."""
    from oracle import tlf_oracle as O
    M = O.Model(w, model.n_heads, model.head_dim, rms_eps=model.rms_eps)
    t0 = time.perf_counter()
    states, lg, _, _ = O.prefill_batch(M, prompts)
    pre = time.perf_counter() - t0
    tok = O.greedy(lg)
    n = 0
    t0 = time.perf_counter()
    while n < 2 or (time.perf_counter() - t0 < budget_s and n < max_steps):
        lg2, _, _ = O.decode(M, states, tok)
        tok = O.greedy(lg2)
        n += 1
    return pre, n, time.perf_counter() - t0


def cpu_baseline(model, w, prompts, budget_s, seqs=8):
    """The oracle (untuned) decoding `seqs` sequences of the same workload on the host."""
    cores = _oracle_threads()
    pre, n, dt = _oracle_decode(model, w, prompts[:seqs], budget_s, model.steps)
    return {"value": seqs * n / dt, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "prefill_s": pre,
            "sample": f"{seqs} of {prompts.shape[0]} sequences: oracle prefill of their {prompts.shape[1]}-token "
                      f"prompts ({pre:.1f} s, timed separately), then {n} batched greedy decode steps timed "
                      f"({dt:.1f} s)"}


def cpu_one_core(synth, budget_s=6.0):
    """The oracle on one host thread (BLAS limited to one thread) for the two
    small decode workloads: the tiny fp32 model at its full batch, and the
    batch 32 x 512 model on a sample of 2 sequences."""
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        return None
    rows = []
    with threadpool_limits(limits=1):
        for name, seqs in (("f32_tiny_b1x32", None), ("bf16_d768_b32x512", 2)):
            m = synth.CONFIGS[name]
            w = synth.make_weights(m)
            prompts = synth.make_prompts(m)
            sample = prompts if seqs is None else prompts[:seqs]
            pre, n, dt = _oracle_decode(m, w, sample, budget_s, m.steps)
            rows.append({"workload": name, "sequences": int(sample.shape[0]), "prompt": int(sample.shape[1]),
                         "prefill_s": pre, "steps": n, "tokens_per_s": sample.shape[0] * n / dt})
    return {"cores": 1, "kind": "oracle", "rows": rows}


def tiny_decode(torch, tlf, synth, warmup=4):
    """The tiny fp32 model (batch 1, 32-token prompt, 32 greedy steps): per-step
    latency of graph-replayed and of kernel-by-kernel decode steps."""
    m = synth.CONFIGS["f32_tiny_b1x32"]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    out = {"workload": "f32_tiny_b1x32 decode: batch 1 x prompt 32, 1-layer d=64 looped block (4x16 heads, "
                       "SwiGLU 256, vocab 512), R=4, float32", "steps": m.steps - warmup}
    for graph in (True, False):
        sess = tlf.Session(m, w, max_batch=1, max_pos=m.max_pos, decode_graph=graph)
        try:
            logits, _ = sess.prefill(torch.from_numpy(prompts).cuda(), want_depths=False)
            first = torch.argmax(logits, dim=-1)
            ms, _ = replay_decode_ms(sess, torch, 1, m.vocab, first, warmup, m.steps - warmup)
        finally:
            sess.close()
        out["us_per_step_graph" if graph else "us_per_step_eager"] = ms * 1e3 / (m.steps - warmup)
    out["tokens_per_s"] = 1e6 / out["us_per_step_graph"]
    return out


def replay_decode_ms(sess, torch, B, V, first_tokens, warmup, steps):
    """ms of `steps` graph-replayed greedy decode steps after `warmup` untimed ones."""
    tok = [first_tokens.to(torch.int32).contiguous(), torch.empty(B, dtype=torch.int32, device=sess.device)]
    out = torch.empty((B, V), dtype=torch.float32, device=sess.device)
    k = 0
    for _ in range(warmup):
        sess.decode_into(tok[k % 2], out, next_tok=tok[(k + 1) % 2])
        k += 1
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        sess.decode_into(tok[k % 2], out, next_tok=tok[(k + 1) % 2])
        k += 1
    e1.record()
    torch.cuda.synchronize()
    st = sess.stats()
    if st["status"] != 0:
        raise RuntimeError(f"device error {st['status']}")
    return e0.elapsed_time(e1), st


def gather_scatter_off(torch, tlf, model, w, prompts, routed_ms_per_step, warmup=4, steps=30):
    """The decode workload with gather-scatter off (dense decode): every loop up
    to the step's deepest token runs all rows, exited rows are discarded at the
    scatter.  Same outputs; the analogue of the paper's latency ablation."""
    B, T = prompts.shape
    sess = tlf.Session(model, w, max_batch=B, max_pos=T + warmup + steps, max_prefill_tokens=65536,
                       dense_decode=True)
    try:
        logits, _ = sess.prefill(torch.from_numpy(prompts).cuda(), want_depths=False)
        first = torch.argmax(logits, dim=-1)
        del logits
        ms, st = replay_decode_ms(sess, torch, B, model.vocab, first, warmup, steps)
    finally:
        sess.close()
        torch.cuda.empty_cache()
    return {"what": "decode with every loop (up to the step's deepest token) run on all rows of the batch, "
                    "exited rows computed and discarded; graph-replayed steps",
            "steps": steps, "ms_per_step": ms / steps, "tokens_per_s": B * steps / (ms / 1e3),
            "latency_increase": (ms / steps) / routed_ms_per_step - 1.0,
            "rows_per_loop_last_step": st["last_step_active_rows"]}


def adaln_decode(torch, tlf, synth, name, routed_ms_per_step, warmup=4, steps=30):
    """The decode workload with AdaLN time/step conditioning: every projection
    row gathers the modulation of its token's (loop, depth) pair."""
    m = synth.CONFIGS[name].replace(adaln=True)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    B, T = prompts.shape
    sess = tlf.Session(m, w, max_batch=B, max_pos=T + warmup + steps, max_prefill_tokens=65536)
    try:
        logits, _ = sess.prefill(torch.from_numpy(prompts).cuda(), want_depths=False)
        first = torch.argmax(logits, dim=-1)
        del logits
        ms, _ = replay_decode_ms(sess, torch, B, m.vocab, first, warmup, steps)
    finally:
        sess.close()
        torch.cuda.empty_cache()
    return {"what": "decode with AdaLN conditioning (synthetic conditioning weights); graph-replayed steps",
            "steps": steps, "ms_per_step": ms / steps, "tokens_per_s": B * steps / (ms / 1e3),
            "overhead": (ms / steps) / routed_ms_per_step - 1.0}


def ttft_sweep(torch, tlf, model, w, synth, lengths=(128, 512, 1024, 2048), chunk=512, reps=5):
    """Time to first token of one request (batch 1): a prefill of T tokens that
    returns the first generated token's logits, for each T; plus the longest
    prompt prefilled in chunks appended to the caches."""
    rows = []
    top = max(lengths)
    sess = tlf.Session(model, w, max_batch=1, max_pos=top, max_prefill_tokens=top)
    try:
        for T in list(lengths) + [("chunked", top)]:
            chunked = isinstance(T, tuple)
            n = top if chunked else T
            toks = torch.from_numpy(synth.make_prompts(model, batch=1, prompt_len=n)).cuda()

            def once():
                if not chunked:
                    return sess.prefill(toks, want_depths=False)[0]
                for a in range(0, n, chunk):
                    lg, _ = sess.prefill(toks[:, a:a + chunk], want_depths=False, append=a > 0)
                return lg
            once()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                lg = once()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            rows.append({"prompt": n, "chunk": chunk if chunked else n, "ttft_ms": ms})
            log(f"ttft T={n}{' chunked by ' + str(chunk) if chunked else ''}: {ms:.2f} ms")
        if sess.stats()["status"] != 0:
            raise RuntimeError("device error in the TTFT sweep")
    finally:
        sess.close()
        torch.cuda.empty_cache()
    return {"workload": f"one request, {model.n_layers}-layer d={model.d_model} looped block, R={model.max_loops}, "
                        f"argmax router; prefill including the first token's logits, mean of {reps} runs",
            "rows": rows}


def threshold_sweep(torch, tlf, synth, name, thresholds=(0.3, 0.4, 0.5, 0.6, 0.7), warmup=4, steps=20):
    """The workload with a two-layer MLP router (hidden width d) and the
    cumulative-probability rule at several thresholds (the analogue of the
    paper's threshold study): depth mix and decode speed per threshold, plus
    the same router under argmax."""
    import numpy as np
    base = synth.CONFIGS[name]
    m = base.replace(router_hidden=base.d_model)
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    B, T = prompts.shape
    rows = []
    for rule, th in [("argmax", None)] + [("cumprob", t) for t in thresholds]:
        sess = tlf.Session(m, w, max_batch=B, max_pos=T + warmup + steps, route_rule=rule,
                           threshold=0.5 if th is None else th, max_prefill_tokens=65536)
        try:
            toks = torch.from_numpy(prompts).cuda()
            logits, _ = sess.prefill(toks, want_depths=False)
            first = torch.argmax(logits, dim=-1)
            del logits
            ms, st = replay_decode_ms(sess, torch, B, m.vocab, first, warmup, steps)
            hist = np.asarray(st["depth_hist"], dtype=np.float64)
            rows.append({"rule": rule, "threshold": th, "tokens_per_s": B * steps / (ms / 1e3),
                         "ms_per_step": ms / steps,
                         "mean_depth": float((hist * np.arange(1, len(hist) + 1)).sum() / hist.sum()),
                         "depth_hist": [int(v) for v in st["depth_hist"]]})
            log(f"router sweep {rule} {th}: {ms / steps:.3f} ms/step, mean depth {rows[-1]['mean_depth']:.2f}")
        finally:
            sess.close()
            torch.cuda.empty_cache()
    return {"workload": f"{name} with a 2-layer MLP router (hidden {m.router_hidden}, SiLU), bias calibrated "
                        f"for the argmax rule; {steps} graph-replayed steps per setting",
            "rows": rows}


def other_workloads(torch, tlf, synth, names=("bf16_d768_b32x512", "bf16_d2048_b64x4096"),
                    warmup=4, steps=20, profiled=4):
    """The other decode workloads of the same family, measured like the main
    one but briefly: decoded tokens/s over graph-replayed steps, the decode
    attention's algorithmic bytes over its event-timed launches, and the same
    kernels at fixed depth R."""
    import numpy as np
    rows = []
    for name in names:
        m = synth.CONFIGS[name]
        w = synth.make_weights(m)
        prompts = synth.make_prompts(m)
        B, T = prompts.shape
        row = {"workload": f"{name} decode: batch {B} x prompt {T}, {m.n_layers}-layer d={m.d_model} looped block "
                           f"({m.n_heads}x{m.head_dim} heads, SwiGLU {m.d_ff}), R={m.max_loops}"}
        for rule in ("argmax", "fixed"):
            ms, (_, st), pre_s, hist = run_config(torch, tlf, m, w, prompts, warmup, steps, profiled,
                                                  route_rule=rule, fixed_depth=m.max_loops)
            gbs = st["attn_algo_bytes"] / (st["attn_ms"] / 1e3) / 1e9
            h = np.asarray(hist, dtype=np.float64)
            rec = {"tokens_per_s": B * steps / (ms / 1e3), "ms_per_step": ms / steps, "attn_achieved_gbs": gbs,
                   "attn_frac": gbs / HBM_PEAK_GBS, "mean_depth": float((h * np.arange(1, len(h) + 1)).sum() / h.sum()),
                   "prefill_s": pre_s}
            row["routed" if rule == "argmax" else "fixed_depth"] = rec
            log(f"{name} {rule}: {ms / steps:.3f} ms/step, attention {gbs:.0f} GB/s")
        rows.append(row)
    return {"steps": steps, "rows": rows}


def prefill_measure(torch, tlf, synth, name):
    """Prefill-only workload: time tlf_prefill and count the algorithmic FLOPs.
    The activations enter the prefill's matrix products as one bf16 part (the
    precision this workload runs at); the same prefill with hi + lo parts is
    timed beside it."""
    import numpy as np
    m = synth.CONFIGS[name]
    w = synth.make_weights(m)
    prompts = synth.make_prompts(m)
    B, T = prompts.shape
    times = {}
    for single in (True, False):
        sess = tlf.Session(m, w, max_batch=B, max_pos=T, max_prefill_tokens=B * T, prefill_act_bf16=single)
        try:
            toks = torch.from_numpy(prompts).cuda()
            sess.prefill(toks)  # warm
            torch.cuda.synchronize()
            reps = 3
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                _, depths = sess.prefill(toks)
            e1.record()
            torch.cuda.synchronize()
            times[single] = e0.elapsed_time(e1) / reps
            dep = depths.cpu().numpy()
            if sess.stats()["status"] != 0:
                raise RuntimeError("device error in the prefill measurement")
        finally:
            sess.close()
            torch.cuda.empty_cache()
    ms = times[True]
    d, F, J, R = m.d_model, m.d_ff, m.n_layers, m.max_loops
    n = np.stack([(dep >= i).sum(axis=1) for i in range(1, R + 1)], axis=1)  # n_{b,i}
    gemm = float(n.sum()) * J * 2 * (4 * d * d + 3 * d * F)
    attn = float((n.astype(np.float64) * (n + 1) / 2).sum()) * J * 4 * d
    head = 2.0 * B * d * m.vocab
    flops = gemm + attn + head
    return {"workload": f"{name} prefill: batch {B} x {T}, d={d}, {m.n_heads}x{m.head_dim} heads, SwiGLU {F}, "
                        f"R={R}, J={J}; activations enter the matrix products as one bf16 part",
            "ms": ms, "tokens_per_s": B * T / ms * 1e3,
            "algorithmic_tflop": flops / 1e12, "tflops": flops / ms / 1e9,
            "mfma_frac": flops / ms / 1e9 / BF16_PEAK_TFLOPS,
            "hi_lo_parts": {"ms": times[False], "tflops": flops / times[False] / 1e9,
                            "mfma_frac": flops / times[False] / 1e9 / BF16_PEAK_TFLOPS}}


def train_gather_scatter(torch, synth, B=8, T=4096, d=1024, R=8, reps=20):
    """Training-side gather-scatter over all R loops of a batch of B x T tokens
    (float32 states of width d, depths drawn from the routed decode's depth
    mix): forward gather + out-of-place (and, separately, in-place) scatter
    per loop, backward gather of
    the state gradient + in-place scatter of the compact gradient per loop.
    Launched from a captured HIP graph (the host enqueues slower than these
    kernels run); HIP events around the replays on the capture's stream."""
    from paper_2609_15160_amd import train
    rows = B * T
    depth = torch.from_numpy(synth.make_train_depths(rows, R)).cuda()
    plans = [train.plan(depth, B, T, i) for i in range(1, R + 1)]
    H = [torch.from_numpy(synth.make_train_states(rows, d)).cuda()]
    H += [torch.empty_like(H[0]) for _ in range(R)]
    gen = torch.Generator(device="cuda").manual_seed(synth.SEED)  # seeded block outputs and gradients
    Y = [torch.randn(p.count, d, device="cuda", generator=gen) for p in plans]
    X = [torch.empty(p.count, d, device="cuda") for p in plans]
    dH = torch.randn(rows, d, device="cuda", generator=gen)
    dY = [torch.empty(p.count, d, device="cuda") for p in plans]

    def forward():
        for i, p in enumerate(plans):
            train.gather_raw(H[i], p, out=X[i])
            train.scatter_raw(H[i], Y[i], p, out=H[i + 1])

    Hin = torch.empty_like(H[0])

    def forward_in_place():
        for i, p in enumerate(plans):
            train.gather_raw(Hin, p, out=X[i])
            train.scatter_raw(Hin, Y[i], p, out=Hin)

    def backward():
        for i in reversed(range(R)):
            train.gather_raw(dH, plans[i], out=dY[i])
            train.scatter_raw(dH, Y[i], plans[i], out=dH)

    def plan_all():
        for i in range(1, R + 1):
            train.tlf.load().tlf_gs_plan(train._ptr(depth), B, T, i, train._ptr(plans[i - 1].index),
                                         train._ptr(plans[i - 1].slot), train._ptr(plans[i - 1].offsets),
                                         train._ptr(plans[i - 1].count_dev), train._stream())

    plan_ws = train.plan_workspace(B, T)

    def plan_all_chunked():
        for i in range(1, R + 1):
            train.tlf.load().tlf_gs_plan_ws(train._ptr(depth), B, T, i, train._ptr(plans[i - 1].index),
                                            train._ptr(plans[i - 1].slot), train._ptr(plans[i - 1].offsets),
                                            train._ptr(plans[i - 1].count_dev), train._ptr(plan_ws),
                                            plan_ws.numel(), train._stream())

    def timed(fn):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            fn()  # warm
        torch.cuda.current_stream().wait_stream(s)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    fwd_ms, bwd_ms, plan_ms = timed(forward), timed(backward), timed(plan_all)
    plan_chunked_ms = timed(plan_all_chunked)
    Hin.copy_(H[0])
    fwi_ms = timed(forward_in_place)
    n = [p.count for p in plans]
    fwd_bytes = sum(4 * c + 2 * 4 * c * d + 4 * rows + 4 * rows * d * 2 + 4 * c * d for c in n)
    bwd_bytes = sum(4 * c + 2 * 4 * c * d + 4 * rows + 3 * 4 * c * d for c in n)
    fwi_bytes = sum(4 * c + 2 * 4 * c * d + 4 * rows + 3 * 4 * c * d for c in n)
    plan_bytes = sum(4 * rows + 4 * c + 4 * rows + 4 * (B + 1) for c in n)
    return {"workload": f"training gather-scatter: batch {B} x {T} tokens, d={d} float32, R={R}, "
                        f"mean depth {float(depth.float().mean()):.2f}",
            "active_rows_per_loop": n,
            "forward_ms": fwd_ms, "forward_gbs": fwd_bytes / fwd_ms / 1e6,
            "forward_in_place_ms": fwi_ms, "forward_in_place_gbs": fwi_bytes / fwi_ms / 1e6,
            "backward_ms": bwd_ms, "backward_gbs": bwd_bytes / bwd_ms / 1e6,
            "plan_us_per_loop": plan_ms * 1e3 / R, "plan_gbs": plan_bytes / plan_ms / 1e6,
            "plan_chunked_us_per_loop": plan_chunked_ms * 1e3 / R,
            "frac": (fwd_bytes + bwd_bytes) / (fwd_ms + bwd_ms) / 1e6 / HBM_PEAK_GBS,
            "frac_in_place": (fwi_bytes + bwd_bytes) / (fwi_ms + bwd_ms) / 1e6 / HBM_PEAK_GBS,
            "what": "per pass over all loops; algorithmic bytes: each gathered row read and written once, "
                    "an out-of-place scatter reads and writes every row and reads each block-output row, "
                    "an in-place scatter reads two and writes one row per active row; indices and slots "
                    "4 bytes each"}


ATTN_SOURCE = os.path.join(ROOT, "paper_2609_15160_amd", "csrc", "attn.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_decode_bf16_d768_b256x2048_traffic.json")
CALIB_BYTES = 1 << 30  # the counted copy reads and writes exactly this many bytes


def source_digest(path=ATTN_SOURCE):
    import hashlib
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def measured_traffic(window, algo_bytes_per_launch):
    """Per-launch HBM bytes of the decode attention from committed rocprofv3
    counter runs.  They are reported only when they were taken on the current
    kernel source and over the same step window (warmup, timed and profiled
    step counts) with the same algorithmic bytes per launch as this run, since
    the work per step drifts with the greedy trajectory.  Returns (bytes or
    None, a record of the stored measurement and its traffic/algorithmic ratio)."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None, None
    info = {"file": os.path.relpath(TRAFFIC_FILE, ROOT), "window": rec.get("window"),
            "algo_bytes_per_launch": rec.get("algo_bytes_per_launch"),
            "traffic_bytes_per_launch": rec.get("traffic_bytes_per_launch")}
    if rec.get("algo_bytes_per_launch"):
        info["ratio"] = rec["traffic_bytes_per_launch"] / rec["algo_bytes_per_launch"]
    if rec.get("attn_source_sha256") != source_digest():
        info["status"] = "not reported: the kernel source changed since the counters were taken"
        return None, info
    same = rec.get("window") == window and rec.get("algo_bytes_per_launch") is not None and \
        abs(rec["algo_bytes_per_launch"] - algo_bytes_per_launch) <= 1e-9 * algo_bytes_per_launch
    if not same:
        info["status"] = "not reported: taken over another step window"
        return None, info
    info["status"] = "same kernel source, step window and algorithmic bytes as this run"
    return rec["traffic_bytes_per_launch"], info


def counter_summary(fetch_csv, write_csv, first, count, bench_json, window):
    """Summarize two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) of
    this benchmark.

    Each counter (KiB per dispatch) is scaled by what it reads for the
    calibration copy of CALIB_BYTES (the first copy kernel of the run), and
    averaged over the decode-attention dispatches [first, first + count) of
    the run, which are the routed run's attention-event pass.  The algorithmic
    bytes per launch of that pass come from the run's own JSON line
    (`bench_json`, the same command's output), together with the step window.
    """
    import csv

    def load(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        copy = next(r for r in rows if "copy" in r["Kernel_Name"])
        attn = [r for r in rows if "k_attn_decode" in r["Kernel_Name"]][first:first + count]
        if len(attn) != count:
            raise SystemExit(f"{path}: {len(attn)} attention dispatches in the window, expected {count}")
        factor = CALIB_BYTES / (float(copy["Counter_Value"]) * 1024.0)
        per = sum(float(r["Counter_Value"]) for r in attn) * 1024.0 * factor / len(attn)
        return factor, per, len(attn), float(copy["Counter_Value"])

    ff, fetch, n, fcopy = load(fetch_csv, "FETCH_SIZE")
    wf, write, n2, wcopy = load(write_csv, "WRITE_SIZE")
    run = json.loads(open(bench_json).read().strip().splitlines()[-1])
    algo = run["roofline"]["algo_bytes_per_launch"]
    return {"attn_source_sha256": source_digest(), "dispatches": n, "window": window,
            "algo_bytes_per_launch": algo,
            "fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
            "traffic_bytes_per_launch": fetch + write, "ratio": (fetch + write) / algo,
            "fetch_scale": ff, "write_scale": wf,
            "calibration": f"copy of {CALIB_BYTES} bytes read {fcopy:.1f} KiB FETCH_SIZE and "
                           f"{wcopy:.1f} KiB WRITE_SIZE"}


def mfma_summary(counter_csv):
    """MFMA activity of the prefill from a rocprofv3 --pmc run of
    `bench.py --prefill-only` that collected MfmaUtil and MfmaFlopsBF16.

    The run holds two sessions of four prefills each (one warm-up, three
    timed): activations as one bf16 part, then as hi + lo parts.  A prefill
    is its embedding kernel with the fill kernels just before it, through its
    last-position LM head (the last GEMM before the next prefill; the second
    session's set-up kernels fall outside).  Per session, over its timed prefills and
    per kernel: the MFMA busy fraction (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE x SIMDs, averaged with each dispatch's duration as the
    weight), the bf16 MFMA work executed (MOPS x 512) and its rate over the
    dispatch durations.  Dispatches run one at a time under counter
    collection, so durations are those of isolated kernels."""
    import csv
    import collections
    disp = {}
    for r in csv.DictReader(open(counter_csv)):
        d = disp.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"],
                                                    "us": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    rows = [disp[k] for k in sorted(disp)]
    starts = [i for i, r in enumerate(rows) if "k_embed_route" in r["name"]]
    if len(starts) != 8:
        raise SystemExit(f"{counter_csv}: {len(starts)} prefills, expected 8 (two sessions of four)")
    bounds = starts + [len(rows)]

    def prefill_rows(p):
        a = bounds[p]
        while a > 0 and "k_fill" in rows[a - 1]["name"]:
            a -= 1
        gemms = [i for i in range(bounds[p], bounds[p + 1]) if "k_gemm" in rows[i]["name"]]
        return rows[a:gemms[-1] + 1]
    out = {}
    for label, first in (("one_part", 1), ("hi_lo_parts", 5)):
        agg = collections.defaultdict(lambda: {"calls": 0, "us": 0.0, "util_us": 0.0, "flop": 0.0})
        for p in range(first, first + 3):
            for r in prefill_rows(p):
                a = agg[r["name"]]
                a["calls"] += 1
                a["us"] += r["us"]
                a["util_us"] += r.get("MfmaUtil", 0.0) * r["us"]
                a["flop"] += r.get("MfmaFlopsBF16", 0.0)
        tot_us = sum(a["us"] for a in agg.values())
        tot_flop = sum(a["flop"] for a in agg.values())
        kernels = sorted(agg.items(), key=lambda kv: -kv[1]["us"])
        out[label] = {
            "prefills": 3, "ms_per_prefill": tot_us / 3e3,
            "mfma_busy_pct": sum(a["util_us"] for a in agg.values()) / tot_us,
            "executed_tflop_per_prefill": tot_flop / 3e12,
            "executed_tflops": tot_flop / (tot_us * 1e6),
            "kernels": [{"name": n, "calls": a["calls"] // 3, "ms_per_prefill": a["us"] / 3e3,
                         "mfma_busy_pct": a["util_us"] / a["us"] if a["us"] else 0.0,
                         "executed_tflop_per_prefill": a["flop"] / 3e12,
                         "executed_tflops": a["flop"] / (a["us"] * 1e6) if a["us"] else 0.0}
                        for n, a in kernels[:10]]}
    return out


def prefill_trace_summary(trace_csv, loops, layers, first=1, count=3):
    """Per-loop kernel durations of `--prefill-only` from a rocprofv3 kernel
    trace: prefills [first, first + count) of the trace (the one-part
    session's timed prefills; prefill k starts at the k-th prefill planner
    dispatch; `first` >= 1), each (loop, layer) running QKV, attention, O,
    gate/up and down in that order; us per call averaged over the prefills
    and layers."""
    import csv
    import collections
    rows = list(csv.DictReader(open(trace_csv)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    plans = [k for k, r in enumerate(rows) if "k_plan_prefill" in r["Kernel_Name"]]
    names = ("qkv", "attn", "o", "gate_up", "down")
    per = collections.defaultdict(list)
    spans = []
    for pf in range(first, first + count):
        a = plans[pf]
        b = plans[pf + 1] if pf + 1 < len(plans) else len(rows)
        blk = [r for r in rows[a + 1:b] if "k_gemm" in r["Kernel_Name"] or "k_attn_prefill" in r["Kernel_Name"]]
        blk = blk[:loops * layers * 5]
        for q, r in enumerate(blk):
            i, rem = divmod(q, layers * 5)
            per[(i, names[rem % 5])].append(dur(r))
        # span: from the first kernel after the previous prefill's last GEMM
        # (its LM head) to this prefill's LM head
        prev = max(k for k in range(plans[pf - 1], a) if "k_gemm" in rows[k]["Kernel_Name"])
        end = max(k for k in range(a, b) if "k_gemm" in rows[k]["Kernel_Name"])
        spans.append((int(rows[end]["End_Timestamp"]) - int(rows[prev + 1]["Start_Timestamp"])) / 1e3)
    table = [{"loop": i + 1, **{n: sum(per[(i, n)]) / len(per[(i, n)]) for n in names if per[(i, n)]}}
             for i in range(loops)]
    return {"prefills": [first, first + count], "span_us": sum(spans) / len(spans),
            "per_prefill_us": {n: layers * sum(t.get(n, 0.0) for t in table) for n in names},
            "per_loop_us": table}


def trace_summary(trace_csv, routed_launches, last_dispatches, loops, layers, first_step, last_step):
    """Per-kernel durations from a rocprofv3 kernel trace of this benchmark,
    the decode attention's average over the routed run's event-timed region
    (its launches are the first `routed_launches` attention dispatches of the
    trace, and the timed region is the last `last_dispatches` of those), and
    the average duration of every (loop, layer, kernel) of the routed run's
    decode steps [first_step, last_step) (step k starts at the k-th decode
    planner dispatch; each (loop, layer) runs QKV, attention, O, gate/up, down)."""
    import csv
    import collections
    rows = list(csv.DictReader(open(trace_csv)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    agg = collections.defaultdict(lambda: [0, 0.0])
    for r in rows:
        agg[r["Kernel_Name"]][0] += 1
        agg[r["Kernel_Name"]][1] += dur(r)
    attn = [r for r in rows if "k_attn_decode" in r["Kernel_Name"]][:routed_launches][-last_dispatches:]
    durs = [dur(r) for r in attn]
    top = sorted(agg.items(), key=lambda kv: -kv[1][1])[:12]
    plans = [k for k, r in enumerate(rows) if "k_plan_decode" in r["Kernel_Name"]]
    names = ("qkv", "attn", "o", "gate_up", "down")
    per = collections.defaultdict(list)
    spans, gaps = [], []
    for st in range(first_step, last_step):
        a = plans[st]
        b = plans[st + 1] if st + 1 < len(plans) else len(rows)
        blk = [r for r in rows[a + 1:b] if "k_attn_decode" in r["Kernel_Name"] or "k_dgemm" in r["Kernel_Name"]]
        blk = blk[:loops * layers * 5]
        for q, r in enumerate(blk):
            i, rem = divmod(q, layers * 5)
            j, p = divmod(rem, 5)
            per[(i, j, names[p])].append(dur(r))
        step_rows = rows[a - 1:b - 1]  # the step's embedding + router kernel precedes its planner
        spans.append((int(step_rows[-1]["End_Timestamp"]) - int(step_rows[0]["Start_Timestamp"])) / 1e3)
        gaps.append(sum((int(y["Start_Timestamp"]) - int(x["End_Timestamp"])) / 1e3
                        for x, y in zip(step_rows, step_rows[1:])))
    table = [{"loop": i + 1, "layer": j + 1,
              **{n: sum(per[(i, j, n)]) / len(per[(i, j, n)]) for n in names if per[(i, j, n)]}}
             for i in range(loops) for j in range(layers)]
    totals = {n: sum(t.get(n, 0.0) for t in table) for n in names}
    return {"kernels": [{"name": n, "calls": c, "total_ms": t / 1e3, "avg_us": t / c} for n, (c, t) in top],
            "attn_routed_timed_region": {"dispatches": len(durs), "avg_us": sum(durs) / max(len(durs), 1)},
            "decode_steps": {"steps": [first_step, last_step],
                             "span_us": sum(spans) / max(len(spans), 1),
                             "gaps_us": sum(gaps) / max(len(gaps), 1),
                             "per_step_us": totals, "per_loop_layer_us": table}}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=80)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--profiled-steps", type=int, default=10,
                    help="steps per profiled pass after the timed region (two passes, launched eagerly: "
                         "events around the loop region, then also around each attention launch)")
    ap.add_argument("--latency-steps", type=int, default=20,
                    help="graph-replayed steps after the profiled passes, each timed on its own (p50/p99)")
    ap.add_argument("--config", default="bf16_d768_b256x2048")
    ap.add_argument("--no-fixed", action="store_true", help="skip the fixed-depth comparison")
    ap.add_argument("--no-graph", action="store_true",
                    help="launch the timed decode steps kernel by kernel instead of replaying a HIP graph")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefill measurement")
    ap.add_argument("--no-sweep", action="store_true", help="skip the MLP-router threshold sweep")
    ap.add_argument("--no-ablation", action="store_true", help="skip the gather-scatter-off decode")
    ap.add_argument("--no-ttft", action="store_true", help="skip the time-to-first-token sweep")
    ap.add_argument("--no-train", action="store_true", help="skip the training-side gather-scatter measurement")
    ap.add_argument("--train-only", action="store_true",
                    help="measure only the training-side gather-scatter and print its JSON")
    ap.add_argument("--no-adaln", action="store_true", help="skip the AdaLN-conditioned decode")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the batch 32 x 512 and batch 64 x 4096 (d=2048) decode workloads")
    ap.add_argument("--prefill-only", action="store_true",
                    help="run only the prefill measurement (batch 8 x 4096) and print its JSON")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help=f"first run a device copy of {CALIB_BYTES} bytes (counter calibration)")
    ap.add_argument("--counter-summary", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "BENCH_JSON"),
                    help="summarize rocprofv3 FETCH_SIZE / WRITE_SIZE runs of this benchmark (run with the same "
                         "--warmup/--steps/--profiled-steps; BENCH_JSON is that run's output) and exit")
    ap.add_argument("--no-tiny", action="store_true", help="skip the tiny fp32 model's per-step latency")
    ap.add_argument("--mfma-summary", metavar="COUNTER_CSV",
                    help="summarize a rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 run of --prefill-only and exit")
    ap.add_argument("--prefill-trace-summary", metavar="TRACE_CSV",
                    help="print per-loop prefill kernel durations from a rocprofv3 kernel trace of --prefill-only")
    ap.add_argument("--trace-summary", metavar="TRACE_CSV",
                    help="summarize a rocprofv3 kernel trace of this benchmark's default run and exit")
    args = ap.parse_args()
    if args.mfma_summary:
        print(json.dumps(mfma_summary(args.mfma_summary)))
        return
    if args.prefill_trace_summary:
        import synth
        m = synth.CONFIGS["bf16_d1024_prefill_b8x4096"]
        print(json.dumps(prefill_trace_summary(args.prefill_trace_summary, m.max_loops, m.n_layers)))
        return
    if args.trace_summary:
        import synth
        m = synth.CONFIGS[args.config]
        per_step = m.max_loops * m.n_layers
        routed = (args.warmup + args.steps + 2 * args.profiled_steps) * per_step
        print(json.dumps(trace_summary(args.trace_summary, routed, args.profiled_steps * per_step,
                                       m.max_loops, m.n_layers, args.warmup, args.warmup + args.steps)))
        return
    if args.counter_summary:
        import synth
        m = synth.CONFIGS[args.config]
        per_step = m.max_loops * m.n_layers  # attention launches per step: R x J
        first = (args.warmup + args.steps + args.profiled_steps) * per_step
        window = {"warmup": args.warmup, "steps": args.steps, "profiled_steps": args.profiled_steps}
        print(json.dumps(counter_summary(*args.counter_summary[:2], first, args.profiled_steps * per_step,
                                         args.counter_summary[2], window)))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (decode shards by sequence "
              "with no exchange; run one process per GPU on its own share of the batch)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import synth
    from paper_2609_15160_amd import tlf

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()
    if args.prefill_only:
        print(json.dumps(prefill_measure(torch, tlf, synth, "bf16_d1024_prefill_b8x4096")), flush=True)
        return
    if args.train_only:
        print(json.dumps(train_gather_scatter(torch, synth)), flush=True)
        return
    base = synth.CONFIGS[args.config]
    if (args.warmup + args.steps + 2 * args.profiled_steps + args.latency_steps > base.steps
            or args.profiled_steps < 1 or args.latency_steps < 0):
        print(f"warmup + steps + 2 x profiled-steps + latency-steps must be <= {base.steps} for {args.config} "
              f"(profiled-steps >= 1)", file=sys.stderr)
        sys.exit(2)
    model = base
    t0 = time.perf_counter()
    w = synth.make_weights(model)
    prompts = synth.make_prompts(model)
    B, T = prompts.shape
    log(f"inputs ready in {time.perf_counter() - t0:.1f}s: batch {B} x prompt {T}")

    ms, (stb, st), prefill_s, hist, lat = run_config(torch, tlf, model, w, prompts, args.warmup, args.steps,
                                                     args.profiled_steps, graph=not args.no_graph,
                                                     latency_steps=args.latency_steps)
    log(f"routed: {ms / args.steps:.3f} ms/step, prefill {prefill_s:.2f}s, depth hist {hist}")
    value = B * args.steps / (ms / 1e3)
    attn_gbs = st["attn_algo_bytes"] / (st["attn_ms"] / 1e3) / 1e9
    per_launch = st["attn_algo_bytes"] / max(st["attn_launches"], 1)
    hot_bytes = hot_path_bytes(stb, model, args.profiled_steps, B)
    hot_gbs = hot_bytes / (stb["block_ms"] / 1e3) / 1e9
    tot_hist = np.asarray(hist, dtype=np.float64)
    mean_depth = float((tot_hist * np.arange(1, len(hist) + 1)).sum() / max(tot_hist.sum(), 1))
    window = {"warmup": args.warmup, "steps": args.steps, "profiled_steps": args.profiled_steps}
    traffic, traffic_info = measured_traffic(window, per_launch)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": model.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, uniform-random prompts, greedy decode)",
        "config": {"workload": f"{args.config} decode: batch {B} x prompt {T}, {model.n_layers}-layer "
                               f"d={model.d_model} looped block ({model.n_heads}x{model.head_dim} heads, "
                               f"SwiGLU {model.d_ff}, vocab {model.vocab}), R={model.max_loops}, "
                               f"argmax router, 16-token KV pages",
                   "batch": B, "prompt": T, "max_loops": model.max_loops, "layers": model.n_layers,
                   "mean_depth": mean_depth},
        "roofline": {"bound": "hbm", "kernel": "k_attn_decode", "achieved": attn_gbs, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": attn_gbs / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_counters": traffic_info,
                     "launches": st["attn_launches"], "avg_launch_us": st["attn_ms"] * 1e3 / st["attn_launches"],
                     "algo_bytes_per_launch": per_launch,
                     "measured": f"HIP events around each attention launch over {args.profiled_steps} decode "
                                 f"steps (the last profiled pass)"},
        "hot_path": {"what": "loop-and-layer region per step: decode attention plus the QKV, O, gate/up "
                             "and down projections with their fused norms, launched kernel by kernel; "
                             "HIP events around the region only",
                     "achieved_gbs": hot_gbs, "frac": hot_gbs / HBM_PEAK_GBS,
                     "ms_per_step": stb["block_ms"] / args.profiled_steps,
                     "algo_bytes_per_step": hot_bytes / args.profiled_steps},
        "prefill_s": prefill_s,
    }
    if lat:
        q = np.percentile(np.asarray(lat), [50, 99])
        out["step_latency_ms"] = {"steps": len(lat), "p50": float(q[0]), "p99": float(q[1]), "max": float(max(lat)),
                                  "mean": float(np.mean(lat)),
                                  "what": "graph-replayed steps after the profiled passes, an event pair "
                                          "around each step"}
    read_gbs = stream_read_gbs(torch, tlf)
    out["stream_read"] = {"gbs": read_gbs,
                          "what": "tlf_probe_read over 4 GiB: the decode attention's 16-byte non-temporal "
                                  "loads, bytes read per second",
                          "attn_frac_of_read": attn_gbs / read_gbs, "hot_path_frac_of_read": hot_gbs / read_gbs}
    log(f"stream read: {read_gbs:.0f} GB/s")
    if not args.no_tiny:
        out["tiny_f32"] = tiny_decode(torch, tlf, synth)
        log(f"tiny f32: {out['tiny_f32']['us_per_step_graph']:.1f} us/step")
    if not args.no_fixed:
        fms, (_, fst), fpre, _ = run_config(torch, tlf, model, w, prompts, args.warmup, args.steps,
                                       args.profiled_steps, route_rule="fixed", fixed_depth=model.max_loops,
                                       graph=not args.no_graph)
        fgbs = fst["attn_algo_bytes"] / (fst["attn_ms"] / 1e3) / 1e9
        out["fixed_depth"] = {"depth": model.max_loops, "value": B * args.steps / (fms / 1e3),
                              "ms_per_step": fms / args.steps, "attn_achieved_gbs": fgbs,
                              "attn_frac": fgbs / HBM_PEAK_GBS, "prefill_s": fpre,
                              "routed_speedup": fms / ms}
        log(f"fixed depth {model.max_loops}: {fms / args.steps:.3f} ms/step")
    if not args.no_ablation:
        out["gather_scatter_off"] = gather_scatter_off(torch, tlf, model, w, prompts, ms / args.steps)
        log(f"gather-scatter off: {out['gather_scatter_off']['ms_per_step']:.3f} ms/step")
    if not args.no_adaln:
        out["adaln"] = adaln_decode(torch, tlf, synth, args.config, ms / args.steps)
        log(f"adaln: {out['adaln']['ms_per_step']:.3f} ms/step")
    if not args.no_others:
        out["other_workloads"] = other_workloads(torch, tlf, synth)
    if not args.no_ttft:
        out["ttft"] = ttft_sweep(torch, tlf, model, w, synth)
    if not args.no_prefill:
        out["prefill"] = prefill_measure(torch, tlf, synth, "bf16_d1024_prefill_b8x4096")
        log(f"prefill 8x4096: {out['prefill']['ms']:.2f} ms")
    if not args.no_train:
        out["train_gather_scatter"] = train_gather_scatter(torch, synth)
        t = out["train_gather_scatter"]
        log(f"train gather-scatter: fwd {t['forward_ms']:.3f} ms {t['forward_gbs']:.0f} GB/s, "
            f"in place {t['forward_in_place_ms']:.3f} ms, bwd {t['backward_ms']:.3f} ms {t['backward_gbs']:.0f} GB/s, "
            f"plan {t['plan_us_per_loop']:.1f} us/loop (chunked {t['plan_chunked_us_per_loop']:.1f})")
    if not args.no_sweep:
        out["router_threshold_sweep"] = threshold_sweep(torch, tlf, synth, args.config)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(model, w, prompts, args.cpu_seconds)
        log(f"cpu baseline: {out['cpu_baseline']['value']:.3f} tokens/s")
        out["cpu_one_core"] = cpu_one_core(synth)
        log("cpu one core: done")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
