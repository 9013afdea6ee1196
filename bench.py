#!/usr/bin/env python3
"""Throughput of the Rift hot path on one MI355X.

One step = one whole scene-query: tile scoring and pruning (rift_score_tiles),
per-tile token selection (rift_select_tokens), varlen compaction (rift_compact)
and the decoder prefill of every retained prompt (rift_prefill), on synthetic
inputs already resident in HBM.  The metric is retained vision tokens
prefilled per second (sum of the per-tile budgets of one query, times steps,
over the timed wall time), with milliseconds per scene-query alongside.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "retained vision tokens prefilled/sec + ms per 400-tile scene query, 1 GPU"
PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
STAGES = ("qkv_rope", "attention", "out_proj", "gate_up_swiglu", "down_proj")
# (each GEMM adds a half-tile tail launch when its last round over the CUs is at most half full)
KERNEL_NAMES = {"qkv_rope": "QKV+RoPE GEMM (gemm_bf16_pp_kernel<0>)",
                "attention": "varlen causal attention (attn_bf16_kernel)",
                "out_proj": "output projection + residual (gemm_bf16_pp_kernel<1>)",
                "gate_up_swiglu": "gate/up+SwiGLU GEMM (gemm_bf16_pp_kernel<2>)",
                "down_proj": "down projection + residual (gemm_bf16_pp_kernel<1>)"}
GEMM_SRC = os.path.join(ROOT, "paper_2609_29029_amd", "csrc", "gemm_bf16.hip")

# HBM traffic of one gate/up+SwiGLU launch at the 400-tile workload with the shared
# system prefix (T = 18,739 packed rows), from two rocprofv3 --pmc runs of this
# script with --traffic-calibration (FETCH_SIZE, then WRITE_SIZE), each scaled
# by what the counter reads for the 1 GiB calibration copy (FETCH_SIZE reads
# half the bytes, WRITE_SIZE all of them): 5.8448 GB fetched + 0.4126 GB written
# (profiles/scene20_l32_counters.md).  Valid only for the GEMM source it was
# measured on, identified by its SHA-256; otherwise reported as null.
TRAFFIC = {"stage": "gate_up_swiglu",
           "gemm_src_sha256": "cb39e4abfd0dc96cef4fed7d068d84fa7a9eb94d172530d4a6ec47f03dc73a45",
           "packed_tokens": 18739,
           "bytes": 6.2574e9}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def stage_flops(T: int, d: int, ffn: int, seq_lens, n_prefix: int = 0) -> dict:
    """Algorithmic flops of one launch of each prefill stage (one layer) over
    T packed rows.  seq_lens are the prompts' whole lengths; with a shared
    prefix of n_prefix rows its causal triangle is computed once, and each
    prompt's own queries attend to the prefix and to their own earlier rows."""
    P = n_prefix
    attn = sum(2 * 2 * d * (L * (L + 1) // 2 - P * (P + 1) // 2) for L in seq_lens)
    attn += 2 * 2 * d * P * (P + 1) // 2   # QK^T and PV over the causal triangles
    return {"qkv_rope": 2 * T * d * 3 * d, "attention": attn, "out_proj": 2 * T * d * d,
            "gate_up_swiglu": 2 * T * d * 2 * ffn, "down_proj": 2 * T * ffn * d}


def _cpu_keys_worker(args):
    """One worker of the CPU baseline: the oracle's per-token keys of a slice
    of tiles (stored values in, float64 keys out)."""
    tiles, dtype, qbank = args
    import synth
    from oracle import rift_oracle as O
    return O.token_keys(synth.to_f64(tiles, dtype), O.query_direction(synth.to_f64(qbank, dtype)))


def cpu_baseline(w, sc, seq_lens_by_tier, n_layers_sample: int) -> dict:
    """The oracle as it stands on the host cores.  Every core in the process's
    affinity set is used, capped at the host share of one GPU (16): BLAS and
    OpenMP pools are set to that count, and the per-token keys of Stage 1 (the
    oracle's cost there) are spread over that many worker processes, a slice
    of tiles each.  Stage 1 (all tiles), selection and compaction run on the
    whole query; the prefill runs `n_layers_sample` decoder layers on one
    prompt of each budget tier and is extrapolated to every prompt and layer
    (every layer costs the same)."""
    import multiprocessing as mp
    from concurrent.futures import ProcessPoolExecutor
    import synth
    from oracle import rift_oracle as O
    cores = max(1, min(len(os.sched_getaffinity(0)), 16))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:  # pragma: no cover
        limiter = None
    m = w.model
    times = {}
    # Stage 1: keys in parallel over tile slices (fresh interpreters: the
    # parent has initialised the GPU, the workers never touch it), then the
    # oracle's pooling, normalisation and ranking on the gathered keys
    t0 = time.perf_counter()
    bounds = np.linspace(0, w.n_tiles, cores + 1).astype(int)
    jobs = [(sc.tokens[a:b], w.dtype, sc.qbank) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
    with ProcessPoolExecutor(max_workers=len(jobs), mp_context=mp.get_context("spawn")) as ex:
        r = np.concatenate(list(ex.map(_cpu_keys_worker, jobs)))
    s = O.tile_scores(r)
    u = O.normalise(s)
    order, n_keep = O.rank_and_keep(s, u, w.keep_count, w.tau)
    times["stage1_s"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    kept = list(order[:n_keep])
    budgets = O.assign_budgets(len(kept), w.levels, w.tier_num, w.tier_den)
    offs, sel = O.select_tokens(r, kept, budgets)
    times["select_s"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    O.compact(sc.tokens, kept, offs, sel, sc.sys, sc.qry)
    times["compact_s"] = time.perf_counter() - t0
    W = {k: synth.to_f64(v, w.dtype) for k, v in synth.make_layer(w, 0).items()}
    rng = np.random.default_rng(0)
    t_prefill = 0.0
    n_ls = max(1, min(n_layers_sample, m.n_layers))
    measured = 0.0
    for L, count in seq_lens_by_tier:
        x = rng.standard_normal((L, m.d))
        t0 = time.perf_counter()
        for _ in range(n_ls):
            x = O.decoder_layer(x, W, m.n_heads, m.head_dim, m.rms_eps, m.rope_base, np.arange(L))
        dt = time.perf_counter() - t0
        measured += dt
        t_prefill += dt * count * m.n_layers / n_ls
    times["prefill_s"] = t_prefill
    if limiter is not None:
        limiter.restore_original_limits()
    total = sum(times.values())
    retained = int(sum(budgets))
    return {"value": retained / total, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "stage_s": {k: round(v, 2) for k, v in times.items()},
            "sample": (f"float64 NumPy oracle on {cores} cores: Stage 1 on all {w.n_tiles} tiles "
                       f"({len(jobs)} worker processes over tile slices), selection and compaction of "
                       f"the whole query, measured; prefill measured as {n_ls} decoder layers on one "
                       f"prompt per budget tier (lengths {[L for L, _ in seq_lens_by_tier]}, "
                       f"{measured:.1f} s) and extrapolated to {sum(c for _, c in seq_lens_by_tier)} "
                       f"prompts x {m.n_layers} layers; {total:.1f} s per query")}


def exhaustive_setup(R, torch, w, tokens, qbank, sysd, qryd, layers, cfg, chunk: int = 50,
                     shared: bool = True):
    """Every tile kept at the full budget n_v: the no-pruning baseline the
    paper compares against.  Same kernels; the prefill runs as consecutive
    calls of `chunk` prompts each (all prompts have the same length), since one
    call is limited to T * max(d, ffn) < 2^31.  With `shared`, as in the Rift
    query, each call's prompts share their system rows (packed once per call).
    Returns a function that enqueues one whole exhaustive query on the current
    stream and returns its status words, and the query's shape."""
    n, nv, d = tokens.shape
    dev = tokens.device
    f64, f32, i32 = torch.float64, torch.float32, torch.int32
    nq = qbank.shape[0]
    fixed = sysd.shape[0] + qryd.shape[0]
    P = sysd.shape[0] if shared else 0
    L = nv + fixed
    Lown = L - P                      # packed rows of a prompt after a shared prefix
    key = torch.empty(n * nv, dtype=f64, device=dev)
    sim = torch.empty(n * nv, nq, dtype=f32, device=dev)
    score = torch.empty(n, dtype=f64, device=dev)
    u = torch.empty(n, dtype=f32, device=dev)
    order = torch.empty(n, dtype=i32, device=dev)
    nkeep = torch.empty(1, dtype=i32, device=dev)
    sws = torch.empty(max(256, R.rift_score_workspace_size(n, nv, d)), dtype=torch.uint8, device=dev)
    budgets = torch.full((n,), nv, dtype=i32, device=dev)
    offs = torch.empty(n + 1, dtype=i32, device=dev)
    sel = torch.empty(n * nv, dtype=i32, device=dev)
    st1 = torch.empty(1, dtype=i32, device=dev)
    chunks = [(c, min(n, c + chunk)) for c in range(0, n, chunk)]
    # one packed batch per prefill call: [system rows once | prompts' own rows]
    Tc = {m: P + m * Lown for m in {b - a for a, b in chunks}}
    T = sum(P + (b - a) * Lown for a, b in chunks)
    packed = torch.empty(max(Tc.values()), d, dtype=tokens.dtype, device=dev)
    cu = torch.empty(chunk + 2, dtype=i32, device=dev)
    pos = torch.empty(max(Tc.values()), dtype=i32, device=dev)
    offs_c = torch.arange(0, chunk + 1, dtype=i32, device=dev) * nv   # every budget is n_v
    st2 = torch.empty(len(chunks), dtype=i32, device=dev)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, max(Tc.values()), L), dtype=torch.uint8, device=dev)
    hid = torch.empty(max(Tc.values()), d, dtype=f32, device=dev)

    def run():
        R.rift_score_tiles(tokens, qbank, n, 0.0, key, sim, score, u, order, nkeep, sws)
        R.rift_select_tokens(key, n, nv, order, budgets, n, offs, sel, st1)
        for c, (a, b) in enumerate(chunks):
            m = b - a
            ncu = m + (2 if shared else 1)
            R.rift_compact(tokens, order[a:b], offs_c[:m + 1], sel[a * nv:b * nv], m, sysd, qryd,
                           packed[:Tc[m]], cu[:ncu], pos[:Tc[m]], st2[c:c + 1], shared_prefix=shared)
            R.rift_prefill(cfg, layers, packed[:Tc[m]], cu[:ncu], pos[:Tc[m]], ncu - 1, L, hid[:Tc[m]], ws,
                           n_prefix=P)
        return st1, st2

    return run, {"packed_tokens": T, "prompts": n, "prefill_calls": len(chunks), "seq_len": L, "n_prefix": P}


def exhaustive_run(run, shape, w, torch) -> dict:
    """One exhaustive query, timed with HIP events on the current stream."""
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    st1, st2 = run()
    e1.record()
    torch.cuda.synchronize()
    assert int(st1.item()) == 0 and int(st2.abs().max().item()) == 0
    ms = e0.elapsed_time(e1)
    m = w.model
    T, L, n = shape["packed_tokens"], shape["seq_len"], shape["prompts"]
    P = shape["n_prefix"]
    per = -(-n // shape["prefill_calls"])
    fl = {k: 0 for k in STAGES}
    for a in range(0, n, per):   # each call's own shared prefix
        mc = min(n, a + per) - a
        for k, v in stage_flops(P + mc * (L - P), m.d, m.ffn, [L] * mc, P).items():
            fl[k] += v
    tflop = sum(fl.values()) * m.n_layers / 1e12
    return {"ms": round(ms, 2), "packed_tokens": T, "prompts": n, "prefill_calls": shape["prefill_calls"],
            "tflop": round(tflop, 1), "frac_bf16_peak": round(tflop / (ms * 1e-3) / PEAK_BF16_TFLOPS, 4)}


def mfma_ceiling(torch, seconds_per_form: float = 0.4) -> dict:
    """bf16 MFMA throughput with nothing but MFMAs on every CU (operands rotating
    over eight register pairs, as in a GEMM), from libriftcalib.so: the
    attainable ceiling under the board power limit, reported beside the
    nominal peak.  Also with all-zero operands (which draw far less power, so
    the clock stays near its maximum): two waves per SIMD, the instruction's
    own rate, and one wave per SIMD, the rate at which a lone wave can issue
    (the ping-pong GEMM loop has one MFMA wave per SIMD at a time).  Last, the
    random-operand MFMAs with the LDS reads (384 bytes per MFMA) and LDS DMA
    (128 bytes per MFMA) of the gate/up loop but none of its waits: the
    ceiling once the loop's data movement shares the power budget.  Three
    timed launches per case, median."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_29029_amd", "libriftcalib.so"))
    lib.rift_calib_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                         ctypes.c_int, ctypes.c_void_p]
    g = torch.Generator(device="cuda").manual_seed(0x52494654)
    src = torch.randn(65536, device="cuda", generator=g).to(torch.bfloat16)
    zero = torch.zeros(65536, device="cuda", dtype=torch.bfloat16)
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.empty(blocks * 512, device="cuda", dtype=torch.float32)
    stream = torch.cuda.current_stream().cuda_stream
    res = {}
    cases = ((0, src, "v_mfma_f32_16x16x32_bf16"), (1, src, "v_mfma_f32_32x32x16_bf16"),
             (0, zero, "v_mfma_f32_16x16x32_bf16 zero operands"),
             (2, zero, "v_mfma_f32_16x16x32_bf16 zero operands, one wave per SIMD"))
    for form, operands, name in cases:
        per_iter = blocks * (4 if form == 2 else 8) * 262144
        iters = max(8, int(seconds_per_form * 1.5e15 / per_iter) // 8 * 8)
        ts = []
        for rep in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            rc = lib.rift_calib_mfma_bf16(form, operands.data_ptr(), out.data_ptr(), blocks, iters, stream)
            e1.record()
            torch.cuda.synchronize()
            if rc != 0:
                raise RuntimeError(f"rift_calib_mfma_bf16 returned {rc}")
            if rep:   # the first launch warms the clocks up
                ts.append(e0.elapsed_time(e1))
        tf = per_iter * iters / (statistics.median(ts) * 1e-3) / 1e12
        res[name] = {"TFLOPs": round(tf, 1), "frac_nominal": round(tf / PEAK_BF16_TFLOPS, 4)}
    # the same MFMAs with the gate/up loop's LDS reads and LDS DMA (no waits or
    # barriers): the ceiling once the loop's own data movement draws power too
    lib.rift_calib_mfma_bf16_moves.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_longlong,
                                               ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    dsrc = torch.randn(1 << 21, device="cuda", generator=g).to(torch.bfloat16)   # 4 MiB
    per_iter = blocks * 8 * 262144
    iters = max(16, int(seconds_per_form * 1.5e15 / per_iter) // 16 * 16)
    ts = []
    for rep in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rc = lib.rift_calib_mfma_bf16_moves(src.data_ptr(), dsrc.data_ptr(), dsrc.numel() * 2, out.data_ptr(),
                                            blocks, iters, stream)
        e1.record()
        torch.cuda.synchronize()
        if rc != 0:
            raise RuntimeError(f"rift_calib_mfma_bf16_moves returned {rc}")
        if rep:
            ts.append(e0.elapsed_time(e1))
    tf = per_iter * iters / (statistics.median(ts) * 1e-3) / 1e12
    res["v_mfma_f32_16x16x32_bf16 with the gate/up loop's LDS reads and LDS DMA"] = {
        "TFLOPs": round(tf, 1), "frac_nominal": round(tf / PEAK_BF16_TFLOPS, 4)}
    return res


class EnergyMeter:
    """Board energy of the GPU from its own accumulator (amdsmi): the counter
    advances in units of `counter_resolution` microjoules and carries the
    timestamp of its last update.  The average power of a workload is the
    difference of two updates that both fall while it runs, over the time
    between them; the poller thread records every update it sees."""

    def __init__(self, torch):
        import amdsmi
        self.smi = amdsmi
        amdsmi.amdsmi_init()
        hs = amdsmi.amdsmi_get_processor_handles()
        bus = torch.cuda.get_device_properties(0).pci_bus_id
        pick = [h for h in hs if int(amdsmi.amdsmi_get_gpu_device_bdf(h).split(":")[1], 16) == bus]
        if len(pick) != 1:
            raise RuntimeError(f"no unique amdsmi device on PCI bus {bus:#x} ({len(hs)} devices)")
        self.h = pick[0]

    def read(self):
        e = self.smi.amdsmi_get_energy_count(self.h)
        return e["energy_accumulator"] * e["counter_resolution"] * 1e-6, e["timestamp"] * 1e-9

    def average_power(self, work, min_seconds: float, min_updates: int = 4) -> dict:
        """Call work() back to back until the counter has updated at least
        `min_updates` times over at least `min_seconds` since the first update
        seen after the loop began; returns watts, the span and the number of
        work() calls per second of wall time."""
        import threading
        ups, stop = [], threading.Event()

        def poll():
            last = None
            while not stop.is_set():
                j, t = self.read()
                if t != last:
                    ups.append((j, t))
                    last = t
                time.sleep(0.005)

        th = threading.Thread(target=poll, daemon=True)
        th.start()
        while not ups:
            time.sleep(0.001)
        t0 = time.perf_counter()
        calls = 0
        while True:
            work()
            calls += 1
            inside = ups[1:]   # ups[0] was read before the loop began
            if len(inside) >= min_updates and inside[-1][1] - inside[0][1] >= min_seconds:
                break
        wall = time.perf_counter() - t0
        stop.set()
        th.join()
        (j0, s0), (j1, s1) = inside[0], inside[-1]
        return {"watts": (j1 - j0) / (s1 - s0), "span_s": s1 - s0, "updates": len(inside),
                "calls": calls, "wall_s_per_call": wall / calls}

    def close(self):
        self.smi.amdsmi_shut_down()


def energy_run(torch, rift_query, ex_run, rift_ms, ex_ms, min_seconds: float) -> dict:
    """Energy per scene-query, Rift against exhaustive: each workload runs back
    to back (one synchronisation per query) while the board's energy counter
    gives its average power; energy per query = average power x wall time per
    query in that loop.  Idle power (no work) is reported for context."""
    try:
        meter = EnergyMeter(torch)
    except Exception as exc:   # amdsmi missing or the device not visible to it
        return {"error": repr(exc)[:200]}
    try:
        def rift():
            rift_query()
            torch.cuda.synchronize()

        def ex():
            ex_run()
            torch.cuda.synchronize()

        idle = meter.average_power(lambda: time.sleep(0.05), min_seconds=2.0, min_updates=3)
        pr = meter.average_power(rift, min_seconds)
        pe = meter.average_power(ex, min_seconds)
    finally:
        meter.close()
    e_r = pr["watts"] * pr["wall_s_per_call"]
    e_e = pe["watts"] * pe["wall_s_per_call"]
    return {"method": "amdsmi energy accumulator: average board power between counter updates "
                      "while the workload runs back to back, times wall time per query",
            "idle_W": round(idle["watts"], 1),
            "rift": {"W": round(pr["watts"], 1), "wall_ms_per_query": round(pr["wall_s_per_call"] * 1e3, 2),
                     "device_ms_per_query": round(rift_ms, 2), "J_per_query": round(e_r, 2),
                     "queries": pr["calls"], "span_s": round(pr["span_s"], 2)},
            "exhaustive": {"W": round(pe["watts"], 1), "wall_ms_per_query": round(pe["wall_s_per_call"] * 1e3, 2),
                           "device_ms_per_query": round(ex_ms, 2), "J_per_query": round(e_e, 2),
                           "queries": pe["calls"], "span_s": round(pe["span_s"], 2)},
            "energy_reduction": round(1 - e_r / e_e, 4)}


def gemm_operand_split(R, torch, q, reps=3) -> dict:
    """One prefill layer at the query's packed shape (shared prefix), per stage:
    once with the query's packed input and first layer's weights, once with the
    input and every weight matrix zero (norm gains one).  The kernels and shapes
    are the same; zero operands barely toggle the matrix cores, so the board
    stays below its power limit and the clock near its maximum, and the ratio of
    the two times is what the power limit costs each GEMM.  Runs alternate;
    median of `reps` per case."""
    sh = q.shape
    cfg = R.model_cfg(sh.d, sh.n_heads, sh.head_dim, sh.ffn, 1, sh.rms_eps, sh.rope_base, R.RIFT_BF16)
    L0 = q.layers[0]
    zl = {k: (torch.ones_like(v) if k.startswith("g_") else torch.zeros_like(v)) for k, v in L0.items()}
    T = q.total_tokens
    x_rand = q.packed
    x_zero = torch.zeros_like(x_rand)
    hid = torch.empty(T, sh.d, dtype=torch.float32, device=x_rand.device)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, q.max_seqlen), dtype=torch.uint8, device=x_rand.device)
    times = {"query_operands": {k: [] for k in STAGES}, "zero_operands": {k: [] for k in STAGES}}
    for _ in range(reps):
        for name, layer, x in (("query_operands", L0, x_rand), ("zero_operands", zl, x_zero)):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(10)]
            R.rift_prefill(cfg, [layer], x, q.cu_seqlens, q.position_ids, q.n_seq, q.max_seqlen, hid, ws,
                           events=ev, n_prefix=q.n_prefix)
            torch.cuda.synchronize()
            for i, k in enumerate(STAGES):
                times[name][k].append(ev[2 * i].elapsed_time(ev[2 * i + 1]))
    out = {name: {k: round(statistics.median(v), 4) for k, v in d.items()} for name, d in times.items()}
    out["zero_over_query_time"] = {k: round(out["zero_operands"][k] / out["query_operands"][k], 4) for k in STAGES}
    return out


def knn_score_timing(R, torch, tokens, qbank, keep_count, m=6, reps=10) -> dict:
    """The scoring call with the optional smoothing over each tile's m most
    similar tiles (median of `reps` calls), for comparison with the plain
    scoring stage the scene-query uses."""
    n, nv, d = tokens.shape
    dev = tokens.device
    key = torch.empty(n * nv, dtype=torch.float64, device=dev)
    sim = torch.empty(n * nv, qbank.shape[0], dtype=torch.float32, device=dev)
    s = torch.empty(n, dtype=torch.float64, device=dev)
    u = torch.empty(n, dtype=torch.float32, device=dev)
    order = torch.empty(n, dtype=torch.int32, device=dev)
    nk = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(R.rift_score_workspace_size(n, nv, d, m), dtype=torch.uint8, device=dev)
    call = lambda: R.rift_score_tiles(tokens, qbank, keep_count, 0.0, key, sim, s, u, order, nk, ws, knn_m=m)
    call()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        call()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return {"m": m, "score_ms": round(statistics.median(ts), 4)}


# Eq. 2 stand-in tables over the paper's budget set for LLaVA-1.5 (accuracy with
# and without the object, energy proportional to the budget); the probability
# p of each kept tile is its normalised score u.
UTILITY = dict(levels=[576, 432, 288, 144, 72], alpha_pos=[0.92, 0.90, 0.85, 0.74, 0.58],
               alpha_neg=[0.95, 0.95, 0.94, 0.93, 0.91],
               energy=[c / 576 for c in (576, 432, 288, 144, 72)], lam=0.1)


def utility_run(R, torch, w, tokens, qbank, sysd, qryd, layers, q, reps=3) -> dict:
    """The scene-query with Eq. 2 utility budgets instead of the rank tiers
    (one read-back of the kept tiles' scores after scoring); wall time per
    query including that synchronisation."""
    from paper_2609_29029_amd.pipeline import SceneQuery
    uq = SceneQuery(tokens, qbank, sysd, qryd, layers, q.shape, w.keep_count, w.tau, w.levels,
                    w.tier_num, w.tier_den, with_sims=True, utility=UTILITY, shared_prefix=q.shared)
    uq.run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        uq.run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    assert uq.check_status() == [0, 0]
    levels, counts = np.unique(uq.budgets_host, return_counts=True)
    return {"ms_per_query": round(ms, 2), "retained_vision_tokens": int(uq.n_selected),
            "tokens_per_s": round(uq.n_selected / (ms * 1e-3), 1),
            "budgets": {int(l): int(c) for l, c in zip(levels, counts)}}


def merge_run(R, torch, w, tokens, qbank, sysd, qryd, layers, q, reps=3) -> dict:
    """The scene-query with each budget split into dominant and contextual
    tokens (VisionZip's merge of the remainder, 54 + 10 at 64): the same
    prompt lengths, plus the merge.  Median device time of the merge call and
    of the whole query over `reps` queries; the merge's float64 work is the
    canonical dot of every non-target remaining token with every target."""
    from paper_2609_29029_amd.pipeline import SceneQuery
    mq = SceneQuery(tokens, qbank, sysd, qryd, layers, q.shape, w.keep_count, w.tau, w.levels,
                    w.tier_num, w.tier_den, with_sims=True, merge=(10, 64), shared_prefix=q.shared)
    mq.run()
    torch.cuda.synchronize()
    tm, tq = [], []
    for _ in range(reps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record()
        mq.score()
        mq.select()
        ev[1].record()
        mq.merge_context()
        ev[2].record()
        mq.compact()
        mq.prefill()
        ev[3].record()
        torch.cuda.synchronize()
        tm.append(ev[1].elapsed_time(ev[2]))
        tq.append(ev[0].elapsed_time(ev[3]))
    assert mq.check_status() == [0, 0, 0]
    dom, ctx = R.rift_split_budgets(mq.budgets_host, w.n_v)
    fma = sum(int(w.n_v - kd - kc) * int(kc) * w.model.d for kd, kc in zip(dom, ctx) if kc > 1)
    ms = statistics.median(tm)
    return {"ms_per_query": round(statistics.median(tq), 2), "merge_ms": round(ms, 4),
            "dominant_tokens": int(mq.n_dominant), "contextual_tokens": int(mq.n_context),
            "retained_vision_tokens": int(mq.n_selected),
            "fp64_fma": fma, "fp64_TFLOPs": round(2 * fma / (ms * 1e-3) / 1e12, 2),
            "frac_fp64_vector_peak": round(2 * fma / (ms * 1e-3) / 1e12 / 78.6, 4)}


def decode_run(R, torch, w, q, steps=8) -> dict:
    """Decode after the scene-query's prefill: the prefill again with its
    key/value cache kept (every layer's rotated keys and values of all
    prompts), then `steps` decode steps, one new token per prompt each
    (synthetic bf16 input embeddings).  A step reads every weight once and
    every cached key and value once: the HBM-bound work per step."""
    m = w.model
    T, n_seq, d = q.total_tokens, q.n_keep, m.d
    kv = torch.empty(m.n_layers, 2, T, d, dtype=torch.bfloat16, device="cuda")
    R.rift_prefill(q.cfg, q.layers, q.packed, q.cu_seqlens, q.position_ids, q.n_seq, q.max_seqlen, q.hidden,
                   q.prefill_ws, kv_cache=kv, n_prefix=q.n_prefix)
    g = torch.Generator(device="cuda").manual_seed(0x52494654)
    x_new = torch.randn(steps, n_seq, d, device="cuda", generator=g).to(torch.bfloat16)
    kv_new = torch.empty(m.n_layers, 2, n_seq, steps, d, dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(R.rift_decode_workspace_size(q.cfg, n_seq, q.max_seqlen, steps), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty(n_seq, d, dtype=torch.float32, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for t in range(steps):
        R.rift_decode_step(q.cfg, q.layers, x_new[t], q.cu_seqlens, T, q.max_seqlen, kv, kv_new, t, out, ws,
                           n_prefix=q.n_prefix)
        ev[t + 1].record()
    torch.cuda.synchronize()
    ms = [ev[t].elapsed_time(ev[t + 1]) for t in range(steps)]
    weight_bytes = m.n_layers * 2 * (4 * d * d + 3 * d * m.ffn + 2 * d)
    keys = T + (n_seq - 1) * q.n_prefix if q.n_prefix > 0 else T   # every prompt reads the shared rows too
    kv_bytes = m.n_layers * 2 * (keys + n_seq * steps / 2) * d * 2
    med = statistics.median(ms)
    del kv, kv_new
    return {"steps": steps, "prompts": n_seq, "ms_per_step": round(med, 3),
            "tokens_per_s": round(n_seq / (med * 1e-3), 1),
            "bytes_per_step": round(weight_bytes + kv_bytes), "GBs": round((weight_bytes + kv_bytes) / (med * 1e-3) / 1e9, 1),
            "frac_hbm": round((weight_bytes + kv_bytes) / (med * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}


def select_batched(R, torch, token_key, order, budgets, n_tiles, n_v, n_keep, copies=64, reps=10, calls=20) -> dict:
    """rift_select_tokens over `copies` scene-queries' keys at once (one call),
    for a bandwidth-meaningful number: the median over `reps` of the mean time
    of `calls` calls enqueued back to back (as inside a query, where the host
    runs ahead of the device; a lone call after a synchronisation also pays
    the host's launch latency, reported as `us_lone_call`)."""
    dev = token_key.device
    keys = token_key.repeat(copies)
    kept = torch.cat([order[:n_keep] + c * n_tiles for c in range(copies)]).contiguous()
    b = budgets[:n_keep].repeat(copies).contiguous()
    total = int(b.sum().item())
    offs = torch.empty(copies * n_keep + 1, dtype=torch.int32, device=dev)
    sel = torch.empty(total, dtype=torch.int32, device=dev)
    st = torch.empty(1, dtype=torch.int32, device=dev)
    for _ in range(2):
        R.rift_select_tokens(keys, copies * n_tiles, n_v, kept, b, copies * n_keep, offs, sel, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    ts, lone = [], []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        R.rift_select_tokens(keys, copies * n_tiles, n_v, kept, b, copies * n_keep, offs, sel, st)
        e1.record()
        torch.cuda.synchronize()
        lone.append(e0.elapsed_time(e1))
        e0.record()
        for _ in range(calls):
            R.rift_select_tokens(keys, copies * n_tiles, n_v, kept, b, copies * n_keep, offs, sel, st)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) / calls)
    assert int(st.item()) == 0
    us = statistics.median(ts) * 1e3
    nbytes = copies * n_keep * n_v * 8 + total * 4 + copies * n_keep * 12
    return {"queries": copies, "kept_tiles": copies * n_keep, "us": round(us, 1),
            "us_lone_call": round(statistics.median(lone) * 1e3, 1), "calls_back_to_back": calls,
            "GBs": round(nbytes / (us * 1e-6) / 1e9, 1),
            "frac_hbm": round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}


def _kernel_label(name: str) -> str:
    """Short kernel name for a rocprofv3 row: namespaces and argument lists
    dropped, template arguments kept."""
    import re
    k = name.replace("void ", "").replace("rift::(anonymous namespace)::", "").replace("rift::", "")
    m = re.match(r"[\w:]+(<[^>]*>)?", k)
    return m.group(0) if m else k[:60]


def trace_report(paths) -> str:
    """Per-kernel durations from rocprofv3 --kernel-trace CSV files: calls,
    total and average microseconds and share of the kernel time, launches of
    one kernel with different grids apart."""
    import csv
    import glob
    files = []
    for p in paths:
        files += sorted(glob.glob(os.path.join(p, "**", "*kernel_trace.csv"), recursive=True)) \
            if os.path.isdir(p) else [p]
    durs: dict = {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                k = (_kernel_label(r["Kernel_Name"]), int(r.get("Grid_Size_X", 0) or 0))
                if k[0].startswith(("at::", "__amd")):
                    continue   # torch's and the runtime's own kernels (input copies, fills)
                durs.setdefault(k, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    grids: dict = {}
    for lab, g in durs:
        grids.setdefault(lab, set()).add(g)
    total = sum(sum(v) for v in durs.values())
    lines = ["| kernel | calls | total us | average us | % |", "|---|---|---|---|---|"]
    for k, v in sorted(durs.items(), key=lambda kv: -sum(kv[1])):
        nm = f"`{k[0]}`" + (f" (grid {k[1]})" if len(grids[k[0]]) > 1 else "")
        lines.append(f"| {nm} | {len(v)} | {sum(v):.0f} | {sum(v) / len(v):.1f} | {100 * sum(v) / total:.2f} |")
    return "\n".join(lines)


def counter_report(paths) -> str:
    """Summarise rocprofv3 --pmc CSV files (one pass per file: the hardware
    collects a few counters per run) as markdown tables per kernel; launches of
    one kernel with different grids are listed apart.  Derived figures:
      clock     GRBM_GUI_ACTIVE / 8 XCDs over the dispatch's duration
      MFMA busy SQ_VALU_MFMA_BUSY_CYCLES over (clock cycles x 1,024 SIMDs)
      SQ busy   SQ_BUSY_CYCLES over (clock cycles x 32 shader engines)
      HBM-side bytes  FETCH_SIZE and WRITE_SIZE (KiB) scaled by what the same
                counters read for the 1 GiB calibration copy (torch.neg over
                2^28 floats: 1 GiB read, 1 GiB written)
      waiting   SQ_WAIT_ANY over SQ_WAVE_CYCLES (share of wave time stalled)
      LDS       SQ_LDS_BANK_CONFLICT over SQ_LDS_IDX_ACTIVE."""
    import csv
    import glob
    files = []
    for p in paths:
        files += sorted(glob.glob(os.path.join(p, "**", "*counter_collection.csv"), recursive=True)) \
            if os.path.isdir(p) else [p]
    vals: dict = {}
    durs: dict = {}
    grids: dict = {}
    for f in files:
        seen = set()
        with open(f) as fh:
            for r in csv.DictReader(fh):
                k = (_kernel_label(r["Kernel_Name"]), int(r.get("Grid_Size", 0) or 0))
                vals.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                key = (f, r["Dispatch_Id"])
                if key not in seen:
                    seen.add(key)
                    durs.setdefault(k, []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    for lab, g in vals:
        grids.setdefault(lab, set()).add(g)

    def name(k):
        return f"`{k[0]}`" + (f" (grid {k[1]})" if len(grids[k[0]]) > 1 else "")
    calib = {c: statistics.mean(v) for k, d in vals.items() if "neg" in k[0] for c, v in d.items()}
    f_scale = (1 << 30) / (calib["FETCH_SIZE"] * 1024) if calib.get("FETCH_SIZE") else None
    w_scale = (1 << 30) / (calib["WRITE_SIZE"] * 1024) if calib.get("WRITE_SIZE") else None

    def fmt(x, nd):
        return "" if x is None else f"{x:.{nd}f}"
    lines = ["| kernel | dispatches | mean us | clock GHz | MFMA busy | SQ busy | fetch GB | write GB | HBM-side GB/s | frac of 8 TB/s |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    stall = ["| kernel | waiting / wave time | VALU instr / wave | SALU instr / wave | LDS instr / wave | LDS bank conflicts / active |",
             "|---|---|---|---|---|---|"]
    for k in sorted(vals):
        if "neg" in k[0] or k[0].startswith("__amd") or k[0].startswith("at::"):
            continue
        d = {c: statistics.mean(v) for c, v in vals[k].items()}
        us = statistics.mean(durs[k]) / 1e3
        cyc = d["GRBM_GUI_ACTIVE"] / 8 if "GRBM_GUI_ACTIVE" in d else None
        clk = cyc / (us * 1e3) if cyc else None
        busy = d["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * 1024) if cyc and "SQ_VALU_MFMA_BUSY_CYCLES" in d else None
        sqb = d["SQ_BUSY_CYCLES"] / (cyc * 32) if cyc and "SQ_BUSY_CYCLES" in d else None
        fgb = d["FETCH_SIZE"] * 1024 * f_scale / 1e9 if f_scale and "FETCH_SIZE" in d else None
        wgb = d["WRITE_SIZE"] * 1024 * w_scale / 1e9 if w_scale and "WRITE_SIZE" in d else None
        gbs = ((fgb or 0) + (wgb or 0)) / (us * 1e-6) if (fgb is not None or wgb is not None) else None
        lines.append(f"| {name(k)} | {len(durs[k])} | {us:.1f} | {fmt(clk, 3)} | "
                     f"{'' if busy is None else f'{busy * 100:.1f}%'} | {fmt(sqb, 2)} | {fmt(fgb, 4)} | {fmt(wgb, 4)} | "
                     f"{fmt(gbs, 0)} | {fmt(gbs and gbs / PEAK_HBM_GBS, 3)} |")
        if "SQ_WAVE_CYCLES" in d or "SQ_INSTS_LDS" in d:
            waves = d.get("SQ_WAVES")
            wait = d["SQ_WAIT_ANY"] / d["SQ_WAVE_CYCLES"] if "SQ_WAIT_ANY" in d and d.get("SQ_WAVE_CYCLES") else None
            per = (lambda c: d[c] / waves if waves and c in d else None)
            conf = (d["SQ_LDS_BANK_CONFLICT"] / d["SQ_LDS_IDX_ACTIVE"]
                    if d.get("SQ_LDS_IDX_ACTIVE") and "SQ_LDS_BANK_CONFLICT" in d else None)
            stall.append(f"| {name(k)} | {'' if wait is None else f'{wait * 100:.1f}%'} | {fmt(per('SQ_INSTS_VALU'), 0)} | "
                         f"{fmt(per('SQ_INSTS_SALU'), 0)} | {fmt(per('SQ_INSTS_LDS'), 0)} | {fmt(conf, 4)} |")
    if f_scale or w_scale:
        lines.append("")
        lines.append(f"Calibration copy (1 GiB read, 1 GiB written): FETCH_SIZE x {f_scale or 0:.3f}, "
                     f"WRITE_SIZE x {w_scale or 0:.3f}.")
    if len(stall) > 2:
        lines += ["", *stall]
    return "\n".join(lines)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="scene20_l32")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-shared-prefix", action="store_true",
                    help="pack the system rows into every prompt instead of prefilling them once")
    ap.add_argument("--cpu-sample-layers", type=int, default=16)
    ap.add_argument("--no-exhaustive", action="store_true",
                    help="skip the every-tile, full-budget comparison run")
    ap.add_argument("--no-energy", action="store_true",
                    help="skip the energy-per-query comparison (board energy counter)")
    ap.add_argument("--energy-seconds", type=float, default=4.0,
                    help="minimum span of energy-counter updates per workload")
    ap.add_argument("--traffic-calibration", action="store_true",
                    help="also run a 1 GiB copy kernel (for HBM counter calibration)")
    ap.add_argument("--core-only", action="store_true",
                    help="time the scene-query and the batched select only (for counter runs)")
    ap.add_argument("--counter-report", nargs="+", metavar="CSV_OR_DIR",
                    help="print a per-kernel summary of rocprofv3 --pmc CSV output and exit (no GPU)")
    ap.add_argument("--trace-report", nargs="+", metavar="CSV_OR_DIR",
                    help="print a per-kernel summary of rocprofv3 --kernel-trace CSV output and exit (no GPU)")
    args = ap.parse_args()
    if args.counter_report:
        print(counter_report(args.counter_report))
        return 0
    if args.trace_report:
        print(trace_report(args.trace_report))
        return 0
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the Rift path here is a single-GPU build "
              "(no collectives); run it with --gpus 1", file=sys.stderr)
        return 2

    import torch
    import synth
    from paper_2609_29029_amd.pipeline import PrefillShape, SceneQuery
    import paper_2609_29029_amd as R

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    R.load()
    w = synth.get(args.workload)
    m = w.model
    t_setup = time.perf_counter()
    sc = synth.make_scene(w)

    def up(a):
        if w.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a)).cuda()

    tokens, qbank, sysd, qryd = up(sc.tokens), up(sc.qbank), up(sc.sys), up(sc.qry)
    layers = []
    for l in range(m.n_layers):
        W = synth.make_layer(w, l)
        layers.append({k: up(v) for k, v in W.items()})
        del W
        if l % 8 == 7:
            log(f"weights: {l + 1}/{m.n_layers} layers on device")
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s")

    shared = not args.no_shared_prefix
    q = SceneQuery(tokens, qbank, sysd, qryd, layers,
                   PrefillShape(m.d, m.n_heads, m.head_dim, m.ffn, m.n_layers, m.rms_eps, m.rope_base),
                   w.keep_count, w.tau, w.levels, w.tier_num, w.tier_den, with_sims=True, shared_prefix=shared)
    T, n_ret = q.total_tokens, q.n_selected
    budgets = [int(b) for b in q.budgets_host]
    seq_lens = [w.n_sys + b + w.n_qry for b in budgets]

    def E():
        return torch.cuda.Event(enable_timing=True)

    for i in range(args.warmup):
        q.run()
        torch.cuda.synchronize()
        log(f"warmup {i + 1}/{args.warmup}")
    if args.warmup:
        assert q.check_status() == [0, 0]

    # Per-launch times of every prefill stage, from untimed queries with an
    # event pair around every stage of every layer.  Each recorded event adds
    # a marker between kernels (320 of them cost about 2.5 ms per query), so
    # the timed loop records only the pairs around the dominant stage.
    n_stage_runs = 2
    lay_all = [[E() for _ in range(10 * m.n_layers)] for _ in range(n_stage_runs)]
    for s in range(n_stage_runs):
        q.score()
        q.select()
        q.compact()
        q.prefill(events=lay_all[s])
    torch.cuda.synchronize()
    per_launch = {}
    for g, name in enumerate(STAGES):
        ds = [lay_all[s][10 * l + 2 * g].elapsed_time(lay_all[s][10 * l + 2 * g + 1])
              for s in range(n_stage_runs) for l in range(m.n_layers)]
        per_launch[name] = sum(ds) / len(ds)
    dom = max(STAGES, key=lambda n: per_launch[n])
    gd = STAGES.index(dom)

    K = args.steps
    top = [[E() for _ in range(5)] for _ in range(K)]
    lay = [[E() if (i % 10) // 2 == gd else None for i in range(10 * m.n_layers)] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(K):
        ev = top[s]
        ev[0].record()
        q.score()
        ev[1].record()
        q.select()
        ev[2].record()
        q.compact()
        ev[3].record()
        q.prefill(events=lay[s])
        ev[4].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    log(f"timed {K} steps: {(t1 - t0) * 1e3 / K:.2f} ms/step")
    assert q.check_status() == [0, 0]
    if args.traffic_calibration:
        # a plain copy of known size (1 GiB read, 1 GiB written) whose FETCH_SIZE and
        # WRITE_SIZE readings scale the counters of the prefill kernels to bytes
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("traffic calibration copy: 1 GiB read + 1 GiB written")

    elapsed = t1 - t0
    ms_step = elapsed * 1e3 / K
    value = n_ret * K / elapsed

    def med(xs):
        return statistics.median(xs)

    stage_ms_total = med([e[0].elapsed_time(e[4]) for e in top])
    stage_ms = {"score": med([e[0].elapsed_time(e[1]) for e in top]),
                "select": med([e[1].elapsed_time(e[2]) for e in top]),
                "compact": med([e[2].elapsed_time(e[3]) for e in top]),
                "prefill": med([e[3].elapsed_time(e[4]) for e in top])}
    # the dominant stage's per-launch average over every layer of the timed steps
    ds = [lay[s][10 * l + 2 * gd].elapsed_time(lay[s][10 * l + 2 * gd + 1])
          for s in range(K) for l in range(m.n_layers)]
    per_launch[dom] = sum(ds) / len(ds)
    fl = stage_flops(T, m.d, m.ffn, seq_lens, q.n_prefix)
    stage_roof = {n: {"ms": round(per_launch[n], 4),
                      "tflops": round(fl[n] / (per_launch[n] * 1e-3) / 1e12, 1),
                      "frac_bf16_peak": round(fl[n] / (per_launch[n] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
                  for n in STAGES}
    # At these prompt lengths attention is bound by HBM, not by the MFMA: it
    # reads q, k and v and writes o once per layer (4 T d storage elements).
    attn_bytes = 4 * T * m.d * (2 if w.dtype == "bf16" else 4)
    stage_roof["attention"].update(
        {"bound": "hbm", "hbm_bytes": attn_bytes,
         "GBs": round(attn_bytes / (per_launch["attention"] * 1e-3) / 1e9, 1),
         "frac_hbm": round(attn_bytes / (per_launch["attention"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)})
    import hashlib
    with open(GEMM_SRC, "rb") as f:
        src_sha = hashlib.sha256(f.read()).hexdigest()
    traffic = (TRAFFIC["bytes"] if dom == TRAFFIC["stage"] and src_sha == TRAFFIC["gemm_src_sha256"]
               and w.name == "scene20_l32" and T == TRAFFIC["packed_tokens"] else None)
    achieved = fl[dom] / (per_launch[dom] * 1e-3) / 1e12
    prefill_flops = sum(fl.values()) * m.n_layers
    # HBM-bound stages: algorithmic bytes
    e = 2 if w.dtype == "bf16" else 4
    score_bytes = w.n_tiles * w.n_v * m.d * e + w.n_tiles * w.n_v * (8 + 4 * (1 + w.n_bg))
    # vision rows read and written, system/query rows written (read once)
    compact_bytes = n_ret * m.d * e * 2 + (T - n_ret) * m.d * e + (w.n_sys + w.n_qry) * m.d * e
    hbm = {"score_GBs": round(score_bytes / (stage_ms["score"] * 1e-3) / 1e9, 1),
           "score_frac": round(score_bytes / (stage_ms["score"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
           "compact_GBs": round(compact_bytes / (stage_ms["compact"] * 1e-3) / 1e9, 1),
           "compact_frac": round(compact_bytes / (stage_ms["compact"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.n_tiles} tiles x {w.n_v} tokens, d={m.d}, keep "
                               f"{w.keep_count}, budgets {list(w.levels)} by score rank, "
                               f"{m.n_layers}-layer LLaMA-7B-shaped varlen prefill",
                   "retained_vision_tokens": n_ret, "packed_tokens": T, "sequences": q.n_keep,
                   "max_seqlen": q.max_seqlen, "prefill_tflop": round(prefill_flops / 1e12, 2),
                   "shared_prefix_rows": q.n_prefix},
        "roofline": {"bound": "mfma", "kernel": KERNEL_NAMES[dom], "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic},
        "stage_ms": {k: round(v, 4) for k, v in stage_ms.items()},
        "prefill_stages": stage_roof,
        "prefill_stages_timing": (f"{dom}: HIP events around each of its launches in the timed steps; other "
                                  f"stages: events around every launch of {n_stage_runs} untimed queries"),
        "prefill_frac_bf16_peak": round(prefill_flops / (stage_ms["prefill"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "hbm": hbm,
    }
    out["packed_tokens_per_s"] = round(T * K / elapsed, 1)
    if args.core_only:
        out["select_batched"] = select_batched(R, torch, q.token_key, q.tile_order, q.budgets, w.n_tiles,
                                               w.n_v, q.n_keep)
        out["select_batched_512"] = select_batched(R, torch, q.token_key, q.tile_order, q.budgets, w.n_tiles,
                                                   w.n_v, q.n_keep, copies=512, reps=3, calls=10)
        print(json.dumps(out), flush=True)
        return 0
    if shared:
        # the same query with the system rows packed into every prompt
        uq = SceneQuery(tokens, qbank, sysd, qryd, layers, q.shape, w.keep_count, w.tau, w.levels,
                        w.tier_num, w.tier_den, with_sims=True, shared_prefix=False)
        uq.run()
        torch.cuda.synchronize()
        t_u = time.perf_counter()
        for _ in range(3):
            uq.run()
        torch.cuda.synchronize()
        ms_u = (time.perf_counter() - t_u) * 1e3 / 3
        assert uq.check_status() == [0, 0]
        out["unshared_prefix"] = {"ms_per_step": round(ms_u, 3), "tokens_per_s": round(n_ret / (ms_u * 1e-3), 1),
                                  "packed_tokens": uq.total_tokens,
                                  "speedup_of_sharing": round(ms_u / ms_step, 4)}
        log(f"unshared prefix: {out['unshared_prefix']}")
        del uq
    ceil = mfma_ceiling(torch)
    out["mfma_ceiling"] = ceil
    c16 = ceil["v_mfma_f32_16x16x32_bf16"]["TFLOPs"]
    out["roofline"]["measured_peak"] = c16
    out["roofline"]["frac_of_measured_peak"] = round(achieved / c16, 4)
    cmv = ceil["v_mfma_f32_16x16x32_bf16 with the gate/up loop's LDS reads and LDS DMA"]["TFLOPs"]
    out["roofline"]["frac_of_data_movement_ceiling"] = round(achieved / cmv, 4)
    if w.dtype == "bf16":
        out["gemm_operand_split"] = gemm_operand_split(R, torch, q)
        log(f"gemm operand split: {out['gemm_operand_split']['zero_over_query_time']}")
    kn = knn_score_timing(R, torch, tokens, qbank, w.keep_count)
    kn["extra_ms_over_plain_score"] = round(kn["score_ms"] - stage_ms["score"], 4)
    out["knn_smoothing"] = kn
    out["utility_policy"] = utility_run(R, torch, w, tokens, qbank, sysd, qryd, layers, q)
    out["contextual_merge"] = merge_run(R, torch, w, tokens, qbank, sysd, qryd, layers, q)
    if w.dtype == "bf16":
        out["decode"] = decode_run(R, torch, w, q)
        log(f"decode: {out['decode']}")
    out["select_batched"] = select_batched(R, torch, q.token_key, q.tile_order, q.budgets, w.n_tiles,
                                           w.n_v, q.n_keep)
    # many rounds of tiles over the CUs: the streaming rate, without the
    # one-round latency of the 64-query call
    out["select_batched_512"] = select_batched(R, torch, q.token_key, q.tile_order, q.budgets, w.n_tiles,
                                               w.n_v, q.n_keep, copies=512, reps=3, calls=10)
    if not args.no_exhaustive:
        log("exhaustive run (every tile at the full budget) ...")
        ex_fn, ex_shape = exhaustive_setup(R, torch, w, tokens, qbank, sysd, qryd, layers, q.cfg, shared=shared)
        ex = exhaustive_run(ex_fn, ex_shape, w, torch)
        ex["rift_ms_over_exhaustive_ms"] = round(stage_ms_total / ex["ms"], 4)
        ex["latency_reduction"] = round(1 - stage_ms_total / ex["ms"], 4)
        out["exhaustive"] = ex
        log(f"exhaustive: {ex['ms']:.1f} ms")
        if not args.no_energy:
            log("energy: idle, Rift and exhaustive loops ...")
            out["energy"] = energy_run(torch, q.run, ex_fn, stage_ms_total, ex["ms"], args.energy_seconds)
            log(f"energy: {out['energy']}")
        del ex_fn
    if not args.no_cpu_baseline:
        tiers = {}
        for L in seq_lens:
            tiers[L] = tiers.get(L, 0) + 1
        t_cpu = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(w, sc, sorted(tiers.items(), reverse=True), args.cpu_sample_layers)
        log(f"cpu baseline {time.perf_counter() - t_cpu:.1f} s")
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
