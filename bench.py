"""Benchmark of the PRECOG hot path on one MI355X.

Headline workload: corpus-chunk encoding -- 64 chunks x 3000 tokens, D=2048,
N=16, bf16 inputs, fp32 state, bf16 y, fp16 captured final states -- the
offline indexing pass of Sec. 4.2.  One step = one precog_scan_encode call
over the whole batch, inputs resident in HBM.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu] [--quick]

Besides the headline, the default run times the other four workloads, each
with its algorithmic bytes, GB/s and fraction of HBM peak and with the oracle
timed beside it on the host cores:

  single_layer   1 x 512 x 128 x 16 fp32, cold and warm, and split at t = 384
  query_path     top-1 retrieval over 10,000 x 384 keys for 256 queries, the
                 retrieved state injected into a 32-token bf16 prefill
                 (injection fused into the scan), cold cache
  long_context   8 x 65,536 x 2048 x 16 bf16 scanned in 256-token chunks
  large_corpus   1024 x 3000 x 1536 x 64 bf16 per layer, state-only, all 24
                 layers timed with per-layer seeded inputs

and the extensions (top-k composition, SMC trajectory / routing /
consolidation, complex-A scan) under "extensions".  --quick times the
headline alone; --only NAME times one of the others alone (for profiling) and
prints its figures instead of the headline line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "SSM prefill scan tokens/s & achieved HBM GB/s (fraction of peak), 1 MI355X"
HBM_PEAK_GBPS = 8000.0
# MI355X fp32 vector peak 157.3 TFLOP/s = 256 CUs x 4 SIMDs x 2.4 GHz x 64
# flops per cycle, i.e. 7.86e13 fused multiply-add issue slots per second.
VALU_PEAK_TFLOPS = 157.3
SLOT_PEAK_PER_S = VALU_PEAK_TFLOPS * 1e12 / 2
# v_exp_f32 issues at a quarter of that slot rate: 1.97e13 exp/s (measured on
# the box: ~8 cycles per wave64 v_exp_f32 per SIMD at 8 waves, the same).
EXP_PEAK_PER_S = SLOT_PEAK_PER_S / 4
# Work per (token, channel, state) of the scan: 1 exp2, 1 multiply (dt A'),
# 1 multiply (u B), 1 FMA (state), 1 FMA (readout) = 6 flops + 1 exp.  As
# issue slots: 4 for the quarter-rate exp + 4 plain = 8.
FLOPS_PER_TDN = 6
SLOTS_PER_TDN = 8
MFMA_F16_PEAK_TFLOPS = 2500.0
PROFILE = os.path.join(ROOT, "profiles", "scan_corpus_encode_b64_l3000_d2048_n16.md")
SCAN_SOURCE = os.path.join(ROOT, "paper_2608_02560_amd", "csrc", "scan_kernels.h")
HOLD_CYCLES = 1_000_000  # spin length of the stream hold (well above one host enqueue)


def scan_bytes(B, L, D, N, in_bytes=2, y_bytes=2, st_bytes=2, readout=True, gate=True,
               h0_bytes=0):
    """Algorithmic bytes of one scan: every input read once, every output
    written once (x, dt, [z] per (t, d); B, [C] per (t, n); y per (t, d);
    hT (and h0 when read) per (d, n); A and Dskip per (d, n) / d)."""
    td = B * L * D
    tn = B * L * N
    total = td * in_bytes * (2 + (1 if (readout and gate) else 0))
    total += tn * in_bytes * (2 if readout else 1)
    if readout:
        total += td * y_bytes + D * 4
    total += B * D * N * (st_bytes + h0_bytes) + D * N * 4
    return total


def measured_traffic():
    """HBM bytes per launch of the corpus-encode scan from the committed
    rocprofv3 counter summary, or None when the kernel source has changed
    since the counters were taken."""
    import hashlib

    try:
        text = open(PROFILE).read()
        src = hashlib.sha256(open(SCAN_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        if ":" in line and line.strip().startswith("- "):
            k, v = line.strip()[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("scan_kernels.h sha256") != src:
        return None
    try:
        return float(fields["traffic bytes per launch"])
    except (KeyError, ValueError):
        return None


def host_cpus():
    """(threads used by the oracle, logical CPUs of the host, CPUs this
    process may run on).  The oracle uses this process's CPUs, at most 16
    (the CPU share of one GPU on the GPU machine)."""
    nproc = os.cpu_count() or 1
    try:
        aff = len(os.sched_getaffinity(0))
    except AttributeError:
        aff = nproc
    return max(1, min(16, aff)), nproc, aff


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_events(fn, reps, flush=None, hold=False):
    """Average duration of fn() in ms, HIP events on torch's current stream
    (the stream every precog call here is enqueued on).  With hold, a bounded
    spin kernel occupies the stream while the host enqueues fn()'s launches,
    so the span between the events is GPU time alone (no host launch
    latency inside it).  One untimed call first takes the first-launch costs
    (code-object load) out of the average."""
    import torch

    fn()
    torch.cuda.synchronize()
    total = 0.0
    for _ in range(reps):
        if flush is not None:
            flush()
        if hold:
            torch.cuda._sleep(HOLD_CYCLES)
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        fn()
        e.record()
        e.synchronize()
        total += s.elapsed_time(e)
    return total / reps


def log(msg):
    """Progress of the run, on stderr (stdout carries the one JSON line)."""
    print("[bench] " + msg, file=sys.stderr, flush=True)


def rates(nbytes, ms):
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"bytes": nbytes, "gbps": gbps, "hbm_frac": gbps / HBM_PEAK_GBPS}


def f64_rows(inp, b0, b1, keys=("x", "dt", "z", "B", "C"), L=None):
    """Batch rows [b0, b1) (first L tokens) of the scan inputs as contiguous
    fp64 numpy arrays (exact widening), plus A and Dskip."""
    import numpy as np

    out = {}
    for k in keys:
        v = inp.get(k)
        out[k] = None if v is None else np.ascontiguousarray(
            v[b0:b1, :L].float().cpu().numpy(), dtype=np.float64)
    out["A"] = inp["A"].double().cpu().numpy()
    out["Dskip"] = None if inp.get("Dskip") is None else inp["Dskip"].double().cpu().numpy()
    return out


def oracle_scan_time(inp, b0, b1, L=None, threads=1, want_y=True, h0=None):
    """Seconds the oracle's scan takes on batch rows [b0, b1) (first L tokens),
    its inputs widened to fp64 beforehand (outside the timing)."""
    import oracle

    a = f64_rows(inp, b0, b1, keys=("x", "dt", "z", "B", "C") if want_y else ("x", "dt", "B"),
                 L=L)
    t0 = time.perf_counter()
    oracle.scan(a["x"], a["dt"], a["A"], a["B"], a.get("C"), a.get("z"), a["Dskip"], h0,
                want_y=want_y, nthreads=threads)
    return time.perf_counter() - t0


# ----------------------------------------------------------------------------
# headline: corpus-chunk encoding
# ----------------------------------------------------------------------------
def bench_corpus(args):
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    wl = synth.CORPUS_ENCODE
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16, wl.dt_mu, wl.dt_sigma)
    y = torch.empty((B, L, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((B, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.BF16, P.F16)
    nws = P.scan_workspace_bytes(desc)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")

    def step():
        P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], None, y, hT, ws, nws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = start.elapsed_time(end) / args.steps
    ms = max(wall * 1e3 / args.steps, ev_ms)
    nbytes = scan_bytes(B, L, D, N)
    tokens = B * L
    tdn = B * L * D * N
    sec = ev_ms * 1e-3
    achieved = nbytes / sec / 1e9
    out = {
        "metric": METRIC,
        "value": tokens / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "io_dtypes": "x/dt/z/B/C bf16, y bf16, state fp32, hT fp16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "seqlen": L, "dim": D, "dstate": N,
                   "chunk": "auto (one pass)", "parallelism": "single GPU"},
        "achieved_gbps": achieved,
        "hbm_frac": achieved / HBM_PEAK_GBPS,
        # the metric's roofline: algorithmic bytes (each input read once,
        # each output written once) over the kernel's event-timed duration
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": measured_traffic(),
                     "kernel": "scan_kernel<16, bf16, bf16, fp16, readout, gate>",
                     "kernel_ms": ev_ms, "bytes_per_launch": nbytes,
                     "bytes_rule": "x, dt, z, y 2 B per (t, d); B, C 2 B per (t, n); "
                                   "hT 2 B per (d, n); A, Dskip once"},
        # what actually bounds the kernel: its vector-ALU work
        "alu": {"flops_per_tdn": FLOPS_PER_TDN, "exp_per_tdn": 1,
                "achieved_tflops": FLOPS_PER_TDN * tdn / sec / 1e12,
                "peak_tflops": VALU_PEAK_TFLOPS,
                "frac": FLOPS_PER_TDN * tdn / sec / 1e12 / VALU_PEAK_TFLOPS,
                "exp_per_s": tdn / sec, "exp_peak_per_s": EXP_PEAK_PER_S,
                "exp_frac": tdn / sec / EXP_PEAK_PER_S,
                "issue_slot_utilisation": {
                    "slots_per_tdn": SLOTS_PER_TDN,
                    "note": "exp = 4 slots (quarter rate), mul, mul, fma, fma = 1 each; "
                            "peak 7.86e13 slots/s = 157.3 TFLOP/s / 2",
                    "achieved_slots_per_s": SLOTS_PER_TDN * tdn / sec,
                    "peak_slots_per_s": SLOT_PEAK_PER_S,
                    "frac": SLOTS_PER_TDN * tdn / sec / SLOT_PEAK_PER_S}},
    }
    cpu = None
    if not args.no_cpu:
        thr, nproc, aff = host_cpus()
        # all 64 chunks with the thread share, eight chunks per call
        t_all = sum(oracle_scan_time(inp, b0, b0 + 8, threads=thr) for b0 in range(0, B, 8))
        # one thread on one chunk (3000 tokens, all channels)
        t_one = oracle_scan_time(inp, 0, 1, threads=1)
        cpu = {"value": tokens / t_all, "unit": "tokens/s", "cores": thr, "kind": "oracle",
               "sample": "the whole workload (64 chunks x 3000 tokens x 2048 channels, N=16), "
                         "fp64, %d threads, %.2f s" % (thr, t_all),
               "nproc": nproc, "affinity_cpus": aff, "cpu": cpu_model(),
               "single_thread": {"value": L / t_one, "unit": "tokens/s", "cores": 1,
                                 "sample": "1 chunk x 3000 tokens x 2048 channels, %.2f s"
                                           % t_one},
               "gpu_over_oracle": (tokens / (ms * 1e-3)) / (tokens / t_all)}
    del inp, y, hT, ws
    torch.cuda.empty_cache()
    return out, cpu


# ----------------------------------------------------------------------------
# the other workloads
# ----------------------------------------------------------------------------
def make_flush():
    import torch

    buf = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device="cuda")
    return buf, (lambda: buf.zero_())  # evicts the 256 MB last-level cache


def bench_single_layer(args, flush):
    """One fp32 layer, B=1, L=512, D=128, N=16 (latency; the whole problem
    fits in the last-level cache), and the same split at t = 384 with the
    intermediate state passed in fp32 (Theorem 1)."""
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    wl = synth.SINGLE_LAYER
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = {k: v.cuda() for k, v in synth.scan_inputs_host(B, L, D, N, wl.seed,
                                                           torch.float32).items()}
    y = torch.empty((B, L, D), dtype=torch.float32, device="cuda")
    hT = torch.empty((B, D, N), dtype=torch.float32, device="cuda")
    h1 = torch.empty((B, D, N), dtype=torch.float32, device="cuda")
    s = 384
    # the automatic chunking (128 channels fill 2 waves, so time is cut into
    # chunks: summary pass, carry fold, replay), and one pass over the sequence
    desc = P.scan_desc(B, L, D, N, P.F32, P.F32, P.F32)
    d1 = P.scan_desc(B, s, D, N, P.F32, P.F32, P.F32)
    d2 = P.scan_desc(B, L - s, D, N, P.F32, P.F32, P.F32)
    one = P.scan_desc(B, L, D, N, P.F32, P.F32, P.F32, chunk=L)
    nws = max(P.scan_workspace_bytes(v) for v in (desc, d1, d2))
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    sl = lambda t, a, b: t[:, a:b]

    def whole(dsc=desc):
        P.scan_encode(dsc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], None, y, hT, ws, nws)

    def split():
        P.scan_encode(d1, sl(inp["x"], 0, s), sl(inp["dt"], 0, s), inp["A"], sl(inp["B"], 0, s),
                      sl(inp["C"], 0, s), sl(inp["z"], 0, s), inp["Dskip"], None,
                      sl(y, 0, s), h1, ws, nws)
        P.scan_encode(d2, sl(inp["x"], s, L), sl(inp["dt"], s, L), inp["A"],
                      sl(inp["B"], s, L), sl(inp["C"], s, L), sl(inp["z"], s, L), inp["Dskip"],
                      h1, sl(y, s, L), hT, ws, nws)

    nb = scan_bytes(B, L, D, N, in_bytes=4, y_bytes=4, st_bytes=4)
    cold = time_events(whole, 20, flush, hold=True)
    warm = time_events(whole, 50, None, hold=True)
    res = {"workload": wl.name + ", y and hT fp32, h0 = 0",
           "timing": "GPU time (stream held while the host enqueues); cold = after a 512 MB "
                     "cache flush",
           "workspace_bytes": nws,
           "cold_us": cold * 1e3, "warm_us": warm * 1e3,
           "one_pass_cold_us": time_events(lambda: whole(one), 20, flush, hold=True) * 1e3,
           "one_pass_warm_us": time_events(lambda: whole(one), 50, None, hold=True) * 1e3,
           "split_384_cold_us": time_events(split, 20, flush, hold=True) * 1e3,
           "split_384_warm_us": time_events(split, 50, None, hold=True) * 1e3,
           "tokens_per_s_warm": L / (warm * 1e-3)}
    res.update(rates(nb, cold))
    res["gbps_warm"] = nb / (warm * 1e-3) / 1e9
    if not args.no_cpu:
        thr = host_cpus()[0]
        t1 = min(oracle_scan_time(inp, 0, 1, threads=1) for _ in range(3))
        tn = min(oracle_scan_time(inp, 0, 1, threads=thr) for _ in range(3))
        res["oracle"] = {"kind": "oracle", "sample": "the whole workload, fp64",
                         "us_1_thread": t1 * 1e6, "us_threads": tn * 1e6, "threads": thr,
                         "tokens_per_s_1_thread": L / t1}
    return res


def bench_query_path(args, flush):
    """Query time (Sec. 4.2): top-1 retrieval of 256 queries over 10,000
    unit-norm 384-dim keys, then the 32-token bf16 prefill starting from the
    retrieved rows of a [10000, 1024, 16] fp16 state store (the injection
    fused into the scan), cold cache."""
    import numpy as np
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    cfg = synth.RETRIEVAL
    Q, M, E = cfg["Q"], cfg["M"], cfg["E"]
    q_h, K_h, _, _ = synth.retrieval_inputs_host(Q, M, E, cfg["planted"], cfg["seed"])
    q, K = q_h.cuda(), K_h.cuda()
    wl = synth.QUERY_PREFILL
    D, N, Lq = wl.dim, wl.dstate, wl.seqlen
    store = synth.state_store(M, D * N, seed=33, device="cuda")
    store3 = store.view(M, D, N)
    idx = torch.empty(Q, dtype=torch.int32, device="cuda")
    nws = P.retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    inp = synth.scan_inputs_device(Q, Lq, D, N, wl.seed, torch.bfloat16)
    h0 = torch.empty((Q, D, N), dtype=torch.float16, device="cuda")
    y = torch.empty((Q, Lq, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((Q, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(Q, Lq, D, N, P.BF16, P.BF16, P.F16)
    prepared = P.prepare_index(K)

    retrieve = lambda: P.retrieve_top1(q, K, idx, ws, nws)
    prefill = lambda: P.scan_encode_indexed(desc, inp["x"], inp["dt"], inp["A"], inp["B"],
                                            inp["C"], inp["z"], inp["Dskip"], store3, M, idx,
                                            y, hT)

    def fused():
        retrieve()
        prefill()

    def fused_prepared():
        P.retrieve_topk_prepared(q, K, prepared, 1, idx, None, ws, nws)
        prefill()

    def separate():
        retrieve()
        P.inject_gather(store, idx, h0.view(Q, -1))
        P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], h0, y, hT)

    nq = P.query_workspace_bytes(desc, M, E)
    wq = torch.empty(max(nq, 16), dtype=torch.uint8, device="cuda")

    def one_call(prep=None):
        P.query_top1_prefill(desc, q, K, store3, idx, inp["x"], inp["dt"], inp["A"], inp["B"],
                             inp["C"], inp["z"], inp["Dskip"], y, hT, wq, nq, prepared=prep)

    r_ms = time_events(retrieve, 20, flush, hold=True)
    p_ms = time_events(prefill, 20, flush, hold=True)
    f_ms = time_events(fused, 20, flush, hold=True)
    fw_ms = time_events(fused, 20, None, hold=True)
    fp_ms = time_events(fused_prepared, 20, flush, hold=True)
    s_ms = time_events(separate, 20, flush, hold=True)
    o_ms = time_events(one_call, 20, flush, hold=True)
    ow_ms = time_events(one_call, 20, None, hold=True)
    op_ms = time_events(lambda: one_call(prepared), 20, flush, hold=True)
    flops = 2.0 * Q * M * E
    rbytes = (Q + M) * E * 4 + Q * 4
    pbytes = scan_bytes(Q, Lq, D, N, h0_bytes=2)  # the injected rows are read once
    res = {"workload": "Q=256 over M=10000 x 384 unit-norm fp32 keys; store [10000, 1024, 16] "
                       "fp16; 32-token bf16 prefill from the retrieved rows, bf16 y, fp16 hT",
           "timing": "GPU time (stream held while the host enqueues), after a 512 MB cache "
                     "flush unless warm",
           "end_to_end_fused_top1_us": f_ms * 1e3,
           "end_to_end_fused_top1_warm_us": fw_ms * 1e3,
           "end_to_end_fused_top1_prepared_index_us": fp_ms * 1e3,
           "end_to_end_separate_gather_us": s_ms * 1e3,
           "one_call_top1_us": o_ms * 1e3,
           "one_call_top1_warm_us": ow_ms * 1e3,
           "one_call_top1_prepared_index_us": op_ms * 1e3,
           "one_call": "precog_query_top1_prefill: retrieval, then the decision and the "
                       "prefill from the decided row in one launch",
           "retrieve_top1_us": r_ms * 1e3,
           "retrieve_bytes": rbytes, "retrieve_gbps": rbytes / (r_ms * 1e-3) / 1e9,
           "retrieve_mfma_frac": flops / (r_ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS,
           "prefill_indexed_us": p_ms * 1e3,
           "queries_per_s": Q / (o_ms * 1e-3)}
    res.update(rates(rbytes + pbytes, o_ms))
    res["prefill_gbps"] = pbytes / (p_ms * 1e-3) / 1e9
    res["prefill_hbm_frac"] = res["prefill_gbps"] / HBM_PEAK_GBPS
    if not args.no_cpu:
        import oracle

        thr = host_cpus()[0]
        store_h = store.cpu()
        a = f64_rows(inp, 0, Q)
        out = {"kind": "oracle", "sample": "the whole workload: fp64 brute-force top-1 over all "
                                           "10,000 keys, gather, fp64 prefill", "threads": thr}
        for name, t in (("1_thread", 1), ("threads", thr)):
            t0 = time.perf_counter()
            ridx, _ = oracle.top1(q_h, K_h, nthreads=t)
            t1 = time.perf_counter()
            h0o = oracle.gather(store_h, ridx).reshape(Q, D, N)
            t2 = time.perf_counter()
            oracle.scan(a["x"], a["dt"], a["A"], a["B"], a["C"], a["z"], a["Dskip"], h0o,
                        nthreads=t)
            t3 = time.perf_counter()
            out["ms_" + name] = (t3 - t0) * 1e3
            out["retrieve_ms_" + name] = (t1 - t0) * 1e3
            out["prefill_ms_" + name] = (t3 - t2) * 1e3
        res["oracle"] = out
        del store_h, a
    del inp, y, hT, h0, store, ws, wq, q, K, prepared
    torch.cuda.empty_cache()
    return res


def bench_long_context(args):
    """8 x 65,536 tokens, D=2048, N=16, bf16, scanned in 256-token chunks
    (summary pass, carry fold, replay)."""
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    wl = synth.LONG_CONTEXT
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16)
    y = torch.empty((B, L, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((B, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.BF16, P.F16, chunk=wl.chunk)
    nws = P.scan_workspace_bytes(desc)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    run = lambda: P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"],
                                inp["z"], inp["Dskip"], None, y, hT, ws, nws)
    ms = time_events(run, 5)
    tdn = B * L * D * N
    res = {"workload": wl.name + ", bf16 y, fp16 hT", "ms": ms,
           "tokens_per_s": B * L / (ms * 1e-3), "workspace_bytes": nws,
           "exp_per_s": 2 * tdn / (ms * 1e-3),
           "exp_note": "two decays per (t, d, n): the summary pass and the replay"}
    res.update(rates(scan_bytes(B, L, D, N), ms))
    if not args.no_cpu:
        thr = host_cpus()[0]
        t_all = sum(oracle_scan_time(inp, b, b + 1, threads=thr) for b in range(B))
        t_one = oracle_scan_time(inp, 0, 1, L=4096, threads=1)
        res["oracle"] = {"kind": "oracle", "threads": thr,
                         "sample": "the whole workload (8 x 65,536 tokens), fp64, one batch "
                                   "row per call, %.1f s" % t_all,
                         "tokens_per_s": B * L / t_all,
                         "tokens_per_s_1_thread": 4096 / t_one,
                         "sample_1_thread": "first 4096 tokens of row 0, all channels"}
    del inp, y, hT, ws
    torch.cuda.empty_cache()
    return res


def bench_large_corpus(args):
    """1024 chunks x 3000 tokens, D=1536, N=64, bf16, state-only (y NULL),
    24 layers each with its own seeded inputs (seed 5000 + layer), every
    layer's final states written into a [1024, 24, 1536, 64] fp16 store."""
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    wl = synth.LARGE_CORPUS
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    nl = synth.LARGE_CORPUS_LAYERS
    store = torch.empty((B, nl, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.F32, P.F16, hT_batch_stride=nl * D * N)
    per_layer = []
    cpu_inp = None
    for layer in range(nl):
        inp = synth.scan_inputs_device(B, L, D, N, wl.seed + layer, torch.bfloat16, wl.dt_mu,
                                       wl.dt_sigma, need_z_c=False)
        run = lambda: P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], None, None,
                                    None, None, None, store[:, layer])
        per_layer.append(time_events(run, 1))
        if layer == 0 and not args.no_cpu:
            cpu_inp = {k: (v[:16].clone() if v is not None and v.dim() == 3 else v)
                       for k, v in inp.items()}
        del inp
    torch.cuda.synchronize()
    total = sum(per_layer)
    tdn = B * L * D * N
    nb = scan_bytes(B, L, D, N, readout=False)
    mean = total / nl
    res = {"workload": wl.name + ", state-only, fp16 states into the 24-layer store",
           "layers": nl, "ms_24_layers": total, "ms_per_layer_mean": mean,
           "ms_per_layer_min": min(per_layer), "ms_per_layer_max": max(per_layer),
           "timing": "each layer's inputs drawn on the device (untimed), one untimed call, "
                     "then one event-timed call; the 24 timed calls summed",
           "chunk_tokens_per_s_24_layers": B * L / (total * 1e-3),
           "tokens_per_s_per_layer": B * L / (mean * 1e-3),
           "exp_per_s": tdn / (mean * 1e-3), "exp_frac": tdn / (mean * 1e-3) / EXP_PEAK_PER_S}
    res.update(rates(nb, mean))
    if cpu_inp is not None:
        thr = host_cpus()[0]
        t16 = oracle_scan_time(cpu_inp, 0, 16, threads=thr, want_y=False)
        t1 = oracle_scan_time(cpu_inp, 0, 1, threads=1, want_y=False)
        res["oracle"] = {"kind": "oracle", "threads": thr,
                         "sample": "layer 0, 16 of 1024 chunks, state-only, fp64, %.2f s; "
                                   "extrapolated linearly to 1024 chunks x 24 layers" % t16,
                         "tokens_per_s_per_layer": 16 * L / t16,
                         "chunk_tokens_per_s_24_layers_extrapolated": 16 * L / t16 / nl,
                         "ms_24_layers_extrapolated": t16 * (B / 16) * nl * 1e3,
                         "tokens_per_s_per_layer_1_thread": L / t1,
                         "sample_1_thread": "layer 0, 1 chunk"}
    del store, cpu_inp
    torch.cuda.empty_cache()
    return res


def bench_extensions(args, flush):
    """Top-k retrieval + softmax composition, the SMC trajectory at three
    dials, SMC routing / consolidation / session start, and the complex-A
    scan on the corpus-encode shape."""
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    res = {}
    cfg = synth.RETRIEVAL
    Q, M, E = cfg["Q"], cfg["M"], cfg["E"]
    q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, cfg["planted"], cfg["seed"])
    q, K = q.cuda(), K.cuda()
    wl = synth.QUERY_PREFILL
    D, N, Lq = wl.dim, wl.dstate, wl.seqlen
    store = synth.state_store(M, D * N, seed=33, device="cuda")
    store3 = store.view(M, D, N)
    nws = P.retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    inp = synth.scan_inputs_device(Q, Lq, D, N, wl.seed, torch.bfloat16)
    y = torch.empty((Q, Lq, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((Q, D, N), dtype=torch.float16, device="cuda")
    h0 = torch.empty((Q, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(Q, Lq, D, N, P.BF16, P.BF16, P.F16)
    kk = 3
    idxk = torch.empty((Q, kk), dtype=torch.int32, device="cuda")
    sck = torch.empty((Q, kk), dtype=torch.float64, device="cuda")
    rk_ms = time_events(lambda: P.retrieve_topk(q, K, kk, idxk, sck, ws, nws), 20, flush,
                        hold=True)
    c_ms = time_events(lambda: P.inject_compose(store, idxk, sck, 1.0, h0.view(Q, -1)), 20,
                       flush, hold=True)

    def fused_k():
        P.retrieve_topk(q, K, kk, idxk, sck, ws, nws)
        P.scan_encode_indexed(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                              inp["Dskip"], store3, M, idxk, y, hT, h0_score=sck, k=kk, tau=1.0)

    # joint retrieval (Sec. 5.4): top-3 from a 500-entry episodic store and
    # from the corpus, fused with the session's semantic state, then the
    # prefill from the fused state
    Me = 500
    _, Ke, _, _ = synth.retrieval_inputs_host(1, Me, E, 0, cfg["seed"] + 1)
    Ke = Ke.cuda()
    se = synth.state_store(Me, D * N, seed=35, device="cuda")
    sem = synth.state_store(20, D * N, seed=36, device="cuda")
    srow = torch.arange(Q, dtype=torch.int32, device="cuda") % 20
    nwe = P.retrieve_workspace_bytes(Q, Me, E)
    wse = torch.empty(nwe, dtype=torch.uint8, device="cuda")
    ie = torch.empty((Q, kk), dtype=torch.int32, device="cuda")
    ve = torch.empty((Q, kk), dtype=torch.float64, device="cuda")
    P.retrieve_topk(q, K, kk, idxk, sck, ws, nws)
    P.retrieve_topk(q, Ke, kk, ie, ve, wse, nwe)
    fuse = lambda: P.inject_fuse(se, ie, ve, store, idxk, sck, kk, 1.0, h0.view(Q, -1), sem, srow,
                                 1.0)
    fu_ms = time_events(fuse, 20, flush, hold=True)

    def joint():
        P.retrieve_topk(q, Ke, kk, ie, ve, wse, nwe)
        P.retrieve_topk(q, K, kk, idxk, sck, ws, nws)
        fuse()
        P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], h0, y, hT)

    # the two retrievals are independent: the episodic one on a second stream
    # (default priority), joined before the fusion
    side = torch.cuda.Stream()

    def joint_two_streams():
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        P.retrieve_topk(q, Ke, kk, ie, ve, wse, nwe, stream=side)
        P.retrieve_topk(q, K, kk, idxk, sck, ws, nws, stream=main)
        main.wait_stream(side)
        fuse()
        P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], h0, y, hT)

    res["joint_query_path"] = {
        "workload": "256 queries: top-3 over a 500-entry episodic store and over the corpus "
                    "(10,000 keys), fused with the session's semantic state (lambda = 1), "
                    "32-token bf16 prefill from the fused state; cold cache, GPU time",
        "fuse_us": fu_ms * 1e3,
        "fuse_gbps": (2 * kk + 2) * Q * D * N * 2 / (fu_ms * 1e-3) / 1e9,
        "end_to_end_us": time_events(joint, 20, flush, hold=True) * 1e3,
        "end_to_end_two_streams_us": time_events(joint_two_streams, 20, flush, hold=True) * 1e3}
    del se, sem, wse, Ke
    res["query_path_top3"] = {
        "workload": "the query path with top-3 retrieval and softmax composition (tau = 1), "
                    "cold cache, GPU time",
        "retrieve_top3_us": rk_ms * 1e3, "compose_us": c_ms * 1e3,
        "compose_gbps": (kk + 1) * Q * D * N * 2 / (c_ms * 1e-3) / 1e9,
        "end_to_end_fused_us": time_events(fused_k, 20, flush, hold=True) * 1e3}
    del inp, y, hT, h0, store, ws, q, K
    torch.cuda.empty_cache()

    wl = synth.SMC_TRAJECTORY
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16, need_z_c=False)
    desc = P.scan_desc(B, L, D, N, P.BF16, P.F32, P.F16)
    traj_res = {"workload": wl.name + ", state-only, fp16 states"}
    for every in synth.SMC_DIALS:
        traj = torch.empty((B, L // every, D, N), dtype=torch.float16, device="cuda")
        run = lambda: P.scan_trajectory(desc, inp["x"], inp["dt"], inp["A"], inp["B"], None, None,
                                        None, None, None, None, traj, every)
        t_ms = time_events(run, 5, hold=True)
        nb = scan_bytes(B, L, D, N, readout=False) - B * D * N * 2 + traj.numel() * 2
        traj_res["every_%d" % every] = {"ms": t_ms, "tokens_per_s": B * L / (t_ms * 1e-3),
                                        "states_kept_per_chunk": L // every, **rates(nb, t_ms)}
        del traj
    res["smc_trajectory"] = traj_res
    del inp
    torch.cuda.empty_cache()

    cfg = synth.SMC
    emb, dom, sub, _, _ = synth.smc_inputs_host(cfg["C"], cfg["E"], cfg["ndom"], cfg["nsub"],
                                                cfg["seed"])
    emb, dom, sub = emb.cuda(), dom.cuda(), sub.cuda()
    R, S = cfg["ndom"] * cfg["nsub"], cfg["S"]
    states = torch.zeros((R, S), dtype=torch.float16, device="cuda")
    contrib = synth.state_store(cfg["C"], S, seed=34, device="cuda")
    outs = [torch.empty(cfg["C"], dtype=torch.int32, device="cuda") for _ in range(3)]
    one = [torch.empty(1, dtype=torch.int32, device="cuda") for _ in range(3)]
    h_init = torch.empty((1, S), dtype=torch.float16, device="cuda")
    ro_ms = time_events(lambda: P.smc_route(emb, dom, sub, *outs), 20, hold=True)
    co_ms = time_events(lambda: P.smc_consolidate(states, contrib, outs[2], 0.2), 20, hold=True)

    def session():
        P.smc_route(emb[:1], dom, sub, *one)
        P.inject_gather(states, one[2], h_init)

    res["smc"] = {
        "workload": "64 chunks routed over 5 domains x 4 sub-clusters (E=384); semantic states "
                    "[20, 24 x 4096] fp16, alpha = 0.2; GPU time",
        "route_us": ro_ms * 1e3, "consolidate_us": co_ms * 1e3,
        "consolidate_gbps": (2 * R * S * 2 + cfg["C"] * S * 2) / (co_ms * 1e-3) / 1e9,
        "session_start_us": time_events(session, 20, hold=True) * 1e3}
    del states, contrib
    torch.cuda.empty_cache()

    wl = synth.COMPLEX_ENCODE
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16)
    A_im = synth.complex_frequencies(D, N).cuda()
    y = torch.empty((B, L, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((B, D, N, 2), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.BF16, P.F16)
    run = lambda: P.scan_complex_raw(desc, inp["x"], inp["dt"], inp["A"], A_im, inp["B"],
                                     inp["C"], inp["z"], inp["Dskip"], None, y, hT)
    x_ms = time_events(run, 5)
    res["complex_encode"] = {"workload": wl.name + ", w_n = pi n, fp16 complex hT",
                             "ms": x_ms, "tokens_per_s": B * L / (x_ms * 1e-3),
                             "transcendentals_per_s": 3 * B * L * D * N / (x_ms * 1e-3),
                             **rates(scan_bytes(B, L, D, N) + B * D * N * 2, x_ms)}
    del inp, y, hT, A_im
    torch.cuda.empty_cache()

    # complex-A scan on the long-context shape, in 256-token chunks
    wl = synth.LONG_CONTEXT
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16)
    A_im = synth.complex_frequencies(D, N).cuda()
    y = torch.empty((B, L, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((B, D, N, 2), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.BF16, P.F16, chunk=wl.chunk)
    nws = P.scan_complex_workspace_bytes(desc)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    run = lambda: P.scan_complex_raw(desc, inp["x"], inp["dt"], inp["A"], A_im, inp["B"],
                                     inp["C"], inp["z"], inp["Dskip"], None, y, hT, ws, nws)
    x_ms = time_events(run, 5)
    res["complex_long_context"] = {"workload": wl.name + ", w_n = pi n, fp16 complex hT",
                                   "ms": x_ms, "tokens_per_s": B * L / (x_ms * 1e-3),
                                   "workspace_bytes": nws,
                                   **rates(scan_bytes(B, L, D, N) + B * D * N * 2, x_ms)}
    del inp, y, hT, A_im, ws
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu", action="store_true", help="skip every oracle timing")
    ap.add_argument("--quick", action="store_true", help="time the headline workload only")
    ap.add_argument("--only", choices=("single_layer", "query_path", "long_context", "large_corpus",
                                       "extensions"),
                    help="time one other workload alone and print its figures (for profiling); "
                         "no headline line")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain 1 GiB device copy (traffic-counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the scan, retrieval and injection "
              "kernels run on a single MI355X and no multi-GPU path is built; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.calibrate_copy:
        n = 1 << 30
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n,
                          "launches": 3}), flush=True)
        return
    if args.only:
        buf, flush = make_flush()
        run = {"single_layer": lambda: bench_single_layer(args, flush),
               "query_path": lambda: bench_query_path(args, flush),
               "long_context": lambda: bench_long_context(args),
               "large_corpus": lambda: bench_large_corpus(args),
               "extensions": lambda: bench_extensions(args, flush)}[args.only]
        print(json.dumps({"only": args.only, args.only: run()}), flush=True)
        return
    t_start = time.perf_counter()
    out, cpu = bench_corpus(args)
    log("corpus encode done (%.1f s)" % (time.perf_counter() - t_start))
    if not args.quick:
        buf, flush = make_flush()
        cfgs = {}
        for name, fn in (("single_layer", lambda: bench_single_layer(args, flush)),
                         ("query_path", lambda: bench_query_path(args, flush)),
                         ("long_context", lambda: bench_long_context(args)),
                         ("large_corpus", lambda: bench_large_corpus(args))):
            cfgs[name] = fn()
            log("%s done (%.1f s)" % (name, time.perf_counter() - t_start))
        out["configs"] = cfgs
        out["extensions"] = bench_extensions(args, flush)
        log("extensions done (%.1f s)" % (time.perf_counter() - t_start))
        del buf
    if cpu is not None:
        out["cpu_baseline"] = cpu
    out["bench_wall_s"] = time.perf_counter() - t_start
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
