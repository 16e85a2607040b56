"""Benchmark of the PRECOG hot path on one MI355X.

Default workload: corpus-chunk encoding -- 64 chunks x 3000 tokens, D=2048,
N=16, bf16 inputs, fp32 state, bf16 y, fp16 captured final states -- the
offline indexing pass of Sec. 4.2.  One step = one precog_scan_encode call
over the whole batch, inputs resident in HBM.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu] [--extra]

--extra also times the query-time path (top-1 retrieval, state injection,
32-token query prefill; the same with the injection fused into the prefill;
and its top-3 variant with softmax composition, separate or fused), the
long-context chunked scan and one layer of the large corpus encode, reported
under "extra".
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
# v_exp_f32 issues at a quarter of the fp32 slot rate: the 157.3 TFLOP/s
# vector peak is 7.86e13 slots/s x 2 flops, so 1.97e13 exp/s (measured on
# the box: ~8 cycles per wave64 v_exp_f32 per SIMD at 8 waves, the same)
EXP_PEAK_PER_S = 157.3e12 / 2 / 4
# MI355X fp32 vector peak: 157.3 TFLOP/s = 7.86e13 FMA issue slots/s (256 CUs x
# 2.4 GHz x 128 lanes).  The scan's algorithmic work per (token, channel,
# state) is 8 issue slots: v_mul (dt A'), v_exp_f32 (quarter rate: 4 slots),
# v_mul (B x dt), v_fma (state), v_fma (readout); expressed as FMA-equivalent
# flops (2 per slot) it is 16 per (t, d, n).
VALU_PEAK_TFLOPS = 157.3
SLOT_FLOPS_PER_TDN = 16
PROFILE = os.path.join(ROOT, "profiles", "scan_corpus_encode_b64_l3000_d2048_n16.md")
SCAN_SOURCE = os.path.join(ROOT, "paper_2608_02560_amd", "csrc", "scan_kernels.h")


def scan_bytes(B, L, D, N, in_bytes=2, y_bytes=2, st_bytes=2, readout=True, gate=True):
    """Algorithmic bytes of one scan: every input read once, every output
    written once (x, dt, [z] per (t, d); B, [C] per (t, n); y per (t, d);
    hT per (d, n); A and Dskip per (d, n) / d)."""
    td = B * L * D
    tn = B * L * N
    total = td * in_bytes * (2 + (1 if (readout and gate) else 0))
    total += tn * in_bytes * (2 if readout else 1)
    if readout:
        total += td * y_bytes + D * 4
    total += B * D * N * st_bytes + D * N * 4
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


def cpu_threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


HOLD_CYCLES = 1_000_000  # spin length of the stream hold (well above one host enqueue)


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


def cpu_baseline_corpus(inp, wl, rows_b):
    """The oracle, as it stands, on the first rows_b chunks of the workload
    (all channels, all tokens), timed on the host cores."""
    import oracle

    nthr = cpu_threads()
    sub = {k: (v[:rows_b].cpu() if v is not None and v.dim() == 3 else
               (v.cpu() if v is not None else None)) for k, v in inp.items()}
    t0 = time.perf_counter()
    oracle.scan(sub["x"], sub["dt"], sub["A"], sub["B"], sub["C"], sub["z"], sub["Dskip"],
                None, nthreads=nthr)
    dt = time.perf_counter() - t0
    tokens = rows_b * wl.seqlen
    return {"value": tokens / dt, "unit": "tokens/s", "cores": nthr, "kind": "oracle",
            "sample": "%d of %d chunks x %d tokens x %d channels, N=%d, fp64, %.1f s wall"
                      % (rows_b, wl.batch, wl.seqlen, wl.dim, wl.dstate, dt),
            "cpu": cpu_model()}


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


def bench_corpus(args):
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    wl = synth.CORPUS_ENCODE
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16, wl.dt_mu, wl.dt_sigma)
    y = torch.empty((B, L, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((B, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.BF16, P.F16, chunk=args.chunk)
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
    achieved = nbytes / (ev_ms * 1e-3) / 1e9
    alu = SLOT_FLOPS_PER_TDN * B * L * D * N / (ev_ms * 1e-3) / 1e12
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
                   "chunk": args.chunk or "auto", "parallelism": "single GPU"},
        "achieved_gbps": achieved,
        "hbm_frac": achieved / HBM_PEAK_GBPS,
        "roofline": {"bound": "alu", "achieved": alu, "peak": VALU_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": alu / VALU_PEAK_TFLOPS,
                     "traffic": measured_traffic(),
                     "kernel": "scan_kernel<16, bf16, bf16, fp16, readout, gate>",
                     "kernel_ms": ev_ms,
                     "work": "16 FMA-equivalent flops (8 fp32 issue slots) per (t, d, n)"},
        "hbm": {"achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBPS, "bytes_per_launch": nbytes},
        # decays exp(-dt A): one v_exp_f32 per (t, d, n); the peak is the
        # quarter-rate transcendental issue of 1024 SIMDs at 2.4 GHz
        "exp": {"achieved": B * L * D * N / (ev_ms * 1e-3), "peak": EXP_PEAK_PER_S,
                "unit": "exp/s", "frac": B * L * D * N / (ev_ms * 1e-3) / EXP_PEAK_PER_S},
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline_corpus(inp, wl, args.cpu_rows)
    del inp, y, hT, ws
    torch.cuda.empty_cache()
    return out


def bench_extra(args):
    import torch

    from paper_2608_02560_amd import precog as P
    from paper_2608_02560_amd import synth

    res = {}
    flush_buf = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device="cuda")
    flush = lambda: flush_buf.zero_()  # evicts the 256 MB last-level cache

    # query-time path
    cfg = synth.RETRIEVAL
    q, K, _, _ = synth.retrieval_inputs_host(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"],
                                             cfg["seed"])
    q, K = q.cuda(), K.cuda()
    wl = synth.QUERY_PREFILL
    D, N = wl.dim, wl.dstate
    store = synth.state_store(cfg["M"], D * N, seed=33, device="cuda")
    idx = torch.empty(cfg["Q"], dtype=torch.int32, device="cuda")
    nws = P.retrieve_workspace_bytes(cfg["Q"], cfg["M"], cfg["E"])
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    inp = synth.scan_inputs_device(wl.batch, wl.seqlen, D, N, wl.seed, torch.bfloat16)
    h0 = torch.empty((wl.batch, D, N), dtype=torch.float16, device="cuda")
    y = torch.empty((wl.batch, wl.seqlen, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((wl.batch, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(wl.batch, wl.seqlen, D, N, P.BF16, P.BF16, P.F16)
    r_ms = time_events(lambda: P.retrieve_top1(q, K, idx, ws, nws), 20, flush, hold=True)
    g_ms = time_events(lambda: P.inject_gather(store, idx, h0.view(wl.batch, -1)), 20, flush,
                       hold=True)
    s_ms = time_events(lambda: P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"],
                                             inp["C"], inp["z"], inp["Dskip"], h0, y, hT), 20,
                       flush, hold=True)

    def pipeline():
        P.retrieve_top1(q, K, idx, ws, nws)
        P.inject_gather(store, idx, h0.view(wl.batch, -1))
        P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], h0, y, hT)

    e_ms = time_events(pipeline, 20, flush, hold=True)

    # the same path with the injection fused into the prefill
    # (precog_scan_encode_indexed reads store[idx] rows directly)
    store3 = store.view(cfg["M"], D, N)
    f_ms = time_events(lambda: P.scan_encode_indexed(desc, inp["x"], inp["dt"], inp["A"], inp["B"],
                                                     inp["C"], inp["z"], inp["Dskip"], store3,
                                                     cfg["M"], idx, y, hT), 20, flush, hold=True)

    def pipeline_fused():
        P.retrieve_top1(q, K, idx, ws, nws)
        P.scan_encode_indexed(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                              inp["Dskip"], store3, cfg["M"], idx, y, hT)

    ef_ms = time_events(pipeline_fused, 20, flush, hold=True)
    eh_ms = time_events(pipeline_fused, 20, flush)
    # the same path with the inputs left in the caches by the previous call
    # (as when the query tokens come straight from the layer before)
    ew_ms = time_events(pipeline_fused, 20, None, hold=True)
    # the same path recorded once in a HIP graph and replayed (cold cache)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pipeline_fused()
    torch.cuda.synchronize()
    eg_ms = time_events(graph.replay, 20, flush, hold=True)
    del graph
    # retrieval over the index prepared once (screen operands and norms made
    # offline, as the keys are), alone and in the fused top-1 path
    prepared = P.prepare_index(K)
    pbytes = prepared.numel()
    rp_ms = time_events(lambda: P.retrieve_topk_prepared(q, K, prepared, 1, idx, None, ws, nws), 20,
                        flush, hold=True)

    def pipeline_fused_prepared():
        P.retrieve_topk_prepared(q, K, prepared, 1, idx, None, ws, nws)
        P.scan_encode_indexed(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                              inp["Dskip"], store3, cfg["M"], idx, y, hT)

    efp_ms = time_events(pipeline_fused_prepared, 20, flush, hold=True)
    flops = 2.0 * cfg["Q"] * cfg["M"] * cfg["E"]
    sbytes = scan_bytes(wl.batch, wl.seqlen, D, N) + wl.batch * D * N * 2
    res["query_path"] = {
        "workload": "Q=256 over M=10000 x 384 keys; store [10000, 1024, 16] fp16; "
                    "32-token bf16 query prefill; cold last-level cache",
        "timing": "GPU time: the stream is held by a bounded spin while the host enqueues "
                  "each timed call; end_to_end_fused_host_ms includes host launch latency; "
                  "end_to_end_fused_warm_ms runs without the cache flush; "
                  "end_to_end_fused_graph_ms replays the path recorded in a HIP graph; "
                  "*_prepared_ms use the index prepared once (precog_retrieve_prepare)",
        "retrieve_ms": r_ms, "retrieve_tflops": flops / (r_ms * 1e-3) / 1e12,
        # the screen's contraction runs as fp16 MFMA (one product per feature):
        # the fraction is taken against the dense fp16 peak
        "retrieve_mfma_frac": flops / (r_ms * 1e-3) / 2500e12,
        "gather_ms": g_ms, "gather_gbps": 2 * wl.batch * D * N * 2 / (g_ms * 1e-3) / 1e9,
        "prefill_ms": s_ms, "prefill_gbps": sbytes / (s_ms * 1e-3) / 1e9,
        "end_to_end_ms": e_ms,
        "fused_inject_prefill_ms": f_ms,
        "end_to_end_fused_ms": ef_ms,
        "end_to_end_fused_host_ms": eh_ms,
        "end_to_end_fused_warm_ms": ew_ms,
        "end_to_end_fused_graph_ms": eg_ms,
        "retrieve_prepared_ms": rp_ms,
        "end_to_end_fused_prepared_ms": efp_ms,
        "prepared_index_bytes": pbytes,
    }

    # top-k variant: top-3 retrieval with scores, softmax composition into h0
    kk = 3
    idxk = torch.empty((cfg["Q"], kk), dtype=torch.int32, device="cuda")
    sck = torch.empty((cfg["Q"], kk), dtype=torch.float64, device="cuda")
    rk_ms = time_events(lambda: P.retrieve_topk(q, K, kk, idxk, sck, ws, nws), 20, flush,
                        hold=True)
    P.retrieve_topk(q, K, kk, idxk, sck, ws, nws)
    c_ms = time_events(lambda: P.inject_compose(store, idxk, sck, 1.0, h0.view(wl.batch, -1)), 20,
                       flush, hold=True)

    def pipeline_k():
        P.retrieve_topk(q, K, kk, idxk, sck, ws, nws)
        P.inject_compose(store, idxk, sck, 1.0, h0.view(wl.batch, -1))
        P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], h0, y, hT)

    ek_ms = time_events(pipeline_k, 20, flush, hold=True)

    # the top-3 path with the composition fused into the prefill
    def pipeline_k_fused():
        P.retrieve_topk(q, K, kk, idxk, sck, ws, nws)
        P.scan_encode_indexed(desc, inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                              inp["Dskip"], store3, cfg["M"], idxk, y, hT, h0_score=sck, k=kk,
                              tau=1.0)

    ekf_ms = time_events(pipeline_k_fused, 20, flush, hold=True)
    res["query_path_topk"] = {
        "workload": "as query_path with top-3 retrieval and softmax composition (tau = 1)",
        "retrieve_topk_ms": rk_ms,
        "compose_ms": c_ms,
        "compose_gbps": (kk + 1) * wl.batch * D * N * 2 / (c_ms * 1e-3) / 1e9,
        "end_to_end_ms": ek_ms,
        "end_to_end_fused_ms": ekf_ms,
    }
    del inp, y, hT, h0, store, ws, q, K, prepared
    torch.cuda.empty_cache()

    # SMC trajectory encode at the fidelity dials (state-only, fp16 states)
    wl = synth.SMC_TRAJECTORY
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16, need_z_c=False)
    desc = P.scan_desc(B, L, D, N, P.BF16, P.F32, P.F16)
    nws = P.scan_workspace_bytes(desc)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device="cuda")
    traj_res = {"workload": wl.name + ", state-only, fp16 states"}
    for every in synth.SMC_DIALS:
        traj = torch.empty((B, L // every, D, N), dtype=torch.float16, device="cuda")
        run = lambda: P.scan_trajectory(desc, inp["x"], inp["dt"], inp["A"], inp["B"], None, None,
                                        None, None, None, None, traj, every, ws, nws)
        t_ms = time_events(run, 5)
        nb = scan_bytes(B, L, D, N, readout=False) - B * D * N * 2 + traj.numel() * 2
        traj_res["every_%d" % every] = {"ms": t_ms, "tokens_per_s": B * L / (t_ms * 1e-3),
                                        "gbps": nb / (t_ms * 1e-3) / 1e9,
                                        "states_kept_per_chunk": L // every}
        del traj
    res["smc_trajectory"] = traj_res
    del inp, ws
    torch.cuda.empty_cache()

    # SMC consolidation: route 64 chunks, fold their final states into the
    # 20 semantic states (24 x 4096, fp16), then a session start (route the
    # opening chunk, inject its semantic state)
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

    se_ms = time_events(session, 20, hold=True)
    res["smc"] = {
        "workload": "64 chunks routed over 5 domains x 4 sub-clusters (E=384); semantic states "
                    "[20, 24 x 4096] fp16, alpha = 0.2",
        "timing": "GPU time: the stream is held by a bounded spin while the host enqueues",
        "route_ms": ro_ms, "consolidate_ms": co_ms,
        "consolidate_gbps": (2 * R * S * 2 + cfg["C"] * S * 2) / (co_ms * 1e-3) / 1e9,
        "session_start_ms": se_ms,
    }
    del states, contrib
    torch.cuda.empty_cache()

    # complex-A scan on the corpus-encode shape (w_n = pi n)
    wl = synth.COMPLEX_ENCODE
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16)
    A_im = synth.complex_frequencies(D, N).cuda()
    y = torch.empty((B, L, D), dtype=torch.bfloat16, device="cuda")
    hT = torch.empty((B, D, N, 2), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.BF16, P.F16)
    run = lambda: P.scan_complex_raw(desc, inp["x"], inp["dt"], inp["A"], A_im, inp["B"],
                                     inp["C"], inp["z"], inp["Dskip"], None, y, hT)
    run()
    x_ms = time_events(run, 5)
    nb = scan_bytes(B, L, D, N) + B * D * N * 2  # hT has two parts
    res["complex_encode"] = {"workload": wl.name + ", w_n = pi n, fp16 complex hT",
                             "ms": x_ms, "tokens_per_s": B * L / (x_ms * 1e-3),
                             "gbps": nb / (x_ms * 1e-3) / 1e9,
                             "transcendentals_per_s": 3 * B * L * D * N / (x_ms * 1e-3)}
    del inp, y, hT, A_im
    torch.cuda.empty_cache()

    # long-context chunked scan (one timed call)
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
    run()
    l_ms = time_events(run, 5)
    nb = scan_bytes(B, L, D, N)
    res["long_context"] = {"workload": wl.name, "ms": l_ms, "tokens_per_s": B * L / (l_ms * 1e-3),
                           "gbps": nb / (l_ms * 1e-3) / 1e9}
    del inp, y, hT, ws
    torch.cuda.empty_cache()

    # one layer of the large corpus encode (state-only)
    wl = synth.LARGE_CORPUS
    B, L, D, N = wl.batch, wl.seqlen, wl.dim, wl.dstate
    inp = synth.scan_inputs_device(B, L, D, N, wl.seed, torch.bfloat16, wl.dt_mu, wl.dt_sigma,
                                   need_z_c=False)
    store = torch.empty((B, 24, D, N), dtype=torch.float16, device="cuda")
    desc = P.scan_desc(B, L, D, N, P.BF16, P.F32, P.F16, hT_batch_stride=24 * D * N)
    run = lambda: P.scan_encode(desc, inp["x"], inp["dt"], inp["A"], inp["B"], None, None,
                                None, None, None, store[:, 0])
    run()
    c_ms = time_events(run, 3)
    nb = scan_bytes(B, L, D, N, readout=False)
    res["large_corpus_layer"] = {"workload": wl.name, "ms": c_ms,
                                 "tokens_per_s": B * L / (c_ms * 1e-3),
                                 "gbps": nb / (c_ms * 1e-3) / 1e9,
                                 "exp_per_s": B * L * D * N / (c_ms * 1e-3),
                                 "exp_frac": B * L * D * N / (c_ms * 1e-3) / EXP_PEAK_PER_S,
                                 # all 24 layers of a chunk batch, one layer per launch
                                 "chunk_tokens_per_s_24_layers": B * L / (24 * c_ms * 1e-3)}
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--chunk", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=32)
    ap.add_argument("--extra", action="store_true")
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
    out = bench_corpus(args)
    if args.extra:
        out["extra"] = bench_extra(args)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
