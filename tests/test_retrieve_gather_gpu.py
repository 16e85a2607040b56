"""Parity of precog_retrieve_top1 (bit-exact indices) and precog_inject_gather
(bit-exact copies) with the oracle, and of the whole query-time path: top-1
retrieval, injection of the retrieved state, then the query prefill."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02560_amd import precog as P
from paper_2608_02560_amd import synth
from precog_testutil import TOL_BF16, err_rms

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _gpu_top1(q, K):
    idx = P.top1(q.to(DEV), K.to(DEV))
    torch.cuda.synchronize()
    return idx.cpu().numpy()


def test_retrieval_workload_bit_exact():
    """Q=256 queries, M=10000 keys of 384 dims, 32 planted queries."""
    cfg = synth.RETRIEVAL
    q, K, pos, rows = synth.retrieval_inputs_host(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"],
                                                  cfg["seed"])
    ref, _ = oracle.top1(q, K, nthreads=8)
    got = _gpu_top1(q, K)
    assert np.array_equal(got, ref)
    assert np.array_equal(got[pos.numpy()], rows.numpy().astype(np.int32))


@pytest.mark.parametrize("Q,M,E", [(1, 1, 4), (3, 33, 16), (65, 1000, 20), (70, 97, 388),
                                   (130, 4099, 64), (8, 20000, 1024), (5, 70001, 8),
                                   (300, 2000, 128), (5000, 700, 64)])
def test_retrieval_ragged_shapes(Q, M, E):
    q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, min(Q, 4), seed=Q * 7 + M + E)
    ref, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(_gpu_top1(q, K), ref)


def test_retrieval_duplicates_and_near_ties():
    """Exact duplicate keys resolve to the lowest row; keys that differ from
    the winner by one fp32 ulp in a few components make fp64 score gaps far
    below fp32 resolution, so only the exact rescoring can order them."""
    g = np.random.default_rng(5)
    q, K, _, _ = synth.retrieval_inputs_host(64, 3000, 384, 0, seed=61)
    K = K.numpy().copy()
    qn = q.numpy()
    win, _ = oracle.top1(qn, K)
    for i, w in enumerate(win[:32]):
        base = K[w].copy()
        # duplicate at a lower and a higher row
        K[(w + 1) % 3000] = base
        lo = int(g.integers(0, 3000))
        # near-tie: nudge 3 components by one ulp towards the query
        near = base.copy()
        for c in g.integers(0, 384, 3):
            near[c] = np.nextafter(near[c], np.float32(np.sign(qn[i, c]) * np.inf))
        K[lo] = near if i % 2 == 0 else base
    ref, best = oracle.top1(qn, K, nthreads=8)
    assert np.array_equal(_gpu_top1(q, torch.from_numpy(K)), ref)


def test_retrieval_equal_real_scores_decided_by_summation_order():
    """Keys that differ from the winner only by two swapped components where
    the query holds equal values: the real inner products are equal, so any
    summation other than the sequential fp64 one of the definition (a tree,
    partial sums) cannot order them; the answer must still be the oracle's."""
    g = np.random.default_rng(66)
    q, K, _, _ = synth.retrieval_inputs_host(48, 2000, 384, 0, seed=66)
    qn, Kn = q.numpy().copy(), K.numpy().copy()
    pairs = [tuple(int(v) for v in g.choice(384, 2, replace=False)) for _ in range(48)]
    for i, (a, b) in enumerate(pairs):
        qn[i, b] = qn[i, a]
    win, _ = oracle.top1(qn, Kn)
    for i, w in enumerate(win):
        a, b = pairs[i]
        twin = Kn[w].copy()
        twin[a], twin[b] = Kn[w, b], Kn[w, a]
        Kn[(w + 1 + i) % 2000] = twin
    ref, _ = oracle.top1(qn, Kn)
    assert np.array_equal(_gpu_top1(torch.from_numpy(qn), torch.from_numpy(Kn)), ref)


def test_retrieval_near_ties_one_ulp_apart():
    """A twin of each query's winner with one component moved by one fp32
    ulp, up or down: both reach the exact rescoring; the real gap is above
    the lane-parallel ordering's error bound (decided by it) or, where the
    query's component is 1e-30, far below it (decided by the sequential fp64
    sums, equal sums going to the lower index)."""
    g = np.random.default_rng(69)
    q, K, _, _ = synth.retrieval_inputs_host(48, 2000, 384, 0, seed=69)
    qn, Kn = q.numpy().copy(), K.numpy().copy()
    cs = [int(v) for v in g.integers(0, 384, 48)]
    for i in range(48):
        if i % 4 >= 2:
            qn[i, cs[i]] = np.float32(1e-30)
    win, _ = oracle.top1(qn, Kn)
    for i, w in enumerate(win):
        twin = Kn[w].copy()
        c = cs[i]
        twin[c] = np.nextafter(twin[c], np.float32(np.inf) if i % 2 else np.float32(-np.inf))
        Kn[(w + 1 + 37 * i) % 2000] = twin
    ref, _ = oracle.top1(qn, Kn)
    assert np.array_equal(_gpu_top1(torch.from_numpy(qn), torch.from_numpy(Kn)), ref)


def test_retrieval_non_unit_rows_and_empty():
    q, K, _, _ = synth.retrieval_inputs_host(40, 500, 64, 8, seed=62)
    scale = torch.from_numpy(np.random.default_rng(1).uniform(0.1, 30.0, (500, 1))).float()
    K2 = K * scale
    ref, _ = oracle.top1(q, K2)
    assert np.array_equal(_gpu_top1(q, K2), ref)
    empty = _gpu_top1(q, K[:0])
    assert np.all(empty == -1)


def test_retrieval_norms_past_the_screen_range():
    """Rows (or a query) whose components could overflow the fp16 screen
    operands: the screen proves nothing, every key is scored in fp64, and
    the answer is still the exact one."""
    q, K, _, _ = synth.retrieval_inputs_host(24, 700, 128, 4, seed=63)
    K2 = K.clone()
    K2[::97] *= 1000.0          # norms 1000: 2^8 |v| can pass 65504
    ref, _ = oracle.top1(q, K2)
    assert np.array_equal(_gpu_top1(q, K2), ref)
    q2 = q.clone()
    q2[5] *= 300.0
    ref, _ = oracle.top1(q2, K)
    assert np.array_equal(_gpu_top1(q2, K), ref)
    # largest norm just inside the range: the screen and its bound hold
    K3 = K.clone()
    K3[::50] *= 200.0
    ref, _ = oracle.top1(q, K3)
    assert np.array_equal(_gpu_top1(q, K3), ref)


def _clustered(Q, M, E, spread, seed):
    """Unit keys and queries around one direction: the smaller `spread`,
    the more 32-key blocks come within the screen's error bound of the best."""
    g = np.random.default_rng(seed)
    base = g.standard_normal(E)
    K = base[None, :] + spread * g.standard_normal((M, E))
    K = (K / np.linalg.norm(K, axis=1, keepdims=True)).astype(np.float32)
    q = base[None, :] + 0.3 * g.standard_normal((Q, E))
    q = (q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32)
    return torch.from_numpy(q), torch.from_numpy(K)


@pytest.mark.parametrize("spread", [1e-3, 3e-2])
def test_retrieval_survivors_past_the_register_groups(spread):
    """40,000 keys = 1,250 blocks, past the 512 whose maxima the decide wave
    holds in registers, with many blocks surviving the block test (all of
    them at spread 1e-3, where every key is a candidate and the candidate
    list is scored in many batches; some at 3e-2); then the same index with
    one key of norm 1000 (every key scored exactly)."""
    q, K = _clustered(8, 40000, 64, spread, 65)
    ref, _ = oracle.top1(q, K)
    assert np.array_equal(_gpu_top1(q, K), ref)
    K2 = K.clone()
    K2[12345] *= 1000.0
    ref, _ = oracle.top1(q, K2)
    assert np.array_equal(_gpu_top1(q, K2), ref)


def test_retrieval_components_below_fp16_normal_range():
    """Keys and queries with many components far below 2^-22 (subnormal or
    zero once scaled into fp16) and near-ties decided by them."""
    g = np.random.default_rng(64)
    q, K, _, _ = synth.retrieval_inputs_host(32, 900, 96, 0, seed=64)
    qn, Kn = q.numpy().copy(), K.numpy().copy()
    tiny = g.random(Kn.shape) < 0.5
    Kn[tiny] *= np.float32(1e-7)
    qn[g.random(qn.shape) < 0.5] *= np.float32(1e-8)
    win, _ = oracle.top1(qn, Kn)
    for i, w in enumerate(win[:16]):
        # a copy of the winner that differs only in components far below the
        # fp16 screen's resolution
        near = Kn[w].copy()
        c = int(g.integers(0, 96))
        near[c] = np.float32(near[c] + np.sign(qn[i, c]) * 1e-9)
        Kn[(w + 7) % 900] = near
    ref, _ = oracle.top1(qn, Kn)
    assert np.array_equal(_gpu_top1(torch.from_numpy(qn), torch.from_numpy(Kn)), ref)


@pytest.mark.parametrize("Q,M,E", [(256, 10000, 384), (65, 1000, 20), (70, 97, 388),
                                   (5, 70001, 8), (40, 300, 4096), (3, 33, 16)])
def test_prepared_index_equals_unprepared(Q, M, E):
    """The prepared index (operands and norms made once) gives the indices
    and fp64 scores of the unprepared calls bit for bit, and the oracle's."""
    q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, min(Q, 4), seed=Q + 3 * M + E)
    qd, Kd = q.to(DEV), K.to(DEV)
    prepared = P.prepare_index(Kd)
    for k in (1, 3):
        i0, s0 = P.topk(qd, Kd, k)
        i1, s1 = P.topk_prepared(qd, Kd, prepared, k)
        torch.cuda.synchronize()
        assert torch.equal(i0, i1) and torch.equal(s0, s1), k
    i2, _ = P.topk_prepared(qd, Kd, prepared, 1, want_score=False)
    torch.cuda.synchronize()
    ref, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(i2[:, 0].cpu().numpy(), ref)


def test_prepared_index_norms_past_the_screen_range():
    q, K, _, _ = synth.retrieval_inputs_host(24, 700, 128, 4, seed=65)
    K2 = K.clone()
    K2[::97] *= 1000.0
    prepared = P.prepare_index(K2.to(DEV))
    i1, _ = P.topk_prepared(q.to(DEV), K2.to(DEV), prepared, 1, want_score=False)
    torch.cuda.synchronize()
    ref, _ = oracle.top1(q, K2)
    assert np.array_equal(i1[:, 0].cpu().numpy(), ref)


@pytest.mark.parametrize("sd,od", [(torch.float16, torch.float16), (torch.float16, torch.float32),
                                   (torch.float32, torch.float32), (torch.float32, torch.float16)])
def test_gather_dtypes(sd, od):
    store = synth.state_store(300, 1024 * 16 + 8, seed=7).to(sd)
    idx = torch.tensor([5, 0, 299, 5, 17, 299], dtype=torch.int32)
    h0 = P.gather(store.to(DEV), idx.to(DEV), out_dtype=od)
    torch.cuda.synchronize()
    ref = oracle.gather(store, idx.numpy())
    if od == torch.float16 and sd == torch.float32:
        ref = oracle.round_f16(ref)
    assert np.array_equal(h0.double().cpu().numpy(), ref)


def test_gather_out_of_range_index_gives_nan_rows():
    store = synth.state_store(10, 64, seed=8).to(DEV)
    idx = torch.tensor([3, -1, 10, 9], dtype=torch.int32, device=DEV)
    h0 = P.gather(store, idx, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.isnan(h0[1]).all() and torch.isnan(h0[2]).all()
    assert torch.equal(h0[0], store[3].float()) and torch.equal(h0[3], store[9].float())


def test_query_time_path_end_to_end():
    """Retrieve the top-1 state of a 10,000-entry fp16 store (D=1024, N=16),
    inject it and prefill 32 bf16 query tokens for 256 queries; compare with
    the oracle doing the same three steps."""
    cfg = synth.RETRIEVAL
    wl = synth.QUERY_PREFILL
    D, N = wl.dim, wl.dstate
    q, K, pos, rows = synth.retrieval_inputs_host(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"],
                                                  cfg["seed"])
    store = synth.state_store(cfg["M"], D * N, seed=33, device=DEV)
    inp = synth.scan_inputs_host(wl.batch, wl.seqlen, D, N, wl.seed, torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    stream = torch.cuda.current_stream()
    idx = P.top1(q.to(DEV), K.to(DEV), stream=stream)
    h0 = P.gather(store, idx, out_dtype=torch.float16, stream=stream).view(wl.batch, D, N)
    y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0,
                   out_dtype=torch.float32, state_dtype=torch.float16, stream=stream)
    torch.cuda.synchronize()
    ref_idx, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    h0_ref = oracle.gather(store.cpu(), ref_idx).reshape(wl.batch, D, N)
    assert np.array_equal(h0.double().cpu().numpy(), h0_ref)
    y_ref, h_ref = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                               inp["Dskip"], h0_ref, nthreads=8)
    assert err_rms(y.double().cpu().numpy(), y_ref) <= TOL_BF16
    assert err_rms(hT.double().cpu().numpy(), h_ref) <= TOL_BF16


@pytest.mark.parametrize("Q,M,E", [(40, 300, 4096), (7, 5, 64), (8, 100000, 384)])
def test_retrieval_extreme_shapes(Q, M, E):
    """The largest feature count (4096: one candidate row per rescoring
    batch), a single partial key block, and a 100,000-key index."""
    q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, min(Q, 3), seed=Q + M + E)
    ref, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(_gpu_top1(q, K), ref)


def test_gather_more_queries_than_one_grid_dimension():
    """Q = 70,000 > 65,535: the launches walk the queries in slices."""
    store = synth.state_store(10, 16, seed=12).to(DEV)
    idx = torch.from_numpy(np.random.default_rng(2).integers(0, 10, 70000).astype(np.int32)).to(DEV)
    h0 = P.gather(store, idx, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = oracle.gather(store.cpu(), idx.cpu().numpy())
    assert np.array_equal(h0.double().cpu().numpy(), ref)


@pytest.mark.parametrize("sd", [torch.float16, torch.float32])
@pytest.mark.parametrize("chunk", [0, 64])
def test_scan_from_store_equals_gather_then_scan(sd, chunk):
    """precog_scan_encode_indexed: batch row b starts from store[idx[b]].
    The injection is fused into the prefill, so y and hT are bitwise those of
    precog_inject_gather followed by precog_scan_encode (one pass and
    chunked); an index outside the store starts its row from NaN, as the
    gather writes NaN for it.  Valid rows also match the oracle."""
    B, L, D, N, M = 6, 300, 256, 16, 40
    inp = synth.scan_inputs_host(B, L, D, N, seed=71, in_dtype=torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    store = torch.from_numpy(np.random.default_rng(8).normal(0, 0.5, (M, D, N))).to(sd).to(DEV)
    idx = torch.tensor([3, 39, -1, 0, 40, 3], dtype=torch.int32, device=DEV)
    y, hT = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store, idx, d["C"], d["z"],
                              d["Dskip"], chunk=chunk)
    h0 = P.gather(store.view(M, D * N), idx, out_dtype=sd).view(B, D, N)
    y2, h2 = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0,
                    state_dtype=sd, chunk=chunk)
    torch.cuda.synchronize()
    ok = torch.tensor([True, True, False, True, False, True])
    assert torch.equal(y[ok], y2[ok]) and torch.equal(hT[ok], h2[ok])
    assert torch.isnan(y[~ok]).all() and torch.isnan(hT[~ok]).all()
    rows = [0, 1, 3, 5]
    h0_ref = store.double().cpu().numpy()[idx.cpu().numpy()[rows]]
    sub = {k: (v[rows] if v.dim() == 3 else v) for k, v in inp.items()}
    y_ref, h_ref = oracle.scan(sub["x"], sub["dt"], sub["A"], sub["B"], sub["C"], sub["z"],
                               sub["Dskip"], h0_ref, nthreads=8)
    assert err_rms(y[rows].double().cpu().numpy(), y_ref) <= TOL_BF16
    assert err_rms(hT[rows].double().cpu().numpy(), h_ref) <= TOL_BF16


def test_scan_from_store_query_workload():
    """The fused query path on the query-time workload: retrieve the top-1
    state of 256 queries, then prefill 32 tokens starting from store[idx]
    directly; bitwise equal to gather + scan."""
    cfg = synth.RETRIEVAL
    wl = synth.QUERY_PREFILL
    D, N = wl.dim, wl.dstate
    q, K, pos, rows = synth.retrieval_inputs_host(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"],
                                                  cfg["seed"])
    store = synth.state_store(cfg["M"], D * N, seed=33, device=DEV)
    inp = synth.scan_inputs_host(wl.batch, wl.seqlen, D, N, wl.seed, torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    idx = P.top1(q.to(DEV), K.to(DEV))
    y, hT = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store.view(cfg["M"], D, N), idx,
                              d["C"], d["z"], d["Dskip"], out_dtype=torch.bfloat16)
    h0 = P.gather(store, idx, out_dtype=torch.float16).view(wl.batch, D, N)
    y2, h2 = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0,
                    out_dtype=torch.bfloat16, state_dtype=torch.float16)
    torch.cuda.synchronize()
    assert torch.equal(y, y2) and torch.equal(hT, h2)
