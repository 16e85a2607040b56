"""Parity of precog_retrieve_topk (bit-exact indices and fp64 scores) and of
precog_inject_compose (within its stated rounding bound) with the oracle,
plus the top-k query-time path: retrieve k states, compose, prefill."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02560_amd import precog as P
from paper_2608_02560_amd import synth
from precog_testutil import TOL_BF16, err_rms

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _gpu_topk(q, K, k):
    idx, sc = P.topk(q.to(DEV), K.to(DEV), k)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), sc.cpu().numpy()


def _check_topk(q, K, k):
    ref_i, ref_s = oracle.topk_scores(q, K, k)
    got_i, got_s = _gpu_topk(q, K, k)
    assert np.array_equal(got_i, ref_i.astype(np.int32))
    # the same sequential fp64 sums: bit-identical scores
    assert np.array_equal(got_s, ref_s)


def test_topk_workload_k3():
    """The retrieval workload (Q=256, M=10000, E=384) at the paper's default k = 3."""
    cfg = synth.RETRIEVAL
    q, K, pos, rows = synth.retrieval_inputs_host(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"],
                                                  cfg["seed"])
    ref_i, ref_s = oracle.topk_scores(q, K, 3)
    got_i, got_s = _gpu_topk(q, K, 3)
    assert np.array_equal(got_i, ref_i.astype(np.int32))
    assert np.array_equal(got_s, ref_s)
    assert np.array_equal(got_i[pos.numpy(), 0], rows.numpy().astype(np.int32))


@pytest.mark.parametrize("spread", [1e-3, 3e-2])
def test_topk_survivors_past_the_register_groups(spread):
    """Top-3 with scores over 40,000 clustered keys (1,250 blocks, many or
    all of them surviving the block test): indices and fp64 scores equal the
    oracle's bit for bit."""
    g = np.random.default_rng(66)
    base = g.standard_normal(64)
    K = base[None, :] + spread * g.standard_normal((40000, 64))
    K = torch.from_numpy((K / np.linalg.norm(K, axis=1, keepdims=True)).astype(np.float32))
    q = base[None, :] + 0.3 * g.standard_normal((8, 64))
    q = torch.from_numpy((q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32))
    _check_topk(q, K, 3)


@pytest.mark.parametrize("Q,M,E,k", [(1, 1, 4, 1), (3, 33, 16, 2), (65, 1000, 20, 5),
                                     (70, 97, 388, 64), (130, 300, 64, 7), (5, 64, 8, 64),
                                     (600, 1500, 96, 3)])
def test_topk_ragged_shapes(Q, M, E, k):
    q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, min(Q, 4), seed=Q * 5 + M + E + k)
    _check_topk(q, K, k)


def test_topk_k1_equals_top1():
    q, K, _, _ = synth.retrieval_inputs_host(50, 2000, 384, 10, seed=71)
    i1 = P.top1(q.to(DEV), K.to(DEV))
    ik, _ = P.topk(q.to(DEV), K.to(DEV), 1)
    torch.cuda.synchronize()
    assert torch.equal(i1.cpu(), ik[:, 0].cpu())


def test_topk_duplicates_and_clustered_keys():
    """Duplicated rows tie exactly (lower row first); a cluster of near
    copies of the winner makes the k best sit inside one 32-key block, the
    case where the k-th block maximum is far below the k-th best score."""
    q, K, _, _ = synth.retrieval_inputs_host(32, 3000, 384, 0, seed=72)
    K = K.numpy().copy()
    qn = q.numpy()
    win, _ = oracle.top1(qn, K)
    g = np.random.default_rng(3)
    for i, w in enumerate(win[:16]):
        base = K[w].copy()
        blk = (int(w) // 32) * 32
        for r in range(blk, min(blk + 32, 3000)):
            if r != w:
                near = base + np.float32(1e-3) * g.standard_normal(384).astype(np.float32)
                K[r] = (near / np.linalg.norm(near)).astype(np.float32)
        K[(w + 97) % 3000] = base  # exact duplicate elsewhere
    _check_topk(q, torch.from_numpy(K), 8)


def _compose_bound(store64, idx, sc, tau):
    """(k + 2) 2^-24 sum_j w_j |h_j| per element: the fp32 weight rounding and
    one rounding per fused multiply-add (the composition's stated bound)."""
    Q, k = idx.shape
    out = np.zeros((Q,) + store64.shape[1:])
    for qi in range(Q):
        lg = sc[qi] / tau
        w = np.exp(lg - lg.max())
        w = w / w.sum()
        for j in range(k):
            out[qi] += w[j] * np.abs(store64[idx[qi, j]])
    return (k + 2) * 2.0 ** -24 * out + 1e-38


@pytest.mark.parametrize("sd,od,k,tau", [(torch.float16, torch.float32, 3, 1.0),
                                         (torch.float32, torch.float32, 5, 0.05),
                                         (torch.float16, torch.float16, 3, 0.2),
                                         (torch.float32, torch.float16, 64, 1.0)])
def test_compose_matches_oracle(sd, od, k, tau):
    q, K, _, _ = synth.retrieval_inputs_host(37, 500, 64, 4, seed=73 + k)
    store = synth.state_store(500, 1024 * 16 + 8, seed=9).to(sd)
    idx, sc = P.topk(q.to(DEV), K.to(DEV), k)
    h0 = P.compose(store.to(DEV), idx, sc, tau=tau, out_dtype=od)
    torch.cuda.synchronize()
    idx_n, sc_n = idx.cpu().numpy(), sc.cpu().numpy()
    ref = oracle.topk_compose(store, idx_n, sc_n, tau)
    bound = _compose_bound(store.double().numpy(), idx_n, sc_n, tau)
    got = h0.double().cpu().numpy()
    if od == torch.float16:
        # the fp32 result is rounded once more, to nearest even fp16: half an
        # fp16 ulp at its magnitude (2^-25 below the normal range)
        mag = np.abs(ref) * (1 + 1e-6) + bound
        bound = bound + np.ldexp(1.0, np.maximum(np.frexp(mag)[1] - 12, -25))
    assert np.all(np.abs(got - ref) <= bound)


def test_compose_k1_is_gather_and_equal_scores_are_mean():
    store = synth.state_store(300, 4096, seed=10).to(DEV)
    idx = torch.tensor([[5], [0], [299]], dtype=torch.int32, device=DEV)
    sc = torch.tensor([[0.3], [-2.0], [7.0]], dtype=torch.float64, device=DEV)
    a = P.compose(store, idx, sc, tau=0.01, out_dtype=torch.float32)
    b = P.gather(store, idx[:, 0].contiguous(), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    idx4 = torch.tensor([[1, 2, 3, 4]], dtype=torch.int32, device=DEV)
    sc4 = torch.zeros((1, 4), dtype=torch.float64, device=DEV)
    m = P.compose(store, idx4, sc4, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = store[1:5].double().mean(0).cpu().numpy()
    assert np.abs(m[0].double().cpu().numpy() - ref).max() <= 6 * 2.0 ** -24 * \
        np.abs(store[1:5].double().cpu().numpy()).mean(0).max()


def test_compose_out_of_range_index_gives_nan_row():
    store = synth.state_store(10, 64, seed=11).to(DEV)
    idx = torch.tensor([[1, 2], [3, 10], [-1, 0]], dtype=torch.int32, device=DEV)
    sc = torch.zeros((3, 2), dtype=torch.float64, device=DEV)
    h0 = P.compose(store, idx, sc, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.isfinite(h0[0]).all()
    assert torch.isnan(h0[1]).all() and torch.isnan(h0[2]).all()


def test_topk_query_path_end_to_end():
    """Top-3 retrieval over the 10,000-entry fp16 store (D=1024, N=16),
    softmax composition into h0, then the 32-token bf16 query prefill for
    256 queries; the oracle runs the same three steps in fp64."""
    cfg = synth.RETRIEVAL
    wl = synth.QUERY_PREFILL
    D, N = wl.dim, wl.dstate
    q, K, _, _ = synth.retrieval_inputs_host(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"],
                                             cfg["seed"])
    store = synth.state_store(cfg["M"], D * N, seed=33, device=DEV)
    inp = synth.scan_inputs_host(wl.batch, wl.seqlen, D, N, wl.seed, torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    idx, sc = P.topk(q.to(DEV), K.to(DEV), 3)
    h0 = P.compose(store, idx, sc, tau=1.0, out_dtype=torch.float32).view(wl.batch, D, N)
    y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0,
                   out_dtype=torch.float32, state_dtype=torch.float32)
    torch.cuda.synchronize()
    ref_i, ref_s = oracle.topk_scores(q, K, 3)
    assert np.array_equal(idx.cpu().numpy(), ref_i.astype(np.int32))
    h0_ref = oracle.topk_compose(store.cpu(), ref_i, ref_s, 1.0).reshape(wl.batch, D, N)
    y_ref, h_ref = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                               inp["Dskip"], h0_ref, nthreads=8)
    assert err_rms(y.double().cpu().numpy(), y_ref) <= TOL_BF16
    assert err_rms(hT.double().cpu().numpy(), h_ref) <= TOL_BF16


@pytest.mark.parametrize("Q,M,E,k", [(20, 300, 4096, 5), (9, 7, 16, 7), (6, 70001, 8, 3)])
def test_topk_extreme_shapes(Q, M, E, k):
    """E = 4096 (one candidate row per rescoring batch), k = M (every key
    ranked) on a single partial key block, and 2,188 key blocks."""
    q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, min(Q, 3), seed=Q * 3 + M + E)
    _check_topk(q, K, k)


def test_compose_more_queries_than_one_grid_dimension():
    store = synth.state_store(12, 16, seed=13).to(DEV)
    g = np.random.default_rng(3)
    idx = torch.from_numpy(g.integers(0, 12, (70000, 2)).astype(np.int32)).to(DEV)
    sc = torch.from_numpy(g.normal(size=(70000, 2))).to(DEV)
    h0 = P.compose(store, idx, sc, tau=0.5, out_dtype=torch.float32)
    torch.cuda.synchronize()
    idx_n, sc_n = idx.cpu().numpy(), sc.cpu().numpy()
    ref = oracle.topk_compose(store.cpu(), idx_n[-500:], sc_n[-500:], 0.5)
    bound = _compose_bound(store.double().cpu().numpy(), idx_n[-500:], sc_n[-500:], 0.5)
    assert np.all(np.abs(h0[-500:].double().cpu().numpy() - ref) <= bound)


@pytest.mark.parametrize("sd", [torch.float16, torch.float32])
@pytest.mark.parametrize("chunk", [0, 64])
def test_scan_from_composed_store_equals_compose_then_scan(sd, chunk):
    """precog_scan_encode_indexed with scores: batch row b starts from the
    softmax composition of its k store rows.  The weights and the fp32 sum
    are the composition kernel's, and the composed state is rounded to the
    state dtype as that kernel stores it, so y and hT are bitwise those of
    precog_inject_compose followed by precog_scan_encode (one pass and
    chunked).  A row with an index outside the store starts from NaN."""
    B, L, D, N, M, k = 5, 300, 256, 16, 40, 3
    inp = synth.scan_inputs_host(B, L, D, N, seed=75, in_dtype=torch.bfloat16)
    d = {key: v.to(DEV) for key, v in inp.items()}
    store = torch.from_numpy(np.random.default_rng(9).normal(0, 0.5, (M, D, N))).to(sd).to(DEV)
    idx = torch.tensor([[3, 39, 0], [7, 7, 1], [5, -1, 2], [0, 1, 2], [9, 40, 8]],
                       dtype=torch.int32, device=DEV)
    sc = torch.from_numpy(np.random.default_rng(10).normal(0.2, 0.05, (B, k))).to(DEV)
    y, hT = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store, idx, d["C"], d["z"],
                              d["Dskip"], score=sc, tau=0.1, chunk=chunk)
    h0 = P.compose(store.view(M, D * N), idx, sc, tau=0.1, out_dtype=sd).view(B, D, N)
    y2, h2 = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0,
                    state_dtype=sd, chunk=chunk)
    torch.cuda.synchronize()
    ok = torch.tensor([True, True, False, True, False])
    assert torch.equal(y[ok], y2[ok]) and torch.equal(hT[ok], h2[ok])
    assert torch.isnan(y[~ok]).all() and torch.isnan(hT[~ok]).all()


def test_scan_from_store_k1_scores_equal_plain_index():
    """k = 1 with a score: the weight is exactly 1, so the start is the row
    itself, as without scores."""
    B, L, D, N, M = 3, 40, 64, 16, 10
    inp = synth.scan_inputs_host(B, L, D, N, seed=76, in_dtype=torch.float32)
    d = {key: v.to(DEV) for key, v in inp.items()}
    store = torch.from_numpy(np.random.default_rng(11).normal(0, 0.5, (M, D, N))).float().to(DEV)
    idx = torch.tensor([[4], [0], [9]], dtype=torch.int32, device=DEV)
    sc = torch.tensor([[0.7], [-3.0], [12.0]], dtype=torch.float64, device=DEV)
    y, hT = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store, idx, d["C"], d["z"],
                              d["Dskip"], score=sc, tau=0.01)
    y2, h2 = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store, idx[:, 0].contiguous(),
                               d["C"], d["z"], d["Dskip"])
    torch.cuda.synchronize()
    assert torch.equal(y, y2) and torch.equal(hT, h2)


@pytest.mark.parametrize("k", [1, 3])
def test_topk_keys_and_queries_of_mixed_norms(k):
    """Keys with norms spread over 1e-3 .. 200 (squared norms below the
    screen's overflow limit, so the per-block and per-key error bounds of the
    decision decide) and queries with norms 1e-2 .. 50: indices and fp64
    scores bit-exact, unprepared and with the prepared index; top-1 also
    through the one-call query path."""
    g = np.random.default_rng(97)
    q, K, _, _ = synth.retrieval_inputs_host(96, 3000, 256, 8, seed=97)
    Kn = K.numpy() * np.exp(g.uniform(np.log(1e-3), np.log(200.0), (3000, 1))).astype(np.float32)
    qn = q.numpy() * np.exp(g.uniform(np.log(1e-2), np.log(50.0), (96, 1))).astype(np.float32)
    q2, K2 = torch.from_numpy(qn.astype(np.float32)), torch.from_numpy(Kn.astype(np.float32))
    assert float((K2.double() ** 2).sum(1).max()) < 60000.0
    _check_topk(q2, K2, k)
    qd, Kd = q2.to(DEV), K2.to(DEV)
    prep = P.prepare_index(Kd)
    i1, s1 = P.topk_prepared(qd, Kd, prep, k)
    torch.cuda.synchronize()
    ref_i, ref_s = oracle.topk_scores(q2, K2, k)
    assert np.array_equal(i1.cpu().numpy(), ref_i.astype(np.int32))
    assert np.array_equal(s1.cpu().numpy(), ref_s)
    if k == 1:
        D, L = 64, 5
        store = synth.state_store(3000, D * 16, seed=98, device=DEV).view(3000, D, 16)
        inp = synth.scan_inputs_host(96, L, D, 16, 99, torch.bfloat16)
        d = {key: v.to(DEV) for key, v in inp.items()}
        idx, _, _ = P.query_prefill(qd, Kd, store, d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"],
                                    d["Dskip"], chunk=L)
        torch.cuda.synchronize()
        assert np.array_equal(idx.cpu().numpy(), ref_i[:, 0].astype(np.int32))
