"""Parity of precog_query_top1_prefill, the query-time path of Sec. 4.2 in one
call (exact top-1 retrieval, injection of the retrieved state, query
prefill): its idx, y and hT are bitwise those of precog_retrieve_top1 (or the
prepared-index retrieval) followed by precog_scan_encode_indexed, and match
the oracle doing the three steps."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02560_amd import precog as P
from paper_2608_02560_amd import synth
from precog_testutil import TOL_BF16, TOL_F32, err_rms

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _bits(t):
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def _case(Q, M, E, L, D, seed, in_dtype=torch.bfloat16):
    q, K, pos, rows = synth.retrieval_inputs_host(Q, M, E, min(Q, 4), seed=seed)
    store = synth.state_store(max(M, 1), D * 16, seed=seed + 1, device=DEV)[:M]
    inp = synth.scan_inputs_host(Q, L, D, 16, seed + 2, in_dtype)
    return q, K, pos, rows, store.reshape(M, D, 16), inp


def _two_calls(desc, qd, Kd, store, d, out_dtype, want_y, prepared=None):
    Q, L, D = d["x"].shape
    M, E = Kd.shape
    idx = torch.empty(Q, dtype=torch.int32, device=DEV)
    nws = P.retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(max(nws, 16), dtype=torch.uint8, device=DEV)
    if prepared is None:
        P.retrieve_top1(qd, Kd, idx, ws, nws)
    else:
        P.retrieve_topk_prepared(qd, Kd, prepared, 1, idx, None, ws, nws)
    y = torch.empty((Q, L, D), dtype=out_dtype, device=DEV) if want_y else None
    hT = torch.empty((Q, D, 16), dtype=store.dtype, device=DEV)
    sws = P.scan_workspace_bytes(desc)
    wss = torch.empty(max(sws, 16), dtype=torch.uint8, device=DEV)
    P.scan_encode_indexed(desc, d["x"], d["dt"], d["A"], d["B"], d["C"] if want_y else None,
                          d["z"] if want_y else None, d["Dskip"] if want_y else None, store, M,
                          idx, y, hT, wss, sws)
    return idx, y, hT


def _one_call(desc, qd, Kd, store, d, out_dtype, want_y, prepared=None, poison=True):
    Q, L, D = d["x"].shape
    M, E = Kd.shape
    idx = torch.full((Q,), -7, dtype=torch.int32, device=DEV)
    y = torch.full((Q, L, D), 3.0, dtype=out_dtype, device=DEV) if want_y else None
    hT = torch.full((Q, D, 16), 5.0, dtype=store.dtype, device=DEV)
    nq = P.query_workspace_bytes(desc, M, E)
    wq = torch.empty(max(nq, 16), dtype=torch.uint8, device=DEV)
    if poison:
        wq.fill_(0x7f)  # nothing may depend on the workspace's previous contents
    P.query_top1_prefill(desc, qd, Kd, store, idx, d["x"], d["dt"], d["A"], d["B"],
                         d["C"] if want_y else None, d["z"] if want_y else None,
                         d["Dskip"] if want_y else None, y, hT, wq, nq, prepared=prepared)
    return idx, y, hT


def _assert_same(a, b):
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0])
    if a[1] is not None:
        assert torch.equal(_bits(a[1]), _bits(b[1]))
    assert torch.equal(_bits(a[2]), _bits(b[2]))


@pytest.mark.parametrize("prepared", [False, True])
def test_query_call_workload_matches_two_calls_and_oracle(prepared):
    """256 queries over 10,000 keys of 384 dims, a [10000, 1024, 16] fp16
    store, 32 bf16 query tokens (the one-launch decision + prefill path)."""
    cfg = synth.RETRIEVAL
    wl = synth.QUERY_PREFILL
    Q, M, E, D, L = cfg["Q"], cfg["M"], cfg["E"], wl.dim, wl.seqlen
    q, K, pos, rows = synth.retrieval_inputs_host(Q, M, E, cfg["planted"], cfg["seed"])
    store = synth.state_store(M, D * 16, seed=33, device=DEV).view(M, D, 16)
    inp = synth.scan_inputs_host(Q, L, D, 16, wl.seed, torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    qd, Kd = q.to(DEV), K.to(DEV)
    prep = P.prepare_index(Kd) if prepared else None
    for out_dtype in (torch.bfloat16, torch.float32):  # fp32 y last: checked against the oracle
        desc = P.scan_desc(Q, L, D, 16, P.BF16, P._DT[out_dtype], P.F16)
        a = _two_calls(desc, qd, Kd, store, d, out_dtype, True, prep)
        b = _one_call(desc, qd, Kd, store, d, out_dtype, True, prep)
        _assert_same(a, b)
    ref_idx, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(b[0].cpu().numpy(), ref_idx)
    assert np.array_equal(ref_idx[pos.numpy()], rows.numpy().astype(np.int32))
    h0_ref = oracle.gather(store.reshape(M, -1).cpu(), ref_idx).reshape(Q, D, 16)
    y_ref, h_ref = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                               inp["Dskip"], h0_ref, nthreads=8)
    assert err_rms(b[1].double().cpu().numpy(), y_ref) <= TOL_BF16
    assert err_rms(b[2].double().cpu().numpy(), h_ref) <= TOL_BF16


@pytest.mark.parametrize("Q,M,E,L,D", [(37, 1000, 64, 23, 1000), (3, 33, 16, 1, 520), (520, 900, 96, 6, 64),
                                       (70, 4099, 388, 40, 64), (1, 1, 4, 9, 8)])
@pytest.mark.parametrize("sd", [torch.float16, torch.float32])
def test_query_call_ragged_one_pass(Q, M, E, L, D, sd):
    """Ragged queries, keys, tokens and channels (waves past D in the last
    workgroup, a partial key block), one pass over time requested so the
    one-launch path runs; fp32 and bf16 y, fp16 and fp32 states; against the
    two calls bitwise and the oracle within tolerance."""
    q, K, _, _, store, inp = _case(Q, M, E, L, D, seed=Q * 13 + M + D)
    store = store.to(sd)
    d = {k: v.to(DEV) for k, v in inp.items()}
    qd, Kd = q.to(DEV), K.to(DEV)
    for out_dtype in (torch.bfloat16, torch.float32):  # fp32 y last: checked against the oracle
        desc = P.scan_desc(Q, L, D, 16, P.BF16, P._DT[out_dtype], P._DT[sd], chunk=L)
        a = _two_calls(desc, qd, Kd, store, d, out_dtype, True)
        b = _one_call(desc, qd, Kd, store, d, out_dtype, True)
        _assert_same(a, b)
    ref_idx, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(b[0].cpu().numpy(), ref_idx)
    h0_ref = oracle.gather(store.reshape(M, -1).cpu(), ref_idx).reshape(Q, D, 16)
    y_ref, h_ref = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                               inp["Dskip"], h0_ref, nthreads=8)
    assert err_rms(b[1].double().cpu().numpy(), y_ref) <= TOL_BF16
    assert err_rms(b[2].double().cpu().numpy(), h_ref) <= TOL_BF16


def test_query_call_state_only_and_fallbacks():
    """y = NULL (state only, one launch); then configurations that run the
    decision and the prefill as two launches: time chunks (the automatic
    choice for few queries) and fp32 inputs.  Every case equals the two calls
    bitwise; the fp32 one also matches the oracle."""
    Q, M, E, L, D = 20, 500, 32, 30, 256
    q, K, _, _, store, inp = _case(Q, M, E, L, D, seed=5)
    d = {k: v.to(DEV) for k, v in inp.items()}
    qd, Kd = q.to(DEV), K.to(DEV)
    desc = P.scan_desc(Q, L, D, 16, P.BF16, P.F32, P.F16, chunk=L)
    _assert_same(_two_calls(desc, qd, Kd, store, d, torch.float32, False),
                 _one_call(desc, qd, Kd, store, d, torch.float32, False))
    desc = P.scan_desc(Q, L, D, 16, P.BF16, P.F32, P.F16)  # automatic: time chunks
    assert P.scan_workspace_bytes(desc) > 0
    _assert_same(_two_calls(desc, qd, Kd, store, d, torch.float32, True),
                 _one_call(desc, qd, Kd, store, d, torch.float32, True))
    inp32 = synth.scan_inputs_host(Q, L, D, 16, 9, torch.float32)
    d32 = {k: v.to(DEV) for k, v in inp32.items()}
    desc = P.scan_desc(Q, L, D, 16, P.F32, P.F32, P.F32, chunk=L)
    s32 = store.float()
    b = _one_call(desc, qd, Kd, s32, d32, torch.float32, True)
    _assert_same(_two_calls(desc, qd, Kd, s32, d32, torch.float32, True), b)
    ref_idx, _ = oracle.top1(q, K, nthreads=8)
    h0_ref = oracle.gather(s32.reshape(M, -1).cpu(), ref_idx).reshape(Q, D, 16)
    y_ref, h_ref = oracle.scan(inp32["x"], inp32["dt"], inp32["A"], inp32["B"], inp32["C"],
                               inp32["z"], inp32["Dskip"], h0_ref, nthreads=8)
    assert err_rms(b[1].double().cpu().numpy(), y_ref) <= TOL_F32
    assert err_rms(b[2].double().cpu().numpy(), h_ref) <= TOL_F32


def test_query_call_empty_index():
    """M = 0: every idx is -1 and every prefill row starts from NaN, as the
    two calls give."""
    Q, E, L, D = 5, 16, 12, 64
    q, _, _, _ = synth.retrieval_inputs_host(Q, 4, E, 0, seed=3)
    inp = synth.scan_inputs_host(Q, L, D, 16, 4, torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    Kd = torch.empty((0, E), dtype=torch.float32, device=DEV)
    store = torch.empty((0, D, 16), dtype=torch.float16, device=DEV)
    desc = P.scan_desc(Q, L, D, 16, P.BF16, P.F32, P.F16, chunk=L)
    a = _two_calls(desc, q.to(DEV), Kd, store, d, torch.float32, True)
    b = _one_call(desc, q.to(DEV), Kd, store, d, torch.float32, True)
    torch.cuda.synchronize()
    assert (b[0] == -1).all() and torch.equal(a[0], b[0])
    assert torch.isnan(b[2].float()).all() and torch.isnan(b[1]).all()
    assert torch.isnan(a[2].float()).all() and torch.isnan(a[1]).all()


def test_query_call_repeated_calls_deterministic():
    """Two calls in a row with the same workspace give the same bits (the
    one-launch path keeps nothing from one call to the next)."""
    Q, M, E, L, D = 64, 2000, 128, 16, 512
    q, K, _, _, store, inp = _case(Q, M, E, L, D, seed=77)
    d = {k: v.to(DEV) for k, v in inp.items()}
    qd, Kd = q.to(DEV), K.to(DEV)
    desc = P.scan_desc(Q, L, D, 16, P.BF16, P.BF16, P.F16, chunk=L)
    a = _one_call(desc, qd, Kd, store, d, torch.bfloat16, True, poison=False)
    b = _one_call(desc, qd, Kd, store, d, torch.bfloat16, True, poison=True)
    _assert_same(a, b)


def _clustered(Q, M, E, spread, seed):
    """Unit keys and queries around one direction: the smaller `spread`, the
    more 32-key blocks come within the screen's error bound of the best."""
    g = np.random.default_rng(seed)
    base = g.standard_normal(E)
    K = base[None, :] + spread * g.standard_normal((M, E))
    K = (K / np.linalg.norm(K, axis=1, keepdims=True)).astype(np.float32)
    q = base[None, :] + 0.3 * g.standard_normal((Q, E))
    q = (q / np.linalg.norm(q, axis=1, keepdims=True)).astype(np.float32)
    return torch.from_numpy(q), torch.from_numpy(K)


def _check_heavy(q, K, L, D, seed, prepared):
    Q, M = q.shape[0], K.shape[0]
    store = synth.state_store(M, D * 16, seed=seed, device=DEV).view(M, D, 16)
    inp = synth.scan_inputs_host(Q, L, D, 16, seed + 1, torch.bfloat16)
    d = {k: v.to(DEV) for k, v in inp.items()}
    qd, Kd = q.to(DEV), K.to(DEV)
    prep = P.prepare_index(Kd) if prepared else None
    desc = P.scan_desc(Q, L, D, 16, P.BF16, P.F32, P.F16, chunk=L)
    a = _two_calls(desc, qd, Kd, store, d, torch.float32, True, prep)
    b = _one_call(desc, qd, Kd, store, d, torch.float32, True, prep)
    _assert_same(a, b)
    ref_idx, _ = oracle.top1(q, K, nthreads=8)
    assert np.array_equal(b[0].cpu().numpy(), ref_idx)


@pytest.mark.parametrize("spread", [1e-3, 3e-2])
def test_query_call_decision_past_the_register_groups(spread):
    """The decision inside the one-launch path (one wave of a 512-thread
    workgroup) with 40,000 keys = 1,250 blocks, past the 512 whose maxima it
    holds in registers: every block survives at spread 1e-3 (every key a
    candidate, the candidate list scored in many batches), some at 3e-2; then
    one key of norm 1000 (every key scored exactly), prepared index too."""
    q, K = _clustered(8, 40000, 64, spread, 65)
    _check_heavy(q, K, 7, 64, 91, prepared=False)
    K2 = K.clone()
    K2[12345] *= 1000.0
    _check_heavy(q, K2, 7, 64, 92, prepared=True)


def test_query_call_largest_feature_count():
    """E = 4096, the largest feature count (one candidate row per rescoring
    batch), inside the one-launch path, unprepared and prepared."""
    q, K, _, _ = synth.retrieval_inputs_host(40, 300, 4096, 3, seed=40 + 300 + 4096)
    _check_heavy(q, K, 11, 192, 93, prepared=False)
    _check_heavy(q, K, 11, 192, 94, prepared=True)
