"""Parity of the HIP scan (precog_scan_encode) with the fp64 oracle.

Small problems are compared element by element over every output; the
workload-sized ones (corpus encode, long context, large corpus) on sampled
(b, d) rows that the oracle recomputes independently, in the same launch
configuration the benchmark times.  Metric: err_rms (max |g - o| over
max(|o|, rms(o))), bars 1e-5 for fp32 inputs and 2e-3 for bf16 inputs with
fp32 state; bf16 outputs must sit within one bf16 ulp of the oracle rounded
to nearest even, fp16 states within one fp16 ulp."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02560_amd import precog as P
from paper_2608_02560_amd import synth
from precog_testutil import TOL_BF16, TOL_F32, err_rms, oracle_rows, sample_rows

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _dev(inp):
    return {k: (v.to(DEV) if v is not None else None) for k, v in inp.items()}


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _full_oracle(inp, h0=None, want_y=True):
    return oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                       inp["Dskip"], h0, want_y=want_y, nthreads=8)


def _bf16_ulp_ok(got_bf16, ref64):
    """|got - RNE_bf16(ref)| <= 1 bf16 ulp of the reference, plus the fp32
    computation's own error on the rms-floored scale of the tolerance metric
    (TOL_F32 x rms(ref)): that term matters only where y cancels to far below
    its rms, where one bf16 ulp of the tiny value is smaller than any fp32
    accumulation can resolve."""
    r = oracle.round_bf16(ref64)
    g = got_bf16.detach().float().cpu().numpy().astype(np.float64)
    rms = np.sqrt(np.mean(np.asarray(ref64, np.float64) ** 2))
    return np.all(np.abs(g - r) <= oracle.bf16_ulp(r) + TOL_F32 * rms)


def _f16_ulp_ok(got_f16, ref64):
    r = oracle.round_f16(ref64)
    g = got_f16.detach().float().cpu().numpy().astype(np.float64)
    _, e = np.frexp(r)
    ulp = np.ldexp(1.0, np.maximum(e, -13) - 11)
    return np.all(np.abs(g - r) <= ulp)


# ---------------------------------------------------------------------------
# Single fp32 layer: B=1, L=512, D=128, N=16 (full comparison)
# ---------------------------------------------------------------------------
def test_single_layer_fp32_full():
    wl = synth.SINGLE_LAYER
    inp = synth.scan_inputs_host(wl.batch, wl.seqlen, wl.dim, wl.dstate, wl.seed, torch.float32)
    y_ref, h_ref = _full_oracle(inp)
    d = _dev(inp)
    for chunk in (0, wl.seqlen, 64, 100, 1):
        y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"],
                       chunk=chunk)
        torch.cuda.synchronize()
        assert err_rms(_np(y), y_ref) <= TOL_F32, chunk
        assert err_rms(_np(hT), h_ref) <= TOL_F32, chunk


def test_single_layer_split_at_384():
    """Theorem 1 on the GPU: scan(c ++ q) == scan(q, h0 = hT(c)), split at
    t = 384 and at points that are not multiples of any tile size."""
    wl = synth.SINGLE_LAYER
    inp = synth.scan_inputs_host(wl.batch, wl.seqlen, wl.dim, wl.dstate, wl.seed, torch.float32)
    y_ref, h_ref = _full_oracle(inp)
    d = _dev(inp)
    y_full, h_full = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"])
    for split in (384, 1, 77, 511):
        part = lambda t, a, b: t[:, a:b].contiguous()
        yc, hc = P.scan(part(d["x"], 0, split), part(d["dt"], 0, split), d["A"],
                        part(d["B"], 0, split), part(d["C"], 0, split),
                        part(d["z"], 0, split), d["Dskip"])
        yq, hq = P.scan(part(d["x"], split, None), part(d["dt"], split, None), d["A"],
                        part(d["B"], split, None), part(d["C"], split, None),
                        part(d["z"], split, None), d["Dskip"], h0=hc)
        torch.cuda.synchronize()
        y_split = torch.cat([yc, yq], dim=1)
        assert err_rms(_np(hq), h_ref) <= TOL_F32
        assert err_rms(_np(y_split), y_ref) <= TOL_F32
        # against the unsplit GPU run: the same recurrence, regrouped
        assert err_rms(_np(hq), _np(h_full)) <= 1e-6
        assert err_rms(_np(y_split), _np(y_full)) <= 1e-6


def test_split_through_fp16_state_within_paper_bound():
    """Passing the intermediate state at fp16 (the paper's storage precision)
    moves the continuation by no more than the rounding of that state,
    carried forward by the decaying recurrence (App. A floating-point note)."""
    wl = synth.SINGLE_LAYER
    inp = synth.scan_inputs_host(wl.batch, wl.seqlen, wl.dim, wl.dstate, wl.seed, torch.float32)
    d = _dev(inp)
    s = 384
    part = lambda t, a, b: t[:, a:b].contiguous()
    _, hc16 = P.scan(part(d["x"], 0, s), part(d["dt"], 0, s), d["A"], part(d["B"], 0, s),
                     part(d["C"], 0, s), part(d["z"], 0, s), d["Dskip"],
                     state_dtype=torch.float16, want_y=False)
    _, hq = P.scan(part(d["x"], s, None), part(d["dt"], s, None), d["A"], part(d["B"], s, None),
                   part(d["C"], s, None), part(d["z"], s, None), d["Dskip"], h0=hc16,
                   state_dtype=torch.float16, want_y=False)
    _, h_ref = _full_oracle(inp, want_y=False)
    _, hc_ref = oracle.scan(inp["x"][:, :s], inp["dt"][:, :s], inp["A"], inp["B"][:, :s],
                            inp["C"][:, :s], want_y=False)
    torch.cuda.synchronize()
    # each stored element moves by <= 2^-11 |h| (RNE), and each later step
    # only shrinks that perturbation (|decay| < 1); the final fp16 store adds
    # its own 2^-11
    bound = 2.0 ** -11 * np.max(np.abs(hc_ref)) + 2.0 ** -11 * np.abs(h_ref) + 1e-6
    assert np.all(np.abs(_np(hq) - h_ref) <= bound)


# ---------------------------------------------------------------------------
# Shapes, options and edge cases (full comparison, small sizes)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("N", [1, 2, 4, 8, 16, 32, 64])
def test_all_state_sizes(N):
    inp = synth.scan_inputs_host(2, 37, 72, N, seed=40 + N, in_dtype=torch.float32, h0_std=1.0)
    y_ref, h_ref = _full_oracle(inp, h0=inp["h0"])
    d = _dev(inp)
    y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=d["h0"])
    torch.cuda.synchronize()
    assert err_rms(_np(y), y_ref) <= TOL_F32
    assert err_rms(_np(hT), h_ref) <= TOL_F32


@pytest.mark.parametrize("B,L,D,N", [(1, 1, 8, 16), (3, 5, 8, 16), (2, 129, 200, 16),
                                     (1, 300, 264, 16), (5, 17, 1032, 16), (2, 150, 72, 64),
                                     (3, 77, 40, 32), (1, 200, 264, 64)])
def test_ragged_shapes(B, L, D, N):
    inp = synth.scan_inputs_host(B, L, D, N, seed=B * 1000 + L + D + N, in_dtype=torch.float32,
                                 h0_std=0.5)
    y_ref, h_ref = _full_oracle(inp, h0=inp["h0"])
    d = _dev(inp)
    for chunk in (0, 7, L):
        y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"],
                       h0=d["h0"], chunk=chunk)
        torch.cuda.synchronize()
        assert err_rms(_np(y), y_ref) <= TOL_F32
        assert err_rms(_np(hT), h_ref) <= TOL_F32


def test_optional_operands():
    inp = synth.scan_inputs_host(2, 50, 64, 16, seed=51, in_dtype=torch.float32, h0_std=1.0)
    d = _dev(inp)
    cases = [dict(z=None), dict(Dskip=None), dict(z=None, Dskip=None), dict(h0=None)]
    for c in cases:
        args = dict(z=inp["z"], Dskip=inp["Dskip"], h0=inp["h0"])
        args.update(c)
        y_ref, h_ref = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"],
                                   args["z"], args["Dskip"], args["h0"])
        dargs = {k: (v.to(DEV) if v is not None else None) for k, v in args.items()}
        y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], **dargs)
        torch.cuda.synchronize()
        assert err_rms(_np(y), y_ref) <= TOL_F32, c
        assert err_rms(_np(hT), h_ref) <= TOL_F32, c
    # state-only encode: y = NULL, C / z / Dskip unread
    _, h_ref = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], h0=inp["h0"],
                           want_y=False)
    _, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], None, None, None, h0=d["h0"], want_y=False)
    torch.cuda.synchronize()
    assert err_rms(_np(hT), h_ref) <= TOL_F32


def test_empty_sequence_copies_state():
    inp = synth.scan_inputs_host(2, 0, 64, 16, seed=52, in_dtype=torch.float32, h0_std=1.0)
    d = _dev(inp)
    _, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=d["h0"])
    _, hz = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"])
    _, h16 = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"],
                    h0=d["h0"].half(), state_dtype=torch.float16)
    torch.cuda.synchronize()
    assert torch.equal(hT, d["h0"])
    assert torch.count_nonzero(hz) == 0
    assert torch.equal(h16.float(), d["h0"].half().float())
    # empty batch and empty channel count are no-ops
    P.scan(d["x"][:0], d["dt"][:0], d["A"], d["B"][:0], d["C"][:0], d["z"][:0], d["Dskip"])


def test_in_place_state_and_strided_store():
    """hT may alias h0 (streaming prefill), and hT may land in a strided slot
    of a [chunks, layers, D, N] store."""
    inp = synth.scan_inputs_host(3, 40, 64, 16, seed=53, in_dtype=torch.float32, h0_std=1.0)
    _, h_ref = _full_oracle(inp, h0=inp["h0"])
    d = _dev(inp)
    for chunk in (0, 8):
        state = d["h0"].clone()
        P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=state, hT=state,
               chunk=chunk)
        torch.cuda.synchronize()
        assert err_rms(_np(state), h_ref) <= TOL_F32
    layers = 4
    store = torch.full((3, layers, 64, 16), -7.0, device=DEV, dtype=torch.float16)
    h0_16 = inp["h0"].half()
    _, h_ref16 = _full_oracle(inp, h0=h0_16)
    for layer in (0, 2):
        P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0_16.to(DEV),
               state_dtype=torch.float16, hT=store[:, layer], hT_batch_stride=layers * 64 * 16)
    torch.cuda.synchronize()
    assert _f16_ulp_ok(store[:, 0], h_ref16) and _f16_ulp_ok(store[:, 2], h_ref16)
    assert torch.all(store[:, 1] == -7.0) and torch.all(store[:, 3] == -7.0)


def test_fp16_state_io():
    inp = synth.scan_inputs_host(2, 60, 128, 16, seed=54, in_dtype=torch.float32, h0_std=1.0)
    h0_16 = inp["h0"].half()
    y_ref, h_ref = _full_oracle(inp, h0=h0_16)
    d = _dev(inp)
    y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"],
                   h0=h0_16.to(DEV), state_dtype=torch.float16)
    torch.cuda.synchronize()
    assert err_rms(_np(y), y_ref) <= TOL_F32
    assert _f16_ulp_ok(hT, h_ref)


def test_deterministic_bitwise():
    inp = synth.scan_inputs_host(4, 300, 256, 16, seed=55, in_dtype=torch.bfloat16)
    d = _dev(inp)
    outs = []
    for _ in range(2):
        outs.append(P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"],
                           out_dtype=torch.bfloat16, state_dtype=torch.float16, chunk=64))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_chunk_sweep_agrees():
    """Any time-chunk length gives the same result up to fp32 reassociation."""
    inp = synth.scan_inputs_host(2, 1000, 128, 16, seed=56, in_dtype=torch.bfloat16)
    y_ref, h_ref = _full_oracle(inp)
    d = _dev(inp)
    for chunk in (0, 1000, 999, 256, 64, 33, 8):
        y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], chunk=chunk)
        torch.cuda.synchronize()
        assert err_rms(_np(y), y_ref) <= 1e-5, chunk
        assert err_rms(_np(hT), h_ref) <= 1e-5, chunk


@pytest.mark.parametrize("B,L,D,N,chunk", [(1, 512, 128, 16, 0), (2, 500, 64, 16, 56),
                                           (2, 500, 64, 16, 16), (3, 300, 40, 16, 5),
                                           (1, 640, 8, 64, 10), (1, 190, 8, 2, 3)])
@pytest.mark.parametrize("sd", [torch.float32, torch.float16])
def test_short_sequence_carries(B, L, D, N, chunk, sd):
    """9 to 64 time chunks over at most 8192 (b, d, n) lanes, where the
    carries come from a scan over the chunks' steps (one wave per lane)
    instead of the sequential fold: the automatic choice for the single
    layer, ragged last chunks, channels past the last full wave, N = 64 and
    N = 2; from a nonzero initial state in fp32 and fp16, against the oracle
    (fp32 bar; an fp16 hT within one fp16 ulp)."""
    inp = synth.scan_inputs_host(B, L, D, N, seed=B * 7 + L + D + N, in_dtype=torch.float32)
    h0 = torch.from_numpy(np.random.default_rng(L).normal(0, 0.5, (B, D, N))).to(sd)
    d = _dev(inp)
    y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0.to(DEV),
                   state_dtype=sd, chunk=chunk)
    torch.cuda.synchronize()
    y_ref, h_ref = _full_oracle(inp, h0.double().numpy())
    assert err_rms(_np(y), y_ref) <= TOL_F32
    if sd == torch.float32:
        assert err_rms(_np(hT), h_ref) <= TOL_F32
    else:
        assert _f16_ulp_ok(hT, h_ref)


def test_short_sequence_carries_from_store():
    """The chunk-step scan with the injected start read inside it: from
    store[idx[b]] and from a softmax composition of k rows, bitwise those of
    gather (compose) + scan in the same chunks; an index outside the store
    gives a NaN row."""
    B, L, D, N, M = 3, 300, 64, 16, 12
    inp = synth.scan_inputs_host(B, L, D, N, seed=79, in_dtype=torch.float32)
    d = _dev(inp)
    store = torch.from_numpy(np.random.default_rng(12).normal(0, 0.5, (M, D, N))).float().to(DEV)
    idx = torch.tensor([5, -1, 11], dtype=torch.int32, device=DEV)
    y, hT = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store, idx, d["C"], d["z"],
                              d["Dskip"], chunk=16)
    h0 = P.gather(store.view(M, D * N), idx, out_dtype=torch.float32).view(B, D, N)
    y2, h2 = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0, chunk=16)
    idx3 = torch.tensor([[1, 2, 3], [4, 12, 5], [0, 0, 1]], dtype=torch.int32, device=DEV)
    sc = torch.tensor([[0.3, 0.2, 0.25], [0.1, 0.2, 0.3], [0.5, 0.5, 0.1]], dtype=torch.float64,
                      device=DEV)
    y3, h3 = P.scan_from_store(d["x"], d["dt"], d["A"], d["B"], store, idx3, d["C"], d["z"],
                               d["Dskip"], score=sc, tau=0.1, chunk=16)
    hc = P.compose(store.view(M, D * N), idx3, sc, tau=0.1, out_dtype=torch.float32).view(B, D, N)
    y4, h4 = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=hc, chunk=16)
    torch.cuda.synchronize()
    ok = torch.tensor([True, False, True])
    for a, b in ((y, y2), (hT, h2), (y3, y4), (h3, h4)):
        assert torch.equal(a[ok], b[ok])
        assert torch.isnan(a[~ok]).all() and torch.isnan(b[~ok]).all()
    y_ref, h_ref = _full_oracle({k: (v[[0, 2]] if v.dim() == 3 else v) for k, v in inp.items()},
                                store.cpu().double().numpy()[[5, 11]])
    assert err_rms(_np(y[[0, 2]]), y_ref) <= TOL_F32
    assert err_rms(_np(hT[[0, 2]]), h_ref) <= TOL_F32


# ---------------------------------------------------------------------------
# Workload-sized runs, sampled rows
# ---------------------------------------------------------------------------
def _device_inputs(wl, need_z_c=True):
    return synth.scan_inputs_device(wl.batch, wl.seqlen, wl.dim, wl.dstate, wl.seed,
                                    torch.bfloat16, wl.dt_mu, wl.dt_sigma, DEV,
                                    need_z_c=need_z_c)


def _check_rows(ref, y=None, hT=None, y_tol=TOL_BF16, bf16_y=False, f16_h=False):
    for (b, d), (yr, hr) in ref.items():
        if y is not None:
            if bf16_y:
                assert _bf16_ulp_ok(y[b, :, d], yr), (b, d)
            else:
                assert err_rms(_np(y[b, :, d]), yr) <= y_tol, (b, d)
        if hT is not None:
            if f16_h:
                assert _f16_ulp_ok(hT[b, d], hr), (b, d)
            else:
                assert err_rms(_np(hT[b, d]), hr) <= TOL_BF16, (b, d)


def test_corpus_encode_full_size_sampled():
    """B=64, L=3000, D=2048, N=16, bf16 in: fp32 y (parity run) and the timed
    form (bf16 y, fp16 hT)."""
    wl = synth.CORPUS_ENCODE
    inp = _device_inputs(wl)
    rows = sample_rows(wl.batch, wl.dim, 40, seed=2)
    ref = oracle_rows(oracle, inp, rows)
    y, hT = P.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"], inp["Dskip"])
    torch.cuda.synchronize()
    _check_rows(ref, y, hT)
    worst = max(err_rms(_np(y[b, :, d]), r[0]) for (b, d), r in ref.items())
    print("corpus encode fp32-y err_rms worst %.3e" % worst)
    del y, hT
    y16, h16 = P.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], out_dtype=torch.bfloat16, state_dtype=torch.float16)
    torch.cuda.synchronize()
    _check_rows(ref, y16, h16, bf16_y=True, f16_h=True)


def test_long_context_chunked_sampled():
    """B=8, L=65536, D=2048, N=16, chunk 256: the inter-chunk carry."""
    wl = synth.LONG_CONTEXT
    inp = _device_inputs(wl)
    rows = sample_rows(wl.batch, wl.dim, 12, seed=4)
    ref = oracle_rows(oracle, inp, rows)
    y, hT = P.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"], inp["Dskip"],
                   chunk=wl.chunk, state_dtype=torch.float32)
    torch.cuda.synchronize()
    _check_rows(ref, y, hT)
    del y, hT
    y16, h16 = P.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                      inp["Dskip"], chunk=wl.chunk, out_dtype=torch.bfloat16,
                      state_dtype=torch.float16)
    torch.cuda.synchronize()
    _check_rows(ref, y16, h16, bf16_y=True, f16_h=True)


def test_chunk_capped_by_32bit_offsets_sampled():
    """One 70,000-token sequence over 8192 channels with a single chunk
    requested: chunk x D x 4 bytes would pass 2^31, so the library splits the
    sequence where its 32-bit buffer offsets still reach (two chunks and a
    carry here); sampled rows match the oracle."""
    B, L, D, N = 1, 70000, 8192, 16
    inp = synth.scan_inputs_device(B, L, D, N, 77, torch.bfloat16)
    rows = sample_rows(B, D, 6, seed=7)
    ref = oracle_rows(oracle, inp, rows)
    y, hT = P.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"], inp["Dskip"],
                   chunk=L, out_dtype=torch.bfloat16, state_dtype=torch.float32)
    torch.cuda.synchronize()
    _check_rows(ref, y, hT, bf16_y=True)


def test_large_corpus_24_layers_into_store():
    """B=1024, L=3000, D=1536, N=64, state-only: all 24 layers, each with its
    own seeded inputs, writing its final states into its slot of one
    [1024, 24, D, N] fp16 store (batch stride 24 D N).  The store starts as
    NaN and is checked after the last launch, on 6 sampled (chunk, channel)
    rows per layer, so every slot is written and no launch touches another
    layer's slot."""
    wl = synth.LARGE_CORPUS
    layers = synth.LARGE_CORPUS_LAYERS
    D, N = wl.dim, wl.dstate
    store = torch.full((wl.batch, layers, D, N), float("nan"), dtype=torch.float16, device=DEV)
    refs = []
    for layer in range(layers):
        inp = synth.scan_inputs_device(wl.batch, wl.seqlen, D, N, wl.seed + layer,
                                       torch.bfloat16, wl.dt_mu, wl.dt_sigma, DEV,
                                       need_z_c=False)
        P.scan(inp["x"], inp["dt"], inp["A"], inp["B"], None, None, None, want_y=False,
               state_dtype=torch.float16, hT=store[:, layer],
               hT_batch_stride=layers * D * N)
        rows = sample_rows(wl.batch, D, 6, seed=layer)
        for (b, d), (_, hr) in oracle_rows(oracle, inp, rows, want_y=False).items():
            refs.append((layer, b, d, hr))
        del inp
    torch.cuda.synchronize()
    for layer, b, d, hr in refs:
        assert _f16_ulp_ok(store[b, layer, d], hr), (layer, b, d)
    assert not torch.isnan(store).any()
