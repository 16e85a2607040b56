"""Pins for the fp64 oracle: each test checks it against something other than
itself -- a closed form, a special case that reduces to a library routine,
an invariant the paper proves, or a brute-force evaluation in mpmath."""
import math

import mpmath
import numpy as np
import pytest
import scipy.linalg
import scipy.special
import torch

import oracle
from paper_2608_02560_amd import synth
from precog_testutil import err_rms


def _rand(B, L, D, N, seed, h0_std=0.0, **kw):
    d = synth.scan_inputs_host(B, L, D, N, seed, torch.float32, h0_std=h0_std, **kw)
    return {k: v.double().numpy() for k, v in d.items()}


# --------------------------------------------------------------------------
# Brute-force unrolling (App. B.1, Eq. unroll), at 50 digits
# --------------------------------------------------------------------------
def _mp_unroll_states(inp, b, d):
    """h_t for t = 1..L from the closed form
    h_t = (prod_{s<=t} a_s) h0 + sum_{r<=t} beta_r prod_{s=r+1..t} a_s,
    with a_s = exp(-dt_s A) and beta_r = B_r x_r dt_r."""
    mpmath.mp.dps = 50
    L = inp["x"].shape[1]
    N = inp["A"].shape[1]
    states = []
    for t in range(L):
        h = []
        for n in range(N):
            A = mpmath.mpf(inp["A"][d, n])
            dts = [mpmath.mpf(inp["dt"][b, s, d]) for s in range(t + 1)]
            total = mpmath.exp(-A * mpmath.fsum(dts)) * mpmath.mpf(inp["h0"][b, d, n])
            for r in range(t + 1):
                beta = (mpmath.mpf(inp["B"][b, r, n]) * mpmath.mpf(inp["x"][b, r, d])
                        * dts[r])
                total += beta * mpmath.exp(-A * mpmath.fsum(dts[r + 1:]))
            h.append(total)
        states.append(h)
    return states


@pytest.mark.parametrize("L,D,N", [(1, 1, 1), (5, 3, 2), (12, 2, 4), (16, 3, 3)])
def test_unroll_bruteforce(L, D, N):
    inp = _rand(2, L, D, N, seed=100 + L, h0_std=1.0)
    y, hT = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"],
                        inp["z"], inp["Dskip"], inp["h0"])
    for b in range(2):
        for d in range(D):
            hs = _mp_unroll_states(inp, b, d)
            for n in range(N):
                ref = float(hs[-1][n])
                assert abs(hT[b, d, n] - ref) <= 1e-13 * max(1.0, abs(ref))
            for t in range(L):
                acc = mpmath.fsum(mpmath.mpf(inp["C"][b, t, n]) * hs[t][n]
                                  for n in range(N))
                zz = mpmath.mpf(inp["z"][b, t, d])
                gate = zz / (1 + mpmath.exp(-zz))
                ref = float((acc + mpmath.mpf(inp["Dskip"][d]) * inp["x"][b, t, d]) * gate)
                assert abs(y[b, t, d] - ref) <= 1e-13 * max(1.0, abs(ref))


def test_hand_worked_two_steps():
    """Two tokens, one channel, one state, worked out by hand from Eq. 1:
    h1 = e^{-dt1 A} h0 + B1 x1 dt1, h2 = e^{-dt2 A} h1 + B2 x2 dt2,
    y_t = (C_t h_t + D x_t) * z_t / (1 + e^{-z_t})."""
    A, h0, D = 0.5, 2.0, 0.25
    dt, x, Bv, Cv, z = [1.0, 2.0], [3.0, -1.0], [0.5, 4.0], [2.0, -1.0], [1.0, -2.0]
    h1 = math.exp(-0.5) * 2.0 + 0.5 * 3.0 * 1.0
    h2 = math.exp(-1.0) * h1 + 4.0 * -1.0 * 2.0
    y1 = (2.0 * h1 + 0.25 * 3.0) * (1.0 / (1.0 + math.exp(-1.0)))
    y2 = (-1.0 * h2 + 0.25 * -1.0) * (-2.0 / (1.0 + math.exp(2.0)))
    a = lambda v: np.array(v, np.float64).reshape(1, 2, 1)
    y, hT = oracle.scan(a(x), a(dt), np.array([[A]]), a(Bv), a(Cv), a(z),
                        np.array([D]), np.array([[[h0]]]))
    assert hT[0, 0, 0] == pytest.approx(h2, rel=1e-15, abs=1e-15)
    assert y[0, :, 0] == pytest.approx([y1, y2], rel=1e-15, abs=1e-15)


# --------------------------------------------------------------------------
# Closed forms and special cases (Eq. 1)
# --------------------------------------------------------------------------
def test_geometric_closed_form():
    """Constant dt, B, x: h_t = a^t h0 + beta (1 - a^t) / (1 - a) with
    a = exp(-dt A), beta = dt B x (the geometric series of Eq. unroll).
    The readout y_t must use h_t, the state after token t."""
    L, D, N = 1000, 3, 4
    g = np.random.default_rng(7)
    A = g.uniform(1, 16, (D, N))
    dtv = np.array([0.03, 0.1, 0.4])
    xv = np.array([1.5, -0.7, 0.2])
    Bv = g.normal(0, 0.25, N)
    Cv = g.normal(0, 0.25, N)
    h0 = g.normal(0, 1, (1, D, N))
    x = np.broadcast_to(xv, (1, L, D)).copy()
    dt = np.broadcast_to(dtv, (1, L, D)).copy()
    B = np.broadcast_to(Bv, (1, L, N)).copy()
    C = np.broadcast_to(Cv, (1, L, N)).copy()
    y, hT = oracle.scan(x, dt, A, B, C, None, None, h0)
    t = np.arange(1, L + 1)[:, None, None]
    a = np.exp(-dtv[:, None] * A)[None]
    beta = (dtv * xv)[:, None] * Bv[None, :]
    h_t = a ** t * h0 + beta[None] * (1 - a ** t) / (1 - a)
    assert err_rms(hT[0], h_t[-1]) < 1e-13
    assert err_rms(y[0], np.einsum("tdn,n->td", h_t, Cv)) < 1e-12


def test_zero_decay_is_cumsum():
    """A = 0: no decay, so h_t = h0 + cumsum_t(dt B x) (numpy.cumsum)."""
    inp = _rand(2, 40, 5, 3, seed=11, h0_std=1.0)
    A0 = np.zeros_like(inp["A"])
    y, hT = oracle.scan(inp["x"], inp["dt"], A0, inp["B"], inp["C"], None, None,
                        inp["h0"])
    beta = inp["dt"][..., None] * inp["x"][..., None] * inp["B"][:, :, None, :]
    h_t = inp["h0"][:, None] + np.cumsum(beta, axis=1)
    assert err_rms(hT, h_t[:, -1]) < 1e-13
    assert err_rms(y, np.einsum("btdn,btn->btd", h_t, inp["C"])) < 1e-12


def test_zero_input_is_pure_decay():
    """x = 0: h_T = h0 * exp(-A * sum_t dt)."""
    inp = _rand(2, 64, 4, 5, seed=12, h0_std=1.0)
    y, hT = oracle.scan(np.zeros_like(inp["x"]), inp["dt"], inp["A"], inp["B"],
                        inp["C"], inp["z"], inp["Dskip"], inp["h0"])
    S = inp["dt"].sum(axis=1)  # [B, D]
    assert err_rms(hT, inp["h0"] * np.exp(-S[:, :, None] * inp["A"][None])) < 1e-12
    # with x = 0 the skip term vanishes too: y = (C . h) silu(z)
    assert np.all(np.isfinite(y))


def test_zero_input_projection_gives_gated_skip():
    """B = 0 and h0 = 0: the state stays zero, y = Dskip x silu(z) where
    silu(z) = z * expit(z) (scipy.special.expit)."""
    inp = _rand(2, 30, 6, 4, seed=13)
    zero = np.zeros_like(inp["B"])
    y, hT = oracle.scan(inp["x"], inp["dt"], inp["A"], zero, inp["C"], inp["z"],
                        inp["Dskip"], None)
    ref = inp["Dskip"] * inp["x"] * inp["z"] * scipy.special.expit(inp["z"])
    assert np.all(hT == 0)
    assert err_rms(y, ref) < 1e-14
    y2, _ = oracle.scan(inp["x"], inp["dt"], inp["A"], zero, inp["C"], None,
                        inp["Dskip"], None)
    assert err_rms(y2, inp["Dskip"] * inp["x"]) == 0.0
    y3, _ = oracle.scan(inp["x"], inp["dt"], inp["A"], zero, inp["C"], None, None, None)
    assert np.all(y3 == 0)


def test_superposition():
    """The update is affine in (h0, x): S(h0, x) = S(h0, 0) + S(0, x)."""
    inp = _rand(2, 50, 4, 4, seed=14, h0_std=1.0)
    args = (inp["dt"], inp["A"], inp["B"], inp["C"])
    _, h_full = oracle.scan(inp["x"], *args, None, None, inp["h0"])
    _, h_free = oracle.scan(np.zeros_like(inp["x"]), *args, None, None, inp["h0"])
    _, h_forced = oracle.scan(inp["x"], *args, None, None, None)
    assert err_rms(h_full, h_free + h_forced) < 1e-13


# --------------------------------------------------------------------------
# Theorem 1 and Proposition 1 (Sec. 4.3, App. A)
# --------------------------------------------------------------------------
def test_split_invariance_bitwise():
    """S(h0, c ++ q) = S(S(h0, c), q): in fp64 the sequential oracle performs
    exactly the same operations, so state and outputs are bit-identical."""
    inp = _rand(1, 512, 16, 16, seed=1)
    keys = ("x", "dt", "B", "C", "z")
    full_y, full_h = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"],
                                 inp["z"], inp["Dskip"], None)
    for split in (1, 100, 384, 511):
        c = {k: inp[k][:, :split] for k in keys}
        q = {k: inp[k][:, split:] for k in keys}
        yc, hc = oracle.scan(c["x"], c["dt"], inp["A"], c["B"], c["C"], c["z"],
                             inp["Dskip"], None)
        yq, hq = oracle.scan(q["x"], q["dt"], inp["A"], q["B"], q["C"], q["z"],
                             inp["Dskip"], hc)
        assert np.array_equal(hq, full_h)
        assert np.array_equal(np.concatenate([yc, yq], axis=1), full_y)


def test_sufficient_statistic():
    """Prop. 1: the continuation depends on the context only through its final
    state.  Build a different context with the same final state (move x along
    the null space of the linear map x_ctx -> h_ctx, from Eq. unroll) and run
    the whole concatenated sequence: outputs on the query part are unchanged
    while outputs on the context part differ."""
    Lc, Lq, D, N = 40, 20, 3, 4
    inp = _rand(1, Lc + Lq, D, N, seed=15)
    x2 = inp["x"].copy()
    for d in range(D):
        dt = inp["dt"][0, :Lc, d]
        S_after = np.cumsum(dt[::-1])[::-1] - dt  # sum_{s>t} dt_s
        Mmap = (np.exp(-np.outer(inp["A"][d], S_after)) * dt[None, :]
                * inp["B"][0, :Lc, :].T)  # [N, Lc]
        null = scipy.linalg.null_space(Mmap)
        x2[0, :Lc, d] += 3.0 * null[:, 0]
    y1, h1 = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                         inp["Dskip"], None)
    y2, h2 = oracle.scan(x2, inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                         inp["Dskip"], None)
    assert np.max(np.abs(y1[:, :Lc] - y2[:, :Lc])) > 1e-3
    assert err_rms(y2[:, Lc:], y1[:, Lc:]) < 1e-12
    assert err_rms(h2, h1) < 1e-12


def test_memory_horizon():
    """App. B.2: tokens older than L_mem (eps = 1e-3) move the final state by
    at most eps times the size of their own contribution."""
    L, D, N = 200, 2, 3
    inp = _rand(1, L, D, N, seed=16)
    eps = 1e-3
    _, h1 = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"])
    for d in range(D):
        # the slowest state decides the horizon of the channel
        amin = inp["A"][d].min()
        logprod = np.cumsum(-inp["dt"][0, ::-1, d] * amin)  # tau = 1..L
        Lmem = int(np.argmax(logprod < np.log(eps))) + 1
        assert 1 <= Lmem < L
        x2 = inp["x"].copy()
        x2[0, : L - Lmem, d] += 10.0
        _, h2 = oracle.scan(x2, inp["dt"], inp["A"], inp["B"], inp["C"])
        bound = eps * np.sum(10.0 * inp["dt"][0, : L - Lmem, d][:, None]
                             * np.abs(inp["B"][0, : L - Lmem, :]), axis=0)
        assert np.all(np.abs(h2[0, d] - h1[0, d]) <= bound + 1e-15)


# --------------------------------------------------------------------------
# Storage rounding (Sec. 4.2 FP16 store; Sec. 4.3 error bound)
# --------------------------------------------------------------------------
def test_round_f16_matches_numpy():
    g = np.random.default_rng(3)
    v = np.concatenate([g.normal(0, 1, 20000), g.normal(0, 1e-6, 2000),
                        np.array([0.0, -0.0, 65504.0, 65519.9, 2.0 ** -24, 2.0 ** -25,
                                  1 + 2.0 ** -11, 1 + 3 * 2.0 ** -11])])
    assert np.array_equal(oracle.round_f16(v), v.astype(np.float16).astype(np.float64))


def test_round_bf16_matches_torch_rne():
    g = np.random.default_rng(4)
    v32 = np.concatenate([g.normal(0, 1, 20000), g.normal(0, 1e-38, 200),
                          np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -1 - 2.0 ** -8])]
                         ).astype(np.float32)
    ref = torch.from_numpy(v32).to(torch.bfloat16).double().numpy()
    assert np.array_equal(oracle.round_bf16(v32.astype(np.float64)), ref)


def test_fp16_state_within_paper_bound():
    """Storing the state at FP16 costs at most 2^-11 relative (round to
    nearest even), inside the ~2^-10 per-element bound of Sec. 4.3."""
    inp = _rand(2, 300, 8, 16, seed=17)
    _, hT = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"])
    normal = np.abs(hT) >= 2.0 ** -14
    q = oracle.round_f16(hT)
    assert np.all(np.abs(q - hT)[normal] <= 2.0 ** -11 * np.abs(hT)[normal])
    assert np.all(np.abs(q - hT)[~normal] <= 2.0 ** -25)


# --------------------------------------------------------------------------
# Retrieval and injection (Sec. 4.2)
# --------------------------------------------------------------------------
def test_top1_matches_numpy_argmax():
    q, K, _, _ = synth.retrieval_inputs_host(64, 3000, 384, 0, seed=21)
    idx, best = oracle.top1(q, K, nthreads=4)
    s = q.double().numpy() @ K.double().numpy().T
    assert np.array_equal(idx, np.argmax(s, axis=1))
    assert np.allclose(best, s.max(axis=1), rtol=0, atol=1e-14)


def test_top1_planted():
    q, K, pos, rows = synth.retrieval_inputs_host(64, 2000, 384, 32, seed=22)
    idx, _ = oracle.top1(q, K)
    assert np.array_equal(idx[pos.numpy()], rows.numpy().astype(np.int32))


def test_top1_duplicates_take_lowest_index():
    q, K, _, _ = synth.retrieval_inputs_host(16, 500, 64, 0, seed=23)
    idx0, _ = oracle.top1(q, K)
    K2 = torch.cat([K, K[idx0[:8].astype(np.int64)]])  # duplicate winners at the end
    K3 = torch.cat([K[idx0[:8].astype(np.int64)], K])  # ... and at the start
    idx2, _ = oracle.top1(q, K2)
    idx3, _ = oracle.top1(q, K3)
    assert np.array_equal(idx2, idx0)
    assert np.array_equal(idx3[:8], np.arange(8))


def test_top1_empty_and_threads():
    q, K, _, _ = synth.retrieval_inputs_host(33, 77, 10, 0, seed=24)
    a, _ = oracle.top1(q, K, nthreads=1)
    b, _ = oracle.top1(q, K, nthreads=7)
    assert np.array_equal(a, b)
    idx, _ = oracle.top1(q[:0], K)
    assert idx.shape == (0,)


def test_gather_is_exact_copy():
    store = synth.state_store(50, 64, seed=5)
    idx = np.array([3, 3, 49, 0])
    out = oracle.gather(store, idx)
    assert np.array_equal(out, store.double().numpy()[[3, 3, 49, 0]])


def test_threads_bitwise_equal():
    inp = _rand(3, 70, 9, 4, seed=18, h0_std=1.0)
    args = [inp[k] for k in ("x", "dt", "A", "B", "C", "z", "Dskip", "h0")]
    y1, h1 = oracle.scan(*args, nthreads=1)
    y2, h2 = oracle.scan(*args, nthreads=5)
    assert np.array_equal(y1, y2) and np.array_equal(h1, h2)


# --------------------------------------------------------------------------
# SMC pieces (Sec. 5)
# --------------------------------------------------------------------------
def test_trajectory_dial_extremes():
    """K = N_c keeps every state (each equals the final state of the prefix);
    K = 1 keeps only the final state, identical to the PRECOG state (Sec. 5.2)."""
    inp = _rand(2, 24, 3, 4, seed=19, h0_std=0.5)
    full = oracle.trajectory(inp["x"], inp["dt"], inp["A"], inp["B"], 1, inp["h0"])
    for t in (1, 7, 24):
        _, h = oracle.scan(inp["x"][:, :t], inp["dt"][:, :t], inp["A"],
                           inp["B"][:, :t], inp["C"][:, :t], None, None, inp["h0"])
        assert np.array_equal(full[:, t - 1], h)
    last = oracle.trajectory(inp["x"], inp["dt"], inp["A"], inp["B"], 24, inp["h0"])
    assert last.shape[1] == 1 and np.array_equal(last[:, 0], full[:, -1])
    every5 = oracle.trajectory(inp["x"], inp["dt"], inp["A"], inp["B"], 5, inp["h0"])
    assert every5.shape[1] == 4 and np.array_equal(every5, full[:, 4::5][:, :4])


def test_topk_compose_limits():
    store = synth.state_store(40, 32, seed=6)
    q, K, _, _ = synth.retrieval_inputs_host(5, 40, 16, 0, seed=25)
    idx, sc = oracle.topk_scores(q, K, 3)
    idx1, _ = oracle.top1(q, K)
    assert np.array_equal(idx[:, 0], idx1)
    # very sharp softmax -> the top-1 state
    sharp = oracle.topk_compose(store, idx, sc, tau=1e-9)
    assert np.allclose(sharp, oracle.gather(store, idx1), atol=1e-12)
    # equal scores -> plain mean of the k states
    flat = oracle.topk_compose(store, idx, np.zeros_like(sc), tau=1.0)
    ref = np.mean([store.double().numpy()[idx[:, j]] for j in range(3)], axis=0)
    assert np.allclose(flat, ref, atol=1e-14)
    # k = 1 is the injection of the top-1 state itself
    one = oracle.topk_compose(store, idx[:, :1], sc[:, :1], tau=0.1)
    assert np.array_equal(one, oracle.gather(store, idx1))


def test_topk_scores_match_sorted_numpy_scores():
    """Ranks against an independent evaluation: numpy's fp64 matrix product
    (a different summation order, so only gaps far above fp64 rounding are
    compared) sorted by (score descending, row ascending)."""
    q, K, _, _ = synth.retrieval_inputs_host(12, 700, 48, 4, seed=26)
    idx, sc = oracle.topk_scores(q, K, 7)
    s = q.double().numpy() @ K.double().numpy().T
    for i in range(12):
        order = np.lexsort((np.arange(700), -s[i]))[:7]
        assert np.array_equal(idx[i], order)
        assert np.allclose(sc[i], s[i, order], rtol=0, atol=1e-14)
    # duplicated rows tie exactly and keep row order
    K2 = torch.cat([K[:5], K[:5]])
    idx2, sc2 = oracle.topk_scores(q[:3], K2, 10)
    for i in range(3):
        assert np.array_equal(sc2[i][0::2], sc2[i][1::2])
        assert np.all(idx2[i][0::2] < idx2[i][1::2])


def test_topk_compose_softmax_by_hand():
    """Two states, scores 0 and log(3) at tau = 1: weights 1/4 and 3/4."""
    store = torch.tensor([[1.0, 2.0, 0.0, 8.0], [5.0, -2.0, 4.0, 0.0]])
    out = oracle.topk_compose(store, np.array([[0, 1]]), np.array([[0.0, np.log(3.0)]]), 1.0)
    assert np.allclose(out, [[4.0, -1.0, 3.0, 2.0]], rtol=0, atol=1e-15)
    # temperature halves the logits: log(3)/2 -> weights 1/(1+sqrt3), sqrt3/(1+sqrt3)
    out2 = oracle.topk_compose(store, np.array([[0, 1]]), np.array([[0.0, np.log(3.0)]]), 2.0)
    w1 = np.sqrt(3.0) / (1.0 + np.sqrt(3.0))
    assert np.allclose(out2[0], (1 - w1) * store[0].numpy() + w1 * store[1].numpy(), atol=1e-15)


def test_fuse_by_hand():
    """Episodic candidates: rows 0, 1 with scores log 3 and -10; corpus
    candidates: rows 0, 1 with scores log 2 and 0.  The three best across
    both stores are (log 3, episodic 0), (log 2, corpus 0), (0, corpus 1):
    weights 3/6, 2/6, 1/6 at tau = 1.  With unit-vector states the fusion
    is [1/2, 1/3, 1/6, 0]; the semantic state [0, 0, 0, 2] at weight 1/2
    adds 1 in the last place."""
    ep = torch.tensor([[1.0, 0.0, 0.0, 0.0], [0.0, 0.0, 0.0, 5.0]])
    co = torch.tensor([[0.0, 1.0, 0.0, 0.0], [0.0, 0.0, 1.0, 0.0]])
    ei, es = np.array([[0, 1]]), np.array([[np.log(3.0), -10.0]])
    ci, cs = np.array([[0, 1]]), np.array([[np.log(2.0), 0.0]])
    h = oracle.fuse(ep, ei, es, co, ci, cs, 3, 1.0)
    assert np.allclose(h, [[0.5, 1 / 3, 1 / 6, 0.0]], rtol=0, atol=1e-15)
    sem = torch.tensor([[9.0, 9.0, 9.0, 9.0], [0.0, 0.0, 0.0, 2.0]])
    h2 = oracle.fuse(ep, ei, es, co, ci, cs, 3, 1.0, sem, np.array([1]), 0.5)
    assert np.allclose(h2, [[0.5, 1 / 3, 1 / 6, 1.0]], rtol=0, atol=1e-15)
    # k = 1: the single best candidate, weight 1; equal scores across the
    # stores go to the episodic one
    one = oracle.fuse(ep, ei, es, co, ci, cs, 1, 1.0)
    assert np.array_equal(one, [[1.0, 0.0, 0.0, 0.0]])
    tie = oracle.fuse(ep, np.array([[1]]), np.array([[0.25]]), co, np.array([[0]]),
                      np.array([[0.25]]), 1, 1.0)
    assert np.array_equal(tie, [[0.0, 0.0, 0.0, 5.0]])


def test_fuse_equals_composition_over_the_joined_index():
    """Fusing the two stores' top-k lists is the top-k composition over one
    index holding the episodic keys then the corpus keys (its lower rows,
    the episodic ones, win equal scores), with the states stacked the same
    way; lam = 0 adds nothing and lam scales the semantic state linearly."""
    g = np.random.default_rng(31)
    Me, Mc, E, S, Q, k = 30, 50, 16, 24, 6, 4
    qe, Ke, _, _ = synth.retrieval_inputs_host(Q, Me, E, 0, seed=32)
    _, Kc, _, _ = synth.retrieval_inputs_host(1, Mc, E, 0, seed=33)
    Kc[7] = Ke[3]  # a corpus key equal to an episodic one: equal scores
    se = synth.state_store(Me, S, seed=34)
    sc_ = synth.state_store(Mc, S, seed=35)
    ie, ve = oracle.topk_scores(qe, Ke, k)
    ic, vc = oracle.topk_scores(qe, Kc, k)
    h = oracle.fuse(se, ie, ve, sc_, ic, vc, k, 0.7)
    ij, vj = oracle.topk_scores(qe, torch.cat([Ke, Kc]), k)
    ref = oracle.topk_compose(torch.cat([se, sc_]), ij, vj, 0.7)
    assert np.allclose(h, ref, rtol=0, atol=1e-13)
    sem = torch.from_numpy(g.normal(size=(5, S)))
    rows = g.integers(0, 5, Q)
    h0 = oracle.fuse(se, ie, ve, sc_, ic, vc, k, 0.7, sem, rows, 0.0)
    h3 = oracle.fuse(se, ie, ve, sc_, ic, vc, k, 0.7, sem, rows, 3.0)
    assert np.array_equal(h0, h)
    assert np.allclose(h3 - h, 3.0 * sem.numpy()[rows], rtol=0, atol=1e-12)
    # very sharp softmax: the single best candidate of either store
    sharp = oracle.fuse(se, ie, ve, sc_, ic, vc, k, 1e-9)
    best = oracle.gather(torch.cat([se, sc_]), ij[:, 0])
    assert np.allclose(sharp, best, rtol=0, atol=1e-12)


def test_route2_matches_numpy():
    g = np.random.default_rng(8)
    E = 24
    emb = synth.unit_rows_host(30, E, g)
    P = synth.unit_rows_host(5, E, g)
    S = synth.unit_rows_host(20, E, g).reshape(5, 4, E)
    m, j = oracle.route2(emb, P, S)
    e64 = emb.astype(np.float64)
    m_ref = np.argmax(e64 @ P.astype(np.float64).T, axis=1)
    assert np.array_equal(m, m_ref)
    j_ref = [np.argmax(S[mm].astype(np.float64) @ e64[c]) for c, mm in enumerate(m_ref)]
    assert np.array_equal(j, j_ref)


def test_ema_fixed_point_and_alpha_one():
    s = np.random.default_rng(9).normal(size=(4, 8))
    h = np.random.default_rng(10).normal(size=(4, 8))
    assert np.array_equal(oracle.ema(s, h, 1.0), h)
    assert np.array_equal(oracle.ema(h, h, 0.3), h * 0.7 + 0.3 * h)
    # repeated consolidation of the same contribution converges to it
    cur = s
    for _ in range(200):
        cur = oracle.ema(cur, h, 0.25)
    assert np.allclose(cur, h, atol=1e-20 + 1e-12)


def test_consolidate_closed_form_and_skips():
    """Repeated deposits into one sub-cluster follow the unrolled EMA,
    s_n = (1-a)^n s_0 + sum_k a (1-a)^(n-1-k) h_k; other rows and
    out-of-table targets change nothing."""
    g = np.random.default_rng(11)
    states = g.normal(size=(4, 6))
    contrib = g.normal(size=(5, 6))
    target = np.array([2, -1, 2, 4, 2])
    a = 0.3
    out = oracle.consolidate(states, contrib, target, a)
    hs = contrib[[0, 2, 4]]
    ref = (1 - a) ** 3 * states[2] + sum(a * (1 - a) ** (2 - k) * hs[k] for k in range(3))
    assert np.allclose(out[2], ref, rtol=0, atol=1e-14)
    for r in (0, 1, 3):
        assert np.array_equal(out[r], states[r])


def test_smc_planted_routes():
    """Chunks planted next to sub-cluster prototypes route to them (Eqs.
    smc-domain and smc-sub), a check that does not use the oracle's scores."""
    emb, dom, sub, pm, pj = synth.smc_inputs_host(64, 384, 5, 4, seed=7)
    m, j = oracle.route2(emb, dom, sub)
    assert np.array_equal(m, pm.numpy()) and np.array_equal(j, pj.numpy())


# --------------------------------------------------------------------------
# Complex diagonal A (Sec. 3: A_k has an imaginary part pi k)
# --------------------------------------------------------------------------
def test_complex_scan_with_zero_frequency_is_the_real_scan():
    inp = _rand(2, 40, 5, 4, seed=27, h0_std=0.7)
    h0c = np.stack([np.asarray(inp["h0"]), np.zeros_like(np.asarray(inp["h0"]))], axis=-1)
    y_c, h_c = oracle.scan_complex(inp["x"], inp["dt"], inp["A"], np.zeros_like(inp["A"]),
                                   inp["B"], inp["C"], inp["z"], inp["Dskip"], h0c)
    y_r, h_r = oracle.scan(inp["x"], inp["dt"], inp["A"], inp["B"], inp["C"], inp["z"],
                           inp["Dskip"], inp["h0"])
    assert np.array_equal(y_c, y_r)
    assert np.array_equal(h_c[..., 0], h_r) and not np.any(h_c[..., 1])


def test_complex_scan_geometric_closed_form():
    """Constant dt, B, x: h_L = alpha^L h0 + beta (1 - alpha^L) / (1 - alpha)
    with the complex alpha = exp(-dt (a + i w)), beta = dt B x; the readout
    takes the real part.  D != N so a transposed A or w fails."""
    L, D, N = 300, 3, 5
    g = np.random.default_rng(28)
    dt, xv = 0.07, 0.9
    a = g.uniform(1, 16, (D, N))
    w = np.pi * np.arange(N)[None, :] * np.ones((D, 1)) + g.uniform(-1, 1, (D, N))
    Bv = g.normal(0, 0.5, N)
    Cv = g.normal(0, 0.5, N)
    h0 = g.normal(size=(1, D, N)) + 1j * g.normal(size=(1, D, N))
    x = np.full((1, L, D), xv)
    dts = np.full((1, L, D), dt)
    Bm = np.tile(Bv, (1, L, 1))
    Cm = np.tile(Cv, (1, L, 1))
    y, hT = oracle.scan_complex(x, dts, a, w, Bm, Cm, None, None,
                                np.stack([h0.real, h0.imag], axis=-1))
    alpha = np.exp(-dt * (a + 1j * w))
    beta = dt * Bv[None, :] * xv
    ref = alpha ** L * h0[0] + beta * (1 - alpha ** L) / (1 - alpha)
    assert np.allclose(hT[0, ..., 0], ref.real, rtol=0, atol=1e-12)
    assert np.allclose(hT[0, ..., 1], ref.imag, rtol=0, atol=1e-12)
    assert np.allclose(y[0, -1], (ref.real * Cv[None, :]).sum(axis=1), rtol=0, atol=1e-12)


def test_complex_scan_pure_rotation():
    """No decay and no input: each state turns by -w * sum(dt), |h| is kept."""
    L, D, N = 50, 2, 3
    g = np.random.default_rng(29)
    dts = g.uniform(0.01, 0.3, (1, L, D))
    w = g.uniform(-5, 5, (D, N))
    h0 = g.normal(size=(1, D, N)) + 1j * g.normal(size=(1, D, N))
    _, hT = oracle.scan_complex(np.zeros((1, L, D)), dts, np.zeros((D, N)), w,
                                np.zeros((1, L, N)), None, None, None,
                                np.stack([h0.real, h0.imag], axis=-1), want_y=False)
    ref = h0[0] * np.exp(-1j * w * dts[0].sum(axis=0)[:, None])
    assert np.allclose(hT[0, ..., 0] + 1j * hT[0, ..., 1], ref, rtol=0, atol=1e-12)
