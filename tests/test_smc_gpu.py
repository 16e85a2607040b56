"""Parity of the SMC steps with the oracle: two-stage routing (bit-exact
routes), semantic consolidation (within its rounding bound; exact where the
arithmetic is exact), and the O(1) session start: route the opening chunk,
inject its sub-cluster's semantic state, prefill the query tokens."""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_02560_amd import precog as P
from paper_2608_02560_amd import synth
from precog_testutil import TOL_BF16, err_rms

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _route(emb, dom, sub):
    m, j, f = P.route(emb.to(DEV), dom.to(DEV), sub.to(DEV))
    torch.cuda.synchronize()
    return m.cpu().numpy(), j.cpu().numpy(), f.cpu().numpy()


def test_route_workload_bit_exact():
    cfg = synth.SMC
    emb, dom, sub, pm, pj = synth.smc_inputs_host(cfg["C"], cfg["E"], cfg["ndom"], cfg["nsub"],
                                                  cfg["seed"])
    m, j, f = _route(emb, dom, sub)
    rm, rj = oracle.route2(emb, dom, sub)
    assert np.array_equal(m, rm) and np.array_equal(j, rj)
    assert np.array_equal(m, pm.numpy()) and np.array_equal(j, pj.numpy())
    assert np.array_equal(f, m * cfg["nsub"] + j)


@pytest.mark.parametrize("C,E,nd,ns", [(1, 4, 1, 1), (7, 20, 64, 3), (33, 388, 5, 64),
                                       (300, 384, 8, 8), (3, 4096, 9, 5), (5, 4, 64, 64)])
def test_route_random_shapes(C, E, nd, ns):
    g = np.random.default_rng(C + E)
    emb = torch.from_numpy(synth.unit_rows_host(C, E, g))
    dom = torch.from_numpy(synth.unit_rows_host(nd, E, g))
    sub = torch.from_numpy(synth.unit_rows_host(nd * ns, E, g).reshape(nd, ns, E))
    m, j, _ = _route(emb, dom, sub)
    rm, rj = oracle.route2(emb, dom, sub)
    assert np.array_equal(m, rm) and np.array_equal(j, rj)


def test_route_ties_go_to_lower_index():
    """Both stages tie exactly: domains 1 and 3 are the same row, and so are
    sub-clusters (1, 0) and (1, 2), all equal to the embedding itself."""
    g = np.random.default_rng(5)
    E = 64
    dom = synth.unit_rows_host(4, E, g)
    dom[3] = dom[1]
    sub = synth.unit_rows_host(16, E, g).reshape(4, 4, E)
    sub[1, 0] = dom[1]
    sub[1, 2] = dom[1]
    emb = np.stack([dom[1], dom[1] + 0.01 * sub[2, 1]]).astype(np.float32)
    m, j, _ = _route(*(torch.from_numpy(np.ascontiguousarray(a)) for a in (emb, dom, sub)))
    rm, rj = oracle.route2(emb, dom, sub)
    assert np.array_equal(m, rm) and np.array_equal(j, rj)
    assert m[0] == 1 and j[0] == 0


def test_route_equal_real_scores_decided_by_summation_order():
    """Prototypes that differ from the winning one only by two swapped
    components where the embedding holds equal values: equal real inner
    products, so only the sequential fp64 sums of the definition can order
    them (both stages, staged-row path)."""
    g = np.random.default_rng(67)
    C, E, nd, ns = 40, 384, 5, 4
    emb = synth.unit_rows_host(C, E, g)
    pairs = [tuple(int(v) for v in g.choice(E, 2, replace=False)) for _ in range(C)]
    for i, (a, b) in enumerate(pairs):
        emb[i, b] = emb[i, a]
    outs = []
    for i in range(C):
        # one embedding per call: its own prototype set with twinned winners
        dom = synth.unit_rows_host(nd, E, g)
        sub = synth.unit_rows_host(nd * ns, E, g).reshape(nd, ns, E)
        rm, _ = oracle.route2(emb[i:i + 1], dom, sub)
        w = int(rm[0])
        a, b = pairs[i]
        twin = dom[w].copy()
        twin[a], twin[b] = dom[w, b], dom[w, a]
        dom[(w + 1) % nd] = twin
        rm, rj = oracle.route2(emb[i:i + 1], dom, sub)
        sw = int(rj[0])
        st = sub[int(rm[0]), sw].copy()
        st[a], st[b] = sub[int(rm[0]), sw, b], sub[int(rm[0]), sw, a]
        sub[int(rm[0]), (sw + 1) % ns] = st
        rm, rj = oracle.route2(emb[i:i + 1], dom, sub)
        m, j, _ = _route(*(torch.from_numpy(np.ascontiguousarray(x)) for x in (emb[i:i + 1], dom, sub)))
        outs.append((m[0] == rm[0]) and (j[0] == rj[0]))
    assert all(outs)


def test_route_near_ties_one_ulp_apart():
    """Domain and sub-cluster prototypes that differ from the winning one in
    a single component by one fp32 ulp, up or down: real scores a hair apart,
    above the lane-parallel sums' error bound (decided by them) or, where the
    embedding's component is 1e-30, far below it (decided by the sequential
    fp64 sums), either way exactly as the definition orders them."""
    g = np.random.default_rng(68)
    C, E, nd, ns = 48, 384, 6, 4
    emb = synth.unit_rows_host(C, E, g)
    for i in range(C):
        dom = synth.unit_rows_host(nd, E, g)
        sub = synth.unit_rows_host(nd * ns, E, g).reshape(nd, ns, E)
        rm, _ = oracle.route2(emb[i:i + 1], dom, sub)
        w = int(rm[0])
        c = int(g.integers(0, E))
        up = bool(i % 2)
        if i % 4 >= 2:
            # the embedding's component there is tiny: the real scores differ
            # far below the error bound, so the sequential sums decide (equal
            # sums go to the lower index)
            emb[i, c] = np.float32(1e-30)
            rm, _ = oracle.route2(emb[i:i + 1], dom, sub)
            w = int(rm[0])
        twin = dom[w].copy()
        twin[c] = np.nextafter(twin[c], np.float32(np.inf) if up else np.float32(-np.inf))
        dom[(w + 1 + i % (nd - 1)) % nd] = twin
        rm, rj = oracle.route2(emb[i:i + 1], dom, sub)
        wm, sw = int(rm[0]), int(rj[0])
        st = sub[wm, sw].copy()
        st[c] = np.nextafter(st[c], np.float32(-np.inf) if up else np.float32(np.inf))
        sub[wm, (sw + 1) % ns] = st
        rm, rj = oracle.route2(emb[i:i + 1], dom, sub)
        m, j, _ = _route(*(torch.from_numpy(np.ascontiguousarray(x)) for x in (emb[i:i + 1], dom, sub)))
        assert m[0] == rm[0] and j[0] == rj[0], (i, m[0], rm[0], j[0], rj[0])


def _cons_bound(states0, contrib, target, alpha, mag_unit):
    """Per-row bound: each fp32 update adds at most 3 units of 2^-24 of the
    magnitudes involved (two roundings of the factors, one of the fused
    multiply-add) and contracts older error by (1 - alpha); fp16 storage
    adds half an fp16 ulp per update."""
    R = states0.shape[0]
    bound = np.zeros(R)
    mx = np.maximum(np.abs(states0).max(axis=1), np.abs(contrib).max())
    for r in range(R):
        n = int(np.sum(target == r))
        bound[r] = n * mag_unit * 2 * mx[r]
    return bound


@pytest.mark.parametrize("sd,hd,alpha", [(torch.float32, torch.float32, 0.25),
                                         (torch.float32, torch.float16, 0.1),
                                         (torch.float16, torch.float16, 0.5),
                                         (torch.float16, torch.float32, 1.0)])
def test_consolidate_matches_oracle(sd, hd, alpha):
    g = np.random.default_rng(12)
    R, S, C = 20, 24 * 4096, 64
    states0 = torch.from_numpy(g.normal(size=(R, S))).to(sd)
    contrib = torch.from_numpy(g.normal(size=(C, S))).to(hd)
    target = torch.from_numpy(g.integers(-1, R + 1, C).astype(np.int32))
    st = states0.to(DEV)
    P.smc_consolidate(st, contrib.to(DEV), target.to(DEV), alpha)
    torch.cuda.synchronize()
    ref = oracle.consolidate(states0, contrib, target.numpy(), alpha)
    got = st.double().cpu().numpy()
    unit = 3 * 2.0 ** -24 + (2.0 ** -11 if sd == torch.float16 else 0.0)
    bound = _cons_bound(states0.double().numpy(), contrib.double().numpy(), target.numpy(),
                        alpha, unit)
    for r in range(R):
        if not np.any(target.numpy() == r):
            assert np.array_equal(got[r], states0[r].double().numpy())  # untouched
        else:
            assert np.abs(got[r] - ref[r]).max() <= bound[r], r
    if alpha == 1.0:
        # alpha = 1 replaces the state with the last contribution routed to it
        for r in range(R):
            hits = np.nonzero(target.numpy() == r)[0]
            if hits.size:
                assert np.array_equal(got[r], contrib[hits[-1]].to(sd).double().numpy())


def test_smc_session_start_end_to_end():
    """Route 64 deposited chunks, consolidate their final states into the
    20 semantic states, then start a session: route the opening utterance,
    inject s_{m*, j*} and prefill 32 query tokens (D=1024, N=16 per state
    row here), all on the stream without host synchronisation."""
    cfg = synth.SMC
    D, N = 1024, 16
    emb, dom, sub, _, _ = synth.smc_inputs_host(cfg["C"] + 1, cfg["E"], cfg["ndom"], cfg["nsub"],
                                                cfg["seed"])
    R = cfg["ndom"] * cfg["nsub"]
    g = np.random.default_rng(13)
    states0 = torch.from_numpy(g.normal(0, 0.3, size=(R, D * N))).float()
    contrib = torch.from_numpy(g.normal(0, 0.3, size=(cfg["C"], D * N))).float()
    wl = synth.scan_inputs_host(1, 32, D, N, seed=14, in_dtype=torch.bfloat16)
    d = {k: v.to(DEV) for k, v in wl.items()}
    st = states0.to(DEV)
    _, _, flat = P.route(emb[:-1].to(DEV), dom.to(DEV), sub.to(DEV))
    P.smc_consolidate(st, contrib.to(DEV), flat, 0.2)
    _, _, f0 = P.route(emb[-1:].to(DEV), dom.to(DEV), sub.to(DEV))
    h0 = P.gather(st, f0, out_dtype=torch.float32).view(1, D, N)
    y, hT = P.scan(d["x"], d["dt"], d["A"], d["B"], d["C"], d["z"], d["Dskip"], h0=h0)
    torch.cuda.synchronize()
    rm, rj = oracle.route2(emb, dom, sub)
    rflat = rm * cfg["nsub"] + rj
    sem = oracle.consolidate(states0, contrib, rflat[:-1], 0.2)
    h0_ref = sem[rflat[-1]].reshape(1, D, N)
    assert err_rms(h0.double().cpu().numpy(), h0_ref) <= 1e-5
    y_ref, h_ref = oracle.scan(wl["x"], wl["dt"], wl["A"], wl["B"], wl["C"], wl["z"], wl["Dskip"],
                               h0_ref, nthreads=8)
    assert err_rms(y.double().cpu().numpy(), y_ref) <= TOL_BF16
    assert err_rms(hT.double().cpu().numpy(), h_ref) <= TOL_BF16
