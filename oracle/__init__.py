"""PRECOG reference oracle -- TEST INFRASTRUCTURE ONLY.

Plain, sequential fp64 implementations of every operation the GPU path
computes.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import this package.  It shares no code with the HIP
path (``paper_2608_02560_amd``) and neither side imports the other; only the
seeded input generators (``paper_2608_02560_amd.synth``) serve both.

What each function follows in the paper (arXiv 2608.02560):

* ``scan``        -- Eq. 1 (Sec. 3) rolled over the sequence (the rollout
  S(h, x_1:T) of App. A), final-state capture of offline indexing (Sec. 4.2)
  and the gated readout read as (C_t . h_t + Dskip x_t) * silu(z_t).
* ``top1``        -- cosine top-1 over unit-norm keys (Sec. 4.2, query time).
* ``gather``      -- state injection h_init <- h^(i*) (Sec. 4.2, query time).
* ``scan_complex`` -- Eq. 1 with the diagonal complex A of Sec. 3.
* ``trajectory``  -- SMC per-step trajectory (Sec. 5.1) thinned by the dial K
  (Sec. 5.2).
* ``topk_compose``-- softmax-weighted composition of the top-k states
  (Sec. 5.4, Eq. smc-fusion; Fig. 1 caption).
* ``fuse``        -- joint episodic + corpus retrieval: the k best candidates
  of both stores composed, plus the session's semantic state as a baseline
  term (Sec. 5.4, Eq. smc-fusion).
* ``route2``, ``ema``, ``consolidate`` -- SMC two-stage routing (Sec. 5.1,
  Eqs. smc-domain, smc-sub) and semantic EMA consolidation (Sec. 5.3,
  Eq. smc-ema), one update and a chunk-ordered sequence of them.
* ``round_bf16``, ``round_f16`` -- round-to-nearest-even storage rounding of
  fp64 values (the paper stores states at FP16, Sec. 4.2).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "precog_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libprecog_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc -O2 (no fast-math); returns the .so path."""
    if force or not os.path.exists(_LIB_PATH) or (
        os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)
    ):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
             "-fno-fast-math", "-ffp-contract=off", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        i64, dp, fp, ip = (ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p)
        lib.oracle_scan_f64.argtypes = [i64, i64, i64, i64] + [dp] * 10 + [ctypes.c_int]
        lib.oracle_scan_f64.restype = ctypes.c_int
        lib.oracle_trajectory_f64.argtypes = [i64] * 5 + [dp] * 6
        lib.oracle_trajectory_f64.restype = ctypes.c_int
        lib.oracle_scan_complex_f64.argtypes = [i64, i64, i64, i64] + [dp] * 11
        lib.oracle_scan_complex_f64.restype = ctypes.c_int
        lib.oracle_top1_f64.argtypes = [i64, i64, i64, fp, fp, ip, dp, ctypes.c_int]
        lib.oracle_top1_f64.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(a):
    """Exact widening of a numpy array or a torch tensor (any float dtype)."""
    if a is None:
        return None
    if hasattr(a, "detach"):  # torch tensor
        a = a.detach().cpu().double().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def scan(x, dt, A, B, C, z=None, Dskip=None, h0=None, want_y=True,
         want_hT=True, nthreads=1):
    """Sequential fp64 selective scan (Eq. 1, Sec. 3).

    Shapes: x, dt, z [Bt, L, D]; A [D, N] (positive: decay exp(-dt*A));
    B, C [Bt, L, N]; Dskip [D]; h0 [Bt, D, N].  Returns (y, hT) as fp64
    arrays (either may be None when not requested).
    """
    x, dt, A, B, C = (_f64(v) for v in (x, dt, A, B, C))
    z, Dskip, h0 = _f64(z), _f64(Dskip), _f64(h0)
    Bt, L, D = x.shape
    N = A.shape[1]
    assert A.shape == (D, N) and dt.shape == x.shape
    assert B.shape == (Bt, L, N)
    if want_y:
        assert C is not None and C.shape == (Bt, L, N)
    if z is not None:
        assert z.shape == x.shape
    if Dskip is not None:
        assert Dskip.shape == (D,)
    if h0 is not None:
        assert h0.shape == (Bt, D, N)
    y = np.zeros((Bt, L, D)) if want_y else None
    hT = np.zeros((Bt, D, N)) if want_hT else None
    rc = _load().oracle_scan_f64(Bt, L, D, N, _ptr(x), _ptr(dt), _ptr(A), _ptr(B),
                                 _ptr(C if want_y else None), _ptr(z), _ptr(Dskip),
                                 _ptr(h0), _ptr(y), _ptr(hT), int(nthreads))
    if rc:
        raise RuntimeError("oracle_scan_f64 failed with code %d" % rc)
    return y, hT


def scan_complex(x, dt, A_re, A_im, B, C, z=None, Dskip=None, h0=None, want_y=True):
    """Eq. 1 with the diagonal complex A of Sec. 3, A = A_re + i A_im
    (A_re > 0): complex state, real input term B x dt, readout of the real
    part of C . h (gated as in ``scan``).  h0 and the returned hT are
    [Bt, D, N, 2] with (real, imaginary) interleaved.  Returns (y, hT)."""
    x, dt, A_re, A_im, B, C, z, Dskip, h0 = (_f64(v) for v in (x, dt, A_re, A_im, B, C, z,
                                                              Dskip, h0))
    Bt, L, D = x.shape
    N = A_re.shape[1]
    y = np.zeros((Bt, L, D)) if want_y else None
    hT = np.zeros((Bt, D, N, 2))
    rc = _load().oracle_scan_complex_f64(Bt, L, D, N, _ptr(x), _ptr(dt), _ptr(A_re),
                                         _ptr(A_im), _ptr(B), _ptr(C), _ptr(z), _ptr(Dskip),
                                         _ptr(h0), _ptr(y), _ptr(hT))
    if rc:
        raise RuntimeError("oracle_scan_complex_f64 failed with code %d" % rc)
    return y, hT


def trajectory(x, dt, A, B, k, h0=None):
    """States after tokens k, 2k, ... of each row (Sec. 5.1-5.2): [Bt, L//k, D, N]."""
    x, dt, A, B, h0 = (_f64(v) for v in (x, dt, A, B, h0))
    Bt, L, D = x.shape
    N = A.shape[1]
    out = np.zeros((Bt, L // k, D, N))
    rc = _load().oracle_trajectory_f64(Bt, L, D, N, int(k), _ptr(x), _ptr(dt),
                                       _ptr(A), _ptr(B), _ptr(h0), _ptr(out))
    if rc:
        raise RuntimeError("oracle_trajectory_f64 failed with code %d" % rc)
    return out


def _f32(a):
    if hasattr(a, "detach"):
        a = a.detach().cpu().float().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def top1(query, index, nthreads=1):
    """Exact cosine top-1 (Sec. 4.2): fp64 inner products summed in index
    order; ties go to the lowest row.  Returns (idx int32 [Q], best fp64 [Q])."""
    q, K = _f32(query), _f32(index)
    Q, E = q.shape
    M = K.shape[0]
    assert K.shape[1] == E
    idx = np.empty(Q, np.int32)
    best = np.empty(Q, np.float64)
    rc = _load().oracle_top1_f64(Q, M, E, _ptr(q), _ptr(K), _ptr(idx),
                                 _ptr(best), int(nthreads))
    if rc:
        raise RuntimeError("oracle_top1_f64 failed with code %d" % rc)
    return idx, best


def gather(store, idx):
    """State injection h0[q] = store[idx[q]] (Sec. 4.2 query time), exact fp64."""
    return _f64(store)[np.asarray(idx, dtype=np.int64)]


def topk_scores(query, index, k):
    """Top-k by fp64 score (products exact, summed in index order), ties to
    the lower row, best first.  Returns (idx [Q, k] int64, score [Q, k])."""
    q = _f32(query).astype(np.float64)
    K = _f32(index).astype(np.float64)
    Q, E = q.shape
    M = K.shape[0]
    idx = np.empty((Q, k), np.int64)
    sc = np.empty((Q, k))
    for qi in range(Q):
        s = np.zeros(M)
        for e in range(E):  # one sequential sum per row, vectorised over rows
            s = s + q[qi, e] * K[:, e]
        order = sorted(range(M), key=lambda i: (-s[i], i))[:k]
        idx[qi] = order
        sc[qi] = s[order]
    return idx, sc


def topk_compose(store, idx, scores, tau):
    """h_init = sum_j w_j h^(j), w = softmax(score / tau) over the k retrieved
    states (Sec. 5.4, Eq. smc-fusion; composition of Fig. 1).  fp64."""
    store = _f64(store)
    Q, k = idx.shape
    out = np.zeros((Q,) + store.shape[1:])
    for qi in range(Q):
        logits = np.asarray(scores[qi], np.float64) / tau
        m = max(logits)
        w = [np.exp(v - m) for v in logits]
        tot = sum(w)
        for j in range(k):
            out[qi] += (w[j] / tot) * store[int(idx[qi, j])]
    return out


def fuse(episodic_store, episodic_idx, episodic_score, corpus_store, corpus_idx, corpus_score, k,
         tau, semantic=None, semantic_row=None, lam=0.0):
    """Joint retrieval at query time (Sec. 5.4, Eq. smc-fusion).  Per query
    the candidates of the episodic store and of the corpus are ranked together
    by score (larger first; equal scores: episodic before corpus, then the
    lower row), the k best are composed with softmax(score / tau) weights,
    and lam times the session's semantic state semantic[semantic_row[q]] is
    added (nothing when semantic is None).  Candidates come as rows
    [Q, k_e] / [Q, k_c] of each store with their scores.  Returns h_init
    [Q, S] in fp64."""
    ep = _f64(episodic_store)
    co = _f64(corpus_store)
    ei = np.asarray(episodic_idx, dtype=np.int64)
    ci = np.asarray(corpus_idx, dtype=np.int64)
    es = np.asarray(episodic_score, dtype=np.float64)
    cs = np.asarray(corpus_score, dtype=np.float64)
    Q = ei.shape[0]
    S = ep.shape[1] if ep.ndim == 2 and ep.shape[0] > 0 else co.shape[1]
    sem = _f64(semantic) if semantic is not None else None
    out = np.zeros((Q, S))
    for qi in range(Q):
        cands = [(-float(es[qi, j]), 0, int(ei[qi, j])) for j in range(ei.shape[1])]
        cands += [(-float(cs[qi, j]), 1, int(ci[qi, j])) for j in range(ci.shape[1])]
        cands.sort()
        top = cands[:k]
        logits = [-c[0] / tau for c in top]
        m = max(logits)
        w = [np.exp(v - m) for v in logits]
        tot = sum(w)
        for (_, src, row), wj in zip(top, w):
            out[qi] += (wj / tot) * (ep if src == 0 else co)[row]
        if sem is not None:
            out[qi] += lam * sem[int(semantic_row[qi])]
    return out


def route2(emb, domain_protos, sub_protos):
    """Two-stage routing (Sec. 5.1, Eqs. smc-domain and smc-sub):
    m* = argmax_m <phi(c), p_m>, then j* = argmax_j <phi(c), q_{m*, j}>.
    sub_protos: [M, J, E].  Ties go to the lower index.  fp64 sums in order."""
    e = _f32(emb).astype(np.float64)
    P = _f32(domain_protos).astype(np.float64)
    S = _f32(sub_protos).astype(np.float64)
    out_m = np.empty(e.shape[0], np.int32)
    out_j = np.empty(e.shape[0], np.int32)
    for c in range(e.shape[0]):
        best, bm = None, -1
        for m in range(P.shape[0]):
            s = 0.0
            for k in range(e.shape[1]):
                s += e[c, k] * P[m, k]
            if bm < 0 or s > best:
                best, bm = s, m
        best, bj = None, -1
        for j in range(S.shape[1]):
            s = 0.0
            for k in range(e.shape[1]):
                s += e[c, k] * S[bm, j, k]
            if bj < 0 or s > best:
                best, bj = s, j
        out_m[c], out_j[c] = bm, bj
    return out_m, out_j


def ema(state, contribution, alpha):
    """Semantic consolidation s <- (1 - alpha) s + alpha h (Sec. 5.3, Eq. smc-ema)."""
    return (1.0 - alpha) * _f64(state) + alpha * _f64(contribution)


def consolidate(states, contrib, target, alpha):
    """Eq. smc-ema applied for every chunk in chunk order (Sec. 5.3): chunk c
    updates the semantic state of its sub-cluster target[c]; targets outside
    the table leave it unchanged.  fp64."""
    out = _f64(states).copy()
    h = _f64(contrib)
    for c, r in enumerate(np.asarray(target, dtype=np.int64)):
        if 0 <= r < out.shape[0]:
            out[r] = ema(out[r], h[c], alpha)
    return out


def round_bf16(a):
    """Round fp64 values to the nearest bfloat16 value, ties to even
    (8 significant bits, exponent range of fp32, subnormals kept)."""
    a = np.asarray(a, dtype=np.float64)
    _, e = np.frexp(a)
    q = np.ldexp(1.0, np.maximum(e, -125) - 8)
    return np.rint(a / q) * q


def round_f16(a):
    """Round fp64 values to the nearest IEEE binary16 value, ties to even
    (11 significant bits, min normal 2^-14, subnormals kept)."""
    a = np.asarray(a, dtype=np.float64)
    _, e = np.frexp(a)
    q = np.ldexp(1.0, np.maximum(e, -13) - 11)
    r = np.rint(a / q) * q
    return np.where(np.abs(r) > 65504.0, np.copysign(np.inf, a), r)


def bf16_ulp(a):
    """Spacing of bfloat16 values at |a| (for one-ulp checks)."""
    a = np.asarray(a, dtype=np.float64)
    _, e = np.frexp(a)
    return np.ldexp(1.0, np.maximum(e, -125) - 8)
