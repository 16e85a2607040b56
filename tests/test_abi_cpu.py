"""Host-only checks of libprecog: it loads, exports every entry point the
public header declares, and rejects malformed arguments with the documented
status before anything touches a GPU (no compute calls are made here)."""
import ctypes
import os
import re

import pytest

from paper_2608_02560_amd import precog as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "precog.h")

OK, ENULL, ESHAPE, EDTYPE, ESTRIDE, EALIGN, EWS = 0, 1, 2, 3, 4, 5, 6

FAKE = 0x10000  # a 16-byte aligned non-null address; never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(precog_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = P.lib()
    names = declared_functions()
    assert set(names) == set(P.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for code in range(9):
        assert P.status_string(code)
    assert P.status_string(99) == "unknown status"


def _encode(desc, x=FAKE, dt=FAKE, A=FAKE, B=FAKE, C=FAKE, z=FAKE, Dskip=FAKE, h0=None,
            y=FAKE, hT=FAKE, ws=None, wsb=0):
    d = desc if desc is None else ctypes.byref(desc)
    return P.lib().precog_scan_encode(d, x, dt, A, B, C, z, Dskip, h0, y, hT, ws, wsb, None)


def _encode_indexed(desc, store=FAKE, rows=4, idx=FAKE, x=FAKE, y=FAKE, hT=FAKE, score=None,
                    k=1, tau=1.0):
    d = desc if desc is None else ctypes.byref(desc)
    return P.lib().precog_scan_encode_indexed(d, x, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, store,
                                              rows, idx, score, k, tau, y, hT, None, 0, None)


def test_indexed_scan_validation_errors():
    good = P.scan_desc(2, 16, 64, 16)
    assert _encode_indexed(None) == ENULL
    assert _encode_indexed(good, idx=None) == ENULL           # the index is the point
    assert _encode_indexed(good, rows=-1) == ESHAPE
    assert _encode_indexed(good, store=None) == ENULL         # rows > 0 need a store
    assert _encode_indexed(good, idx=FAKE + 4) == EALIGN
    assert _encode_indexed(good, store=FAKE + 8) == EALIGN
    assert _encode_indexed(P.scan_desc(2, 16, 64, 16, h0_batch_stride=64 * 16 - 8)) == ESTRIDE
    assert _encode_indexed(P.scan_desc(0, 16, 64, 16), idx=None) == OK  # nothing to compute
    assert _encode_indexed(good, k=2) == ESHAPE                 # k > 1 needs scores
    assert _encode_indexed(good, score=FAKE, k=0) == ESHAPE
    assert _encode_indexed(good, score=FAKE, k=65) == ESHAPE
    assert _encode_indexed(good, score=FAKE, k=3, tau=0.0) == ESHAPE
    assert _encode_indexed(good, score=FAKE, k=3, tau=float("inf")) == ESHAPE
    assert _encode_indexed(good, score=FAKE + 8, k=3) == EALIGN


def test_scan_validation_errors():
    good = P.scan_desc(2, 16, 64, 16)
    assert _encode(None) == ENULL
    assert _encode(P.scan_desc(-1, 16, 64, 16)) == ESHAPE
    assert _encode(P.scan_desc(2, -1, 64, 16)) == ESHAPE
    assert _encode(P.scan_desc(2, 16, 64, 3)) == ESHAPE        # N not supported
    assert _encode(P.scan_desc(2, 16, 64, 128)) == ESHAPE
    assert _encode(P.scan_desc(2, 16, 60, 16)) == EALIGN       # D % 8
    assert _encode(P.scan_desc(2, 16, 64, 16, in_dtype=P.F16)) == EDTYPE
    assert _encode(P.scan_desc(2, 16, 64, 16, out_dtype=P.F16)) == EDTYPE
    assert _encode(P.scan_desc(2, 16, 64, 16, state_dtype=P.BF16)) == EDTYPE
    assert _encode(P.scan_desc(2, 16, 64, 16, h0_batch_stride=64 * 16 - 8)) == ESTRIDE
    assert _encode(P.scan_desc(2, 16, 64, 16, hT_batch_stride=4)) == ESTRIDE
    assert _encode(P.scan_desc(2, 16, 64, 16, hT_batch_stride=64 * 16 + 4)) == EALIGN
    assert _encode(good, x=None) == ENULL
    assert _encode(good, dt=None) == ENULL
    assert _encode(good, A=None) == ENULL
    assert _encode(good, B=None) == ENULL
    assert _encode(good, C=None) == ENULL                       # C needed for y
    assert _encode(good, x=FAKE + 2) == EALIGN
    assert _encode(good, hT=FAKE + 8) == EALIGN
    # chunked scans need workspace
    chunked = P.scan_desc(2, 1024, 64, 16, chunk=128)
    need = P.scan_workspace_bytes(chunked)
    assert need > 0
    assert _encode(chunked) == EWS
    assert _encode(chunked, ws=FAKE, wsb=need - 1) == EWS


def test_scan_noops_return_ok_without_device():
    # nothing to compute: empty batch, empty channels, or no output requested
    assert _encode(P.scan_desc(0, 16, 64, 16)) == OK
    assert _encode(P.scan_desc(2, 16, 0, 16)) == OK
    assert _encode(P.scan_desc(2, 16, 64, 16), y=None, hT=None) == OK
    # y = NULL makes C, z and Dskip optional
    st = _encode(P.scan_desc(0, 16, 64, 16), C=None, z=None, Dskip=None, y=None)
    assert st == OK


def test_scan_workspace_sizes():
    assert P.scan_workspace_bytes(P.scan_desc(64, 3000, 2048, 16)) == 0  # one pass
    d = P.scan_desc(8, 65536, 2048, 16, chunk=256)
    C = 256
    carry = 8 * C * 2048 * 16 * 4
    dts = 8 * C * 2048 * 4
    assert P.scan_workspace_bytes(d) == carry + dts
    # chunk >= L is one pass
    assert P.scan_workspace_bytes(P.scan_desc(2, 100, 64, 16, chunk=100)) == 0
    assert P.scan_workspace_bytes(P.scan_desc(2, 100, 64, 16, chunk=1000)) == 0
    # invalid descriptor reports 0
    assert P.scan_workspace_bytes(P.scan_desc(2, 100, 60, 16)) == 0


def test_chunk_cap_covers_the_coefficient_streams():
    """Chunks are capped so every per-token stream stays addressable with
    32-bit buffer offsets: chunk * max(D, N) * 4 < 2^31.  With D = 8 and
    N = 64 the coefficient rows B_t, C_t are the wider ones, so a one-chunk
    request over 3 * 2^23 tokens is cut into 4 chunks (the cap is
    (2^31 - 1) / 256 = 2^23 - 1 tokens), which shows in the carry workspace."""
    L = 3 * (1 << 23)
    d = P.scan_desc(1, L, 8, 64, chunk=L)
    nch = -(-L // ((2 ** 31 - 1) // (64 * 4)))
    assert nch == 4
    carry = nch * 8 * 64 * 4
    dts = -(-(nch * 8 * 4) // 256) * 256
    assert P.scan_workspace_bytes(d) == carry + dts
    # D wider than N: the cap follows D, (2^31 - 1) / (512 * 4) = 2^20 - 1 tokens
    assert P.scan_workspace_bytes(P.scan_desc(1, (1 << 20) - 1, 512, 16, chunk=1 << 20)) == 0
    assert P.scan_workspace_bytes(P.scan_desc(1, 1 << 20, 512, 16, chunk=1 << 20)) > 0


def test_retrieve_validation_errors():
    L = P.lib()
    ws = P.retrieve_workspace_bytes(4, 10, 16)
    assert ws >= 4 * 9 + 10 * 4
    # the workspace scales with Q M / 32 (block summaries), not with Q M
    assert P.retrieve_workspace_bytes(256, 10000, 384) < 256 * 10000 * 4 // 8
    call = lambda q=FAKE, k=FAKE, Q=4, M=10, E=16, idx=FAKE, w=FAKE, wb=ws: \
        L.precog_retrieve_top1(q, k, Q, M, E, idx, w, wb, None)
    assert call(Q=-1) == ESHAPE
    assert call(E=2) == ESHAPE
    assert call(E=8192) == ESHAPE
    assert call(E=18) == EALIGN
    assert call(q=None) == ENULL
    assert call(k=None) == ENULL
    assert call(idx=None) == ENULL
    assert call(w=None) == EWS
    assert call(wb=ws - 1) == EWS
    assert call(q=FAKE + 4) == EALIGN
    assert call(Q=0) == OK


def _query(desc, q=FAKE, K=FAKE, prepared=None, pbytes=0, M=100, E=64, store=FAKE, idx=FAKE,
           x=FAKE, y=FAKE, hT=FAKE, ws=FAKE, wsb=None):
    d = desc if desc is None else ctypes.byref(desc)
    if wsb is None:
        wsb = P.query_workspace_bytes(desc, M, E) if desc is not None else 0
    return P.lib().precog_query_top1_prefill(d, q, K, prepared, pbytes, M, E, store, idx, x, FAKE,
                                             FAKE, FAKE, FAKE, FAKE, FAKE, y, hT, ws, wsb, None)


def test_query_call_validation_errors():
    """precog_query_top1_prefill checks every argument of both halves (the
    retrieval and the prefill from the store) before the device."""
    good = P.scan_desc(8, 16, 64, 16, P.BF16, P.BF16, P.F16)
    assert _query(None) == ENULL
    assert _query(good, q=None) == ENULL
    assert _query(good, idx=None) == ENULL
    assert _query(good, K=None) == ENULL
    assert _query(good, store=None) == ENULL        # M > 0 rows need a store
    assert _query(good, x=None) == ENULL             # the prefill's inputs
    assert _query(good, E=6) == EALIGN
    assert _query(good, E=2) == ESHAPE
    assert _query(good, M=-1) == ESHAPE
    assert _query(good, q=FAKE + 4) == EALIGN
    assert _query(good, store=FAKE + 8) == EALIGN
    assert _query(good, hT=FAKE + 2) == EALIGN
    assert _query(good, ws=None) == EWS
    assert _query(good, wsb=P.retrieve_workspace_bytes(8, 100, 64) - 1) == EWS
    assert _query(good, prepared=FAKE, pbytes=P.retrieve_index_bytes(100, 64) - 1) == EWS
    assert _query(P.scan_desc(8, 16, 64, 16, P.F16)) == EDTYPE
    assert _query(P.scan_desc(8, 16, 60, 16)) == EALIGN
    assert _query(P.scan_desc(8, 16, 64, 3)) == ESHAPE
    # time chunks need the scan's workspace after the retrieval's
    few = P.scan_desc(2, 4096, 64, 16)
    need = P.query_workspace_bytes(few, 100, 64)
    assert need > P.retrieve_workspace_bytes(2, 100, 64) and P.scan_workspace_bytes(few) > 0
    assert _query(few, wsb=need - 1) == EWS
    # nothing to do: no queries
    assert _query(P.scan_desc(0, 16, 64, 16), q=None, idx=None, ws=None, wsb=0) == OK


def test_query_workspace_bytes():
    desc = P.scan_desc(256, 32, 1024, 16, P.BF16, P.BF16, P.F16)
    r = P.retrieve_workspace_bytes(256, 10000, 384)
    assert P.query_workspace_bytes(desc, 10000, 384) == (r + 255) // 256 * 256
    assert P.scan_workspace_bytes(desc) == 0  # 4096 waves: one pass
    assert P.query_workspace_bytes(P.scan_desc(2, 16, 60, 16), 10, 64) == 0   # invalid desc
    assert P.query_workspace_bytes(desc, 10, 6) == 0                         # invalid E


def test_trajectory_validation_errors():
    L = P.lib()
    good = P.scan_desc(2, 16, 64, 16)

    def call(desc=good, traj=FAKE, every=4, x=FAKE):
        return L.precog_scan_trajectory(ctypes.byref(desc), x, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                        None, FAKE, FAKE, traj, every, None, 0, None)
    assert call(every=0) == ESHAPE
    assert call(every=-3) == ESHAPE
    assert call(traj=None) == ENULL
    assert call(traj=FAKE + 4) == EALIGN
    assert call(x=None) == ENULL
    assert call(P.scan_desc(2, 16, 60, 16)) == EALIGN
    assert call(P.scan_desc(0, 16, 64, 16)) == OK      # empty batch
    # nothing to capture (L < every) and no other output: NULL traj is fine
    assert L.precog_scan_trajectory(ctypes.byref(good), FAKE, FAKE, FAKE, FAKE, None, None, None,
                                    None, None, None, None, 17, None, 0, None) == OK


def test_complex_scan_validation_errors():
    L = P.lib()

    def call(desc, x=FAKE, Aim=FAKE, h0=None, ws=None, wsb=0):
        return L.precog_scan_complex(ctypes.byref(desc), x, FAKE, FAKE, Aim, FAKE, FAKE, FAKE,
                                     FAKE, h0, FAKE, FAKE, ws, wsb, None)
    assert call(P.scan_desc(2, 16, 64, 32)) == ESHAPE          # N > 16
    assert call(P.scan_desc(2, 16, 64, 16, h0_batch_stride=64 * 16)) == ESTRIDE  # < 2 D N
    assert call(P.scan_desc(2, 16, 64, 16), Aim=None) == ENULL
    assert call(P.scan_desc(2, 16, 64, 16), x=None) == ENULL
    assert call(P.scan_desc(2, 16, 60, 16)) == EALIGN
    assert call(P.scan_desc(2, 16, 64, 16), h0=FAKE + 4) == EALIGN
    assert call(P.scan_desc(0, 16, 64, 16)) == OK
    # chunked complex scans need workspace: carries [B, C, D, N, 2] fp32 and
    # chunk dt sums [B, C, D] fp32, each 256-byte aligned
    chunked = P.scan_desc(2, 1024, 64, 16, chunk=128)
    need = P.scan_complex_workspace_bytes(chunked)
    assert need == 2 * 8 * 64 * 16 * 2 * 4 + 2 * 8 * 64 * 4
    assert call(chunked) == EWS
    assert call(chunked, ws=FAKE, wsb=need - 1) == EWS
    assert call(chunked, ws=FAKE + 8, wsb=need) == EALIGN
    assert P.scan_complex_workspace_bytes(P.scan_desc(2, 1024, 64, 16, chunk=1024)) == 0
    assert P.scan_complex_workspace_bytes(P.scan_desc(2, 1024, 64, 32)) == 0  # invalid: N > 16


def test_complex_chunk_cap_keeps_32bit_offsets():
    """A one-chunk request whose per-token streams would pass 2^31 bytes
    (70,000 tokens x 8200 channels x 4 bytes) is cut at
    (2^31 - 1) / (8200 * 4) = 65,472 tokens into two chunks, so it takes a
    workspace instead of wrapping the kernels' 32-bit offsets."""
    L = 70000
    d = P.scan_desc(1, L, 8200, 16, in_dtype=P.F32, out_dtype=P.F32, chunk=L)
    cap = (2 ** 31 - 1) // (8200 * 4)
    assert cap == 65472 and -(-L // cap) == 2
    assert P.scan_complex_workspace_bytes(d) == 2 * 8200 * 16 * 2 * 4 + 2 * 8200 * 4 + 192


def test_topk_validation_errors():
    L = P.lib()
    ws = P.retrieve_workspace_bytes(4, 10, 16)
    call = lambda q=FAKE, K=FAKE, Q=4, M=10, E=16, k=3, idx=FAKE, sc=FAKE, w=FAKE, wb=ws: \
        L.precog_retrieve_topk(q, K, Q, M, E, k, idx, sc, w, wb, None)
    assert call(k=0) == ESHAPE
    assert call(k=65, M=100) == ESHAPE
    assert call(k=11) == ESHAPE          # more than M keys
    assert call(M=0, k=1) == ESHAPE
    assert call(E=18) == EALIGN
    assert call(idx=None) == ENULL
    assert call(sc=FAKE + 8) == EALIGN
    assert call(w=None) == EWS
    assert call(Q=0) == OK


def test_prepared_index_validation_errors():
    L = P.lib()
    nb = P.retrieve_index_bytes(10, 16)
    # 16-byte operand entries for ceil(10/32) blocks x ceil(16/16) steps x 64,
    # then the norms, each part 256-byte aligned
    assert nb == 1024 + 256 + 256
    assert P.retrieve_index_bytes(0, 16) == 0
    assert P.retrieve_index_bytes(10, 18) == 0
    prep = lambda K=FAKE, M=10, E=16, out=FAKE, b=nb: L.precog_retrieve_prepare(K, M, E, out, b, None)
    assert prep(M=0) == ESHAPE
    assert prep(E=4100) == ESHAPE
    assert prep(E=18) == EALIGN
    assert prep(K=None) == ENULL
    assert prep(out=None) == ENULL
    assert prep(out=FAKE + 8) == EALIGN
    assert prep(b=nb - 1) == EWS
    ws = P.retrieve_workspace_bytes(4, 10, 16)
    call = lambda q=FAKE, K=FAKE, pr=FAKE, pb=nb, Q=4, M=10, E=16, k=3, idx=FAKE, sc=FAKE, \
        w=FAKE, wb=ws: L.precog_retrieve_topk_prepared(q, K, pr, pb, Q, M, E, k, idx, sc, w, wb,
                                                       None)
    assert call(k=0) == ESHAPE
    assert call(k=11) == ESHAPE
    assert call(pr=None) == ENULL
    assert call(pb=nb - 1) == EWS
    assert call(pr=FAKE + 8) == EALIGN
    assert call(E=18) == EALIGN
    assert call(w=None) == EWS
    assert call(Q=0) == OK


def test_compose_validation_errors():
    L = P.lib()
    call = lambda s=FAKE, sd=P.F16, M=10, S=64, idx=FAKE, sc=FAKE, Q=3, k=3, tau=1.0, h=FAKE, \
        hd=P.F32: L.precog_inject_compose(s, sd, M, S, idx, sc, Q, k, tau, h, hd, None)
    assert call(k=0) == ESHAPE
    assert call(k=65) == ESHAPE
    assert call(tau=0.0) == ESHAPE
    assert call(tau=-1.0) == ESHAPE
    assert call(tau=float("nan")) == ESHAPE
    assert call(tau=float("inf")) == ESHAPE
    assert call(sd=P.BF16) == EDTYPE
    assert call(S=12) == EALIGN
    assert call(sc=None) == ENULL
    assert call(idx=None) == ENULL
    assert call(sc=FAKE + 8) == EALIGN
    assert call(Q=0) == OK


def test_fuse_validation_errors():
    L = P.lib()

    def call(es=FAKE, er=10, ei=FAKE, esc=FAKE, ek=3, cs=FAKE, cr=20, ci=FAKE, csc=FAKE, ck=3,
             sd=P.F16, S=64, Q=3, k=3, tau=1.0, sem=None, srow=None, sr=0, lam=1.0, h=FAKE,
             hd=P.F32):
        return L.precog_inject_fuse(es, er, ei, esc, ek, cs, cr, ci, csc, ck, sd, S, Q, k, tau, sem,
                                    srow, sr, lam, h, hd, None)
    assert call(k=0) == ESHAPE
    assert call(k=7) == ESHAPE                 # more than the two lists hold
    assert call(ek=65) == ESHAPE
    assert call(ck=-1) == ESHAPE
    assert call(er=-1) == ESHAPE
    assert call(tau=0.0) == ESHAPE
    assert call(tau=float("inf")) == ESHAPE
    assert call(lam=float("nan")) == ESHAPE
    assert call(sd=P.BF16) == EDTYPE
    assert call(hd=P.BF16) == EDTYPE
    assert call(S=12) == EALIGN
    assert call(ei=None) == ENULL
    assert call(csc=None) == ENULL
    assert call(cs=None) == ENULL
    assert call(sem=FAKE, srow=None, sr=4) == ENULL
    assert call(h=None) == ENULL
    assert call(esc=FAKE + 8) == EALIGN
    assert call(srow=FAKE + 4, sem=FAKE, sr=4) == EALIGN
    assert call(Q=0) == OK
    # an empty list needs none of its pointers
    assert call(ck=0, ci=None, csc=None, cs=None, Q=0) == OK


def test_smc_validation_errors():
    L = P.lib()
    route = lambda e=FAKE, C=3, E=16, d=FAKE, nd=5, s=FAKE, ns=4, mo=FAKE, so=FAKE, fo=None: \
        L.precog_smc_route(e, C, E, d, nd, s, ns, mo, so, fo, None)
    assert route(nd=0) == ESHAPE
    assert route(ns=65) == ESHAPE
    assert route(E=2) == ESHAPE
    assert route(E=18) == EALIGN
    assert route(d=None) == ENULL
    assert route(so=None) == ENULL
    assert route(fo=FAKE + 4) == EALIGN
    assert route(C=0) == OK
    cons = lambda st=FAKE, sd=P.F16, R=20, S=64, h=FAKE, hd=P.F16, t=FAKE, C=3, a=0.25: \
        L.precog_smc_consolidate(st, sd, R, S, h, hd, t, C, a, None)
    assert cons(a=0.0) == ESHAPE
    assert cons(a=1.5) == ESHAPE
    assert cons(a=float("nan")) == ESHAPE
    assert cons(R=70000) == ESHAPE
    assert cons(sd=P.BF16) == EDTYPE
    assert cons(S=12) == EALIGN
    assert cons(t=None) == ENULL
    assert cons(h=FAKE + 2) == EALIGN
    assert cons(C=0) == OK
    assert cons(a=1.0, C=0) == OK


def test_gather_validation_errors():
    L = P.lib()
    call = lambda s=FAKE, sd=P.F16, M=10, S=64, idx=FAKE, Q=3, h=FAKE, hd=P.F32: \
        L.precog_inject_gather(s, sd, M, S, idx, Q, h, hd, None)
    assert call(M=-1) == ESHAPE
    assert call(sd=P.BF16) == EDTYPE
    assert call(hd=7) == EDTYPE
    assert call(S=12) == EALIGN
    assert call(s=None) == ENULL
    assert call(idx=None) == ENULL
    assert call(h=None) == ENULL
    assert call(h=FAKE + 2) == EALIGN
    assert call(Q=0) == OK
    assert call(S=0) == OK


def test_descriptor_layout_matches_header():
    # int64 x4, three 4-byte enums (+4 padding), int64 x3
    assert ctypes.sizeof(P.ScanDesc) == 4 * 8 + 3 * 4 + 4 + 3 * 8
    assert P.ScanDesc.h0_batch_stride.offset == 48
