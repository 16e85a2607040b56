"""Python binding of libprecog (the C ABI in include/precog.h).

Argument marshalling only: every step of the computation runs in the gfx950
kernels of libprecog.so.  PyTorch supplies device memory and the current
HIP stream.  There is no fallback: if the library is missing or the device is
not a gfx950, the calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# Always the in-tree build: tests, smoke and bench measure the library built
# from this tree's sources.
LIB_PATH = os.path.join(_HERE, "libprecog.so")

F32, BF16, F16 = 0, 1, 2
_DT = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}

STATUS = {0: "PRECOG_OK", 1: "PRECOG_ERR_NULL", 2: "PRECOG_ERR_SHAPE", 3: "PRECOG_ERR_DTYPE",
          4: "PRECOG_ERR_STRIDE", 5: "PRECOG_ERR_ALIGN", 6: "PRECOG_ERR_WORKSPACE",
          7: "PRECOG_ERR_ARCH", 8: "PRECOG_ERR_HIP"}

EXPORTS = ("precog_scan_workspace_bytes", "precog_scan_encode", "precog_scan_encode_indexed",
           "precog_scan_trajectory",
           "precog_scan_complex", "precog_scan_complex_workspace_bytes",
           "precog_retrieve_workspace_bytes", "precog_retrieve_top1",
           "precog_retrieve_top1_noalloc",
           "precog_retrieve_topk", "precog_retrieve_index_bytes", "precog_retrieve_prepare",
           "precog_retrieve_topk_prepared", "precog_query_workspace_bytes",
           "precog_query_top1_prefill", "precog_inject_gather", "precog_inject_compose",
           "precog_inject_fuse",
           "precog_smc_route", "precog_smc_consolidate", "precog_status_string")


class PrecogError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__("%s failed: %s (%s)" % (fn, STATUS.get(status, status),
                                                 status_string(status)))


class ScanDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seqlen", ctypes.c_int64),
                ("dim", ctypes.c_int64), ("dstate", ctypes.c_int64),
                ("in_dtype", ctypes.c_int), ("out_dtype", ctypes.c_int),
                ("state_dtype", ctypes.c_int),
                ("h0_batch_stride", ctypes.c_int64), ("hT_batch_stride", ctypes.c_int64),
                ("chunk", ctypes.c_int64)]


_lib = None


def lib():
    """The loaded libprecog.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libprecog.so is not built (%s); run "
                               "`python -m paper_2608_02560_amd.build`" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
        L.precog_scan_workspace_bytes.argtypes = [ctypes.POINTER(ScanDesc)]
        L.precog_scan_workspace_bytes.restype = sz
        L.precog_scan_encode.argtypes = [ctypes.POINTER(ScanDesc)] + [vp] * 11 + [sz, vp]
        L.precog_scan_encode.restype = ctypes.c_int
        L.precog_scan_encode_indexed.argtypes = [ctypes.POINTER(ScanDesc)] + [vp] * 8 + \
            [i64, vp, vp, i64, ctypes.c_double, vp, vp, vp, sz, vp]
        L.precog_scan_encode_indexed.restype = ctypes.c_int
        L.precog_scan_trajectory.argtypes = [ctypes.POINTER(ScanDesc)] + [vp] * 11 + \
            [i64, vp, sz, vp]
        L.precog_scan_trajectory.restype = ctypes.c_int
        L.precog_scan_complex.argtypes = [ctypes.POINTER(ScanDesc)] + [vp] * 12 + [sz, vp]
        L.precog_scan_complex.restype = ctypes.c_int
        L.precog_scan_complex_workspace_bytes.argtypes = [ctypes.POINTER(ScanDesc)]
        L.precog_scan_complex_workspace_bytes.restype = sz
        L.precog_retrieve_workspace_bytes.argtypes = [i64, i64, i64]
        L.precog_retrieve_workspace_bytes.restype = sz
        L.precog_retrieve_top1.argtypes = [vp, vp, i64, i64, i64, vp, vp, sz, vp]
        L.precog_retrieve_top1.restype = ctypes.c_int
        L.precog_retrieve_top1_noalloc.argtypes = [vp, vp, i64, i64, i64, vp, vp]
        L.precog_retrieve_top1_noalloc.restype = ctypes.c_int
        L.precog_retrieve_topk.argtypes = [vp, vp, i64, i64, i64, i64, vp, vp, vp, sz, vp]
        L.precog_retrieve_topk.restype = ctypes.c_int
        L.precog_retrieve_index_bytes.argtypes = [i64, i64]
        L.precog_retrieve_index_bytes.restype = sz
        L.precog_retrieve_prepare.argtypes = [vp, i64, i64, vp, sz, vp]
        L.precog_retrieve_prepare.restype = ctypes.c_int
        L.precog_retrieve_topk_prepared.argtypes = [vp, vp, vp, sz, i64, i64, i64, i64, vp, vp, vp,
                                                    sz, vp]
        L.precog_retrieve_topk_prepared.restype = ctypes.c_int
        L.precog_query_workspace_bytes.argtypes = [ctypes.POINTER(ScanDesc), i64, i64]
        L.precog_query_workspace_bytes.restype = sz
        L.precog_query_top1_prefill.argtypes = [ctypes.POINTER(ScanDesc), vp, vp, vp, sz, i64, i64,
                                                vp, vp] + [vp] * 9 + [vp, sz, vp]
        L.precog_query_top1_prefill.restype = ctypes.c_int
        L.precog_inject_gather.argtypes = [vp, ctypes.c_int, i64, i64, vp, i64, vp,
                                           ctypes.c_int, vp]
        L.precog_inject_gather.restype = ctypes.c_int
        L.precog_inject_compose.argtypes = [vp, ctypes.c_int, i64, i64, vp, vp, i64, i64,
                                            ctypes.c_double, vp, ctypes.c_int, vp]
        L.precog_inject_compose.restype = ctypes.c_int
        L.precog_inject_fuse.argtypes = [vp, i64, vp, vp, i64, vp, i64, vp, vp, i64, ctypes.c_int,
                                         i64, i64, i64, ctypes.c_double, vp, vp, i64,
                                         ctypes.c_double, vp, ctypes.c_int, vp]
        L.precog_inject_fuse.restype = ctypes.c_int
        L.precog_smc_route.argtypes = [vp, i64, i64, vp, i64, vp, i64, vp, vp, vp, vp]
        L.precog_smc_route.restype = ctypes.c_int
        L.precog_smc_consolidate.argtypes = [vp, ctypes.c_int, i64, i64, vp, ctypes.c_int, vp, i64,
                                             ctypes.c_double, vp]
        L.precog_smc_consolidate.restype = ctypes.c_int
        L.precog_status_string.argtypes = [ctypes.c_int]
        L.precog_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().precog_status_string(int(status)).decode()


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(fn, st):
    if st != 0:
        raise PrecogError(fn, st)


def scan_desc(batch, seqlen, dim, dstate, in_dtype=BF16, out_dtype=F32, state_dtype=F32,
              h0_batch_stride=0, hT_batch_stride=0, chunk=0) -> ScanDesc:
    return ScanDesc(batch, seqlen, dim, dstate, in_dtype, out_dtype, state_dtype,
                    h0_batch_stride, hT_batch_stride, chunk)


def scan_workspace_bytes(desc: ScanDesc) -> int:
    return int(lib().precog_scan_workspace_bytes(ctypes.byref(desc)))


def scan_encode(desc: ScanDesc, x, dt, A, B, C=None, z=None, Dskip=None, h0=None, y=None,
                hT=None, workspace=None, workspace_bytes=0, stream=None):
    """precog_scan_encode on device tensors (or raw device pointers)."""
    st = lib().precog_scan_encode(ctypes.byref(desc), _ptr(x), _ptr(dt), _ptr(A), _ptr(B),
                                  _ptr(C), _ptr(z), _ptr(Dskip), _ptr(h0), _ptr(y), _ptr(hT),
                                  _ptr(workspace), int(workspace_bytes), _stream(stream))
    _check("precog_scan_encode", st)


def scan_encode_indexed(desc: ScanDesc, x, dt, A, B, C=None, z=None, Dskip=None, store=None,
                        store_rows=0, h0_idx=None, y=None, hT=None, workspace=None,
                        workspace_bytes=0, stream=None, h0_score=None, k=1, tau=1.0):
    """precog_scan_encode_indexed on device tensors (or raw device pointers)."""
    st = lib().precog_scan_encode_indexed(ctypes.byref(desc), _ptr(x), _ptr(dt), _ptr(A), _ptr(B),
                                          _ptr(C), _ptr(z), _ptr(Dskip), _ptr(store),
                                          int(store_rows), _ptr(h0_idx), _ptr(h0_score), int(k),
                                          float(tau), _ptr(y), _ptr(hT), _ptr(workspace),
                                          int(workspace_bytes), _stream(stream))
    _check("precog_scan_encode_indexed", st)


def scan_trajectory(desc: ScanDesc, x, dt, A, B, C=None, z=None, Dskip=None, h0=None, y=None,
                    hT=None, traj=None, every=1, workspace=None, workspace_bytes=0, stream=None):
    """precog_scan_trajectory on device tensors (or raw device pointers)."""
    st = lib().precog_scan_trajectory(ctypes.byref(desc), _ptr(x), _ptr(dt), _ptr(A), _ptr(B),
                                      _ptr(C), _ptr(z), _ptr(Dskip), _ptr(h0), _ptr(y), _ptr(hT),
                                      _ptr(traj), int(every), _ptr(workspace),
                                      int(workspace_bytes), _stream(stream))
    _check("precog_scan_trajectory", st)


def scan_complex_workspace_bytes(desc: ScanDesc) -> int:
    return int(lib().precog_scan_complex_workspace_bytes(ctypes.byref(desc)))


def scan_complex_raw(desc: ScanDesc, x, dt, A_re, A_im, B, C=None, z=None, Dskip=None, h0=None,
                     y=None, hT=None, workspace=None, workspace_bytes=0, stream=None):
    """precog_scan_complex on device tensors (or raw device pointers)."""
    st = lib().precog_scan_complex(ctypes.byref(desc), _ptr(x), _ptr(dt), _ptr(A_re), _ptr(A_im),
                                   _ptr(B), _ptr(C), _ptr(z), _ptr(Dskip), _ptr(h0), _ptr(y),
                                   _ptr(hT), _ptr(workspace), int(workspace_bytes),
                                   _stream(stream))
    _check("precog_scan_complex", st)


def retrieve_workspace_bytes(Q, M, E) -> int:
    return int(lib().precog_retrieve_workspace_bytes(Q, M, E))


def retrieve_top1(query, index, idx, workspace, workspace_bytes=None, stream=None):
    Q, E = query.shape
    M = index.shape[0]
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib().precog_retrieve_top1(_ptr(query), _ptr(index), Q, M, E, _ptr(idx),
                                    _ptr(workspace), int(workspace_bytes), _stream(stream))
    _check("precog_retrieve_top1", st)


def retrieve_top1_noalloc(query, index, idx, stream=None):
    """precog_retrieve_top1_noalloc: top-1 with the library's fixed device
    array as workspace (nothing allocated)."""
    Q, E = query.shape
    M = index.shape[0]
    st = lib().precog_retrieve_top1_noalloc(_ptr(query), _ptr(index), Q, M, E, _ptr(idx),
                                            _stream(stream))
    _check("precog_retrieve_top1_noalloc", st)


NOALLOC_SCRATCH_BYTES = 32 << 20


def retrieve_topk(query, index, k, idx, score, workspace, workspace_bytes=None, stream=None):
    Q, E = query.shape
    M = index.shape[0]
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib().precog_retrieve_topk(_ptr(query), _ptr(index), Q, M, E, int(k), _ptr(idx),
                                    _ptr(score), _ptr(workspace), int(workspace_bytes),
                                    _stream(stream))
    _check("precog_retrieve_topk", st)


def retrieve_index_bytes(M, E) -> int:
    return int(lib().precog_retrieve_index_bytes(M, E))


def retrieve_prepare(index, prepared, stream=None):
    """precog_retrieve_prepare: the prepared form of index [M, E] into `prepared`."""
    M, E = index.shape
    nbytes = prepared.numel() * prepared.element_size()
    st = lib().precog_retrieve_prepare(_ptr(index), M, E, _ptr(prepared), int(nbytes),
                                       _stream(stream))
    _check("precog_retrieve_prepare", st)


def retrieve_topk_prepared(query, index, prepared, k, idx, score, workspace, workspace_bytes=None,
                           stream=None):
    Q, E = query.shape
    M = index.shape[0]
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    pbytes = prepared.numel() * prepared.element_size()
    st = lib().precog_retrieve_topk_prepared(_ptr(query), _ptr(index), _ptr(prepared), int(pbytes),
                                             Q, M, E, int(k), _ptr(idx), _ptr(score),
                                             _ptr(workspace), int(workspace_bytes),
                                             _stream(stream))
    _check("precog_retrieve_topk_prepared", st)


def query_workspace_bytes(desc: ScanDesc, M, E) -> int:
    return int(lib().precog_query_workspace_bytes(ctypes.byref(desc), int(M), int(E)))


def query_top1_prefill(desc: ScanDesc, query, index, store, idx, x, dt, A, B, C=None, z=None,
                       Dskip=None, y=None, hT=None, workspace=None, workspace_bytes=None,
                       prepared=None, stream=None):
    """precog_query_top1_prefill: exact top-1 of each query, then the prefill
    of batch row b from store row idx[b] (one call)."""
    M, E = index.shape
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    pbytes = prepared.numel() * prepared.element_size() if prepared is not None else 0
    st = lib().precog_query_top1_prefill(ctypes.byref(desc), _ptr(query), _ptr(index),
                                         _ptr(prepared), int(pbytes), int(M), int(E), _ptr(store),
                                         _ptr(idx), _ptr(x), _ptr(dt), _ptr(A), _ptr(B), _ptr(C),
                                         _ptr(z), _ptr(Dskip), _ptr(y), _ptr(hT), _ptr(workspace),
                                         int(workspace_bytes), _stream(stream))
    _check("precog_query_top1_prefill", st)


def inject_compose(store, idx, score, tau, h0, stream=None):
    M = store.shape[0]
    S = store[0].numel() if M > 0 else h0[0].numel()
    Q, k = idx.shape
    st = lib().precog_inject_compose(_ptr(store), _DT[store.dtype], M, S, _ptr(idx), _ptr(score),
                                     Q, k, float(tau), _ptr(h0), _DT[h0.dtype], _stream(stream))
    _check("precog_inject_compose", st)


def inject_gather(store, idx, h0, stream=None):
    M = store.shape[0]
    S = store[0].numel() if M > 0 else h0[0].numel()
    st = lib().precog_inject_gather(_ptr(store), _DT[store.dtype], M, S, _ptr(idx),
                                    idx.shape[0], _ptr(h0), _DT[h0.dtype], _stream(stream))
    _check("precog_inject_gather", st)


def inject_fuse(episodic_store, episodic_idx, episodic_score, corpus_store, corpus_idx,
                corpus_score, k, tau, h0, semantic=None, semantic_row=None, lam=1.0,
                stream=None):
    """precog_inject_fuse: stores [M, ...] (same dtype), candidate lists
    [Q, k_e] / [Q, k_c] (int32 rows, fp64 scores), h0 [Q, ...]."""
    Q = h0.shape[0]
    S = h0[0].numel() if Q > 0 else 0
    ke = episodic_idx.shape[1] if episodic_idx is not None else 0
    kc = corpus_idx.shape[1] if corpus_idx is not None else 0
    st = lib().precog_inject_fuse(_ptr(episodic_store), episodic_store.shape[0],
                                  _ptr(episodic_idx), _ptr(episodic_score), ke,
                                  _ptr(corpus_store), corpus_store.shape[0], _ptr(corpus_idx),
                                  _ptr(corpus_score), kc, _DT[episodic_store.dtype], S, Q, int(k),
                                  float(tau), _ptr(semantic), _ptr(semantic_row),
                                  semantic.shape[0] if semantic is not None else 0, float(lam),
                                  _ptr(h0), _DT[h0.dtype], _stream(stream))
    _check("precog_inject_fuse", st)


def smc_route(emb, domain_protos, sub_protos, domain_out, sub_out, flat_out=None, stream=None):
    C, E = emb.shape
    st = lib().precog_smc_route(_ptr(emb), C, E, _ptr(domain_protos), domain_protos.shape[0],
                                _ptr(sub_protos), sub_protos.shape[1], _ptr(domain_out),
                                _ptr(sub_out), _ptr(flat_out), _stream(stream))
    _check("precog_smc_route", st)


def smc_consolidate(states, contrib, target, alpha, stream=None):
    R = states.shape[0]
    S = states[0].numel() if R > 0 else 0
    C = target.shape[0]
    st = lib().precog_smc_consolidate(_ptr(states), _DT[states.dtype], R, S, _ptr(contrib),
                                      _DT[contrib.dtype], _ptr(target), C, float(alpha),
                                      _stream(stream))
    _check("precog_smc_consolidate", st)


# ----------------------------------------------------------------------------
# Convenience wrappers that allocate outputs and workspace with torch.
# ----------------------------------------------------------------------------
def scan(x, dt, A, B, C=None, z=None, Dskip=None, h0=None, *, out_dtype=torch.float32,
         state_dtype=torch.float32, want_y=True, want_hT=True, chunk=0, hT=None,
         hT_batch_stride=0, h0_batch_stride=0, stream=None):
    """Runs the scan; returns (y, hT) (None where not requested)."""
    Bt, L, D = x.shape
    N = A.shape[1]
    desc = scan_desc(Bt, L, D, N, _DT[x.dtype], _DT[out_dtype], _DT[state_dtype],
                     h0_batch_stride, hT_batch_stride, chunk)
    y = torch.empty((Bt, L, D), dtype=out_dtype, device=x.device) if want_y else None
    if want_hT and hT is None:
        hT = torch.empty((Bt, D, N), dtype=state_dtype, device=x.device)
    nbytes = scan_workspace_bytes(desc)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device) if nbytes else None
    scan_encode(desc, x, dt, A, B, C, z, Dskip, h0, y, hT if want_hT else None, ws, nbytes,
                stream)
    return y, (hT if want_hT else None)


def scan_from_store(x, dt, A, B, store, idx, C=None, z=None, Dskip=None, *, score=None, tau=1.0,
                    out_dtype=torch.float32, want_y=True, want_hT=True, chunk=0, stream=None):
    """Runs the scan with batch row b starting from store[idx[b]] (store
    [M, D, N] in the state dtype, idx [B] int32), or, with score [B, k] fp64
    and idx [B, k], from the softmax composition of those k rows; returns
    (y, hT)."""
    Bt, L, D = x.shape
    N = A.shape[1]
    state_dtype = store.dtype
    desc = scan_desc(Bt, L, D, N, _DT[x.dtype], _DT[out_dtype], _DT[state_dtype], 0, 0, chunk)
    y = torch.empty((Bt, L, D), dtype=out_dtype, device=x.device) if want_y else None
    hT = torch.empty((Bt, D, N), dtype=state_dtype, device=x.device) if want_hT else None
    nbytes = scan_workspace_bytes(desc)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device) if nbytes else None
    k = 1 if score is None else score.shape[1]
    scan_encode_indexed(desc, x, dt, A, B, C, z, Dskip, store, store.shape[0], idx, y, hT, ws,
                        nbytes, stream, h0_score=score, k=k, tau=tau)
    return y, hT


def query_prefill(query, index, store, x, dt, A, B, C=None, z=None, Dskip=None, *,
                  prepared=None, out_dtype=torch.float32, want_y=True, want_hT=True, chunk=0,
                  stream=None):
    """The query-time path in one call: idx = exact top-1 of each query row
    over index, then the scan of batch row b from store[idx[b]] (store
    [M, D, N] in the state dtype); returns (idx, y, hT)."""
    Bt, L, D = x.shape
    N = A.shape[1]
    M, E = index.shape
    desc = scan_desc(Bt, L, D, N, _DT[x.dtype], _DT[out_dtype], _DT[store.dtype], 0, 0, chunk)
    idx = torch.empty(Bt, dtype=torch.int32, device=x.device)
    y = torch.empty((Bt, L, D), dtype=out_dtype, device=x.device) if want_y else None
    hT = torch.empty((Bt, D, N), dtype=store.dtype, device=x.device) if want_hT else None
    nbytes = query_workspace_bytes(desc, M, E)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=x.device)
    query_top1_prefill(desc, query, index, store, idx, x, dt, A, B, C, z, Dskip, y, hT, ws, nbytes,
                       prepared, stream)
    return idx, y, hT


def trajectory(x, dt, A, B, every, C=None, z=None, Dskip=None, h0=None, *,
               out_dtype=torch.float32, state_dtype=torch.float32, want_y=False, want_hT=False,
               chunk=0, stream=None):
    """Runs the scan keeping every `every`-th state; returns (traj, y, hT)."""
    Bt, L, D = x.shape
    N = A.shape[1]
    desc = scan_desc(Bt, L, D, N, _DT[x.dtype], _DT[out_dtype], _DT[state_dtype], 0, 0, chunk)
    # every < 1 is left to the library to reject
    traj = torch.empty((Bt, L // every if every >= 1 else 0, D, N), dtype=state_dtype,
                       device=x.device)
    y = torch.empty((Bt, L, D), dtype=out_dtype, device=x.device) if want_y else None
    hT = torch.empty((Bt, D, N), dtype=state_dtype, device=x.device) if want_hT else None
    nbytes = scan_workspace_bytes(desc)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device) if nbytes else None
    scan_trajectory(desc, x, dt, A, B, C, z, Dskip, h0, y, hT, traj, every, ws, nbytes, stream)
    return traj, y, hT


def scan_complex(x, dt, A_re, A_im, B, C=None, z=None, Dskip=None, h0=None, *,
                 out_dtype=torch.float32, state_dtype=torch.float32, want_y=True, want_hT=True,
                 chunk=0, stream=None):
    """Complex-A scan; returns (y, hT) with hT [Bt, D, N, 2] (None where not requested)."""
    Bt, L, D = x.shape
    N = A_re.shape[1]
    desc = scan_desc(Bt, L, D, N, _DT[x.dtype], _DT[out_dtype], _DT[state_dtype], chunk=chunk)
    y = torch.empty((Bt, L, D), dtype=out_dtype, device=x.device) if want_y else None
    hT = torch.empty((Bt, D, N, 2), dtype=state_dtype, device=x.device) if want_hT else None
    nbytes = scan_complex_workspace_bytes(desc)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device) if nbytes else None
    scan_complex_raw(desc, x, dt, A_re, A_im, B, C, z, Dskip, h0, y, hT, ws, nbytes, stream)
    return y, hT


def top1(query, index, stream=None):
    Q, E = query.shape
    M = index.shape[0]
    idx = torch.empty(Q, dtype=torch.int32, device=query.device)
    nbytes = retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=query.device)
    retrieve_top1(query, index, idx, ws, nbytes, stream)
    return idx


def topk(query, index, k, stream=None):
    """Exact top-k: returns (idx int32 [Q, k], score fp64 [Q, k])."""
    Q, E = query.shape
    M = index.shape[0]
    idx = torch.empty((Q, k), dtype=torch.int32, device=query.device)
    score = torch.empty((Q, k), dtype=torch.float64, device=query.device)
    nbytes = retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=query.device)
    retrieve_topk(query, index, k, idx, score, ws, nbytes, stream)
    return idx, score


def prepare_index(index, stream=None):
    """The prepared form of index [M, E] (a uint8 device tensor)."""
    M, E = index.shape
    prepared = torch.empty(max(retrieve_index_bytes(M, E), 16), dtype=torch.uint8,
                           device=index.device)
    retrieve_prepare(index, prepared, stream)
    return prepared


def topk_prepared(query, index, prepared, k, want_score=True, stream=None):
    """Exact top-k over a prepared index: (idx int32 [Q, k], score fp64 [Q, k] or None)."""
    Q, E = query.shape
    M = index.shape[0]
    idx = torch.empty((Q, k), dtype=torch.int32, device=query.device)
    score = torch.empty((Q, k), dtype=torch.float64, device=query.device) if want_score else None
    nbytes = retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=query.device)
    retrieve_topk_prepared(query, index, prepared, k, idx, score, ws, nbytes, stream)
    return idx, score


def compose(store, idx, score, tau=1.0, out_dtype=None, stream=None):
    out_dtype = out_dtype or store.dtype
    h0 = torch.empty((idx.shape[0],) + tuple(store.shape[1:]), dtype=out_dtype,
                     device=store.device)
    inject_compose(store, idx, score, tau, h0, stream)
    return h0


def route(emb, domain_protos, sub_protos, stream=None):
    """Two-stage routing: returns (domain int32 [C], sub int32 [C], flat int32 [C])."""
    C = emb.shape[0]
    outs = [torch.empty(C, dtype=torch.int32, device=emb.device) for _ in range(3)]
    smc_route(emb, domain_protos, sub_protos, *outs, stream=stream)
    return tuple(outs)


def gather(store, idx, out_dtype=None, stream=None):
    out_dtype = out_dtype or store.dtype
    h0 = torch.empty((idx.shape[0],) + tuple(store.shape[1:]), dtype=out_dtype,
                     device=store.device)
    inject_gather(store, idx, h0, stream)
    return h0
