"""precog_retrieve_top1_noalloc, the retrieval entry point for callers that
cannot allocate device memory, against precog_retrieve_top1 with a
caller-supplied workspace: bit-identical indices on two calls in a row, the
second with a smaller input (the library's array then still holds the first
call's larger contents), both also equal to the oracle's argmax."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2608_02560_amd import precog as P
from paper_2608_02560_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _with_workspace(q, K):
    Q, E = q.shape
    M = K.shape[0]
    idx = torch.full((Q,), -7, dtype=torch.int32, device=DEV)
    nbytes = P.retrieve_workspace_bytes(Q, M, E)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    st = P.lib().precog_retrieve_top1(q.data_ptr(), K.data_ptr(), Q, M, E, idx.data_ptr(),
                                      ws.data_ptr(), nbytes,
                                      torch.cuda.current_stream().cuda_stream)
    assert st == 0, P.status_string(st)
    torch.cuda.synchronize()
    return idx.cpu().numpy()


def _noalloc(q, K):
    Q, E = q.shape
    M = K.shape[0]
    idx = torch.full((Q,), -7, dtype=torch.int32, device=DEV)
    st = P.lib().precog_retrieve_top1_noalloc(q.data_ptr(), K.data_ptr(), Q, M, E,
                                              idx.data_ptr(),
                                              torch.cuda.current_stream().cuda_stream)
    assert st == 0, P.status_string(st)
    torch.cuda.synchronize()
    return idx.cpu().numpy()


def test_noalloc_matches_workspace_entry_point_twice():
    cfg = synth.RETRIEVAL
    cases = [(cfg["Q"], cfg["M"], cfg["E"], cfg["planted"], cfg["seed"]),  # the query workload
             (40, 2500, 128, 4, 71)]                                       # then a smaller one
    for Q, M, E, planted, seed in cases:
        assert P.retrieve_workspace_bytes(Q, M, E) <= P.NOALLOC_SCRATCH_BYTES
        q, K, _, _ = synth.retrieval_inputs_host(Q, M, E, planted, seed)
        ref, _ = oracle.top1(q, K, nthreads=8)
        qd, Kd = q.to(DEV), K.to(DEV)
        a = _with_workspace(qd, Kd)
        b = _noalloc(qd, Kd)
        print("noalloc case Q=%d M=%d E=%d" % (Q, M, E), flush=True)
        assert np.array_equal(b, a)
        assert np.array_equal(b, ref)


def test_noalloc_rejects_workspace_past_the_array():
    # the block summaries of 16384 queries x 100,000 keys (9 bytes per query
    # and 32-key block, 460 MB) exceed the 32 MiB array
    Q, M = 16384, 100000
    assert P.retrieve_workspace_bytes(Q, M, 64) > P.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((Q, 64), dtype=torch.float32, device=DEV)
    K = torch.zeros((M, 64), dtype=torch.float32, device=DEV)
    idx = torch.full((Q,), -7, dtype=torch.int32, device=DEV)
    st = P.lib().precog_retrieve_top1_noalloc(q.data_ptr(), K.data_ptr(), Q, M, 64,
                                              idx.data_ptr(), None)
    assert st == 6  # PRECOG_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert int(idx.min()) == -7 and int(idx.max()) == -7  # nothing was enqueued
