"""Seeded synthetic inputs shaped like the paper's workloads.

This module draws inputs only; it holds none of the scan, retrieval or
injection arithmetic, so both the HIP path and the fp64 oracle can use it.

Distributions (one recipe for every workload):

* x, z ~ N(0, 1)
* dt = softplus(N(mu, sigma)) computed in fp64, then rounded to the input
  dtype (the selective timescale is positive, Sec. 3; (mu, sigma) = (-2, 0.5)
  for the corpus chunks, (-3, 1) for the large corpus encode)
* A ~ U[1, 16] per (d, n), fp32 (positive: the decay is exp(-dt * A) < 1)
* B, C ~ N(0, 1/N) per (b, t, n), shared across channels
* Dskip ~ N(0, 1) per channel, fp32
* index keys and queries: N(0, 1) rows normalised in fp64, then rounded to
  fp32 (unit-norm, so the inner product is the cosine); a set of queries is
  planted as normalize(k_j + 0.05 * noise) so their answer j is known
* stored states ~ N(0, 1), fp16

Host draws use numpy PCG64 with the draw order x, z, dt, A, B, C, Dskip.
Bulk workloads (hundreds of MB per tensor) are drawn on the device with a
seeded torch generator in the same order.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class ScanWorkload:
    name: str
    batch: int
    seqlen: int
    dim: int
    dstate: int
    in_dtype: torch.dtype = torch.bfloat16
    dt_mu: float = -2.0
    dt_sigma: float = 0.5
    chunk: int = 0
    seed: int = 0

    @property
    def tokens(self) -> int:
        return self.batch * self.seqlen


# The five workloads: a single fp32 layer, corpus-chunk encoding, the query
# prefill of query-time injection, a long-context scan and a large corpus
# encode (per layer; 24 layers use seeds 5000 + layer); then the SMC
# trajectory encode.
SINGLE_LAYER = ScanWorkload("single_layer_b1_l512_d128_n16_f32", 1, 512, 128, 16,
                            torch.float32, seed=1)
CORPUS_ENCODE = ScanWorkload("corpus_encode_b64_l3000_d2048_n16_bf16", 64, 3000,
                             2048, 16, seed=2)
QUERY_PREFILL = ScanWorkload("query_prefill_q256_l32_d1024_n16_bf16", 256, 32,
                             1024, 16, seed=3)
LONG_CONTEXT = ScanWorkload("long_context_b8_l65536_d2048_n16_bf16_chunk256", 8,
                            65536, 2048, 16, chunk=256, seed=4)
LARGE_CORPUS = ScanWorkload("large_corpus_b1024_l3000_d1536_n64_bf16_per_layer",
                            1024, 3000, 1536, 64, dt_mu=-3.0, dt_sigma=1.0,
                            seed=5000)
LARGE_CORPUS_LAYERS = 24
# SMC trajectory encode: 512-token conversation chunks (the paper's N_c), one
# layer, captured at the fidelity dial's every = 1 (K = N_c), 8 and 512 (K = 1).
SMC_TRAJECTORY = ScanWorkload("smc_trajectory_b64_l512_d2048_n16_bf16", 64, 512,
                              2048, 16, seed=6)
SMC_DIALS = (1, 8, 512)

RETRIEVAL = dict(Q=256, M=10000, E=384, planted=32, seed=3)
STATE_STORE = dict(M=10000, D=1024, N=16)


# Complex-A variant: the corpus-encode shape with frequencies w_n = pi n
# (Sec. 3), complex fp32 state.
COMPLEX_ENCODE = ScanWorkload("complex_encode_b64_l3000_d2048_n16_bf16", 64, 3000,
                              2048, 16, seed=8)


def complex_frequencies(D: int, N: int) -> torch.Tensor:
    """A_im[d, n] = pi n, the paper's imaginary part of A (Sec. 3), fp32."""
    return torch.from_numpy(np.tile(np.pi * np.arange(N, dtype=np.float64), (D, 1))).float()


def _softplus64(v: np.ndarray) -> np.ndarray:
    return np.logaddexp(0.0, v)


def scan_inputs_host(B: int, L: int, D: int, N: int, seed: int,
                     in_dtype: torch.dtype = torch.float32,
                     dt_mu: float = -2.0, dt_sigma: float = 0.5,
                     h0_std: float = 0.0):
    """Scan inputs drawn on the host (numpy PCG64).  Returns a dict of CPU
    torch tensors: x, dt, z, B, C in ``in_dtype``; A, Dskip in fp32; h0 fp32
    (zeros unless h0_std > 0)."""
    g = np.random.Generator(np.random.PCG64(seed))
    x = g.standard_normal((B, L, D))
    z = g.standard_normal((B, L, D))
    dt = _softplus64(g.normal(dt_mu, dt_sigma, (B, L, D)))
    A = g.uniform(1.0, 16.0, (D, N))
    Bm = g.normal(0.0, 1.0 / np.sqrt(N), (B, L, N))
    Cm = g.normal(0.0, 1.0 / np.sqrt(N), (B, L, N))
    Dskip = g.standard_normal(D)
    h0 = g.standard_normal((B, D, N)) * h0_std if h0_std > 0 else np.zeros((B, D, N))

    def t(a, dtype):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dtype)

    return dict(x=t(x, in_dtype), dt=t(dt, in_dtype), z=t(z, in_dtype),
                A=t(A, torch.float32), B=t(Bm, in_dtype), C=t(Cm, in_dtype),
                Dskip=t(Dskip, torch.float32), h0=t(h0, torch.float32))


def scan_inputs_device(B: int, L: int, D: int, N: int, seed: int,
                       in_dtype: torch.dtype = torch.bfloat16,
                       dt_mu: float = -2.0, dt_sigma: float = 0.5,
                       device: str = "cuda", need_z_c: bool = True):
    """Same recipe, drawn on the device with a seeded torch generator (for
    workloads too large to draw on the host).  Tensors are generated in
    slices of the batch so the fp32 temporaries stay small."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = {}

    def normal_(shape, mean=0.0, std=1.0):
        dst = torch.empty(shape, dtype=in_dtype, device=device)
        for b0 in range(0, shape[0], 8):
            tmp = torch.randn((min(8, shape[0] - b0),) + tuple(shape[1:]),
                              generator=g, device=device, dtype=torch.float32)
            dst[b0:b0 + tmp.shape[0]] = (tmp * std + mean).to(in_dtype)
            del tmp
        return dst

    out["x"] = normal_((B, L, D))
    out["z"] = normal_((B, L, D)) if need_z_c else None
    dt = torch.empty((B, L, D), dtype=in_dtype, device=device)
    for b0 in range(0, B, 8):
        tmp = torch.randn((min(8, B - b0), L, D), generator=g, device=device,
                          dtype=torch.float32)
        dt[b0:b0 + tmp.shape[0]] = torch.nn.functional.softplus(
            tmp * dt_sigma + dt_mu).to(in_dtype)
        del tmp
    out["dt"] = dt
    out["A"] = torch.rand((D, N), generator=g, device=device,
                          dtype=torch.float32) * 15.0 + 1.0
    out["B"] = normal_((B, L, N), std=1.0 / float(np.sqrt(N)))
    out["C"] = normal_((B, L, N), std=1.0 / float(np.sqrt(N))) if need_z_c else None
    out["Dskip"] = torch.randn((D,), generator=g, device=device, dtype=torch.float32)
    return out


def unit_rows_host(rows: int, E: int, g: np.random.Generator) -> np.ndarray:
    v = g.standard_normal((rows, E))
    v /= np.sqrt(np.sum(v * v, axis=1, keepdims=True))
    return v.astype(np.float32)


def retrieval_inputs_host(Q: int, M: int, E: int, planted: int, seed: int):
    """(queries [Q, E] fp32, index [M, E] fp32, planted_pos [P], planted_row [P]).
    The last ``planted`` queries are normalize(k_j + 0.05 noise) for random j."""
    g = np.random.Generator(np.random.PCG64(seed))
    index = unit_rows_host(M, E, g)
    queries = unit_rows_host(Q, E, g)
    planted = min(planted, Q)
    pos = np.arange(Q - planted, Q)
    rows = g.integers(0, max(M, 1), planted) if M > 0 else np.zeros(0, np.int64)
    for p, r in zip(pos, rows):
        v = index[r].astype(np.float64) + 0.05 * g.standard_normal(E)
        queries[p] = (v / np.sqrt(np.sum(v * v))).astype(np.float32)
    return (torch.from_numpy(queries), torch.from_numpy(index),
            torch.from_numpy(pos), torch.from_numpy(rows))


# SMC memory: M = 5 cognitive domains x J = 4 sub-clusters with 384-dim
# prototypes, semantic states of 24 layers x 4096 (192 KB at fp16, Sec. 5.3),
# 64 chunks deposited per consolidation call.
SMC = dict(C=64, E=384, ndom=5, nsub=4, S=24 * 4096, seed=7)


def smc_inputs_host(C: int, E: int, ndom: int, nsub: int, seed: int, spread: float = 0.3):
    """Unit-norm domain prototypes p_m, sub-cluster prototypes q_{m,j} =
    normalize(p_m + spread * noise), and chunk embeddings planted near a
    drawn sub-cluster: phi(c) = normalize(q_{m,j} + 0.05 * noise).  Returns
    (emb [C, E], dom [ndom, E], sub [ndom, nsub, E], planted_m [C],
    planted_j [C]); the plants make the expected routes known independently
    of any scoring code."""
    g = np.random.Generator(np.random.PCG64(seed))
    dom = unit_rows_host(ndom, E, g).astype(np.float64)
    sub = np.empty((ndom, nsub, E))
    for m in range(ndom):
        v = dom[m] + spread * g.standard_normal((nsub, E)) / np.sqrt(E)
        sub[m] = v / np.linalg.norm(v, axis=1, keepdims=True)
    pm = g.integers(0, ndom, C)
    pj = g.integers(0, nsub, C)
    v = sub[pm, pj] + 0.05 * g.standard_normal((C, E)) / np.sqrt(E)
    emb = v / np.linalg.norm(v, axis=1, keepdims=True)
    f = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return f(emb), f(dom), f(sub), torch.from_numpy(pm), torch.from_numpy(pj)


def state_store(M: int, S: int, seed: int, device: str = "cpu",
                dtype: torch.dtype = torch.float16):
    """A store of M precomputed states of S elements each, N(0, 1)."""
    if device == "cpu":
        g = np.random.Generator(np.random.PCG64(seed))
        return torch.from_numpy(g.standard_normal((M, S))).to(dtype)
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = torch.empty((M, S), dtype=dtype, device=device)
    for m0 in range(0, M, 1024):
        m1 = min(M, m0 + 1024)
        out[m0:m1] = torch.randn((m1 - m0, S), generator=g, device=device).to(dtype)
    return out
