// Internal declarations shared by the HIP kernels and the C-ABI layer of
// libprecog (not part of the public interface, which is include/precog.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "precog.h"

namespace precog {

// Storage tags.  bf16 and fp16 are both 16-bit; the tags keep them apart.
struct bf16_t { uint16_t bits; };
struct f16_t { uint16_t bits; };

enum ScanFlags : int {
  kHasZ = 1,   // gate z present
  kHasD = 2,   // Dskip present
  kHasH0 = 4,  // initial state present
  kHasHT = 8,  // final state requested
  kBalance = 16,  // balance the progress of waves sharing a SIMD (scan_kernel)
};

// Everything one scan launch needs.  Passed by value as the kernel argument.
struct ScanParams {
  const void* x;
  const void* dt;
  const void* z;
  const void* Bm;
  const void* Cm;
  const float* A;
  const float* A_im;  // imaginary part of A (complex-A launches only)
  const float* Dskip;
  const void* h0;
  const int32_t* h0_idx;    // non-null: batch row b starts from store rows h0_idx[b * h0_k + j]
  int64_t h0_rows;          // rows of that store (h0); an index outside [0, h0_rows) gives NaN
  const double* h0_score;   // non-null: [B, h0_k] scores, the start is their softmax composition
  int h0_k;                 // rows composed per batch row (1 without scores)
  double h0_inv_tau;        // 1 / temperature of that composition
  void* y;
  void* hT;
  float* carry;   // [B, C, D, N] fp32 ([B, C, D, N, 2] for complex A): slot 0 = h0,
                  // slot c = state entering chunk c
  float* dtsum;   // [B, C, D] fp32: slot c = sum of dt over chunk c (c < C-1)
  void* traj;     // [B, traj_count, D, N] state dtype (trajectory launches only)
  int64_t traj_every, traj_count;
  int64_t B, L, D;
  int64_t chunk;  // tokens per time chunk
  int64_t h0_stride, hT_stride;
  int nchunks;    // C
  int dblocks;    // ceil(D / 256)
  int flags;
};

// Threads per workgroup of the real-A scan kernels: 8 waves, so that the two
// waves sharing a SIMD at two waves per SIMD belong to one workgroup and can
// see each other's progress in LDS (see scan_kernels.h).
constexpr int kScanThreads = 512;

// Launchers (return the HIP launch status).  in/out/state dtypes are the
// precog_dtype codes of the public header.
hipError_t launch_scan(const ScanParams& p, int N, int in_dtype, int out_dtype,
                       int state_dtype, hipStream_t s);
hipError_t launch_scan_traj(const ScanParams& p, int N, int in_dtype, int out_dtype,
                            int state_dtype, hipStream_t s);
// Complex diagonal A: N <= 16, states interleaved (re, im); chunked like the
// real scan (summary, carry fold, replay) when p.nchunks > 1.
hipError_t launch_scan_complex(const ScanParams& p, int N, int in_dtype, int out_dtype,
                               int state_dtype, hipStream_t s);

struct RetrieveParams {
  const float* q;      // [Q, E]
  const float* K;      // [M, E]
  void* qop;           // fp16(2^8 q) in operand order (workspace)
  const void* kop;     // prepared index operands, or null (keys read as fp32)
  float* blockmax;     // [Q, nkb] largest screen score per 32-key block (workspace)
  float* blocksec;     // [Q, nkb] largest screen score of the block's other keys (workspace)
  uint8_t* blockarg;   // [Q, nkb] key of the largest, 0..31 within its block (workspace)
  float* rownorm2;     // [M] squared key norms (workspace)
  float* blocknorm2;   // [nkb] largest squared key norm per block (workspace)
  int32_t* idx;        // [Q, k]
  double* score;       // [Q, k] exact scores of idx, or null
  int64_t Q, M, E;
  int nkb;             // ceil(M / 32)
  int nqg;             // 32-query groups, padded to whole screen workgroups
  int nks;             // ceil(E / 16): 16-feature steps
  int k;               // keys kept per query, 1..kMaxTopK
  // error-bound constants of the decide (set by launch_retrieve from E)
  double err_g, err_h, err_tiny, err_gs;
};
// Screen workgroup: kRetWaves waves of 32 queries each, over kRetBlocks
// blocks of 32 keys.
constexpr int kRetWaves = 8;
constexpr int kRetBlocks = 2;
constexpr int kMaxTopK = 64;
hipError_t launch_retrieve(const RetrieveParams& p, hipStream_t s);
// The two halves of launch_retrieve: query operands and screen (also sets
// p's error-bound constants), then the decision.
hipError_t launch_retrieve_screen(RetrieveParams& p, hipStream_t s);
hipError_t launch_retrieve_decide(const RetrieveParams& p, hipStream_t s);
// The query-time prefill that decides its own query's top-1 (batch row b =
// query b of `rp`, whose screen has run) and starts from that store row:
// N = 16, bf16 inputs, one pass, readout with gate or state only.  Returns
// hipErrorInvalidValue for any other configuration, without launching.
hipError_t launch_query_scan(const ScanParams& p, const RetrieveParams& rp, int out_dtype,
                             int state_dtype, hipStream_t s);
// Body of the retrieval entry points (precog_abi.cpp): validates the
// arguments, lays out `workspace` and launches; `prepared` may be null.
// Validation and parameters of a retrieval call (nothing launched); with
// Q == 0 it returns PRECOG_OK and p is not used.  Without dev_check it stops
// after the argument checks (no device query, p not filled).
precog_status retrieve_setup(const float* query_emb, const float* index_emb, const void* prepared,
                             int64_t Q, int64_t M, int64_t E, int64_t k, int32_t* idx,
                             double* score, void* workspace, size_t workspace_bytes,
                             RetrieveParams& p, bool dev_check);
precog_status retrieve_entry(const float* query_emb, const float* index_emb, const void* prepared,
                             int64_t Q, int64_t M, int64_t E, int64_t k, int32_t* idx,
                             double* score, void* workspace, size_t workspace_bytes,
                             void* stream);
// Prepared index: p.kop, p.rownorm2 and p.blocknorm2 are written from p.K.
hipError_t launch_retrieve_prepare(const RetrieveParams& p, hipStream_t s);

struct GatherParams {
  const void* store;  // [M, S]
  const int32_t* idx; // [Q]
  void* out;          // [Q, S]
  int64_t M, S, Q;
};
hipError_t launch_gather(const GatherParams& p, int store_dtype, int out_dtype,
                         hipStream_t s);

struct ComposeParams {
  const void* store;     // [M, S]
  const int32_t* idx;    // [Q, k]
  const double* score;   // [Q, k]
  void* out;             // [Q, S]
  int64_t M, S, Q;
  int k;
  double inv_tau;        // 1 / temperature
};
hipError_t launch_compose(const ComposeParams& p, int store_dtype, int out_dtype,
                          hipStream_t s);

struct FuseParams {
  const void* store[2];     // episodic [rows[0], S] and corpus [rows[1], S] states
  int64_t rows[2];
  const int32_t* idx[2];    // [Q, kk[s]] candidate rows of store s
  const double* score[2];   // [Q, kk[s]] their scores
  int kk[2];                // candidates per query in each list, 0..kMaxTopK
  const void* sem;          // [sem_rows, S] semantic states, or null
  const int32_t* sem_row;   // [Q] row of the session's semantic state
  int64_t sem_rows;
  float lambda;             // weight of the semantic state
  void* out;                // [Q, S]
  int64_t S, Q;
  int k;                    // candidates composed, 1..kMaxTopK
  double inv_tau;           // 1 / temperature
};
hipError_t launch_fuse(const FuseParams& p, int store_dtype, int out_dtype, hipStream_t s);

struct RouteParams {
  const float* emb;    // [C, E] chunk embeddings
  const float* dom;    // [ndom, E] domain prototypes
  const float* sub;    // [ndom, nsub, E] sub-cluster prototypes
  int32_t* dom_out;    // [C]
  int32_t* sub_out;    // [C]
  int32_t* flat_out;   // [C] dom * nsub + sub, or null
  int64_t C, E;
  int ndom, nsub;      // 1..64 each
};
hipError_t launch_route(const RouteParams& p, hipStream_t s);

struct EmaParams {
  void* states;          // [R, S] semantic states, updated in place
  const void* contrib;   // [C, S] chunk contributions
  const int32_t* target; // [C] row of states per chunk; outside [0, R): none
  int64_t R, S, C;
  float alpha, one_minus_alpha;
};
hipError_t launch_ema(const EmaParams& p, int state_dtype, int contrib_dtype, hipStream_t s);

// Raw buffer descriptor over [base, base + bytes): loads at or past `bytes`
// return zero and stores there are dropped by the hardware range check.
constexpr int kBufWord3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)
constexpr uint32_t kDropOffset = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes), kBufWord3);
}

// Maps a hardware workgroup id to a logical one so that logically adjacent
// workgroups run on the same XCD (the dispatcher deals workgroups to the 8
// XCDs round-robin, and each XCD has its own L2).
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int kXcd = 8;
  const int xcd = bid % kXcd;
  const int local = bid / kXcd;
  const int per = nblocks / kXcd;
  const int rem = nblocks % kXcd;
  return xcd < rem ? xcd * (per + 1) + local
                   : rem * (per + 1) + (xcd - rem) * per + local;
}

}  // namespace precog
