// Exact cosine top-1 retrieval for gfx950 (query time, Sec. 4.2).
//
// The answer is defined in fp64: score(q, i) = sum_e q_e k_{i,e} summed in
// index order (products of fp32 values are exact in fp64), idx = the lowest i
// attaining the maximum.  Two kernels reach it exactly:
//
//   screen   fp32 matrix-core pass (v_mfma_f32_16x16x4_f32): S~ = Q K^T for
//            every (query, row), plus the squared norm of every key row.
//   decide   one workgroup per query: m = max_i S~_i at i0, then every row
//            whose screen score could still be the fp64 maximum,
//              S~_i + e_i >= m - e_i0,   e_i = g |q| |k_i| + tiny,
//            is rescored in fp64 in index order, and the best (score, lowest
//            index) wins.  g bounds the error of any fp32 evaluation order
//            of an E-term dot product (gamma_E = E u / (1 - E u), u = 2^-24,
//            with the sum of |q_e k_e| bounded by |q| |k_i| via
//            Cauchy-Schwarz), inflated to cover the fp32 norms and the fp64
//            rounding of the reference scores.  The fp64 argmax therefore
//            always sits in the candidate set, and ties resolve exactly as
//            in the definition.
#include "precog_kernels.h"

namespace precog {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kRows = 32;   // key rows per screen workgroup
constexpr int kQW = 64;     // queries per wave pass
constexpr int kScreenBlock = 256;

// Screen: workgroup = kRows key rows x all queries; wave w takes query
// blocks w, w+4, ...; per pass a wave computes 64 queries x 32 rows as
// 4 x 2 tiles of 16 x 16.  Within a step of 16 feature indices, lane l
// (row/col l % 16, slot l / 16) loads a float4 of features
// [e0 + 4 slot, e0 + 4 slot + 4) and feeds component j to MFMA j: the same
// permutation of the feature index on both operands leaves the dot product
// unchanged.
__global__ __launch_bounds__(kScreenBlock) void screen_kernel(const RetrieveParams p) {
  const int64_t r0 = static_cast<int64_t>(xcd_remap(blockIdx.x, gridDim.x)) * kRows;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = lane & 15;
  const int slot = lane >> 4;
  const int64_t E = p.E;

  // Squared norms of this block's rows (fp32, index order).
  if (threadIdx.x < kRows && r0 + threadIdx.x < p.M) {
    const float* kr = p.K + (r0 + threadIdx.x) * E;
    float acc = 0.f;
    for (int64_t e = 0; e < E; e += 4) {
      const float4 v = *reinterpret_cast<const float4*>(kr + e);
      acc = fmaf(v.x, v.x, acc);
      acc = fmaf(v.y, v.y, acc);
      acc = fmaf(v.z, v.z, acc);
      acc = fmaf(v.w, v.w, acc);
    }
    p.rownorm2[r0 + threadIdx.x] = acc;
  }

  // Key rows this lane feeds as the B operand (clamped; results of clamped
  // rows are never stored).
  const float* krow[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t r = min(r0 + j * 16 + col, p.M - 1);
    krow[j] = p.K + r * E;
  }

  for (int64_t qb = static_cast<int64_t>(wave) * kQW; qb < p.Q; qb += 4 * kQW) {
    const float* qrow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t q = min(qb + i * 16 + col, p.Q - 1);
      qrow[i] = p.q + q * E;
    }
    floatx4 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    for (int64_t e0 = 0; e0 < E; e0 += 16) {
      const int64_t e = e0 + 4 * slot;
      const bool in = e < E;
      float4 av[4], bv[2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        av[i] = in ? *reinterpret_cast<const float4*>(qrow[i] + e) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        bv[j] = in ? *reinterpret_cast<const float4*>(krow[j] + e) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].x, bv[j].x, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].y, bv[j].y, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].z, bv[j].z, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].w, bv[j].w, acc[i][j], 0, 0, 0);
        }
    }
    // Output tile (i, j): lane l holds rows 4 (l / 16) + r (queries) of
    // column l % 16 (key rows), r = 0..3.
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int64_t key = r0 + j * 16 + col;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t q = qb + i * 16 + 4 * slot + r;
          if (q < p.Q && key < p.M) p.scores[q * p.ld_scores + key] = acc[i][j][r];
        }
      }
  }
}

constexpr int kDecideBlock = 256;

__device__ __forceinline__ bool better(double s, int64_t i, double bs, int64_t bi) {
  return bi < 0 || s > bs || (s == bs && i < bi);
}

// One workgroup per query.
__global__ __launch_bounds__(kDecideBlock) void decide_kernel(const RetrieveParams p) {
  const int64_t q = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t E = p.E;
  const int64_t M = p.M;
  __shared__ float qs[4096];
  __shared__ float red_f[kDecideBlock];
  __shared__ int64_t red_i[kDecideBlock];
  __shared__ double red_d[kDecideBlock];

  const float* qg = p.q + q * E;
  float nq = 0.f;
  for (int64_t e = tid; e < E; e += kDecideBlock) {
    const float v = qg[e];
    qs[e] = v;
    nq = fmaf(v, v, nq);
  }
  red_f[tid] = nq;
  __syncthreads();
  for (int w = kDecideBlock / 2; w > 0; w >>= 1) {
    if (tid < w) red_f[tid] += red_f[tid + w];
    __syncthreads();
  }
  const float qnorm = sqrtf(red_f[0]);
  __syncthreads();

  // Max screen score and the lowest index attaining it.
  const float* srow = p.scores + q * p.ld_scores;
  float m = -INFINITY;
  int64_t mi = -1;
  for (int64_t i = tid; i < M; i += kDecideBlock) {
    const float v = srow[i];
    if (mi < 0 || v > m) { m = v; mi = i; }
  }
  red_f[tid] = m;
  red_i[tid] = mi;
  __syncthreads();
  for (int w = kDecideBlock / 2; w > 0; w >>= 1) {
    if (tid < w) {
      const float vo = red_f[tid + w];
      const int64_t io = red_i[tid + w];
      if (io >= 0 && (red_i[tid] < 0 || vo > red_f[tid] || (vo == red_f[tid] && io < red_i[tid]))) {
        red_f[tid] = vo;
        red_i[tid] = io;
      }
    }
    __syncthreads();
  }
  const float mmax = red_f[0];
  const int64_t i0 = red_i[0];
  __syncthreads();
  if (i0 < 0) {  // M == 0
    if (tid == 0) p.idx[q] = -1;
    return;
  }

  // Error margin of one fp32 screen score (see the file comment).
  const double u = 5.9604644775390625e-08;  // 2^-24
  const double gam = (static_cast<double>(E) * u) / (1.0 - static_cast<double>(E) * u);
  const double g = gam * 1.001 + 1e-12;
  const double tiny = 1e-30;
  const double e_i0 = g * static_cast<double>(qnorm) * sqrt(static_cast<double>(p.rownorm2[i0])) + tiny;
  const double thresh = static_cast<double>(mmax) - e_i0;

  double best = -INFINITY;
  int64_t bi = -1;
  for (int64_t i = tid; i < M; i += kDecideBlock) {
    const double ei = g * static_cast<double>(qnorm) * sqrt(static_cast<double>(p.rownorm2[i])) + tiny;
    if (static_cast<double>(srow[i]) + ei >= thresh) {
      const float* kr = p.K + i * E;
      double s = 0.0;
      for (int64_t e = 0; e < E; ++e)
        s = s + static_cast<double>(qs[e]) * static_cast<double>(kr[e]);
      if (better(s, i, best, bi)) { best = s; bi = i; }
    }
  }
  red_d[tid] = best;
  red_i[tid] = bi;
  __syncthreads();
  for (int w = kDecideBlock / 2; w > 0; w >>= 1) {
    if (tid < w) {
      const double so = red_d[tid + w];
      const int64_t io = red_i[tid + w];
      if (io >= 0 && better(so, io, red_d[tid], red_i[tid])) {
        red_d[tid] = so;
        red_i[tid] = io;
      }
    }
    __syncthreads();
  }
  if (tid == 0) p.idx[q] = static_cast<int32_t>(red_i[0]);
}

}  // namespace

hipError_t launch_retrieve(const RetrieveParams& p, hipStream_t s) {
  if (p.M > 0) {
    const int64_t blocks = (p.M + kRows - 1) / kRows;
    hipLaunchKernelGGL(screen_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kScreenBlock), 0, s, p);
  }
  hipLaunchKernelGGL(decide_kernel, dim3(static_cast<unsigned>(p.Q)), dim3(kDecideBlock), 0, s, p);
  return hipGetLastError();
}

}  // namespace precog
