// State injection for gfx950 (query time, Sec. 4.2): h0[q] = store[idx[q]],
// its top-k generalisation, the softmax-weighted composition
// h0[q] = sum_j w_j store[idx[q, j]] (Sec. 5.4 Eq. smc-fusion; Fig. 1), and
// the joint retrieval of Sec. 5.4: the k best candidates of an episodic and a
// corpus store composed the same way, plus lambda times the session's
// semantic state.
//
// Each lane moves 8 consecutive elements (16 bytes of fp16 or 32 bytes of
// fp32) so every wave access is a contiguous 1-2 KiB segment.  fp16 -> fp32
// widening is exact; fp32 -> fp16 rounds to nearest even.  An index outside
// [0, M) reads nothing and writes NaN.
#include "compose.h"
#include "precog_kernels.h"

namespace precog {
namespace {

constexpr int kBlock = 256;
constexpr int kVec = 8;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float8 __attribute__((ext_vector_type(8)));

template <typename T> struct Vec8;
template <> struct Vec8<float> {
  static __device__ __forceinline__ float8 load(const void* base, int64_t i) {
    return *reinterpret_cast<const float8*>(static_cast<const float*>(base) + i);
  }
  static __device__ __forceinline__ void store(void* base, int64_t i, float8 v) {
    *reinterpret_cast<float8*>(static_cast<float*>(base) + i) = v;
  }
};
template <> struct Vec8<f16_t> {
  static __device__ __forceinline__ float8 load(const void* base, int64_t i) {
    const half8 h = *reinterpret_cast<const half8*>(static_cast<const _Float16*>(base) + i);
    return __builtin_convertvector(h, float8);
  }
  static __device__ __forceinline__ void store(void* base, int64_t i, float8 v) {
    *reinterpret_cast<half8*>(static_cast<_Float16*>(base) + i) = __builtin_convertvector(v, half8);
  }
};

template <typename TS, typename TO>
__global__ __launch_bounds__(kBlock) void gather_kernel(const GatherParams p) {
  const int64_t q = blockIdx.y;
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * kVec;
  if (e >= p.S) return;
  const int32_t src = p.idx[q];
  float8 v;
  if (src >= 0 && src < p.M) {
    v = Vec8<TS>::load(p.store, static_cast<int64_t>(src) * p.S + e);
  } else {
    const float nan = __builtin_nanf("");
    v = float8{nan, nan, nan, nan, nan, nan, nan, nan};
  }
  Vec8<TO>::store(p.out, q * p.S + e, v);
}

// Same-dtype copy: move raw 16-byte words, no conversion.
__global__ __launch_bounds__(kBlock) void gather_raw_kernel(const GatherParams p, int64_t words_per_row,
                                                            int elem_bytes) {
  const int64_t q = blockIdx.y;
  const int64_t w = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (w >= words_per_row) return;
  const int32_t src = p.idx[q];
  uint4 v;
  if (src >= 0 && src < p.M) {
    v = reinterpret_cast<const uint4*>(p.store)[static_cast<int64_t>(src) * words_per_row + w];
  } else {
    const uint32_t nan = elem_bytes == 4 ? 0x7fc00000u : 0x7e007e00u;
    v = make_uint4(nan, nan, nan, nan);
  }
  reinterpret_cast<uint4*>(p.out)[q * words_per_row + w] = v;
}

// Composition: wave 0 of each workgroup turns the k scores of its query into
// fp32 weights (compose.h: fp64 softmax, sum in rank order, rounded once);
// then every lane sums w_j h_j in fp32 in rank order (j = 0 first), one fma
// per term.  k = 1 gives w = 1 exactly, so the result equals the plain
// gather bit for bit.
template <typename TS, typename TO>
__global__ __launch_bounds__(kBlock) void compose_kernel(const ComposeParams p) {
  const int64_t q = blockIdx.y;
  const int k = p.k;
  __shared__ float w[kMaxTopK];
  __shared__ int32_t src[kMaxTopK];
  __shared__ int bad;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const bool on = lane < k;
    const double* srow = p.score + q * k;
    const SoftmaxDen den = softmax_den(srow, k, p.inv_tau);
    const int32_t ij = on ? p.idx[q * k + lane] : 0;
    const bool oob = on && (ij < 0 || ij >= p.M);
    const uint64_t badmask = __ballot(oob);
    if (on) {
      w[lane] = softmax_weight(srow[lane], den, p.inv_tau);
      src[lane] = ij;
    }
    if (lane == 0) bad = badmask != 0;
  }
  __syncthreads();
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * kVec;
  if (e >= p.S) return;
  float8 acc;
  if (bad) {
    const float nan = __builtin_nanf("");
    acc = float8{nan, nan, nan, nan, nan, nan, nan, nan};
  } else {
    acc = float8{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const float8 v = Vec8<TS>::load(p.store, static_cast<int64_t>(src[j]) * p.S + e);
      const float wj = w[j];
#pragma unroll
      for (int c = 0; c < kVec; ++c) acc[c] = fmaf(wj, v[c], acc[c]);
    }
  }
  Vec8<TO>::store(p.out, q * p.S + e, acc);
}

__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(__double2loint(v)), lane);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(__double2hiint(v)), lane);
  return __hiloint2double(hi, lo);
}

// Candidate order of the joint retrieval: larger score first (NaN last),
// then the episodic store (0) before the corpus (1), then the lower row,
// then the earlier list position; a total order, so ranks are distinct.
struct Cand {
  double s;
  int src, row, pos;
};
__device__ __forceinline__ bool cand_before(const Cand& a, const Cand& b) {
  const double sa = a.s != a.s ? -INFINITY : a.s;
  const double sb = b.s != b.s ? -INFINITY : b.s;
  if (sa != sb) return sa > sb;
  if (a.src != b.src) return a.src < b.src;
  if (a.row != b.row) return a.row < b.row;
  return a.pos < b.pos;
}

// Joint retrieval (Sec. 5.4, Eq. smc-fusion): wave 0 of each workgroup ranks
// the query's candidates of both stores (lane j holds entry j of each list;
// every lane counts, from one broadcast element per step, the elements
// ordered before its own), keeps the k best in rank order in LDS and turns
// their scores into fp32 weights (compose.h, as the composition does); then
// every lane sums w_j h_j in fp32 in rank order, one fma per term, and adds
// lambda times the session's semantic state with one more fma.  A candidate
// or semantic row outside its store gives a NaN row.
template <typename TS, typename TO>
__global__ __launch_bounds__(kBlock) void fuse_kernel(const FuseParams p) {
  const int64_t q = blockIdx.y;
  const int k = p.k;
  __shared__ double ss[kMaxTopK];
  __shared__ float w[kMaxTopK];
  __shared__ int32_t srow[kMaxTopK];
  __shared__ int32_t ssrc[kMaxTopK];
  __shared__ int bad;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    Cand mine[2];
    bool have[2];
#pragma unroll
    for (int l = 0; l < 2; ++l) {
      have[l] = lane < p.kk[l];
      mine[l].s = have[l] ? p.score[l][q * p.kk[l] + lane] : 0.0;
      mine[l].row = have[l] ? p.idx[l][q * p.kk[l] + lane] : 0;
      mine[l].src = l;
      mine[l].pos = lane;
    }
    int rank[2] = {0, 0};
#pragma unroll
    for (int l = 0; l < 2; ++l) {
      for (int i = 0; i < p.kk[l]; ++i) {
        Cand o;
        o.s = readlane_f64(mine[l].s, i);
        o.row = __builtin_amdgcn_readlane(mine[l].row, i);
        o.src = l;
        o.pos = i;
        rank[0] += cand_before(o, mine[0]) ? 1 : 0;
        rank[1] += cand_before(o, mine[1]) ? 1 : 0;
      }
    }
#pragma unroll
    for (int l = 0; l < 2; ++l) {
      if (have[l] && rank[l] < k) {
        ss[rank[l]] = mine[l].s;
        srow[rank[l]] = mine[l].row;
        ssrc[rank[l]] = l;
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the list is in LDS
    __builtin_amdgcn_wave_barrier();
    const SoftmaxDen den = softmax_den(ss, k, p.inv_tau);
    const bool on = lane < k;
    bool oob = false;
    if (on) {
      w[lane] = softmax_weight(ss[lane], den, p.inv_tau);
      oob = srow[lane] < 0 || srow[lane] >= (ssrc[lane] == 0 ? p.rows[0] : p.rows[1]);
    }
    if (lane == 0 && p.sem != nullptr) {
      const int32_t r = p.sem_row[q];
      oob = oob || r < 0 || r >= p.sem_rows;
    }
    const uint64_t badmask = __ballot(oob);
    if (lane == 0) bad = badmask != 0;
  }
  __syncthreads();
  const int64_t e = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * kVec;
  if (e >= p.S) return;
  float8 acc;
  if (bad) {
    const float nan = __builtin_nanf("");
    acc = float8{nan, nan, nan, nan, nan, nan, nan, nan};
  } else {
    acc = float8{0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const void* base = ssrc[j] == 0 ? p.store[0] : p.store[1];
      const float8 v = Vec8<TS>::load(base, static_cast<int64_t>(srow[j]) * p.S + e);
      const float wj = w[j];
#pragma unroll
      for (int c = 0; c < kVec; ++c) acc[c] = fmaf(wj, v[c], acc[c]);
    }
    if (p.sem != nullptr) {
      const float8 v = Vec8<TS>::load(p.sem, static_cast<int64_t>(p.sem_row[q]) * p.S + e);
#pragma unroll
      for (int c = 0; c < kVec; ++c) acc[c] = fmaf(p.lambda, v[c], acc[c]);
    }
  }
  Vec8<TO>::store(p.out, q * p.S + e, acc);
}

}  // namespace

hipError_t launch_gather(const GatherParams& p, int store_dtype, int out_dtype, hipStream_t s) {
  if (store_dtype == out_dtype) {
    const int eb = store_dtype == 0 ? 4 : 2;
    const int64_t words = p.S * eb / 16;
    const dim3 grid(static_cast<unsigned>((words + kBlock - 1) / kBlock), static_cast<unsigned>(p.Q));
    hipLaunchKernelGGL(gather_raw_kernel, grid, dim3(kBlock), 0, s, p, words, eb);
  } else {
    const dim3 grid(static_cast<unsigned>((p.S / kVec + kBlock - 1) / kBlock), static_cast<unsigned>(p.Q));
    if (store_dtype == 2)
      hipLaunchKernelGGL((gather_kernel<f16_t, float>), grid, dim3(kBlock), 0, s, p);
    else
      hipLaunchKernelGGL((gather_kernel<float, f16_t>), grid, dim3(kBlock), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_compose(const ComposeParams& p, int store_dtype, int out_dtype, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>((p.S / kVec + kBlock - 1) / kBlock), static_cast<unsigned>(p.Q));
  if (store_dtype == 2 && out_dtype == 2)
    hipLaunchKernelGGL((compose_kernel<f16_t, f16_t>), grid, dim3(kBlock), 0, s, p);
  else if (store_dtype == 2)
    hipLaunchKernelGGL((compose_kernel<f16_t, float>), grid, dim3(kBlock), 0, s, p);
  else if (out_dtype == 2)
    hipLaunchKernelGGL((compose_kernel<float, f16_t>), grid, dim3(kBlock), 0, s, p);
  else
    hipLaunchKernelGGL((compose_kernel<float, float>), grid, dim3(kBlock), 0, s, p);
  return hipGetLastError();
}

}  // namespace precog

namespace precog {
hipError_t launch_fuse(const FuseParams& p, int store_dtype, int out_dtype, hipStream_t s) {
  const dim3 grid(static_cast<unsigned>((p.S / kVec + kBlock - 1) / kBlock), static_cast<unsigned>(p.Q));
  if (store_dtype == 2 && out_dtype == 2)
    hipLaunchKernelGGL((fuse_kernel<f16_t, f16_t>), grid, dim3(kBlock), 0, s, p);
  else if (store_dtype == 2)
    hipLaunchKernelGGL((fuse_kernel<f16_t, float>), grid, dim3(kBlock), 0, s, p);
  else if (out_dtype == 2)
    hipLaunchKernelGGL((fuse_kernel<float, f16_t>), grid, dim3(kBlock), 0, s, p);
  else
    hipLaunchKernelGGL((fuse_kernel<float, float>), grid, dim3(kBlock), 0, s, p);
  return hipGetLastError();
}
}  // namespace precog
