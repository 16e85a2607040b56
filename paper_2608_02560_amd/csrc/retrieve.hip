// Exact cosine top-1 retrieval for gfx950 (query time, Sec. 4.2).
//
// The answer is defined in fp64: score(q, i) = sum_e q_e k_{i,e} summed in
// index order (products of fp32 values are exact in fp64), idx = the lowest i
// attaining the maximum.  Three kernels reach it exactly:
//
//   prep     rounds every query value v to fp16(2^8 v) (round to nearest
//            even; the power-of-two scale is exact and lifts unit-norm
//            components clear of the fp16 subnormal range) and stores the
//            values in the order the matrix-core operands are consumed, so a
//            wave's operand load is one contiguous 1 KiB segment.
//   screen   workgroup = 64 keys x 256 queries: the keys are read
//            row-contiguously, rounded the same way and staged in LDS; each
//            wave computes 32 queries against them with
//            v_mfma_f32_32x32x16_f16 (each product of two fp16 values is
//            exact in fp32) and scales back by 2^-16.  For every (query,
//            32-key block) it keeps the largest screen score S~, its key, and
//            the largest S~ of the block's other keys; and the squared norm
//            of every key and the largest one of every block.
//   decide   one wave per query: m = the largest screen score.  A key can
//            still be the fp64 maximum only if S~_i + e(i) >= m - e(i0), where
//            e(i) = g |q| |k_i| + h (|q| + |k_i|) + tiny bounds the error of
//            its screen score (g bounds the fp16 rounding and the fp32
//            accumulation, taken at twice its round-to-nearest bound, per
//            unit of sum |q_e k_e|, which Cauchy-Schwarz bounds by |q| |k_i|;
//            h bounds values below the fp16 normal range per unit of the
//            1-norms; both are inflated for the fp32 norms and the fp64
//            rounding of the reference).  Blocks are tested first with their
//            maxima and norm bounds; of a surviving block only its largest
//            key is a candidate unless its second largest passes too, then
//            every key of the block is; every candidate is scored exactly in
//            fp64 in index order and the best (score, lowest index) wins, so
//            the result is exact.  A query or key of norm 245 or more could
//            leave the fp16 range (2^8 |v| past 65504); then the screen
//            proves nothing and every key is scored in fp64.
#include <cmath>

#include "decide.h"
#include "precog_kernels.h"
#include "wave_ops.h"

namespace precog {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx4 __attribute__((ext_vector_type(4)));

// operands are fp16(kScale v); screen scores come back as kUnscale S
constexpr float kScale = 256.f;
constexpr float kUnscale = 1.f / 65536.f;

// features per chunk: the wave preloads its query operands for a whole chunk
// (kFC / 16 x 4 VGPRs)
constexpr int kFC = 128;
constexpr int kKS = kFC / 16; // 16-feature MFMA steps per chunk

__device__ __forceinline__ halfx4 to_op(const float4& v) {
  const floatx4 f = {v.x * kScale, v.y * kScale, v.z * kScale, v.w * kScale};
  return __builtin_convertvector(f, halfx4);
}

// prep: entry ((g * nks + ks) * 2 + h) * 32 + r holds features
// [16 ks + 8 h, 16 ks + 8 h + 8) of query 32 g + r (zero past Q or E).
__global__ __launch_bounds__(256) void prep_kernel(const RetrieveParams p) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = static_cast<int64_t>(p.nqg) * p.nks * 64;
  if (t >= total) return;
  const int r = static_cast<int>(t & 31);
  const int h = static_cast<int>((t >> 5) & 1);
  const int64_t gk = t >> 6;
  const int ks = static_cast<int>(gk % p.nks);
  const int64_t g = gk / p.nks;
  const int64_t q = g * 32 + r;
  halfx4 o[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int64_t e = 16 * ks + 8 * h + 4 * c;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (q < p.Q && e < p.E) v = *reinterpret_cast<const float4*>(p.q + q * p.E + e);
    o[c] = to_op(v);
  }
  const halfx8 o8 = {o[0][0], o[0][1], o[0][2], o[0][3], o[1][0], o[1][1], o[1][2], o[1][3]};
  reinterpret_cast<halfx8*>(p.qop)[t] = o8;
}

// screen: workgroup (kg, qg) = key blocks [kRetBlocks kg, kRetBlocks kg +
// kRetBlocks) (32 keys each) x query groups [kRetWaves qg, kRetWaves qg +
// kRetWaves) (32 queries each), wave w taking query group kRetWaves qg + w.
// Per 128-feature chunk the workgroup stages its blocks' key rows in LDS,
// rounded to fp16(2^8 k) and laid out in operand order [kb][ks][h][row],
// the row XOR-swizzled with (2 ks + h) so the staging writes and the operand
// reads hit distinct banks; every wave loads its own query operands.  The
// loads of chunk c + 1 are issued before chunk c is staged (two register
// buffers, two LDS tiles), so a chunk's memory round trip overlaps the
// previous chunk's staging and matrix work.  MFMA operands: keys are
// the rows (A), queries the columns (B); lane l supplies row / column
// l mod 32 and the 8 features of half h = l / 32 of the 16-feature step, so
// each dot product is the same whatever order the instruction consumes
// features in.  Output register r of lane l holds key row 8 (r / 4) + 4 h +
// (r mod 4) and query column l mod 32, so the 32 keys of a block for one
// query sit in the 16 registers of lanes l and l xor 32: the block's largest
// screen score, its key and the largest of the other keys are found in
// registers and one exchange between the two halves.  Per (query, block) the
// screen stores those three (block maxima, second maxima, keys), not the
// scores themselves.
template <bool PREP>
__global__ __launch_bounds__(64 * kRetWaves) void screen_kernel(const RetrieveParams p) {
  constexpr int kT = 64 * kRetWaves;        // threads
  constexpr int kRows = kKB * kRetBlocks;   // key rows per workgroup
  constexpr int kC4 = kFC / 4;              // float4 columns per row and chunk
  constexpr int kStage = kRows * kC4 / kT;  // float4 staged per thread and chunk
  constexpr int kPK = kRetBlocks * kKS * 64 / kT;  // prepared entries per thread and chunk
  static_assert(kRows * kC4 % kT == 0 && kRetBlocks * kKS * 64 % kT == 0,
                "staging must divide evenly");
  static_assert(kT % kC4 == 0, "a thread stages one column of several rows");
  const int nqwg = static_cast<int>((p.Q + 32 * kRetWaves - 1) / (32 * kRetWaves));
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int kg = lb / nqwg;
  const int qg = lb - kg * nqwg;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave-uniform, so the operand descriptors below live in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31;
  const int half = lane >> 5;
  const int64_t E = p.E;
  const int64_t k0 = static_cast<int64_t>(kg) * kRows;  // first key of the workgroup
  const int64_t qw = (static_cast<int64_t>(qg) * kRetWaves + wave) * 32;  // first query of the wave
  const bool active = qw < p.Q;
  // its 32-query group in the split layout (clamped for waves past Q, whose
  // loads stay in bounds and whose results are discarded)
  const int64_t g = active ? qw / 32 : p.nqg - 1;

  // two LDS tiles of a chunk's keys (double buffer, see below)
  __shared__ halfx8 kop[2][kRetBlocks][kKS][2][32];
  __shared__ float nsum[kRows];

  // thread t stages float4 column t mod kC4 of rows t / kC4 + (kT / kC4) j
  const int c4 = tid % kC4;
  const int srow0 = tid / kC4;
  const int64_t nrows = p.M - k0 < kRows ? p.M - k0 : kRows;  // rows past M read as zero
  const __amdgpu_buffer_rsrc_t kres =
      make_rsrc(p.K + k0 * E, static_cast<uint32_t>(nrows * E * 4));
  float n2[kStage];  // this thread's share of its rows' squared norms
#pragma unroll
  for (int j = 0; j < kStage; ++j) n2[j] = 0.f;
  // the wave's 32-query group of operands: nks entries of 1 KiB
  const uint32_t gbytes = static_cast<uint32_t>(p.nks) * 1024u;
  const __amdgpu_buffer_rsrc_t ores = make_rsrc(static_cast<const char*>(p.qop) + g * gbytes, gbytes);
  const uint32_t lane_off = static_cast<uint32_t>(lane) * 16u;

  floatx16 acc[kRetBlocks];
#pragma unroll
  for (int b = 0; b < kRetBlocks; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[b][r] = 0.f;

  // Two chunks in flight: chunk c + 1's loads (keys and query operands,
  // into the other register buffer) are issued before chunk c is staged,
  // and chunk c + 1 is staged into the other LDS tile, so one barrier per
  // chunk separates the staging from the reads.
  struct Chunk {
    halfx8 pk[PREP ? kPK : 1];
    float4 kv[PREP ? 1 : kStage];
    halfx8 aq[kKS];
  };
  auto issue = [&](Chunk& ch, int64_t fc) {
    const int nks = fc < E ? static_cast<int>((E - fc + 15) / 16 < kKS ? (E - fc + 15) / 16 : kKS) : 0;
    if constexpr (PREP) {
#pragma unroll
      for (int j = 0; j < kPK; ++j) {
        const int i = tid + kT * j;
        const int b = i / (kKS * 64);
        const int w = i - b * (kKS * 64);
        const int64_t kb = static_cast<int64_t>(kg) * kRetBlocks + b;
        if (w < nks * 64 && kb < p.nkb)
          ch.pk[j] = static_cast<const halfx8*>(p.kop)[(kb * p.nks + fc / 16) * 64 + w];
        else
          ch.pk[j] = halfx8{};
      }
    } else {
#pragma unroll
      for (int j = 0; j < kStage; ++j) {
        const int row = srow0 + (kT / kC4) * j;
        const int64_t e = fc + 4 * c4;
        const uint32_t off = e < E ? static_cast<uint32_t>((row * E + e) * 4) : kDropOffset;
        ch.kv[j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(kres, off, 0, 0));
      }
    }
#pragma unroll
    for (int i = 0; i < kKS; ++i) {
      const int64_t ks = fc / 16 + i;
      ch.aq[i] = ks < p.nks ? __builtin_bit_cast(halfx8, __builtin_amdgcn_raw_buffer_load_b128(
                                                             ores, lane_off,
                                                             static_cast<uint32_t>(ks) * 1024u, 0))
                            : halfx8{};
    }
  };
  auto consume = [&](const Chunk& ch, int64_t fc, int slot) {
    if constexpr (PREP) {
      halfx8* dst = &kop[slot][0][0][0][0];
#pragma unroll
      for (int j = 0; j < kPK; ++j) dst[tid + kT * j] = ch.pk[j];
    } else {
#pragma unroll
      for (int j = 0; j < kStage; ++j) {
        const int row = srow0 + (kT / kC4) * j;
        const float4 v = ch.kv[j];
        n2[j] = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, n2[j]))));
        const int b = row / kKB;
        const int r = row % kKB;
        const int ks = c4 >> 2;
        const int h = (c4 >> 1) & 1;
        const int sub = c4 & 1;
        const int srow = r ^ ((2 * ks + h) & 31);
        reinterpret_cast<halfx4*>(&kop[slot][b][ks][h][srow])[sub] = to_op(v);
      }
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
        if (fc + 16 * ks < E) {
          const int srow = r32 ^ ((2 * ks + half) & 31);
#pragma unroll
          for (int b = 0; b < kRetBlocks; ++b)
            acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kop[slot][b][ks][half][srow], ch.aq[ks],
                                                            acc[b], 0, 0, 0);
        }
      }
    }
  };
  Chunk ca, cb;
  issue(ca, 0);
  for (int64_t f0 = 0; f0 < E; f0 += 2 * kFC) {
    const bool second = f0 + kFC < E;
    if (second) issue(cb, f0 + kFC);
    consume(ca, f0, 0);
    if (second) {
      if (f0 + 2 * kFC < E) issue(ca, f0 + 2 * kFC);
      consume(cb, f0 + kFC, 1);
    }
  }
  if (active) {
    const int64_t q = qw + r32;
#pragma unroll
    for (int b = 0; b < kRetBlocks; ++b) {
      const int64_t kb = static_cast<int64_t>(kg) * kRetBlocks + b;
      // largest (m1, its key i1) and the largest of the other keys (m2) over
      // this lane's 16 rows; a tie with m1 goes to m2, keys past M rank last
      float m1 = -INFINITY, m2 = -INFINITY;
      int i1 = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 8 * (r >> 2) + 4 * half + (r & 3);
        const float v = kb * kKB + row < p.M ? acc[b][r] * kUnscale : -INFINITY;
        if (v > m1) {
          m2 = m1;
          m1 = v;
          i1 = row;
        } else {
          m2 = fmaxf(m2, v);
        }
      }
      // merge with the other half's (rows 4 apart in each group of 8)
      const float o1 = xor_shfl(m1, 32);
      const float o2 = xor_shfl(m2, 32);
      const int oi = __builtin_bit_cast(int, xor_shfl(__builtin_bit_cast(float, i1), 32));
      const bool mine = m1 > o1 || (m1 == o1 && i1 < oi);
      const float s1 = mine ? m1 : o1;
      const float s2 = mine ? fmaxf(m2, o1) : fmaxf(o2, m1);
      const int si = mine ? i1 : oi;
      if (half == 0 && q < p.Q && kb < p.nkb) {
        p.blockmax[q * p.nkb + kb] = s1;
        p.blocksec[q * p.nkb + kb] = s2;
        p.blockarg[q * p.nkb + kb] = static_cast<uint8_t>(si);
      }
    }
  }
  // squared key norms (workgroups with qg == 0; a prepared index holds
  // them): the kC4 threads staging a row hold disjoint parts of it, adjacent
  // lanes of one wave; combined in a fixed order
  if (!PREP && qg == 0) {
#pragma unroll
    for (int j = 0; j < kStage; ++j) {
      float v = n2[j];
#pragma unroll
      for (int m = 1; m < kC4; m <<= 1) v += xor_shfl(v, m);
      if (c4 == 0) nsum[srow0 + (kT / kC4) * j] = v;
    }
    __syncthreads();
    if (tid < kRows) {
      const int64_t key = k0 + tid;
      if (key < p.M) p.rownorm2[key] = nsum[tid];
    }
    if (tid < kRetBlocks * kKB) {
      const int64_t kb = static_cast<int64_t>(kg) * kRetBlocks + tid / kKB;
      float mx = k0 + tid < p.M ? nsum[tid] : 0.f;
      mx = fmaxf(mx, xor_shfl(mx, 1));
      mx = fmaxf(mx, xor_shfl(mx, 2));
      mx = fmaxf(mx, xor_shfl(mx, 4));
      mx = fmaxf(mx, xor_shfl(mx, 8));
      mx = fmaxf(mx, xor_shfl(mx, 16));
      if ((tid & 31) == 0 && kb < p.nkb) p.blocknorm2[kb] = mx;
    }
  }
}

// the rank order: larger score first, then lower index
// Prepared index, operands: entry ((kb * nks + ks) * 2 + h) * 32 + r' holds
// features [16 ks + 8 h, 16 ks + 8 h + 8) of key 32 kb + r as fp16(2^8 k)
// (zero past M or E), at r' = r xor ((2 (ks mod kKS) + h) mod 32): the order
// and swizzle of the screen's LDS tile, so a chunk's tile is one contiguous
// copy.
__global__ __launch_bounds__(256) void prep_index_kernel(const RetrieveParams p) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t total = static_cast<int64_t>(p.nkb) * p.nks * 64;
  if (t >= total) return;
  const int r = static_cast<int>(t & 31);
  const int h = static_cast<int>((t >> 5) & 1);
  const int64_t bk = t >> 6;
  const int ks = static_cast<int>(bk % p.nks);
  const int64_t kb = bk / p.nks;
  const int64_t key = kb * kKB + r;
  halfx4 o[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int64_t e = 16 * ks + 8 * h + 4 * c;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (key < p.M && e < p.E) v = *reinterpret_cast<const float4*>(p.K + key * p.E + e);
    o[c] = to_op(v);
  }
  const int rs = r ^ ((2 * (ks % kKS) + h) & 31);
  const halfx8 o8 = {o[0][0], o[0][1], o[0][2], o[0][3], o[1][0], o[1][1], o[1][2], o[1][3]};
  static_cast<halfx8*>(const_cast<void*>(p.kop))[(bk * 2 + h) * 32 + rs] = o8;
}

// Prepared index, norms: one wave per 32-key block; lane l < 32 sums the
// squares of key 32 kb + l, the block keeps the largest.
__global__ __launch_bounds__(64) void prep_norms_kernel(const RetrieveParams p) {
  const int64_t kb = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t key = kb * kKB + (lane & 31);
  const bool ok = lane < kKB && key < p.M;
  float n2 = 0.f;
  if (ok) {
    const float4* row = reinterpret_cast<const float4*>(p.K + key * p.E);
    for (int64_t e4 = 0; e4 < p.E / 4; ++e4) {
      const float4 v = row[e4];
      n2 = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, n2))));
    }
    p.rownorm2[key] = n2;
  }
  float mx = ok ? n2 : 0.f;
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) mx = fmaxf(mx, xor_shfl(mx, m));
  if (lane == 0) p.blocknorm2[kb] = mx;
}

// FL: row loads in flight when a whole block is rescored.  Top-1 keeps 16
// (24 took its decision from 7.1 to 7.5 us: more registers on its short
// path); top-k, which rescores whole blocks more often, takes 24.
template <int FL>
__global__ __launch_bounds__(64) void decide_kernel(const RetrieveParams p) {
  __shared__ DecideShared sh;
  decide_query<FL>(p, blockIdx.x, sh);
}

}  // namespace

// The constants of the decide's error bounds, from E alone.
// Screen scores: each operand value w = fp16(2^8 v) / 2^8 has |w - v| <=
// a |v| + bs with a = 2^-11 (round to nearest in the fp16 normal range) and
// bs = 2^-22 (below it, whether rounded to a subnormal or flushed to zero).
// So |q~ k~ - q k| <= (2a + a^2) |q k| + bs (1 + a) (|q| + |k|) + bs^2 per
// feature; summed with Cauchy-Schwarz for the products and |v|_1 <= sqrt(E)
// |v| for the 1-norms.  The fp32 sum of the E exact products adds at most
// 2 gamma_E times their absolute sum (twice the round-to-nearest bound, so
// additions that truncate, or align the products of one instruction to the
// largest, are covered too); the 2^-16 scale back is exact (or below
// 2^-149).  The factor 1.01 covers the fp32 norms (relative error
// ~gamma_E) and 1e-12 the fp64 reference's own rounding.  A norm past
// kMaxNorm2 could overflow fp16 (2^8 |v| >= 65520): then every key is
// scored exactly.
// Lane-parallel fp64 sums (top-1 fast ordering): a sum of E / 64 features
// per lane followed by a 6-level tree is within gamma_{E/64+7} sum |p_e| of
// the exact sum, the sequential sum of the definition within gamma_E
// sum |p_e|; err_gs bounds both together per unit of |q| |k| (1.01 for the
// fp32 norms).
static void error_bound_constants(RetrieveParams& p) {
  const double u = 5.9604644775390625e-08;  // 2^-24
  const double a = 4.8828125e-04;           // 2^-11
  const double bs = 2.384185791015625e-07;  // 2^-22
  const double en = static_cast<double>(p.E);
  const double gam2 = 2.0 * (en * u) / (1.0 - en * u);
  p.err_g = 1.01 * (2.0 * a + a * a + gam2 * (1.0 + 2.0 * a + a * a)) + 1e-12;
  p.err_h = 1.01 * (1.0 + gam2) * bs * (1.0 + a) * std::sqrt(en);
  p.err_tiny = 1.01 * (1.0 + gam2) * en * bs * bs + 1e-30;
  const double u53 = 1.1102230246251565e-16;  // 2^-53
  const double nf = static_cast<double>(p.E / 64 + 7);
  p.err_gs = 1.01 * (nf * u53 / (1.0 - nf * u53) + en * u53 / (1.0 - en * u53));
}

hipError_t launch_retrieve_screen(RetrieveParams& p, hipStream_t s) {
  error_bound_constants(p);
  if (p.nkb > 0) {
    const int64_t entries = static_cast<int64_t>(p.nqg) * p.nks * 64;
    hipLaunchKernelGGL(prep_kernel, dim3(static_cast<unsigned>((entries + 255) / 256)), dim3(256), 0, s, p);
    const int64_t nqwg = (p.Q + 32 * kRetWaves - 1) / (32 * kRetWaves);
    const int64_t nkbg = (p.nkb + kRetBlocks - 1) / kRetBlocks;
    const dim3 grid(static_cast<unsigned>(nkbg * nqwg));
    if (p.kop != nullptr)
      hipLaunchKernelGGL(screen_kernel<true>, grid, dim3(64 * kRetWaves), 0, s, p);
    else
      hipLaunchKernelGGL(screen_kernel<false>, grid, dim3(64 * kRetWaves), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_retrieve_decide(const RetrieveParams& p, hipStream_t s) {
  if (p.k == 1)
    hipLaunchKernelGGL(decide_kernel<16>, dim3(static_cast<unsigned>(p.Q)), dim3(64), 0, s, p);
  else
    hipLaunchKernelGGL(decide_kernel<24>, dim3(static_cast<unsigned>(p.Q)), dim3(64), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_retrieve(const RetrieveParams& pin, hipStream_t s) {
  RetrieveParams p = pin;
  const hipError_t e = launch_retrieve_screen(p, s);
  if (e != hipSuccess) return e;
  return launch_retrieve_decide(p, s);
}

hipError_t launch_retrieve_prepare(const RetrieveParams& p, hipStream_t s) {
  const int64_t entries = static_cast<int64_t>(p.nkb) * p.nks * 64;
  hipLaunchKernelGGL(prep_index_kernel, dim3(static_cast<unsigned>((entries + 255) / 256)), dim3(256), 0, s, p);
  hipLaunchKernelGGL(prep_norms_kernel, dim3(static_cast<unsigned>(p.nkb)), dim3(64), 0, s, p);
  return hipGetLastError();
}

}  // namespace precog
