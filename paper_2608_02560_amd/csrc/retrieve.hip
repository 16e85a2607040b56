// Exact cosine top-1 retrieval for gfx950 (query time, Sec. 4.2).
//
// The answer is defined in fp64: score(q, i) = sum_e q_e k_{i,e} summed in
// index order (products of fp32 values are exact in fp64), idx = the lowest i
// attaining the maximum.  Three kernels reach it exactly:
//
//   prep     splits every query value v into hi = bf16(v) and lo = bf16(v - hi)
//            (round to nearest even; v - hi is exact in fp32) and stores them
//            in the order the matrix-core operands are consumed, so a wave's
//            operand load is one contiguous 1 KiB segment.
//   screen   workgroup = 32 keys x 128 queries: the keys are read
//            row-contiguously, split the same way and staged in LDS; each wave
//            computes a 32 x 32 tile with v_mfma_f32_32x32x16_bf16, summing
//            q_hi k_hi + q_hi k_lo + q_lo k_hi in fp32 (each product exact).
//            It stores every screen score S~_i, the maximum of each
//            (query, 32-key block), and the squared norm of every key and the
//            largest one of every block.
//   decide   one wave per query: m = the largest screen score.  A key can
//            still be the fp64 maximum only if S~_i + e(i) >= m - e(i0), where
//            e(i) = g |q| |k_i| + tiny bounds the error of its screen score
//            (g bounds the split error and the fp32 accumulation of the
//            screen per unit of sum |q_e k_e|, which Cauchy-Schwarz bounds
//            by |q| |k_i|; it is inflated for the fp32 norms, rounding inside
//            the matrix core, and the fp64 rounding of the reference).  Blocks
//            are tested first with their maxima and norm bounds, then the keys
//            of surviving blocks one by one; every candidate is scored exactly
//            in fp64 in index order and the best (score, lowest index) wins,
//            so the result is exact.
#include "precog_kernels.h"

namespace precog {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kKB = 32;       // keys per block (screen workgroup, block maxima)
constexpr int kQW = 32;       // queries per wave (one 32 x 32 tile)
constexpr int kQWG = 4 * kQW; // queries per workgroup
// features per chunk: the wave preloads its query operands for a whole chunk
// (2 x kFC / 16 x 4 VGPRs); 128 leaves room for three waves per SIMD
#ifndef PRECOG_RET_FC
#define PRECOG_RET_FC 128
#endif
constexpr int kFC = PRECOG_RET_FC;
constexpr int kKS = kFC / 16; // 16-feature MFMA steps per chunk

__device__ __forceinline__ float xor_shfl(float v, int m) {
  const int src = (static_cast<int>(threadIdx.x & 63) ^ m) * 4;
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, v)));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += xor_shfl(v, m);
  return v;
}

__device__ __forceinline__ void split4(const float4& v, bf16x4& hi, bf16x4& lo) {
  const floatx4 f = {v.x, v.y, v.z, v.w};
  hi = __builtin_convertvector(f, bf16x4);
  lo = __builtin_convertvector(f - __builtin_convertvector(hi, floatx4), bf16x4);
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
  bf16x4 hi[2], lo[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int64_t e = 16 * ks + 8 * h + 4 * c;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (q < p.Q && e < p.E) v = *reinterpret_cast<const float4*>(p.q + q * p.E + e);
    split4(v, hi[c], lo[c]);
  }
  const bf16x8 h8 = {hi[0][0], hi[0][1], hi[0][2], hi[0][3], hi[1][0], hi[1][1], hi[1][2], hi[1][3]};
  const bf16x8 l8 = {lo[0][0], lo[0][1], lo[0][2], lo[0][3], lo[1][0], lo[1][1], lo[1][2], lo[1][3]};
  reinterpret_cast<bf16x8*>(p.qhi)[t] = h8;
  reinterpret_cast<bf16x8*>(p.qlo)[t] = l8;
}

// screen: workgroup (kb, qg) = key block kb (keys 32 kb + 0..31) x queries
// [128 qg, 128 qg + 128), wave w taking 32 of them.  Per feature chunk the
// workgroup loads the block's key rows row-contiguously and every wave its
// query operands, all before the first wait (one memory latency per chunk);
// the keys are split and stored in LDS in operand order
// [ks][h][row], the row index XOR-swizzled with (2 ks + h) so both the
// staging writes and the operand reads hit distinct banks.  MFMA operands:
// lane l supplies row / column l mod 32 and the 8 features of half
// h = l / 32 of the 16-feature step, for queries and keys alike, so each dot
// product is unchanged whatever order the instruction consumes features in.
// Output register r holds query row 8 (r / 4) + 4 h + (r mod 4), key column
// l mod 32; screen scores are stored as 128-byte runs of 32 keys.
__global__ __launch_bounds__(256) void screen_kernel(const RetrieveParams p) {
  const int nqwg = static_cast<int>((p.Q + kQWG - 1) / kQWG);
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int kb = lb / nqwg;
  const int qg = lb - kb * nqwg;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave-uniform, so the operand descriptors below live in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r32 = lane & 31;
  const int half = lane >> 5;
  const int64_t E = p.E;
  const int64_t k0 = static_cast<int64_t>(kb) * kKB;
  const int64_t qw = static_cast<int64_t>(qg) * kQWG + wave * kQW;  // first query of the wave
  const bool active = qw < p.Q;
  // its 32-query group in the split layout (clamped for waves past Q, whose
  // loads stay in bounds and whose results are discarded)
  const int64_t g = active ? qw / 32 : p.nqg - 1;

  // double-buffered: chunk c is staged in buffer c mod 2, so one barrier per
  // chunk separates the staging of c from the reads of c - 1 and c - 2
  __shared__ bf16x8 khi[2][kKS][2][32];
  __shared__ bf16x8 klo[2][kKS][2][32];
  __shared__ float nsum[2][kKB];

  const int srow_base = (tid >> 2) & 31;  // key row this thread stages
  // the block's rows through a descriptor: rows past M read as zero
  const int64_t nrows = p.M - k0 < kKB ? p.M - k0 : kKB;
  const __amdgpu_buffer_rsrc_t kres =
      make_rsrc(p.K + k0 * E, static_cast<uint32_t>(nrows * E * 4));
  const uint32_t krow_off = static_cast<uint32_t>(srow_base * E * 4);
  float n2 = 0.f;                         // its share of that row's squared norm
  // the wave's 32-query group of split operands: nks entries of 1 KiB
  const uint32_t gbytes = static_cast<uint32_t>(p.nks) * 1024u;
  const __amdgpu_buffer_rsrc_t hres = make_rsrc(static_cast<const char*>(p.qhi) + g * gbytes, gbytes);
  const __amdgpu_buffer_rsrc_t lres = make_rsrc(static_cast<const char*>(p.qlo) + g * gbytes, gbytes);
  const uint32_t lane_off = static_cast<uint32_t>(lane) * 16u;

  floatx16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;

  int buf = 0;
  for (int64_t fc = 0; fc < E; fc += kFC, buf ^= 1) {
    const int nks = static_cast<int>((E - fc + 15) / 16 < kKS ? (E - fc + 15) / 16 : kKS);
    const uint32_t ks0 = static_cast<uint32_t>(fc / 16);
    // issue every load of the chunk before waiting on any: the key float4s
    // (thread t takes row (t / 4) mod 32 and the float4 columns
    // t mod 4 + 4 (t / 128) + 8 j, so four lanes read 64 contiguous bytes
    // of a row and the wave covers 16 rows per load), then the wave's query
    // operands (entries past the group's nks read as zero)
    float4 kv[kFC / 32];
#pragma unroll
    for (int j = 0; j < kFC / 32; ++j) {
      const int c4 = (tid & 3) + 4 * (tid >> 7) + 8 * j;
      const int64_t e = fc + 4 * c4;
      const uint32_t off = e < E ? krow_off + static_cast<uint32_t>(e * 4) : kDropOffset;
      kv[j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(kres, off, 0, 0));
    }
    bf16x8 ah[kKS], al[kKS];
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) {
      const uint32_t so = (ks0 + ks) * 1024u;
      ah[ks] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(hres, lane_off, so, 0));
      al[ks] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(lres, lane_off, so, 0));
    }
#pragma unroll
    for (int j = 0; j < kFC / 32; ++j) {
      const int c4 = (tid & 3) + 4 * (tid >> 7) + 8 * j;
      const float4 v = kv[j];
      n2 = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, n2))));
      bf16x4 hi, lo;
      split4(v, hi, lo);
      const int ks = c4 >> 2;
      const int h = (c4 >> 1) & 1;
      const int sub = c4 & 1;
      const int srow = srow_base ^ ((2 * ks + h) & 31);
      reinterpret_cast<bf16x4*>(&khi[buf][ks][h][srow])[sub] = hi;
      reinterpret_cast<bf16x4*>(&klo[buf][ks][h][srow])[sub] = lo;
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
        if (ks < nks) {
          const int srow = r32 ^ ((2 * ks + half) & 31);
          const bf16x8 bh = khi[buf][ks][half][srow];
          const bf16x8 bl = klo[buf][ks][half][srow];
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[ks], bh, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[ks], bl, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[ks], bh, acc, 0, 0, 0);
        }
      }
    }
  }
  if (active) {
    const int64_t key = k0 + r32;
    const bool key_ok = key < p.M;
    float mx[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t q = qw + 8 * (r >> 2) + 4 * half + (r & 3);
      if (q < p.Q && key_ok) p.scores[q * p.ld_scores + key] = acc[r];
      mx[r] = key_ok ? acc[r] : -INFINITY;
    }
    // maximum over the 32 keys (lanes) of each half-wave, step-major so the
    // 16 shuffles of a step are in flight together
#pragma unroll
    for (int m = 1; m < 32; m <<= 1) {
      float t[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) t[r] = xor_shfl(mx[r], m);
#pragma unroll
      for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], t[r]);
    }
    if (r32 == 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t q = qw + 8 * (r >> 2) + 4 * half + (r & 3);
        if (q < p.Q) p.blockmax[q * p.nkb + kb] = mx[r];
      }
    }
  }
  // squared key norms (workgroups with qg == 0): the eight threads staging
  // a row hold disjoint parts of it; combined in a fixed order
  if (qg == 0) {
    n2 += xor_shfl(n2, 1);
    n2 += xor_shfl(n2, 2);
    if ((tid & 3) == 0) nsum[tid >> 7][srow_base] = n2;
    __syncthreads();
    if (tid < kKB) {
      const float r2 = nsum[0][tid] + nsum[1][tid];
      const bool ok = k0 + tid < p.M;
      if (ok) p.rownorm2[k0 + tid] = r2;
      float mx = ok ? r2 : 0.f;
      mx = fmaxf(mx, xor_shfl(mx, 1));
      mx = fmaxf(mx, xor_shfl(mx, 2));
      mx = fmaxf(mx, xor_shfl(mx, 4));
      mx = fmaxf(mx, xor_shfl(mx, 8));
      mx = fmaxf(mx, xor_shfl(mx, 16));
      if (tid == 0) p.blocknorm2[kb] = mx;
    }
  }
}

__device__ __forceinline__ bool better(double s, int64_t i, double bs, int64_t bi) {
  return bi < 0 || s > bs || (s == bs && i < bi);
}

constexpr int kMaxE = 4096;

__device__ __forceinline__ double shfl_d(double v, int src_lane) {
  const int lo = __builtin_amdgcn_ds_bpermute(src_lane * 4, static_cast<int>(__double2loint(v)));
  const int hi = __builtin_amdgcn_ds_bpermute(src_lane * 4, static_cast<int>(__double2hiint(v)));
  return __hiloint2double(hi, lo);
}

__device__ __forceinline__ int shfl_i(int v, int src_lane) {
  return __builtin_amdgcn_ds_bpermute(src_lane * 4, v);
}

// (value, index) order of the block-maximum pass: larger value first, then
// lower index.  NaN values are never ranked.
__device__ __forceinline__ bool before(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

constexpr int kCand = 64;             // candidate list capacity (indices)
constexpr int kRowWords = 8192;       // LDS words for staged candidate rows

// decide: one 64-lane workgroup per query (see the file comment).  For the
// k best keys the bound uses t_k, the k-th largest block maximum: k distinct
// blocks hold a key with screen score >= t_k, so k keys have exact scores
// >= t_k - e_max and every key of the exact top k has S~_i + e(i) >= that.
// (k = 1: t_1 = m.)  Blocks are discarded with their maxima and norm bounds,
// then keys one by one; surviving keys are collected in an LDS list and
// scored exactly in batches: the wave stages a batch of rows in LDS (row
// pitch E + 4 words, 16-byte aligned)
// and lane j sums row j in fp64 in feature order (fma equals
// multiply-then-add here: the product of two fp32 values is exact in fp64),
// so the chains of a batch run side by side.  Scores enter a rank list
// spread over the lanes (lane j holds rank j), ordered by score, then by
// lower index; the order of insertion does not change the list.
__global__ __launch_bounds__(64) void decide_kernel(const RetrieveParams p) {
  const int64_t q = blockIdx.x;
  const int lane = threadIdx.x;
  const int E = static_cast<int>(p.E);
  const int nkb = p.nkb;
  const int k = p.k;
  __shared__ __attribute__((aligned(16))) float qs[kMaxE];
  __shared__ __attribute__((aligned(16))) float rs[kRowWords];
  __shared__ int cand[kCand];
  const float4* qg4 = reinterpret_cast<const float4*>(p.q + q * p.E);
  const float* bm = p.blockmax + q * nkb;
  const float* sc = p.scores + q * p.ld_scores;

  float nq = 0.f;
#pragma unroll 4
  for (int e4 = lane; e4 < E / 4; e4 += 64) {
    const float4 v = qg4[e4];
    *reinterpret_cast<float4*>(qs + 4 * e4) = v;
    nq = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, nq))));
  }
  const float qnorm = sqrtf(wave_sum(nq));

  // t_k: k rounds, each taking the first (value, index) pair after the
  // previous one (the first round also takes the largest block norm); fewer
  // than k ranked blocks leave t_k = -inf (every key is then a candidate)
  float nmax = 0.f;
  float tv = INFINITY;
  int ti = -1;
  bool found = true;
  for (int r = 0; r < k && found; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    bool any = false;
    for (int kb0 = 0; kb0 < nkb; kb0 += 256) {
      float b[4], n[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kb = kb0 + 64 * j + lane;
        b[j] = kb < nkb ? bm[kb] : __builtin_nanf("");
        n[j] = (r == 0 && kb < nkb) ? p.blocknorm2[kb] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kb = kb0 + 64 * j + lane;
        nmax = fmaxf(nmax, n[j]);
        if (before(tv, ti, b[j], kb) && (!any || before(b[j], kb, bv, bi))) {
          bv = b[j];
          bi = kb;
          any = true;
        }
      }
    }
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
      const float ov = xor_shfl(bv, s);
      const int oi = __builtin_amdgcn_ds_bpermute((lane ^ s) * 4, bi);
      const bool oany = __builtin_amdgcn_ds_bpermute((lane ^ s) * 4, static_cast<int>(any)) != 0;
      if (oany && (!any || before(ov, oi, bv, bi))) {
        bv = ov;
        bi = oi;
        any = true;
      }
    }
    found = any;
    if (any) {
      tv = bv;
      ti = bi;
    }
  }
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) nmax = fmaxf(nmax, xor_shfl(nmax, s));
  const float tk = found ? tv : -INFINITY;

  // Screen-score error bound per unit of |q| |k_i|: dropped split terms
  // q_lo k_lo + (q_hi + q_lo) dk + dq k <= 3.05 * 2^-16 (bf16 rounding 2^-8
  // relative, twice), plus fp32 accumulation of 3E exact products, gamma_3E
  // (with 1.008 for |hi| + |lo| > |v|); doubled for any rounding the matrix
  // core performs inside one instruction, the fp32 norms and the fp64
  // reference's own rounding.
  const double u = 5.9604644775390625e-08;  // 2^-24
  const double n3 = 3.0 * static_cast<double>(E);
  const double gam = (n3 * u) / (1.0 - n3 * u);
  const double g = 2.0 * (1.008 * gam + 3.05 * 1.52587890625e-05) + 1e-12;
  const double tiny = 1e-30;
  const double gq = g * static_cast<double>(qnorm);
  const double thresh = static_cast<double>(tk) - (gq * sqrt(static_cast<double>(nmax)) + tiny);

  // rank list: lane j < k holds the j-th best (score, index) so far
  double ls = -INFINITY;
  int64_t li = -1;
  auto insert = [&](double s, int64_t ii) {
    const bool ahead = lane < k && li >= 0 && better(ls, li, s, ii);
    const int pos = __builtin_popcountll(__ballot(ahead));
    if (pos < k) {
      const double ps = shfl_d(ls, lane > 0 ? lane - 1 : 0);
      const int pil = shfl_i(static_cast<int>(li), lane > 0 ? lane - 1 : 0);
      if (lane > pos) {
        ls = ps;
        li = pil;
      } else if (lane == pos) {
        ls = s;
        li = ii;
      }
    }
  };

  // exact scores of the listed candidates, a batch of rows at a time
  const int pitch = E + 4;  // E is a multiple of 4: rows stay 16-byte aligned
  const int batch_max = kRowWords / pitch < 64 ? kRowWords / pitch : 64;
  int ncand = 0;
  auto flush = [&]() {
    for (int c0 = 0; c0 < ncand; c0 += batch_max) {
      const int nb = ncand - c0 < batch_max ? ncand - c0 : batch_max;
      __syncthreads();  // previous batch consumed, list and qs complete
      // one flat (row, float4) space, so the loads of several rows are in
      // flight together
      const int e4n = E / 4;
#pragma unroll 8
      for (int f = lane; f < nb * e4n; f += 64) {
        const int r = f / e4n;
        const int e4 = f - r * e4n;
        const float4 v =
            reinterpret_cast<const float4*>(p.K + static_cast<int64_t>(cand[c0 + r]) * p.E)[e4];
        *reinterpret_cast<float4*>(rs + r * pitch + 4 * e4) = v;
      }
      __syncthreads();
      // the chain stays one fma per feature in feature order; reading four
      // features per 16-byte LDS access (the query's a broadcast) and
      // unrolling lets the reads run ahead of the dependent fp64 chain
      double s = 0.0;
      if (lane < nb) {
        const float* row = rs + lane * pitch;
#pragma unroll 4
        for (int e = 0; e < E; e += 4) {
          const float4 qv = *reinterpret_cast<const float4*>(qs + e);
          const float4 rv = *reinterpret_cast<const float4*>(row + e);
          s = fma(static_cast<double>(qv.x), static_cast<double>(rv.x), s);
          s = fma(static_cast<double>(qv.y), static_cast<double>(rv.y), s);
          s = fma(static_cast<double>(qv.z), static_cast<double>(rv.z), s);
          s = fma(static_cast<double>(qv.w), static_cast<double>(rv.w), s);
        }
      }
      for (int r = 0; r < nb; ++r) {
        const int lo = __builtin_amdgcn_ds_bpermute(r * 4, static_cast<int>(__double2loint(s)));
        const int hi = __builtin_amdgcn_ds_bpermute(r * 4, static_cast<int>(__double2hiint(s)));
        insert(__hiloint2double(hi, lo), cand[c0 + r]);
      }
    }
    ncand = 0;
  };

  for (int kb0 = 0; kb0 < nkb; kb0 += 256) {
    uint64_t bmask[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kb = kb0 + 64 * j + lane;
      float b = -INFINITY, n = 0.f;
      if (kb < nkb) {
        b = bm[kb];
        n = p.blocknorm2[kb];
      }
      const bool pass = kb < nkb && static_cast<double>(b) + gq * sqrt(static_cast<double>(n)) + tiny >= thresh;
      bmask[j] = __ballot(pass);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      while (bmask[j]) {
        const int blk = kb0 + 64 * j + __builtin_ctzll(bmask[j]);
        bmask[j] &= bmask[j] - 1;
        const int64_t i = static_cast<int64_t>(blk) * kKB + (lane & (kKB - 1));
        bool cand_ok = false;
        if (lane < kKB && i < p.M)
          cand_ok = static_cast<double>(sc[i]) + gq * sqrt(static_cast<double>(p.rownorm2[i])) + tiny >= thresh;
        const uint64_t cmask = __ballot(cand_ok);
        if (!cmask) continue;
        if (ncand + kKB > kCand) flush();
        if (cand_ok) cand[ncand + __builtin_popcountll(cmask & ((1ull << lane) - 1))] = static_cast<int>(i);
        ncand += __builtin_popcountll(cmask);
      }
    }
  }
  flush();
  if (lane < k) {
    p.idx[q * k + lane] = static_cast<int32_t>(li);
    if (p.score) p.score[q * k + lane] = ls;
  }
}

}  // namespace

hipError_t launch_retrieve(const RetrieveParams& p, hipStream_t s) {
  if (p.nkb > 0) {
    const int64_t entries = static_cast<int64_t>(p.nqg) * p.nks * 64;
    hipLaunchKernelGGL(prep_kernel, dim3(static_cast<unsigned>((entries + 255) / 256)), dim3(256), 0, s, p);
    const int64_t nqwg = (p.Q + kQWG - 1) / kQWG;
    hipLaunchKernelGGL(screen_kernel, dim3(static_cast<unsigned>(p.nkb * nqwg)), dim3(256), 0, s, p);
  }
  hipLaunchKernelGGL(decide_kernel, dim3(static_cast<unsigned>(p.Q)), dim3(64), 0, s, p);
  return hipGetLastError();
}

}  // namespace precog
