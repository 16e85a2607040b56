// Selective-SSM scan with the diagonal complex A of Sec. 3, A = a + i w
// (a > 0 in this sign convention, the paper's w_k = pi k being one choice):
//   h_t[n] = exp(-dt_t (a[n] + i w[n])) h_{t-1}[n] + B_t[n] x_t dt_t
//   y_t    = (sum_n C_t[n] Re h_t[n] + Dskip x_t) * silu(z_t)
// with the complex state kept as (real, imaginary) fp32 pairs in VGPRs and
// stored interleaved.
//
// Same work decomposition as the real scan (one lane per (b, d) channel, 64
// adjacent channels per wave, buffer loads, B_t / C_t reaching every lane as
// DPP row_newbcast operands).  Per (t, d, n): exp2 of dt a' for the
// magnitude; the angle dt w / (2 pi) in revolutions, reduced to [0, 1) by
// v_fract_f32, then v_cos_f32 / v_sin_f32 (which take revolutions); then the
// complex multiply-add
//   re' = c re + s im + B u,   im' = c im - s re,   (c, s) = |decay| (cos, sin).
//
// Long sequences over few channels are cut into time chunks as in the real
// scan (two levels):
//   pass 1 (summary): each chunk but the last is scanned from a zero state;
//          its complex end state and its sum of dt go to the workspace;
//   pass 2 (carry):   per (b, d, n), H_c = exp(-S_{c-1} (a + i w)) H_{c-1}
//          + s_{c-1}, sequential over chunks: the composition of the affine
//          maps h -> r h + s that each chunk applies, whose factor is the
//          product of its tokens' decays, exp(-(a + i w) sum dt);
//   pass 3 (replay):  each chunk is rescanned from its carried-in state,
//          producing y and, for the last chunk, hT.
#include "scan_kernels.h"

namespace precog {
namespace {

constexpr float kInv2Pi = 0.15915494309189535f;

template <int N, int... m>
__device__ __forceinline__ void ctoken(float (&hr)[N], float (&hi)[N], const float (&a2)[N],
                                       const float (&w1)[N], float dtv, float u, float bv,
                                       std::integer_sequence<int, m...>) {
  ((void)[&] {
    const float mag = __builtin_amdgcn_exp2f(dtv * a2[m]);
    const float rev = __builtin_amdgcn_fractf(dtv * w1[m]);
    const float c = mag * __builtin_amdgcn_cosf(rev);
    const float s = mag * __builtin_amdgcn_sinf(rev);
    const float re = hr[m];
    hr[m] = fmaf(c, re, fmaf(s, hi[m], u * row_bcast<m>(bv)));
    hi[m] = fmaf(c, hi[m], -(s * re));
  }(), ...);
}

template <int N, typename TSt>
__device__ __forceinline__ void load_cstate(float (&hr)[N], float (&hi)[N], const TSt* src) {
#pragma unroll
  for (int n = 0; n < N; ++n) {
    hr[n] = to_f32(src[2 * n]);
    hi[n] = to_f32(src[2 * n + 1]);
  }
}

template <int N, typename TSt>
__device__ __forceinline__ void store_cstate(TSt* dst, const float (&hr)[N], const float (&hi)[N]) {
  float v[2 * N];
#pragma unroll
  for (int n = 0; n < N; ++n) {
    v[2 * n] = hr[n];
    v[2 * n + 1] = hi[n];
  }
  store_state_vec<2 * N>(dst, v);
}

// One lane = one (b, d) channel over one time chunk.  HASZ: gate present.
//   KIND == kReadout:   y and (last chunk) hT
//   KIND == kStateOnly: hT only (y == NULL: C, z, Dskip unread)
//   KIND == kSummary:   chunk end state from zero -> carry slot c+1, sum dt
template <int N, typename TIn, typename TOut, typename TSt, int KIND, bool HASZ>
__global__ __launch_bounds__(kSBlock) void scan_complex_kernel(
    const TIn* __restrict__ xg, const TIn* __restrict__ dtg, const TIn* __restrict__ zg,
    const TIn* __restrict__ Bg, const TIn* __restrict__ Cg, TOut* __restrict__ yg,
    const ScanParams p) {
  constexpr int kPer = N < 16 ? N : 16;
  constexpr bool kRead = KIND == kReadout;
  const int lb = xcd_remap(blockIdx.x, gridDim.x);
  const int dblk = lb % p.dblocks;
  const int rest = lb / p.dblocks;
  const int b = rest % static_cast<int>(p.B);
  const int c = rest / static_cast<int>(p.B);
  const int64_t D = p.D;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t wave_d0 = static_cast<int64_t>(dblk) * kSBlock + wave * 64;
  // progress balancing between the two waves of a SIMD (scan_kernels.h)
  const bool fair = balance_enabled(p);
  __shared__ int progress[kSWaves];
  if (fair) balance_init(progress, wave);  // uniform over the workgroup
  if (wave_d0 >= D) return;
  const int64_t dtrue = wave_d0 + lane;
  const bool live = dtrue < D;
  const int64_t d = live ? dtrue : D - 1;

  const int64_t t0 = static_cast<int64_t>(c) * p.chunk;
  const int64_t t1 = min(p.L, t0 + p.chunk);
  const int nsteps = static_cast<int>(t1 > t0 ? t1 - t0 : 0);

  float a2[N], w1[N];
  load_state<N>(a2, p.A + d * N);
  load_state<N>(w1, p.A_im + d * N);
#pragma unroll
  for (int n = 0; n < N; ++n) {
    a2[n] *= -kLog2e;
    w1[n] *= kInv2Pi;
  }
  // carry slots hold (re, im) pairs: [B, C, D, N, 2]
  const int64_t DN2 = 2 * D * N;
  float hr[N], hi[N];
  if constexpr (KIND == kSummary) {
#pragma unroll
    for (int n = 0; n < N; ++n) hr[n] = hi[n] = 0.f;
  } else if (p.nchunks > 1) {
    load_cstate<N>(hr, hi, p.carry + (static_cast<int64_t>(b) * p.nchunks + c) * DN2 + 2 * d * N);
  } else if (p.flags & kHasH0) {
    load_cstate<N>(hr, hi, static_cast<const TSt*>(p.h0) + b * p.h0_stride + 2 * d * N);
  } else {
#pragma unroll
    for (int n = 0; n < N; ++n) hr[n] = hi[n] = 0.f;
  }
  const float dsk = (kRead && (p.flags & kHasD)) ? p.Dskip[d] : 0.f;

  // descriptors over this chunk's rows of x, dt, z, y ([nsteps, D]) and B, C
  // ([nsteps, N]); lane offsets in bytes
  using SI = Stream<TIn>;
  using SO = Stream<TOut>;
  const int64_t row0 = static_cast<int64_t>(b) * p.L + t0;
  const uint32_t in_row = static_cast<uint32_t>(D * sizeof(TIn));
  const uint32_t out_row = static_cast<uint32_t>(D * sizeof(TOut));
  const uint32_t bc_row = static_cast<uint32_t>(N * sizeof(TIn));
  const uint32_t ns = static_cast<uint32_t>(nsteps > 0 ? nsteps : 1);
  const auto rx = make_rsrc(xg + row0 * D, ns * in_row);
  const auto rd = make_rsrc(dtg + row0 * D, ns * in_row);
  const auto rz = make_rsrc(zg + row0 * D, ns * in_row);
  const auto rb = make_rsrc(Bg + row0 * N, ns * bc_row);
  const auto rc = make_rsrc(Cg + row0 * N, ns * bc_row);
  const auto ry = make_rsrc(yg + row0 * D, ns * out_row);
  const uint32_t dl = static_cast<uint32_t>(d) * sizeof(TIn);
  const uint32_t dly = live ? static_cast<uint32_t>(d) * sizeof(TOut) : kDropOffset;
  const int lane16 = lane & 15;
  const uint32_t el = static_cast<uint32_t>(lane16 < N ? lane16 : N - 1) * sizeof(TIn);

  struct Tile {
    typename SI::raw x[kPFWide], dt[kPFWide], z[kPFWide], b[kPFWide], c[kPFWide];
  };
  Tile t0b, t1b;
  const int last = nsteps > 0 ? nsteps - 1 : 0;
  auto fetch = [&](Tile& tb, int tile) {
#pragma unroll
    for (int k = 0; k < kPFWide; ++k) {
      int st = tile * kPFWide + k;
      st = st < last ? st : last;
      const uint32_t so = static_cast<uint32_t>(st) * in_row;
      tb.x[k] = SI::load(rx, dl, so);
      tb.dt[k] = SI::load(rd, dl, so);
      if constexpr (HASZ) tb.z[k] = SI::load(rz, dl, so);
      const uint32_t sb = static_cast<uint32_t>(st) * bc_row;
      tb.b[k] = SI::load(rb, el, sb);
      if constexpr (kRead) tb.c[k] = SI::load(rc, el, sb);
    }
  };
  float dtacc = 0.f;
  auto step = [&](const Tile& tb, int k, int st) {
    const float xv = SI::f32(tb.x[k]);
    const float dtv = SI::f32(tb.dt[k]);
    const float u = dtv * xv;
    ctoken<N>(hr, hi, a2, w1, dtv, u, SI::f32(tb.b[k]), std::make_integer_sequence<int, kPer>{});
    if constexpr (kRead) {
      float acc = 0.f;
      readout_group<N, 0>(acc, SI::f32(tb.c[k]), hr);
      float out = fmaf(dsk, xv, acc);
      if constexpr (HASZ) {
        const float zv = SI::f32(tb.z[k]);
        const float e = __builtin_amdgcn_exp2f(-kLog2e * zv);
        out *= zv * __builtin_amdgcn_rcpf(1.f + e);
      }
      SO::store(ry, dly, static_cast<uint32_t>(st) * out_row, out);
    }
    if constexpr (KIND == kSummary) dtacc += dtv;
  };
  auto run_tile = [&](const Tile& tb, int tile) {
#pragma unroll
    for (int k = 0; k < kPFWide; ++k) step(tb, k, tile * kPFWide + k);
  };
  auto run_tile_guarded = [&](const Tile& tb, int tile) {
#pragma unroll
    for (int k = 0; k < kPFWide; ++k)
      if (tile * kPFWide + k < nsteps) step(tb, k, tile * kPFWide + k);
  };

  if (nsteps > 0) {
    fetch(t0b, 0);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): tile 0 in before tile 1 is requested
    int tile = 0;
    for (; (tile + 2) * kPFWide <= nsteps; tile += 2) {
      if (fair) balance_step(progress, wave, tile);
      fetch(t1b, tile + 1);
      run_tile(t0b, tile);
      fetch(t0b, tile + 2);
      run_tile(t1b, tile + 1);
    }
    fetch(t1b, tile + 1);
    run_tile_guarded(t0b, tile);
    run_tile_guarded(t1b, tile + 1);
  }

  if (!live) return;
  if constexpr (KIND == kSummary) {
    store_cstate<N>(p.carry + (static_cast<int64_t>(b) * p.nchunks + c + 1) * DN2 + 2 * d * N, hr,
                    hi);
    p.dtsum[(static_cast<int64_t>(b) * p.nchunks + c) * D + d] = dtacc;
  } else {
    if ((p.flags & kHasHT) && c == p.nchunks - 1)
      store_cstate<N>(static_cast<TSt*>(p.hT) + b * p.hT_stride + 2 * d * N, hr, hi);
  }
}

// Pass 2: per (b, d, n) lane, fold the chunk summaries in time order.
// carry[b, 0] = h0; carry[b, c] = exp(-S_{c-1} (a + i w)) carry[b, c-1]
// + s_{c-1}, where pass 1 left s_{c-1} in carry[b, c] and S_{c-1} in
// dtsum[b, c-1].  The magnitude is exp2(a' S) as in the tokens; the angle
// S w / (2 pi) is formed and reduced to [0, 1) revolutions in fp64 (it
// reaches hundreds of revolutions over a long chunk, where fp32 would keep
// too few fraction bits), then cos / sin as in the tokens.
template <typename TSt>
__global__ __launch_bounds__(256) void complex_carry_kernel(const ScanParams p, int N) {
  const int64_t DN = p.D * N;
  const int64_t gid = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (gid >= p.B * DN) return;
  const int64_t b = gid / DN;
  const int64_t dn = gid - b * DN;
  const int64_t d = dn / N;
  const float a2 = -kLog2e * p.A[dn];
  const double w1 = static_cast<double>(p.A_im[dn]) * 0.15915494309189535;  // 1 / (2 pi)
  float Hr = 0.f, Hi = 0.f;
  if (p.flags & kHasH0) {
    const TSt* src = static_cast<const TSt*>(p.h0) + b * p.h0_stride + 2 * dn;
    Hr = to_f32(src[0]);
    Hi = to_f32(src[1]);
  }
  float* cp = p.carry + b * p.nchunks * 2 * DN + 2 * dn;
  const float* sp = p.dtsum + b * p.nchunks * p.D + d;
  cp[0] = Hr;
  cp[1] = Hi;
  constexpr int kU = 4;
  for (int c0 = 1; c0 < p.nchunks; c0 += kU) {
    float sr[kU], si[kU], Sv[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      if (c0 + k < p.nchunks) {
        sr[k] = cp[(c0 + k) * 2 * DN];
        si[k] = cp[(c0 + k) * 2 * DN + 1];
        Sv[k] = sp[(c0 + k - 1) * p.D];
      }
    }
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      if (c0 + k < p.nchunks) {
        const double turns = static_cast<double>(Sv[k]) * w1;
        const float rev = static_cast<float>(turns - floor(turns));
        const float mag = __builtin_amdgcn_exp2f(a2 * Sv[k]);
        const float cs = mag * __builtin_amdgcn_cosf(rev);
        const float sn = mag * __builtin_amdgcn_sinf(rev);
        const float re = Hr;
        Hr = fmaf(cs, re, fmaf(sn, Hi, sr[k]));
        Hi = fmaf(cs, Hi, fmaf(-sn, re, si[k]));
        cp[(c0 + k) * 2 * DN] = Hr;
        cp[(c0 + k) * 2 * DN + 1] = Hi;
      }
    }
  }
}

template <int N, typename TIn, typename TOut, typename TSt>
hipError_t launch_c(const ScanParams& p, hipStream_t s) {
  const int64_t rows_blocks = static_cast<int64_t>(p.dblocks) * p.B;
  const TIn* X = static_cast<const TIn*>(p.x);
  const TIn* DT = static_cast<const TIn*>(p.dt);
  const TIn* Z = static_cast<const TIn*>(p.z);
  const TIn* BB = static_cast<const TIn*>(p.Bm);
  const TIn* CC = static_cast<const TIn*>(p.Cm);
  if (p.nchunks > 1) {
    const dim3 g1(static_cast<unsigned>(rows_blocks * (p.nchunks - 1)));
    hipLaunchKernelGGL((scan_complex_kernel<N, TIn, float, float, kSummary, false>), g1,
                       dim3(kSBlock), 0, s, X, DT, Z, BB, CC, static_cast<float*>(nullptr), p);
    const int64_t lanes = p.B * p.D * N;
    hipLaunchKernelGGL((complex_carry_kernel<TSt>), dim3(static_cast<unsigned>((lanes + 255) / 256)),
                       dim3(256), 0, s, p, N);
  }
  const dim3 grid(static_cast<unsigned>(rows_blocks * p.nchunks));
  if (p.y != nullptr && (p.flags & kHasZ))
    hipLaunchKernelGGL((scan_complex_kernel<N, TIn, TOut, TSt, kReadout, true>), grid, dim3(kSBlock),
                       0, s, X, DT, Z, BB, CC, static_cast<TOut*>(p.y), p);
  else if (p.y != nullptr)
    hipLaunchKernelGGL((scan_complex_kernel<N, TIn, TOut, TSt, kReadout, false>), grid,
                       dim3(kSBlock), 0, s, X, DT, Z, BB, CC, static_cast<TOut*>(p.y), p);
  else
    hipLaunchKernelGGL((scan_complex_kernel<N, TIn, float, TSt, kStateOnly, false>), grid,
                       dim3(kSBlock), 0, s, X, DT, Z, BB, CC, static_cast<float*>(nullptr), p);
  return hipGetLastError();
}

template <int N, typename TIn, typename TOut>
hipError_t c_state(const ScanParams& p, int state_dtype, hipStream_t s) {
  return state_dtype == 0 ? launch_c<N, TIn, TOut, float>(p, s) : launch_c<N, TIn, TOut, f16_t>(p, s);
}

template <int N, typename TIn>
hipError_t c_out(const ScanParams& p, int out_dtype, int state_dtype, hipStream_t s) {
  return out_dtype == 0 ? c_state<N, TIn, float>(p, state_dtype, s)
                        : c_state<N, TIn, bf16_t>(p, state_dtype, s);
}

template <int N>
hipError_t c_in(const ScanParams& p, int in_dtype, int out_dtype, int state_dtype, hipStream_t s) {
  return in_dtype == 0 ? c_out<N, float>(p, out_dtype, state_dtype, s)
                       : c_out<N, bf16_t>(p, out_dtype, state_dtype, s);
}

}  // namespace

hipError_t launch_scan_complex(const ScanParams& p, int N, int in_dtype, int out_dtype,
                               int state_dtype, hipStream_t s) {
  switch (N) {
    case 1: return c_in<1>(p, in_dtype, out_dtype, state_dtype, s);
    case 2: return c_in<2>(p, in_dtype, out_dtype, state_dtype, s);
    case 4: return c_in<4>(p, in_dtype, out_dtype, state_dtype, s);
    case 8: return c_in<8>(p, in_dtype, out_dtype, state_dtype, s);
    case 16: return c_in<16>(p, in_dtype, out_dtype, state_dtype, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace precog
