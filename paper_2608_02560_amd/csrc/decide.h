// Exact top-k decision of the retrieval (Sec. 4.2) for one query, run by one
// wave: the margin tests on the screen's block summaries, the proven fast
// ordering and the fp64 rescoring described in retrieve.hip.  Used by the
// retrieval's decide kernel and by the query-time prefill that decides its
// own query before scanning (scan_kernels.h).
#pragma once

#include <cmath>

#include "precog_kernels.h"
#include "wave_ops.h"

namespace precog {
namespace {

constexpr int kKB = 32;  // keys per block (one MFMA tile's rows; block summaries)

__device__ __forceinline__ float xor_shfl(float v, int m) {
  const int src = (static_cast<int>(threadIdx.x & 63) ^ m) * 4;
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, v)));
}

__device__ __forceinline__ bool ranks_before(double s, int i, double bs, int bi) {
  return s > bs || (s == bs && i < bi);
}


constexpr int kMaxE = 4096;

// (value, index) order of the block-maximum pass: larger value first, then
// lower index.  NaN values are never ranked.
__device__ __forceinline__ bool before(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

constexpr int kCand = 256;            // candidate list capacity (indices)
constexpr int kBList = 512;           // surviving-block list capacity (>= 2 groups of 256)
// squared norm below which 2^8 |v| stays under the fp16 overflow threshold
// for every component v (|v| < 245)
constexpr float kMaxNorm2 = 60000.f;
constexpr int kRowWords = 8192;       // LDS words for staged candidate rows
constexpr int kCacheGroups = 2;       // 256-block groups whose maxima stay in registers

// LDS of one deciding wave.  The query in fp64 takes the first E doubles
// of `qr`; the staged candidate rows take the rest (so a short query leaves
// room for more rows per batch: 40 rows of 384 features instead of 21).
constexpr int kQRWords = 2 * kMaxE + kRowWords;  // 4-byte words of `qr`
struct DecideShared {
  float qr[kQRWords] __attribute__((aligned(16)));
  int cand[kCand];
  int blist[kBList];
  double slot_s[64];
  int slot_i[64];
};

// The deciding wave's lanes exchange values through LDS: a compiler barrier
// keeps every LDS access on its side, and the LDS unit performs one wave's
// accesses in issue order.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// decide: one wave per query (the decision of the retrieval file's comment).  For the
// k best keys the bound uses t_k, the k-th largest block maximum: k distinct
// blocks hold a key with screen score >= t_k, so k keys have exact scores
// >= t_k - e_max and every key of the exact top k has S~_i + e(i) >= that.
// (k = 1: t_1 = m.)  Blocks are discarded with their maxima and norm bounds,
// then keys one by one; surviving keys are collected in an LDS list and
// scored exactly in batches: the wave stages a batch of rows in LDS (row
// pitch E + 4 words, 16-byte aligned)
// and lane j sums row j in fp64 in feature order (fma equals
// multiply-then-add here: the product of two fp32 values is exact in fp64),
// so the chains of a batch run side by side.  Each scored batch is merged
// into a rank list spread over the lanes (lane j holds rank j), ordered by
// score, then by lower index; the order of the batches does not change the
// list.
// FL: row loads in flight per round when a whole block is rescored in fp32
// (as many as the caller's register budget allows).
template <int FL>
__device__ __forceinline__ int32_t decide_query(const RetrieveParams& p, int64_t q,
                                                DecideShared& sh) {
  const int lane = threadIdx.x & 63;
  const int E = static_cast<int>(p.E);
  const int nkb = p.nkb;
  const int k = p.k;
  // the query (exact in fp64) first, the staged rows after it; E is a
  // multiple of 4, so the rows stay 16-byte aligned
  double* const qs = reinterpret_cast<double*>(sh.qr);
  float* const rs = sh.qr + 2 * E;
  const int row_words = kQRWords - 2 * E;
  int* const cand = sh.cand;
  int* const blist = sh.blist;
  double* const slot_s = sh.slot_s;
  int* const slot_i = sh.slot_i;
  const float4* qg4 = reinterpret_cast<const float4*>(p.q + q * p.E);
  const float* bm = p.blockmax + q * nkb;
  const float* bsec = p.blocksec + q * nkb;
  const uint8_t* barg = p.blockarg + q * nkb;

  // the block maxima and norms of the first kCacheGroups x 256 blocks,
  // loaded once (in flight with the query row) and held in registers for
  // the t_k rounds and the block tests; blocks past nkb hold NaN / 0
  float cb[4 * kCacheGroups], cn[4 * kCacheGroups];
#pragma unroll
  for (int g = 0; g < kCacheGroups; ++g) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kb = 256 * g + 64 * j + lane;
      cb[4 * g + j] = kb < nkb ? bm[kb] : __builtin_nanf("");
      cn[4 * g + j] = kb < nkb ? p.blocknorm2[kb] : 0.f;
    }
  }

  // fixed-width groups of predicated loads, so every load of a group is in
  // flight before the first is consumed
  const int e4n = E / 4;
  float nq = 0.f;
  for (int g0 = 0; g0 < e4n; g0 += 4 * 64) {
    float4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e4 = g0 + 64 * u + lane;
      v[u] = e4 < e4n ? qg4[e4] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e4 = g0 + 64 * u + lane;
      if (e4 < e4n) {
        reinterpret_cast<double2*>(qs + 4 * e4)[0] = make_double2(v[u].x, v[u].y);
        reinterpret_cast<double2*>(qs + 4 * e4)[1] = make_double2(v[u].z, v[u].w);
      }
      nq = fmaf(v[u].x, v[u].x, fmaf(v[u].y, v[u].y, fmaf(v[u].z, v[u].z, fmaf(v[u].w, v[u].w, nq))));
    }
  }
  const float qnorm2 = wave_sum(nq);
  const float qnorm = sqrtf(qnorm2);

  // t_k: k rounds, each taking the first (value, index) pair after the
  // previous one (the first round also takes the largest block norm); fewer
  // than k ranked blocks leave t_k = -inf (every key is then a candidate)
  float nmax = 0.f;
#pragma unroll
  for (int c = 0; c < 4 * kCacheGroups; ++c) nmax = fmaxf(nmax, cn[c]);
  float tv = INFINITY;
  int ti = -1;
  bool found = true;
  for (int r = 0; r < k && found; ++r) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    bool any = false;
    auto consider = [&](float b, int kb) {
      if (before(tv, ti, b, kb) && (!any || before(b, kb, bv, bi))) {
        bv = b;
        bi = kb;
        any = true;
      }
    };
#pragma unroll
    for (int c = 0; c < 4 * kCacheGroups; ++c) consider(cb[c], 64 * c + lane);
    for (int kb0 = 256 * kCacheGroups; kb0 < nkb; kb0 += 256) {
      float b[4], n[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kb = kb0 + 64 * j + lane;
        b[j] = kb < nkb ? bm[kb] : __builtin_nanf("");
        n[j] = (r == 0 && kb < nkb) ? p.blocknorm2[kb] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        nmax = fmaxf(nmax, n[j]);
        consider(b[j], kb0 + 64 * j + lane);
      }
    }
    // the wave's first pair: the largest value, then the lowest index among
    // the lanes holding it (lanes without a pair take no part)
    const float m = wave_max(any ? bv : -INFINITY);
    const int mi = wave_min(any && bv == m ? bi : 0x7fffffff);
    found = __ballot(any) != 0;
    if (found) {
      tv = m;
      ti = mi;
    }
  }
  nmax = wave_max(nmax);
  const float tk = found ? tv : -INFINITY;

  // Screen-score error bound e(i) = g |q| |k_i| + h (|q| + |k_i|) + tiny;
  // g, h and tiny depend on E only (error_bound_constants, on the host)
  const double qn = static_cast<double>(qnorm);
  const double gq = p.err_g * qn + p.err_h;
  const double hq = p.err_h * qn + p.err_tiny;
  // error bound of a screen score whose key has squared norm <= n2.  The
  // root is the fp32 one (v_sqrt_f32, within 1 ulp) of n2 raised to at
  // least the smallest normal, widened by 2^-16 in fp64: never below the
  // true root, so the bound stays an upper bound (the tests only ever pass
  // more keys), without an fp64 root per block (NaN stays NaN)
  auto err = [&](float n2) {
    const float r = __builtin_amdgcn_sqrtf(n2 < 0x1p-126f ? 0x1p-126f : n2);
    return gq * (static_cast<double>(r) * (1.0 + 0x1p-16)) + hq;
  };
  const bool exhaustive = !(qnorm2 < kMaxNorm2) || !(nmax < kMaxNorm2);
  const double thresh = exhaustive ? -INFINITY : static_cast<double>(tk) - err(nmax);

  // rank list: lane j < nl holds the j-th best (score, index) so far
  double ls = -INFINITY;
  int li = -1;
  int nl = 0;
  // merge a scored batch (lane r < nb: score s of key ci) into the list:
  // every element counts the elements of both sets ordered before it
  // (broadcast one pair per step), so its new rank is known at once, and
  // the elements with rank < k go through LDS to the lane of their rank.
  // Keys are distinct, so ranks are distinct.
  auto merge = [&](double s, int ci, int nb) {
    const double sk = s != s ? -INFINITY : s;  // NaN scores rank last
    int before_new = 0;                        // for this lane's batch element
    int new_before_old = 0;                    // for this lane's list element
    const int steps = nl > nb ? nl : nb;
    for (int i = 0; i < steps; ++i) {
      if (i < nl) {
        const double es = readlane_d(ls, i);
        const int ei = __builtin_amdgcn_readlane(li, i);
        before_new += (lane < nb && ranks_before(es, ei, sk, ci)) ? 1 : 0;
      }
      if (i < nb) {
        const double ns = readlane_d(sk, i);
        const int ni = __builtin_amdgcn_readlane(ci, i);
        before_new += (lane < nb && i != lane && ranks_before(ns, ni, sk, ci)) ? 1 : 0;
        new_before_old += (lane < nl && ranks_before(ns, ni, ls, li)) ? 1 : 0;
      }
    }
    wave_sync();  // the previous merge has read its slots
    if (lane < nl && lane + new_before_old < k) {
      slot_s[lane + new_before_old] = ls;
      slot_i[lane + new_before_old] = li;
    }
    if (lane < nb && before_new < k) {
      slot_s[before_new] = sk;
      slot_i[before_new] = ci;
    }
    wave_sync();
    nl = nl + nb < k ? nl + nb : k;
    if (lane < nl) {
      ls = slot_s[lane];
      li = slot_i[lane];
    }
  };

  // exact scores of the listed candidates, a batch of rows at a time
  const int pitch = E + 4;  // E is a multiple of 4: rows stay 16-byte aligned
  const uint64_t inv_e4n = ((1ull << 32) + static_cast<uint64_t>(e4n) - 1) / static_cast<uint64_t>(e4n);
  const int batch_max = row_words / pitch < 64 ? row_words / pitch : 64;
  int ncand = 0;
  bool early = false;  // a batch was scored before the list was complete
  // rows cand[c0 .. c0 + nb) into rs (row pitch `pitch`): one flat
  // (row, float4) space in fixed-width groups of predicated loads, so the
  // loads of several rows are in flight together (f / e4n as a 64-bit
  // multiply-high: exact for f < 2^17, e4n <= 1024)
  auto stage_rows = [&](int c0, int nb) {
    wave_sync();  // previous batch consumed, list and qs complete
    const int tot = nb * e4n;
    for (int f0 = 0; f0 < tot; f0 += 8 * 64) {
      float4 v[8];
      int off[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int f = f0 + 64 * u + lane;
        const int r = f < tot ? static_cast<int>((static_cast<uint64_t>(f) * inv_e4n) >> 32) : 0;
        const int e4 = f - r * e4n;
        off[u] = f < tot ? r * pitch + 4 * e4 : -1;
        v[u] = f < tot ? reinterpret_cast<const float4*>(p.K + static_cast<int64_t>(cand[c0 + r]) * p.E)[e4]
                       : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (off[u] >= 0) *reinterpret_cast<float4*>(rs + off[u]) = v[u];
    }
    wave_sync();
  };
  auto flush = [&]() {
    for (int c0 = 0; c0 < ncand; c0 += batch_max) {
      const int nb = ncand - c0 < batch_max ? ncand - c0 : batch_max;
      stage_rows(c0, nb);
      // the chain stays one fma per feature in feature order; the query is
      // held in fp64 (converted once, exactly), so a feature costs one
      // conversion of the key value and the fma; reading four key values
      // per 16-byte LDS access (the query's two 16-byte broadcasts) and
      // unrolling lets the reads run ahead of the dependent fp64 chain
      double s = 0.0;
      if (lane < nb) {
        const float* row = rs + lane * pitch;
#pragma unroll 4
        for (int e = 0; e < E; e += 4) {
          const double2 q01 = *reinterpret_cast<const double2*>(qs + e);
          const double2 q23 = *reinterpret_cast<const double2*>(qs + e + 2);
          const float4 rv = *reinterpret_cast<const float4*>(row + e);
          s = fma(q01.x, static_cast<double>(rv.x), s);
          s = fma(q01.y, static_cast<double>(rv.y), s);
          s = fma(q23.x, static_cast<double>(rv.z), s);
          s = fma(q23.y, static_cast<double>(rv.w), s);
        }
      }
      merge(s, lane < nb ? cand[c0 + lane] : -1, nb);
    }
    ncand = 0;
  };

  // Surviving blocks go, in ascending order, to an LDS list, tested 64 per
  // round (lane j takes entry i0 + j, its summary loads in flight together
  // with the other lanes').  A key other than the block's largest has a
  // screen score of at most the block's second largest, so if that second
  // largest fails the test with the block's norm bound, the largest is the
  // block's only candidate (tested with its own norm).  Otherwise every key
  // of the block is rescored in fp32 from its fp32 row (lane l: key l mod 32,
  // every other float4 of the features from l / 32 on, the two halves
  // added): that sum differs from the exact score by at most
  // gamma_{E+1} |q| |k_i|, far inside the screen's bound e(i), so the keys
  // passing the same test with it are the block's candidates.
  int nbl = 0;
  auto test_list = [&]() __attribute__((always_inline)) {
    wave_sync();  // the list entries written by other lanes are in
    for (int i0 = 0; i0 < nbl; i0 += 64) {
      const bool on = i0 + lane < nbl;
      const int kb = on ? blist[i0 + lane] : 0;
      const float s1 = on ? bm[kb] : -INFINITY;
      const float s2 = on ? bsec[kb] : -INFINITY;
      const int a1 = on ? static_cast<int>(barg[kb]) : 0;
      const float bn = on ? p.blocknorm2[kb] : 0.f;
      const int64_t key1 = static_cast<int64_t>(kb) * kKB + a1;
      const bool key_ok = on && key1 < p.M;
      const float kn = key_ok ? p.rownorm2[key1] : 0.f;
      const bool full = on && (exhaustive || static_cast<double>(s2) + err(bn) >= thresh);
      const bool single =
          key_ok && !full && static_cast<double>(s1) + err(kn) >= thresh;
      const uint64_t smask = __ballot(single);
      if (smask) {
        if (ncand + 64 > kCand) {
          early = true;
          flush();
        }
        if (single) cand[ncand + __builtin_popcountll(smask & ((1ull << lane) - 1))] = static_cast<int>(key1);
        ncand += __builtin_popcountll(smask);
      }
      uint64_t fmask = __ballot(full);
      while (fmask) {
        const int j = __builtin_ctzll(fmask);
        fmask &= fmask - 1;
        const int64_t b0 = static_cast<int64_t>(__builtin_amdgcn_readlane(kb, j)) * kKB;
        const int cnt = static_cast<int>(p.M - b0 < kKB ? p.M - b0 : kKB);
        const int r = lane & (kKB - 1);
        const bool kok = r < cnt;
        float part[4] = {0.f, 0.f, 0.f, 0.f};
        if (kok) {
          // FL 16-byte loads of the row in flight per round (the sum's
          // order is free: any order stays within gamma_{E+1})
          const float4* row = reinterpret_cast<const float4*>(p.K + (b0 + r) * p.E);
          for (int e0 = lane >> 5; e0 < e4n; e0 += 2 * FL) {
            float4 v[FL];
#pragma unroll
            for (int u = 0; u < FL; ++u) {
              const int f = e0 + 2 * u;
              v[u] = f < e4n ? row[f] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int u = 0; u < FL; ++u) {
              const int f = e0 + 2 * u;
              if (f < e4n) {
                const double2 q01 = *reinterpret_cast<const double2*>(qs + 4 * f);
                const double2 q23 = *reinterpret_cast<const double2*>(qs + 4 * f + 2);
                float& a = part[u & 3];
                a = fmaf(static_cast<float>(q01.x), v[u].x, a);
                a = fmaf(static_cast<float>(q01.y), v[u].y, a);
                a = fmaf(static_cast<float>(q23.x), v[u].z, a);
                a = fmaf(static_cast<float>(q23.y), v[u].w, a);
              }
            }
          }
        }
        float tot = (part[0] + part[1]) + (part[2] + part[3]);
        tot += xor_shfl(tot, 32);
        const bool ok = lane < kKB && kok &&
                        (exhaustive || static_cast<double>(tot) +
                                           err(p.rownorm2[b0 + r]) >= thresh);
        const uint64_t cmask = __ballot(ok);
        if (cmask) {
          if (ncand + kKB > kCand) {
            early = true;
            flush();
          }
          if (ok) cand[ncand + __builtin_popcountll(cmask & ((1ull << lane) - 1))] = static_cast<int>(b0 + r);
          ncand += __builtin_popcountll(cmask);
        }
      }
    }
    wave_sync();  // every list entry is read before the list is refilled
    nbl = 0;
  };
  // one group of 256 blocks: lane l holds the maxima and norms of blocks
  // kb0 + 64 j + l
  auto add_group = [&](int kb0, const float (&b4)[4], const float (&n4)[4]) {
    if (nbl > kBList - 256) test_list();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kb = kb0 + 64 * j + lane;
      const bool pass = kb < nkb && (exhaustive || static_cast<double>(b4[j]) + err(n4[j]) >= thresh);
      const uint64_t bmask = __ballot(pass);
      if (pass) blist[nbl + __builtin_popcountll(bmask & ((1ull << lane) - 1))] = kb;
      nbl += __builtin_popcountll(bmask);
    }
  };
#pragma unroll
  for (int g = 0; g < kCacheGroups; ++g) {
    if (256 * g < nkb) {
      const float b4[4] = {cb[4 * g], cb[4 * g + 1], cb[4 * g + 2], cb[4 * g + 3]};
      const float n4[4] = {cn[4 * g], cn[4 * g + 1], cn[4 * g + 2], cn[4 * g + 3]};
      add_group(256 * g, b4, n4);
    }
  }
  for (int kb0 = 256 * kCacheGroups; kb0 < nkb; kb0 += 256) {
    float b4[4], n4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kb = kb0 + 64 * j + lane;
      b4[j] = kb < nkb ? bm[kb] : -INFINITY;
      n4[j] = kb < nkb ? p.blocknorm2[kb] : 0.f;
    }
    add_group(kb0, b4, n4);
  }
  if (nbl > 0) test_list();
  // Top-1 without scores: the candidate list provably holds the exact
  // argmax, so a single candidate is the answer.  With several, each is
  // scored by a lane-parallel fp64 sum (every product exact; each lane sums
  // its E / 64 features, then a 6-level tree), which differs from the
  // exact real sum by at most gamma_{E/64+7} sum |p_e|; the sequential sum
  // of the definition by at most gamma_E sum |p_e|; and sum |p_e| <=
  // |q| |k_i| (1.01 covers the fp32 norms).  If the best candidate's lower
  // end beats every other's upper end, it is the sequential argmax;
  // otherwise (near or exact ties) the sequential rescoring below decides.
  bool done = false;
  if (k == 1 && p.score == nullptr && !early && ncand > 0) {
    if (ncand == 1) {
      li = cand[0];
      done = true;
    } else {
      const double gs = p.err_gs;
      double best = 0.0, best_mu = 0.0, others = -INFINITY;
      int best_i = -1;
      for (int c0 = 0; c0 < ncand; c0 += batch_max) {
        const int nb = ncand - c0 < batch_max ? ncand - c0 : batch_max;
        // the batch's squared norms, one lane each, in flight with its rows
        // (the list is complete: test_list ended with a wave_sync)
        const float cn2 = lane < nb ? p.rownorm2[cand[c0 + lane]] : 0.f;
        stage_rows(c0, nb);
        for (int r = 0; r < nb; ++r) {
          const float* row = rs + r * pitch;
          double part = 0.0;
          for (int e = lane; e < E; e += 64)
            part = fma(qs[e], static_cast<double>(row[e]), part);
          const double a = wave_sum_d(part);
          const int ci = cand[c0 + r];
          const float n2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cn2), r));
          const double mu = gs * qn * sqrt(static_cast<double>(n2)) + 1e-300;
          if (best_i < 0 || a > best || (a == best && ci < best_i)) {
            if (best_i >= 0) others = fmax(others, best + best_mu);
            best = a;
            best_mu = mu;
            best_i = ci;
          } else {
            others = fmax(others, a + mu);
          }
        }
      }
      if (best - best_mu > others) {
        li = best_i;
        done = true;
      }
    }
  }
  if (!done) flush();
  if (lane < k) {
    p.idx[q * k + lane] = static_cast<int32_t>(li);
    if (p.score) p.score[q * k + lane] = ls;
  }
  return __builtin_amdgcn_readfirstlane(li);
}

}  // namespace
}  // namespace precog
