// Device routines of the draw shared by the per-sequence kernel and the
// vocabulary-shard kernels: the draw job, fp64 helpers of the latency-bound
// steps, the combine of chunk partials, and the per-chunk passes of the draw
// (residual max(0, p - q), p, bonus exponentials, bonus argmax) with their
// sub-block totals.
#pragma once

#include <math.h>

#include "common.hpp"
#include "lanes.hpp"
#include "row_io.hpp"

namespace dsde {
namespace {

constexpr int kVirt = kThreads / 64;          // chunk-layout threads played by one lane (4)

// How many of a lane's chunk-layout threads one loop iteration handles: as
// many as the registers allow loads in flight for.
template <int DT, bool VEC>
constexpr int kVirtUnroll = !VEC ? 1 : DT == DSDE_BF16 ? kVirt : 2;

// What the draw of one sequence needs, decided by the acceptance.
struct DrawJob {
  int32_t kind;          // 0: residual of the first rejected pair, 1: bonus row, 2: greedy, token known,
                         // 3: greedy, argmax of the bonus row, -1: nothing (flagged)
  int32_t accepted;      // a_b
  int32_t target_row;
  int32_t draft_row;     // -1 for the bonus row
  float scale;           // c = log2(e) / T_b
  float mt, md;          // row reference shifts of the rejected pair
  float inv_sp, inv_sq;  // 1 / row sums of the rejected pair
  float u;               // draw uniform
  int32_t token;         // greedy: the emitted token when it is already known
};

// The draw job as read from LDS, moved to scalar registers (it is the same in
// every lane), which frees vector registers for the draw stream's loads.
__device__ __forceinline__ float uniform_f(float v) {
  return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(v)));
}
__device__ __forceinline__ DrawJob uniform_job(const DrawJob &j) {
  DrawJob u;
  u.kind = __builtin_amdgcn_readfirstlane(j.kind);
  u.accepted = __builtin_amdgcn_readfirstlane(j.accepted);
  u.target_row = __builtin_amdgcn_readfirstlane(j.target_row);
  u.draft_row = __builtin_amdgcn_readfirstlane(j.draft_row);
  u.scale = uniform_f(j.scale);
  u.mt = uniform_f(j.mt);
  u.md = uniform_f(j.md);
  u.inv_sp = uniform_f(j.inv_sp);
  u.inv_sq = uniform_f(j.inv_sq);
  u.u = uniform_f(j.u);
  u.token = __builtin_amdgcn_readfirstlane(j.token);
  return u;
}

// 2^x in double for the latency-bound steps: x = n + r with n = rint(x) and
// |r| <= 1/2; e^(r ln 2) by its Taylor series to degree 10 (remainder below
// 0.35^11 / 11! * e^0.35 < 4e-13 relative), scaled by 2^n.
__device__ __forceinline__ double exp2_taylor(double x) {
  if (!(x >= -1100.0)) return x != x ? x : 0.0;  // NaN stays NaN; below 2^-1074 is 0
  if (x > 1100.0) return HUGE_VAL;
  const double n = rint(x);
  const double y = (x - n) * kLn2;
  double p = 1.0 / 3628800.0;
  p = fma(p, y, 1.0 / 362880.0);
  p = fma(p, y, 1.0 / 40320.0);
  p = fma(p, y, 1.0 / 5040.0);
  p = fma(p, y, 1.0 / 720.0);
  p = fma(p, y, 1.0 / 120.0);
  p = fma(p, y, 1.0 / 24.0);
  p = fma(p, y, 1.0 / 6.0);
  p = fma(p, y, 0.5);
  p = fma(p, y, 1.0);
  p = fma(p, y, 1.0);
  return ldexp(p, int(n));
}

// log2 of a positive row sum in double: s = m 2^e with m in [1/2, 1); the
// hardware log2 (v_log_f32) gives y0 = log2 m to about 1.5e-7, and one
// correction step finishes it: m 2^-y0 = 1 + d with |d| < 3e-7, and
// log2(1 + d) = (d - d^2 / 2) / ln 2 up to d^3 (below 1e-20).  Used for the
// KLD, the entropy and the log-normalisers; the acceptance test takes no
// logarithm.
__device__ __forceinline__ double log2_rowsum(double s) {
  int e;
  const double m = frexp(s, &e);
  const double y0 = double(__builtin_amdgcn_logf(float(m)));
  const double d = m * exp2_taylor(-y0) - 1.0;
  return double(e) + y0 + (d - 0.5 * d * d) * (1.0 / kLn2);
}

// 1 / s in double: the hardware estimate and two Newton steps.
__device__ __forceinline__ double rcp_newton(double s) {
  double r = __builtin_amdgcn_rcp(s);
  r = fma(fma(-s, r, 1.0), r, r);
  r = fma(fma(-s, r, 1.0), r, r);
  return r;
}

// reductions inside aligned groups of G lanes (G = 16, 32 or 64)
template <int G>
__device__ __forceinline__ float group_max(float v) {
  return lanes::group_reduce<G>(v, lanes::Max{});
}
template <int G>
__device__ __forceinline__ double group_sum(double v) {
  return lanes::group_reduce<G>(v, lanes::Add{});
}

// Folds the statistics (mt, md, sp, sq, a, h) of one more part of a row pair
// (a chunk, or a vocabulary slice) into a running set: both are rescaled to
// the larger reference shifts; the KL and entropy accumulators take the shift
// of the log-ratio along (a = sum 2^at (at - ad) with at, ad relative to the
// references).
__device__ __forceinline__ void fold_pair_stats(float &lmt, float &lmd, double &lsp, double &lsq, double &la,
                                                double &lh, float qmt, float qmd, double qsp, double qsq, double qa,
                                                double qh) {
  const float nt = fmaxf(lmt, qmt), nd = fmaxf(lmd, qmd);
  const double d0t = double(lmt) - nt, d0d = double(lmd) - nd;
  const double d1t = double(qmt) - nt, d1d = double(qmd) - nd;
  const double f0t = exp2_taylor(d0t), f0d = exp2_taylor(d0d), f1t = exp2_taylor(d1t), f1d = exp2_taylor(d1d);
  la = f0t * (la + lsp * (d0t - d0d)) + f1t * (qa + qsp * (d1t - d1d));
  lh = f0d * (lh + lsq * d0d) + f1d * (qh + qsq * d1d);
  lsp = f0t * lsp + f1t * qsp;
  lsq = f0d * lsq + f1d * qsq;
  lmt = nt;
  lmd = nd;
}

// Combines the chunk partials of every drafted pair of one sequence (stored
// under slots slot0 + j): groups of G lanes, one pair per group, lane g of a
// group folds chunks g, g + G, ...  Results go to LDS (st_*[j] for position j;
// st_zmax, when given, receives the greedy rows' largest raw target logit).
template <int G, int WAVES>
__device__ inline void combine_pairs(const PairChunk *__restrict__ part, int64_t slot0, int32_t s, int32_t nc,
                                     const PairChunk &q0, const ChunkArg *__restrict__ chunk_arg, ChunkArg arg0,
                                     float *st_mt, float *st_md, double *st_sp, double *st_sq, double *st_a,
                                     double *st_h, int *st_bad, int *st_arg, float *st_zmax = nullptr) {
  constexpr int P = 64 / G;  // pairs per wavefront
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane % G;
  for (int32_t base = 0; base < s; base += WAVES * P) {
    const int32_t j = base + wave * P + lane / G;
    float lmt = -INFINITY, lmd = -INFINITY;
    double lsp = 0.0, lsq = 0.0, la = 0.0, lh = 0.0;
    // greedy: the largest raw logit among this lane's chunks and its token
    float lz = -INFINITY;
    int32_t larg = 0x7fffffff;
    if (j < s) {
      for (int32_t ch = g; ch < nc; ch += G) {
        // the first chunk of the first round was fetched at kernel start
        const bool pre = base == 0 && ch == g;
        const PairChunk q = pre ? q0 : part[(slot0 + j) * nc + ch];
        if (chunk_arg) {
          const ChunkArg qa = pre ? arg0 : chunk_arg[(slot0 + j) * nc + ch];
          // chunks come in ascending order: on equal maxima the earlier wins
          if (larg == 0x7fffffff || qa.zmax > lz) {
            lz = qa.zmax;
            larg = qa.idx;
          }
        }
        if (lmt == -INFINITY) {
          lmt = q.mt;
          lmd = q.md;
          lsp = q.sp;
          lsq = q.sq;
          la = q.a;
          lh = q.h;
        } else {
          fold_pair_stats(lmt, lmd, lsp, lsq, la, lh, q.mt, q.md, q.sp, q.sq, q.a, q.h);
        }
      }
    }
    const float mt = group_max<G>(lmt), md = group_max<G>(lmd);
    double tsp = 0.0, tsq = 0.0, ta = 0.0, th = 0.0;
    if (lmt != -INFINITY) {
      const double dt = double(lmt) - double(mt), dd = double(lmd) - double(md);
      const double ft = exp2_taylor(dt), fd = exp2_taylor(dd);
      tsp = lsp * ft;
      tsq = lsq * fd;
      ta = ft * (la + lsp * (dt - dd));
      th = fd * (lh + lsq * dd);
    }
    tsp = group_sum<G>(tsp);
    tsq = group_sum<G>(tsq);
    ta = group_sum<G>(ta);
    th = group_sum<G>(th);
    int32_t arg = 0x7fffffff;
    float zm = -INFINITY;
    if (chunk_arg) {  // the row argmax: smallest token among the chunks holding the row maximum
      zm = group_max<G>(lz);
      arg = larg != 0x7fffffff && lz == zm ? larg : 0x7fffffff;
      arg = lanes::group_reduce<G>(arg, lanes::Min{});
    }
    if (j < s && g == 0) {
      st_mt[j] = mt;
      st_md[j] = md;
      st_sp[j] = tsp;
      st_sq[j] = tsq;
      st_a[j] = ta;
      st_h[j] = th;
      st_bad[j] = !(isfinite(mt) && isfinite(md) && isfinite(tsp) && isfinite(tsq) && isfinite(ta));
      st_arg[j] = arg;
      if (st_zmax) st_zmax[j] = zm;
    }
  }
}

// Raw bf16 chunk loads of the draw stream: the loads of issue_raw_bf16 and
// the padding of pad_raw_bf16, with 32-bit word indices off a uniform row
// base (word i0 + 256 q of the row, clamped to the last word), so that each
// load takes one offset register and no 64-bit address arithmetic.
__device__ __forceinline__ RawBf16 issue_row_bf16(const char *row, uint32_t i0, uint32_t last) {
  const uint4 *p = (const uint4 *)row;
  RawBf16 r;
  r.v0 = stream_load(p + min(i0, last));
  r.v1 = stream_load(p + min(i0 + 256u, last));
  r.v2 = stream_load(p + min(i0 + 512u, last));
  r.v3 = stream_load(p + min(i0 + 768u, last));
  return r;
}
__device__ __forceinline__ RawBf16 pad_row_bf16(const RawBf16 &a, uint32_t i0, uint32_t last) {
  const uint4 pad = make_uint4(kPadBf16x2, kPadBf16x2, kPadBf16x2, kPadBf16x2);
  RawBf16 r;
  r.v0 = i0 <= last ? a.v0 : pad;
  r.v1 = i0 + 256u <= last ? a.v1 : pad;
  r.v2 = i0 + 512u <= last ? a.v2 : pad;
  r.v3 = i0 + 768u <= last ? a.v3 : pad;
  return r;
}

// Sub-blocks: each chunk splits into 16 runs of 512 consecutive logits, and
// the draw keeps the weight total of every run, so that after the chunk
// search only one run (one 16-byte load per lane and row for bf16) has to be
// read again and scanned.  Slot i of chunk-layout thread lane + 64 k lies in
// sub-block sub_of(i, k) (from the layouts: bf16 16-byte rows put slot group
// i / 8 of thread t at 2048 (i / 8) + 8 t, fp32 16-byte rows group i / 4 at
// 1024 (i / 4) + 4 t, other rows slot i at 256 i + t).
constexpr int kSubs = 16;
constexpr int kSubLen = kChunk / kSubs;  // 512
template <int DT, bool VEC>
__device__ constexpr int sub_of(int i, int k) {
  return VEC ? (DT == DSDE_BF16 ? 4 * (i / 8) + k : 2 * (i / 4) + (k >> 1)) : (i >> 1);
}

// The draw weights, each evaluated by one routine wherever it is needed (the
// chunk totals and the final scan), with no contraction of the product into
// a neighbouring sum, so that both places see the same bits.
__device__ __forceinline__ float residual_weight(float zt, float zd, const DrawJob &job) {
#pragma clang fp contract(off)
  const float p = fast_exp2(fmaf(zt, job.scale, -job.mt)) * job.inv_sp;
  // p - q as one fused operation: p - 2^(z_d c - md) / S_q
  return fmaxf(fmaf(-fast_exp2(fmaf(zd, job.scale, -job.md)), job.inv_sq, p), 0.0f);  // padding: 0
}
__device__ __forceinline__ float target_p_weight(float zt, const DrawJob &job) {
#pragma clang fp contract(off)
  return fast_exp2(fmaf(zt, job.scale, -job.mt)) * job.inv_sp;
}
__device__ __forceinline__ float bonus_weight(float z, float scale, float ref) {
  return fast_exp2(fmaf(z, scale, -ref));
}

// Per-lane sub-block sums -> the chunk's 64 row partials in LDS (sub-block j
// total = out[j] + out[16 + j] + out[32 + j] + out[48 + j]) and the chunk
// total.
__device__ __forceinline__ double finish_chunk(const float (&a)[kSubs], float *out) {
  const float r = lanes::row_transpose_sum16(a);
  out[threadIdx.x & 63] = r;
  return double(lanes::wave_sum(r));
}

// Chunk of one or two rows as 32 floats per chunk-layout thread, for the
// generic layouts, calling f(i, k, zt, zd) per slot.  fp32 16-byte rows
// handle two chunk-layout threads per iteration (register pressure); the
// sub-block of a slot then depends on the iteration, so the sums of one
// iteration go to kSubs / 2 partials first.
template <int DT, bool VEC, bool TWO, typename F>
__device__ __forceinline__ void generic_chunk_sums(const char *trow, const char *drow, int64_t V, int64_t ch,
                                                   float (&a)[kSubs], F f) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < kSubs; ++j) a[j] = 0.f;
  if constexpr (VEC && DT == DSDE_FP32) {
    for (int kk = 0; kk < 2; ++kk) {
      float b[kSubs / 2];
#pragma unroll
      for (int g = 0; g < kSubs / 2; ++g) b[g] = 0.f;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        float zt[kEltsPerThread], zd[kEltsPerThread];
        load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * (2 * kk + k2), zt);
        if constexpr (TWO) load_chunk_f32<DT, VEC>(drow, V, ch, lane + 64 * (2 * kk + k2), zd);
#pragma unroll
        for (int i = 0; i < kEltsPerThread; ++i) b[i / 4] += f(zt[i], TWO ? zd[i] : 0.f);
      }
#pragma unroll
      for (int g = 0; g < kSubs / 2; ++g) {  // sub-block 2 g + kk
        a[2 * g] = kk == 0 ? b[g] : a[2 * g];
        a[2 * g + 1] = kk == 1 ? b[g] : a[2 * g + 1];
      }
    }
  } else {
#pragma unroll kVirtUnroll<DT, VEC>
    for (int k = 0; k < kVirt; ++k) {
      float zt[kEltsPerThread], zd[kEltsPerThread];
      load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * k, zt);
      if constexpr (TWO) load_chunk_f32<DT, VEC>(drow, V, ch, lane + 64 * k, zd);
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) a[sub_of<DT, VEC>(i, k)] += f(zt[i], TWO ? zd[i] : 0.f);
    }
  }
}

// Total of the residual weights max(0, p - q) over one chunk of the rejected
// pair, by one wavefront (lane l plays the chunk-layout threads l + 64 k), and
// its sub-block partials.
template <int DT, bool VEC>
__device__ inline double residual_chunk(const char *trow, const char *drow, int64_t V, int64_t ch,
                                        const DrawJob &job, float *sub) {
  const int lane = threadIdx.x & 63;
  float a[kSubs];
  if constexpr (DT == DSDE_BF16 && VEC) {
    // every load of the chunk (both rows, all four chunk-layout threads: 32 KiB
    // per wavefront) is issued before any value is used; each chunk-layout
    // thread's four sub-block sums then go into one wave sum as well, which
    // keeps the compiler's order of use equal to the order of issue (loads
    // return in that order) and gives the chunk total
    RawBf16 rt[kVirt], rd[kVirt];
#pragma unroll
    for (int k = 0; k < kVirt; ++k) {
      rt[k] = issue_raw_bf16(trow, V, ch, lane + 64 * k);
      rd[k] = issue_raw_bf16(drow, V, ch, lane + 64 * k);
    }
    float sw[kVirt];
#pragma unroll
    for (int k = 0; k < kVirt; ++k) {
      const RawBf16 t_ = pad_raw_bf16(rt[k], V, ch, lane + 64 * k), d_ = pad_raw_bf16(rd[k], V, ch, lane + 64 * k);
      float tk = 0.f;
#pragma unroll
      for (int g = 0; g < kEltsPerThread / 8; ++g) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) s += residual_weight(pick_bf16(t_, 8 * g + e), pick_bf16(d_, 8 * g + e), job);
        a[sub_of<DT, VEC>(8 * g, k)] = s;
        tk += s;
      }
      sw[k] = wave_sum(tk);
    }
    sub[lane] = lanes::row_transpose_sum16(a);
    double w = 0.0;
#pragma unroll
    for (int k = 0; k < kVirt; ++k) w += double(sw[k]);
    return w;
  } else {
    generic_chunk_sums<DT, VEC, true>(trow, drow, V, ch, a,
                                      [&](float zt, float zd) { return residual_weight(zt, zd, job); });
  }
  return finish_chunk(a, sub);
}

// Total of p over one chunk of the rejected pair's target row (the draw's
// fallback when the residual has no mass), and its sub-block partials.
template <int DT, bool VEC>
__device__ inline double target_p_chunk(const char *trow, int64_t V, int64_t ch, const DrawJob &job, float *sub) {
  float a[kSubs];
  generic_chunk_sums<DT, VEC, false>(trow, nullptr, V, ch, a,
                                     [&](float zt, float) { return target_p_weight(zt, job); });
  return finish_chunk(a, sub);
}

// Bonus row, one chunk, by one wavefront: the chunk reference ref = max(z) c,
// the total of 2^(z c - ref) and its sub-block partials, and whether a NaN or
// +-inf logit was seen (+inf shows in the max, NaN in the sum, -inf in the
// min; padding is finite).
template <int DT, bool VEC>
__device__ inline void bonus_chunk(const char *trow, int64_t V, int64_t ch, float scale, double *w_out,
                                   float *ref_out, int *bad_out, float *sub) {
  const int lane = threadIdx.x & 63;
  float m = -INFINITY, lo = INFINITY;
  float a[kSubs];
  if constexpr (VEC && DT == DSDE_BF16) {
    // one load: the raw chunk stays in registers for both passes
    const uint32_t last = uint32_t(V / 8 - 1), i0 = uint32_t(ch) * 1024u + uint32_t(lane);
    RawBf16 r[kVirt];
#pragma unroll
    for (int k = 0; k < kVirt; ++k) r[k] = issue_row_bf16(trow, i0 + 64u * k, last);
#pragma unroll
    for (int k = 0; k < kVirt; ++k) r[k] = pad_row_bf16(r[k], i0 + 64u * k, last);
#pragma unroll
    for (int k = 0; k < kVirt; ++k)
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) {
        const float z = pick_bf16(r[k], i);
        m = fmaxf(m, z);
        lo = fminf(lo, z);
      }
    const float ref = wave_max(m) * scale;
#pragma unroll
    for (int k = 0; k < kVirt; ++k)
#pragma unroll
      for (int g = 0; g < kEltsPerThread / 8; ++g) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) s += bonus_weight(pick_bf16(r[k], 8 * g + e), scale, ref);
        a[sub_of<DT, VEC>(8 * g, k)] = s;
      }
    *ref_out = ref;
  } else {
    // first pass: max and min; second pass over the same logits (now in
    // cache): the exponentials against the chunk reference
#pragma unroll kVirtUnroll<DT, VEC>
    for (int k = 0; k < kVirt; ++k) {
      float z[kEltsPerThread];
      load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * k, z);
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) {
        m = fmaxf(m, z[i]);
        lo = fminf(lo, z[i]);
      }
    }
    const float ref = wave_max(m) * scale;
    generic_chunk_sums<DT, VEC, false>(trow, nullptr, V, ch, a,
                                       [&](float z, float) { return bonus_weight(z, scale, ref); });
    *ref_out = ref;
  }
  const double w = finish_chunk(a, sub);
  const int bad = __ballot(m == INFINITY || lo == -INFINITY) != 0;
  *w_out = w;
  *bad_out = bad || !isfinite(w) || !isfinite(*ref_out);
}


// Greedy bonus row, one chunk, by one wavefront: the largest raw logit, the
// smallest token id holding it, and whether a NaN or +-inf logit was seen.
template <int DT, bool VEC>
__device__ inline void bonus_argmax_chunk(const char *trow, int64_t V, int64_t ch, float *zmax_out, int32_t *idx_out,
                                          int *bad_out) {
  const int lane = threadIdx.x & 63;
  if constexpr (VEC && DT == DSDE_BF16) {
    // pass 1 over the raw chunk in registers: max, min, and a sum that a NaN
    // propagates through (|z| <= 2^64 keeps finite sums finite); pass 2: the
    // lanes holding the maximum find its first token (slots of one
    // chunk-layout thread ascend in token order)
    RawBf16 r[kVirt];
#pragma unroll
    for (int k = 0; k < kVirt; ++k) r[k] = load_raw_bf16(trow, V, ch, lane + 64 * k);
    float m = -INFINITY, lo = INFINITY, sum = 0.f;
#pragma unroll
    for (int k = 0; k < kVirt; ++k)
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) {
        const float z = pick_bf16(r[k], i);
        m = fmaxf(m, z);
        lo = fminf(lo, z);
        sum += z;
      }
    const float M = wave_max(m);
    uint32_t best = 0xffffffffu;
    if (m == M) {
#pragma unroll
      for (int k = 0; k < kVirt; ++k)
#pragma unroll
        for (int i = kEltsPerThread - 1; i >= 0; --i)
          if (pick_bf16(r[k], i) == M) {
            const uint32_t idx = uint32_t(Layout<DT, VEC>::index(ch, i, lane + 64 * k));
            best = idx < best ? idx : best;
          }
    }
    best = lanes::wave_min(best);
    *zmax_out = M;
    *idx_out = int32_t(best);
    *bad_out = __ballot(m == INFINITY || lo == -INFINITY || sum != sum) != 0;
  } else {
    float m = -INFINITY;
    uint32_t best = 0xffffffffu;
    int bad = 0;
#pragma unroll kVirtUnroll<DT, VEC>
    for (int k = 0; k < kVirt; ++k) {
      float z[kEltsPerThread];
      load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * k, z);
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) {
        const float v = z[i];  // padding is finite and below every admissible logit
        if (!isfinite(v)) bad = 1;
        const uint32_t idx = uint32_t(Layout<DT, VEC>::index(ch, i, lane + 64 * k));
        if (v > m || (v == m && idx < best)) {
          m = v;
          best = idx;
        }
      }
    }
    const float M = wave_max(m);
    uint32_t cand = m == M ? best : 0xffffffffu;
    cand = lanes::wave_min(cand);
    *zmax_out = M;
    *idx_out = int32_t(cand);
    *bad_out = __ballot(bad) != 0;
  }
}


// The inverse-CDF draw inside one row, by one wavefront, from the totals a
// chunk pass left behind: weight(ch) is chunk ch's draw weight (fp64, in the
// row's scale), subs holds 64 row partials of the 16 sub-block totals per
// chunk (chunk-major), and target is the weight to pass, in [0, row total).
// The rule at every level (chunk, sub-block, element) is the draw's: the last
// position with positive weight whose exclusive prefix is <= the target.
// Bonus rows (mode 2) carry a reference per chunk, chunk_ref(ch), and the row
// scale row_ref.  Returns the row-local token id in every lane.
template <int DT, bool VEC, typename WF, typename RF>
__device__ inline int32_t draw_in_row(int32_t nc, WF weight, RF chunk_ref, float row_ref, double target,
                                      const float *subs, const char *trow, const char *drow, int64_t V, int mode,
                                      const DrawJob &job) {
  const int lane = threadIdx.x & 63;
  int32_t best = -1;
  double best_excl = 0.0, base = 0.0;
  for (int32_t c0 = 0; c0 < nc; c0 += 64) {
    const int32_t ch = c0 + lane;
    const double w = ch < nc ? weight(ch) : 0.0;
    const lanes::Scan<double> sc = lanes::wave_scan(w);
    const double incl = base + sc.incl;
    const double excl = lane == 0 ? base : base + sc.excl;
    const uint64_t cand = __ballot(ch < nc && w > 0.0 && excl <= target);
    if (cand) {
      const int l = 63 - __builtin_clzll(cand);
      best = c0 + l;
      best_excl = lanes::readlane(excl, l);
    }
    base = lanes::readlane(incl, 63);
  }
  const int32_t chunk = best >= 0 ? best : 0;
  double rem = target - best_excl;
  if (rem < 0.0) rem = 0.0;
  const float ref = mode == 2 ? chunk_ref(chunk) : 0.f;
  if (mode == 2) rem *= exp2_taylor(double(row_ref) - double(ref));  // into the chunk's own scale

  // the sub-block
  double sbw = 0.0;
  if (lane < kSubs) {
    const float *r = subs + int64_t(chunk) * 64;
    sbw = double(((r[lane] + r[16 + lane]) + r[32 + lane]) + r[48 + lane]);
  }
  const lanes::Scan<double> ss = lanes::wave_scan(sbw);
  const uint64_t scand = __ballot(lane < kSubs && sbw > 0.0 && ss.excl <= rem);
  const int sb = scand ? 63 - __builtin_clzll(scand) : 0;
  double rem2 = rem - lanes::readlane(ss.excl, sb);
  if (rem2 < 0.0) rem2 = 0.0;

  // its 512 logits, 8 consecutive per lane
  const int64_t run0 = int64_t(chunk) * kChunk + int64_t(sb) * kSubLen + 8 * lane;
  float w[8];
  {
    float zt[8];
    load_run<DT, VEC, 8>(trow, V, run0, zt);
    if (mode == 0) {
      float zd[8];
      load_run<DT, VEC, 8>(drow, V, run0, zd);
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = residual_weight(zt[i], zd[i], job);
    } else if (mode == 1) {
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = target_p_weight(zt[i], job);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = bonus_weight(zt[i], job.scale, ref);
    }
  }
  double run_total = 0.0;
  int last = -1;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    run_total += double(w[i]);
    if (w[i] > 0.0f) last = i;
  }
  const lanes::Scan<double> sr = lanes::wave_scan(run_total);
  const uint64_t cand = __ballot(last >= 0 && sr.excl <= rem2);
  const int winner = cand ? 63 - __builtin_clzll(cand) : 0;
  int pick = last >= 0 ? last : 0;
  double acc = sr.excl;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    acc += double(w[i]);
    if (acc > rem2) {
      pick = i;
      break;
    }
  }
  return lanes::readlane(int32_t(run0 + pick), winner);
}
}  // namespace
}  // namespace dsde
