// Batched speculative verification with ragged per-sequence speculation
// lengths on gfx950 (speculative sampling, Sec. 2.1; ragged layout, bonus and
// pad, Sec. 3.2; per-token KLD of the SL adapter, Sec. 3.1.2).
//
// Kernels, in launch order on the caller's stream:
//   setup_kernel, stats_kernel   (stats.hip) layout check, work list, and the
//                      row statistics of every drafted pair, chunk by chunk.
//   seq_kernel         one workgroup per sequence: combines the chunk partials
//                      of its drafted pairs (fp64), KLD, acceptance u < p(x)/q(x)
//                      (fp64) up to the first rejection, then the draw: the
//                      residual max(0, p - q) of the rejected pair (or the bonus
//                      row) streamed one wavefront per chunk with the chunk
//                      and sub-block totals in LDS, then one wavefront: a
//                      fixed-order fp64 prefix to the chunk holding u' * Z, the
//                      same over its 16 sub-blocks, and an ordered scan of the
//                      512 logits of the sub-block found.
//                      Fused step: one wavefront also runs the signal update.
//   next_sl_kernel     (signal.hip, fused step only) batch cap and next lengths.
//
// Every reduction runs in a fixed order, so results are bitwise reproducible.
#include <math.h>

#include "common.hpp"
#include "row_io.hpp"
#include "signal_device.hpp"

namespace dsde {
namespace {

// ---------------------------------------------------------------------------
// per-sequence kernel: acceptance, draw weights and draw
// ---------------------------------------------------------------------------

// Threads per sequence: 512 (8 wavefronts) when every sequence has a CU of its
// own, 256 when sequences outnumber the CUs (then three workgroups share a CU
// and each one's latency-bound phases overlap the others' row streams).
constexpr int kSeqThreadsWide = 512;
constexpr int kSeqThreadsNarrow = 256;
constexpr int kVirt = kThreads / 64;          // chunk-layout threads played by one lane (4)

// How many of a lane's chunk-layout threads one loop iteration handles: as
// many as the registers allow loads in flight for.
template <int DT, bool VEC>
constexpr int kVirtUnroll = !VEC ? 1 : DT == DSDE_BF16 ? kVirt : 2;

struct StepParams {
  const void *target, *draft;
  int64_t V;
  int32_t B, k_max, nc, pad_id;
  const int32_t *sl, *cu_sl, *draft_tokens;
  const float *temperature, *u_acc, *u_res;
  int32_t *accepted, *tokens;
  float *kld;
  uint32_t *seq_err;
  double *row_lse;
  float *entropy;  // draft entropy per drafted position (nats), may be null
  const PairChunk *part;
  const Gathered *gathered;
  const ChunkArg *chunk_arg;  // greedy pairs: the target row's maximum and argmax per chunk
};

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

// Combines the chunk partials of every drafted pair of one sequence (stored
// under slots slot0 + j): groups of G lanes, one pair per group, lane g of a
// group folds chunks g, g + G, ...  Results go to LDS (st_*[j] for position j).
template <int G, int WAVES>
__device__ inline void combine_pairs(const PairChunk *__restrict__ part, int64_t slot0, int32_t s, int32_t nc,
                                     const PairChunk &q0, const ChunkArg *__restrict__ chunk_arg, ChunkArg arg0,
                                     float *st_mt, float *st_md, double *st_sp, double *st_sq, double *st_a,
                                     double *st_h, int *st_bad, int *st_arg) {
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
          const float nt = fmaxf(lmt, q.mt), nd = fmaxf(lmd, q.md);
          const double d0t = double(lmt) - nt, d0d = double(lmd) - nd;
          const double d1t = double(q.mt) - nt, d1d = double(q.md) - nd;
          const double f0t = exp2_taylor(d0t), f0d = exp2_taylor(d0d), f1t = exp2_taylor(d1t), f1d = exp2_taylor(d1d);
          la = f0t * (la + lsp * (d0t - d0d)) + f1t * (q.a + q.sp * (d1t - d1d));
          lh = f0d * (lh + lsq * d0d) + f1d * (q.h + q.sq * d1d);
          lsp = f0t * lsp + f1t * q.sp;
          lsq = f0d * lsq + f1d * q.sq;
          lmt = nt;
          lmd = nd;
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
    if (chunk_arg) {  // the row argmax: smallest token among the chunks holding the row maximum
      const float zm = group_max<G>(lz);
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

// One workgroup per sequence.
//   1. all wavefronts: combine the chunk partials of the drafted pairs (fp64);
//      wavefront 0: input checks, acceptance u < p(x)/q(x) (fp64), the
//      accepted tokens and the draw job.  The last wavefront then writes the
//      KLD (and entropy, log-normalisers) of every position and, fused, runs
//      the signal update of the sequence.
//   2. wavefront w: the draw-weight totals of chunks w, w + 8, ... (residual
//      max(0, p - q) of the first rejected pair, or the bonus row), into LDS.
//   3. wavefront 0: fixed-order fp64 prefix over the chunk totals to the chunk
//      holding u' * Z, the same over that chunk's sub-block totals, then the
//      ordered scan of the sub-block (the other wavefronts are done).
template <int DT, bool VEC, bool FUSED, int NT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(NT == kSeqThreadsNarrow ? 3 : 1))) void seq_kernel(
    const StepParams P, const SignalArgs S) {
  constexpr int kSeqWaves = NT / 64;
  constexpr int kSignalWave = kSeqWaves - 1;  // wavefront of the KLD outputs and the fused signal update
  __shared__ float st_mt[DSDE_MAX_K + 1], st_md[DSDE_MAX_K + 1];
  __shared__ double st_sp[DSDE_MAX_K + 1], st_sq[DSDE_MAX_K + 1], st_a[DSDE_MAX_K + 1], st_h[DSDE_MAX_K + 1];
  __shared__ int st_bad[DSDE_MAX_K + 1], st_arg[DSDE_MAX_K + 1];
  __shared__ uint32_t s_err_in, s_err;  // error bits before and after the row checks
  __shared__ double ch_w[kMaxChunks], ch_p[kMaxChunks];
  __shared__ float ch_ref[kMaxChunks];
  __shared__ int ch_bad[kMaxChunks];
  __shared__ int32_t ch_arg[kMaxChunks];
  extern __shared__ float s_sub[];  // 64 row partials of the 16 sub-block totals, per chunk
  __shared__ DrawJob s_job;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // uniform: chunk indices and addresses stay scalar
  const int32_t b = blockIdx.x;
  const int32_t width = P.k_max + 1;
  int32_t *tok = P.tokens + int64_t(b) * width;
  // first round trip: everything whose address depends on the sequence index
  // alone - this sequence's chunk partials and gathered logits (stored by slot
  // b * k_max + j; positions past SL_b are fetched and ignored), and the
  // per-sequence inputs
  const int G = P.nc <= 16 ? 16 : P.nc <= 32 ? 32 : 64;
  const int32_t j0 = wave * (64 / G) + lane / G, g0 = lane % G;
  const int64_t slot0 = int64_t(b) * P.k_max;
  PairChunk q0{};
  if (j0 < P.k_max && g0 < P.nc) q0 = P.part[(slot0 + j0) * P.nc + g0];
  ChunkArg arg0{0.f, 0};  // greedy pairs only; fetched regardless, it costs no extra round trip
  if (j0 < P.k_max && g0 < P.nc) arg0 = P.chunk_arg[(slot0 + j0) * P.nc + g0];
  Gathered gz{0.f, 0.f};
  if (wave == 0 && lane < P.k_max) gz = P.gathered[slot0 + lane];
  uint32_t err = P.seq_err[b];  // the set-up's layout verdict
  const int32_t s = P.sl[b], first = P.cu_sl[b];
  const float T = P.temperature[b], ur = P.u_res[b];
  // one wait for the whole first round trip: every load above is issued
  // before any of the pins below asks for its value
  asm volatile("" ::: "memory");
  pin(q0.mt);
  pin(q0.md);
  pin(q0.sp);
  pin(q0.sq);
  pin(q0.a);
  pin(gz.zt);
  pin(gz.zd);
  pin(arg0.zmax);
  pin(arg0.idx);
  if (err & DSDE_ERR_LAYOUT) {
    if (t < width) tok[t] = P.pad_id;
    if (t == 0) {
      P.accepted[b] = 0;
      if constexpr (FUSED) S.mu_last[b] = S.var_short[b] = S.var_long[b] = S.wvir[b] = S.sf[b] = NAN;
    }
    return;
  }
  // T_b = 0: greedy verification (statistics at T = 1, uniforms unused)
  const bool greedy = T == 0.0f;
  const ChunkArg *cargs = greedy ? P.chunk_arg : nullptr;
  // per-position inputs of wavefront 0 (lane j = drafted position j)
  int32_t x = 0;
  float u = 0.f;
  if (wave == 0 && lane < s) {
    x = P.draft_tokens[first + lane];
    u = P.u_acc[first + lane];
  }

  // ---- 1. acceptance
  // row statistics of every drafted pair (read even for a flagged sequence:
  // the layout is valid, so every access stays in bounds)
  if (s > 0) {
    if (G == 16)
      combine_pairs<16, kSeqWaves>(P.part, slot0, s, P.nc, q0, cargs, arg0, st_mt, st_md, st_sp, st_sq, st_a,
                                    st_h, st_bad, st_arg);
    else if (G == 32)
      combine_pairs<32, kSeqWaves>(P.part, slot0, s, P.nc, q0, cargs, arg0, st_mt, st_md, st_sp, st_sq, st_a,
                                    st_h, st_bad, st_arg);
    else
      combine_pairs<64, kSeqWaves>(P.part, slot0, s, P.nc, q0, cargs, arg0, st_mt, st_md, st_sp, st_sq, st_a,
                                    st_h, st_bad, st_arg);
  }
  __syncthreads();
  if (wave == 0) {
    {  // per-sequence input checks
      uint32_t e = 0;
      if (lane < s) {
        if (x < 0 || int64_t(x) >= P.V) e |= DSDE_ERR_TOKEN;
        if (!greedy && !(u >= 0.0f && u < 1.0f)) e |= DSDE_ERR_UNIFORM;
      }
      if (lane == 0 && !greedy) {
        if (!(T >= kMinTemp && T <= kMaxTemp)) e |= DSDE_ERR_TEMP;
        if (!(ur >= 0.0f && ur < 1.0f)) e |= DSDE_ERR_UNIFORM;
      }
      err |= lanes::wave_or(e);
    }
    const float c = greedy ? kLog2e : kLog2e / T;  // the same values as the set-up's scale
    const bool active = lane < s && !err;
    bool ok = false, bad = false;
    float my_mt = 0.f, my_md = 0.f, my_isp = 0.f, my_isq = 0.f;
    int32_t my_arg = 0;
    if (lane == 0) s_err_in = err;  // the KLD wavefront writes the log-normalisers of unflagged sequences
    if (active) {
      bad = st_bad[lane] != 0;
      const double sp = st_sp[lane], sq = st_sq[lane];
      my_mt = st_mt[lane];
      my_md = st_md[lane];
      my_arg = st_arg[lane];
      my_isp = float(rcp_newton(sp));
      my_isq = float(rcp_newton(sq));
      if (greedy) {
        ok = x == my_arg;  // accept iff the drafted token is the target row's argmax
      } else {
        // u < p(x) / q(x) with p(x) = 2^(z_t(x) c - mt) / S_p and q(x) = 2^(z_d(x) c - md) / S_q,
        // tested as u S_p < 2^D S_q (no logarithm on this path; z c is exact in double)
        const double D = (double(gz.zt) * double(c) - double(my_mt)) - (double(gz.zd) * double(c) - double(my_md));
        ok = double(u) * sp < exp2_taylor(D) * sq;
      }
    }
    if (__ballot(bad)) err |= DSDE_ERR_LOGIT;
    const uint64_t mask = __ballot(ok);
    int32_t a = int32_t(__builtin_ctzll(~mask));
    if (a > s) a = s;
    if (err) a = 0;
    if (lane == 0) s_err = err;
    if (lane < width) tok[lane] = lane < a ? x : P.pad_id;
    // the first rejected position's row values, from its lane
    const float a_mt = lanes::readlane(my_mt, a), a_md = lanes::readlane(my_md, a);
    const float a_isp = lanes::readlane(my_isp, a), a_isq = lanes::readlane(my_isq, a);
    const int32_t a_arg = lanes::readlane(my_arg, a);
    if (lane == 0) {
      P.accepted[b] = a;
      DrawJob j{};
      j.kind = -1;
      if (!err && greedy) {
        j.accepted = a;
        j.target_row = first + b + a;
        j.draft_row = -1;
        if (a < s) {  // the argmax of the first rejected row is known already
          j.kind = 2;
          j.token = a_arg;
          tok[a] = a_arg;
        } else {      // the argmax of the bonus row
          j.kind = 3;
        }
      } else if (!err) {
        j.accepted = a;
        j.scale = c;
        j.u = ur;
        if (a < s) {
          j.kind = 0;
          j.target_row = first + b + a;
          j.draft_row = first + a;
          j.mt = a_mt;
          j.md = a_md;
          j.inv_sp = a_isp;
          j.inv_sq = a_isq;
        } else {
          j.kind = 1;
          j.target_row = first + b + s;
          j.draft_row = -1;
        }
      }
      s_job = j;
    }
  }
  __syncthreads();
  const DrawJob job = uniform_job(s_job);

  // ---- 2. draw-weight totals of every chunk
  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const int32_t nc = P.nc;
  if (job.kind == 3) {
    const char *trow = (const char *)P.target + size_t(job.target_row) * size_t(P.V) * esz;
    for (int32_t ch = wave; ch < nc; ch += kSeqWaves) {
      float zmax;
      int32_t idx;
      int bad;
      bonus_argmax_chunk<DT, VEC>(trow, P.V, ch, &zmax, &idx, &bad);
      if (lane == 0) {
        ch_ref[ch] = zmax;
        ch_arg[ch] = idx;
        ch_bad[ch] = bad;
      }
    }
    __syncthreads();
  } else if (job.kind == 0 || job.kind == 1) {
    const char *trow = (const char *)P.target + size_t(job.target_row) * size_t(P.V) * esz;
    if (job.kind == 0) {
      const char *drow = (const char *)P.draft + size_t(job.draft_row) * size_t(P.V) * esz;
      for (int32_t ch = wave; ch < nc; ch += kSeqWaves) {
        const double w = residual_chunk<DT, VEC>(trow, drow, P.V, ch, job, s_sub + int64_t(ch) * 64);
        if (lane == 0) ch_w[ch] = w;
      }
    } else {
      for (int32_t ch = wave; ch < nc; ch += kSeqWaves) {
        double w;
        float ref;
        int bad;
        bonus_chunk<DT, VEC>(trow, P.V, ch, job.scale, &w, &ref, &bad, s_sub + int64_t(ch) * 64);
        if (lane == 0) {
          ch_w[ch] = w;
          ch_ref[ch] = ref;
          ch_bad[ch] = bad;
        }
      }
    }
    __syncthreads();
    if (job.kind == 0) {
      // the residual's total mass, evaluated identically by every wavefront;
      // without mass the draw falls back to p, whose chunk totals come next
      double part = 0.0;
      for (int32_t ch = lane; ch < nc; ch += 64) part += ch_w[ch];
      if (!(wave_sum_f64(part) > 0.0)) {
        for (int32_t ch = wave; ch < nc; ch += kSeqWaves) {
          const double p = target_p_chunk<DT, VEC>(trow, P.V, ch, job, s_sub + int64_t(ch) * 64);
          if (lane == 0) ch_p[ch] = p;
        }
        __syncthreads();
      }
    }
  }

  if (wave == kSignalWave) {
    // the KLD of every drafted position (lane j: position j), its draft
    // entropy and row log-normalisers, and in the fused step the signal update
    // of Sec. 3.1.2 on those KLD values: on the last wavefront after the last
    // barrier, beside wavefront 0's chunk search and final scan, so that none
    // of it delays the draw (the draw stream is VALU-bound: work added to any
    // wavefront before the barrier lengthens it)
    // the ring state, fetched here: its round trip overlaps the KLD arithmetic
    RingPrefetch rp{};
    if constexpr (FUSED) rp = wave_ring_prefetch(S.hist + int64_t(b) * S.W, S.head + b, S.count + b, S.W);
    const uint32_t e_in = s_err_in, e_all = s_err;
    float my_kld = NAN, my_h = NAN;
    if (lane < s && !e_in) {
      const double sp = st_sp[lane], sq = st_sq[lane];
      const double l2sp = log2_rowsum(sp), l2sq = log2_rowsum(sq);
      // KL in log2 units: E_p[(z_t c - mt) - (z_d c - md)] - log2 S_p + log2 S_q
      const double kl = (st_a[lane] * rcp_newton(sp) - l2sp + l2sq) * kLn2;
      // draft entropy in log2 units: log2 S_q - E_q[z_d c - md]
      const double h = (l2sq - st_h[lane] * rcp_newton(sq)) * kLn2;
      if (!e_all) {
        my_kld = kl > 0.0 ? float(kl) : 0.0f;
        my_h = float(h);
      }
      if (!st_bad[lane] && P.row_lse) {
        P.row_lse[2 * (first + lane)] = (double(st_mt[lane]) + l2sp) * kLn2;
        P.row_lse[2 * (first + lane) + 1] = (double(st_md[lane]) + l2sq) * kLn2;
      }
    }
    if (lane < s) P.kld[first + lane] = my_kld;
    if (lane < s && P.entropy) P.entropy[first + lane] = my_h;
    if constexpr (FUSED) {
      const uint32_t e = wave_signal_update(s, first, nullptr, my_kld, rp, S.hist + int64_t(b) * S.W, S.head + b,
                                            S.count + b, S.W, S.n_short, S.n_long, S.delta, S.eps, S.mu_last + b,
                                            S.var_short + b, S.var_long + b, S.wvir + b, S.sf + b);
      if (e && lane == 0) atomicOr(&P.seq_err[b], e);
    }
  }

  if (job.kind < 0 || job.kind == 2) {  // flagged, or a greedy token already emitted
    if (err && wave == 0 && lane == 0) atomicOr(&P.seq_err[b], err);
    return;
  }
  if (job.kind == 3) {
    // greedy bonus: the chunk holding the row maximum (the earliest on ties)
    if (wave == 0) {
      float best = -INFINITY;
      int32_t bch = 0x7fffffff;
      int bad = 0;
      for (int32_t ch = lane; ch < nc; ch += 64) {
        bad |= ch_bad[ch];
        if (bch == 0x7fffffff || ch_ref[ch] > best) {
          best = ch_ref[ch];
          bch = ch;
        }
      }
      bad = lanes::wave_or(bad);
      const float M = wave_max(best);
      int32_t cand = bch != 0x7fffffff && best == M ? bch : 0x7fffffff;
      cand = lanes::wave_min(cand);
      if (bad) {
        // a NaN or infinite logit in the bonus row: no token is emitted
        if (lane < width) tok[lane] = P.pad_id;
        if (lane == 0) {
          P.accepted[b] = 0;
          atomicOr(&P.seq_err[b], DSDE_ERR_LOGIT);
        }
      } else if (lane == 0) {
        tok[job.accepted] = ch_arg[cand];
      }
    }
    return;
  }

  if (wave != 0) return;

  // ---- 3. wavefront 0: the chunk holding u' * Z (lanes over chunks,
  // fixed-order fp64), the sub-block inside it, and the token inside that
  int mode = job.kind == 0 ? 0 : 2;  // 0: residual weights, 1: p of the rejected pair, 2: bonus exponentials
  float ref_max = -INFINITY;
  if (mode == 2) {
    int bad = 0;
    for (int32_t ch = lane; ch < nc; ch += 64) {
      bad |= ch_bad[ch];
      ref_max = fmaxf(ref_max, ch_ref[ch]);
    }
    ref_max = wave_max(ref_max);
    if (lanes::wave_or(bad)) {
      // a NaN or infinite logit in the bonus row: no token is emitted
      if (lane < width) tok[lane] = P.pad_id;
      if (lane == 0) {
        P.accepted[b] = 0;
        atomicOr(&P.seq_err[b], err | DSDE_ERR_LOGIT);
      }
      return;
    }
  }
  auto weight = [&](int32_t ch, int m) -> double {
    return m == 0 ? ch_w[ch] : m == 1 ? ch_p[ch] : ch_w[ch] * exp2_taylor(double(ch_ref[ch]) - double(ref_max));
  };
  double part = 0.0;
  for (int32_t ch = lane; ch < nc; ch += 64) part += weight(ch, mode);
  double Z = wave_sum_f64(part);
  if (mode == 0 && !(Z > 0.0)) {  // no residual mass: p of the same target row
    mode = 1;
    part = 0.0;
    for (int32_t ch = lane; ch < nc; ch += 64) part += weight(ch, 1);
    Z = wave_sum_f64(part);
  }
  const double target_mass = double(job.u) * Z;
  // inclusive scan 64 chunks at a time; the chunk holding the target is the
  // last one with positive weight whose exclusive prefix is <= the target
  // (prefixes tile exactly: each chunk's start is the previous chunk's end),
  // which also covers rounding past the total
  int32_t best = -1;
  double best_excl = 0.0, base = 0.0;
  for (int32_t c0 = 0; c0 < nc; c0 += 64) {
    const int32_t ch = c0 + lane;
    const double w = ch < nc ? weight(ch, mode) : 0.0;
    const lanes::Scan<double> sc = lanes::wave_scan(w);
    const double incl = base + sc.incl;
    const double excl = lane == 0 ? base : base + sc.excl;
    const uint64_t cand = __ballot(ch < nc && w > 0.0 && excl <= target_mass);
    if (cand) {
      const int l = 63 - __builtin_clzll(cand);
      best = c0 + l;
      best_excl = lanes::readlane(excl, l);
    }
    base = lanes::readlane(incl, 63);
  }
  const int32_t chunk = best >= 0 ? best : 0;
  double rem = target_mass - best_excl;
  if (rem < 0.0) rem = 0.0;
  const float ref = mode == 2 ? ch_ref[chunk] : 0.f;
  if (mode == 2) rem *= exp2_taylor(double(ref_max) - double(ref));  // into the chunk's own scale

  // the sub-block: the same rule over the chunk's 16 sub-block totals
  double sbw = 0.0;
  if (lane < kSubs) {
    const float *r = s_sub + int64_t(chunk) * 64;
    sbw = double(((r[lane] + r[16 + lane]) + r[32 + lane]) + r[48 + lane]);
  }
  const lanes::Scan<double> ss = lanes::wave_scan(sbw);
  const uint64_t scand = __ballot(lane < kSubs && sbw > 0.0 && ss.excl <= rem);
  const int sb = scand ? 63 - __builtin_clzll(scand) : 0;
  double rem2 = rem - lanes::readlane(ss.excl, sb);
  if (rem2 < 0.0) rem2 = 0.0;

  // ---- 4. the 512 logits of that sub-block, 8 consecutive per lane, with the
  // weights evaluated by the routines of the totals; the lane holding the
  // target walks its own eight
  const int64_t run0 = int64_t(chunk) * kChunk + int64_t(sb) * kSubLen + 8 * lane;
  const char *trow = (const char *)P.target + size_t(job.target_row) * size_t(P.V) * esz;
  float w[8];
  {
    float zt[8];
    load_run<DT, VEC, 8>(trow, P.V, run0, zt);
    if (mode == 0) {
      float zd[8];
      const char *drow = (const char *)P.draft + size_t(job.draft_row) * size_t(P.V) * esz;
      load_run<DT, VEC, 8>(drow, P.V, run0, zd);
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
  int last = -1;  // this lane's last positive weight
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    run_total += double(w[i]);
    if (w[i] > 0.0f) last = i;
  }
  const lanes::Scan<double> sr = lanes::wave_scan(run_total);
  // the last lane with positive weight whose exclusive prefix is <= the target
  // (rounding past the sub-block's total lands on its last positive weight)
  const uint64_t cand = __ballot(last >= 0 && sr.excl <= rem2);
  const int winner = cand ? 63 - __builtin_clzll(cand) : 0;
  if (lane == winner) {
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
    tok[job.accepted] = int32_t(run0 + pick);
    if (err) atomicOr(&P.seq_err[b], err);
  }
}

}  // namespace

// Largest dynamic LDS a launch of `kernel` may ask for: the CU's LDS less the
// kernel's static LDS (0 when the runtime does not tell).  Set up once per
// kernel.
template <typename K>
static size_t dynamic_lds_limit(K kernel) {
  int dev = 0, lds = 0;
  hipFuncAttributes attr{};
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) != hipSuccess ||
      hipFuncGetAttributes(&attr, reinterpret_cast<const void *>(kernel)) != hipSuccess || lds <= 0 ||
      size_t(lds) <= attr.sharedSizeBytes) {
    (void)hipGetLastError();
    return 0;
  }
  const size_t bytes = size_t(lds) - attr.sharedSizeBytes;
  if (hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                          int(bytes)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return bytes;
}

template <typename K>
static int launch_one_seq(K kernel, size_t limit, size_t need, size_t spread, int B, int threads,
                          const StepParams &P, const SignalArgs &S, hipStream_t stream) {
  if (need > limit) return DSDE_DEVICE_ERROR;  // cannot happen within the vocabulary limit
  const size_t dyn = spread > need && spread <= limit ? spread : need;
  kernel<<<dim3(unsigned(B)), dim3(unsigned(threads)), dyn, stream>>>(P, S);
  return DSDE_OK;
}

template <int DT, bool VEC>
static int launch_seq(const VerifyArgs &a, const StepParams &P, const SignalArgs &S) {
  // Dynamic LDS: the sub-block partials, 256 bytes per chunk.  With no more
  // sequences than CUs: 512 threads per sequence, one sequence per CU.  Two
  // such workgroups would fit on one CU, and the dispatcher could pair them
  // up on half of the CUs, each pair then sharing one CU's load bandwidth;
  // asking for more than half of the CU's LDS per workgroup places one
  // sequence per CU.  With more sequences: 256 threads per sequence and only
  // the LDS needed, so that several share a CU.
  static const size_t lim_wide_fused = dynamic_lds_limit(seq_kernel<DT, VEC, true, kSeqThreadsWide>);
  static const size_t lim_wide_plain = dynamic_lds_limit(seq_kernel<DT, VEC, false, kSeqThreadsWide>);
  static const size_t lim_narrow_fused = dynamic_lds_limit(seq_kernel<DT, VEC, true, kSeqThreadsNarrow>);
  static const size_t lim_narrow_plain = dynamic_lds_limit(seq_kernel<DT, VEC, false, kSeqThreadsNarrow>);
  int dev = 0, ncu = 0, lds = 0;
  const bool known = hipGetDevice(&dev) == hipSuccess &&
                     hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                     hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) ==
                         hipSuccess;
  (void)hipGetLastError();
  const bool few = known && a.B <= ncu;
  const size_t need = size_t(P.nc) * 64 * sizeof(float);
  const size_t spread = known ? size_t(lds) / 2 + 1 : 0;
  if (few) {
    if (a.signal)
      return launch_one_seq(seq_kernel<DT, VEC, true, kSeqThreadsWide>, lim_wide_fused, need, spread, a.B,
                            kSeqThreadsWide, P, S, a.stream);
    return launch_one_seq(seq_kernel<DT, VEC, false, kSeqThreadsWide>, lim_wide_plain, need, spread, a.B,
                          kSeqThreadsWide, P, S, a.stream);
  }
  if (a.signal)
    return launch_one_seq(seq_kernel<DT, VEC, true, kSeqThreadsNarrow>, lim_narrow_fused, need, 0, a.B,
                          kSeqThreadsNarrow, P, S, a.stream);
  return launch_one_seq(seq_kernel<DT, VEC, false, kSeqThreadsNarrow>, lim_narrow_plain, need, 0, a.B,
                        kSeqThreadsNarrow, P, S, a.stream);
}

int launch_verify(const VerifyArgs &a) {
  const WorkspaceLayout L = workspace_layout(a.B, a.N, a.V, a.k_max);
  const int32_t nc = int32_t(num_chunks(a.V));
  char *ws = (char *)a.workspace;
  WorkItem *work = (WorkItem *)(ws + L.work);
  PairChunk *part = (PairChunk *)(ws + L.pair_chunk);
  Gathered *gath = (Gathered *)(ws + L.gathered);
  (void)hipGetLastError();
  ChunkArg *cargs = (ChunkArg *)(ws + L.chunk_arg);
  launch_stats_pass(a, work, part, gath, cargs);
  const bool vec = rows_vectorizable(a);
  StepParams P;
  P.target = a.target;
  P.draft = a.draft;
  P.V = a.V;
  P.B = a.B;
  P.k_max = a.k_max;
  P.nc = nc;
  P.pad_id = a.pad_id;
  P.sl = a.sl;
  P.cu_sl = a.cu_sl;
  P.draft_tokens = a.draft_tokens;
  P.temperature = a.temperature;
  P.u_acc = a.u_acc;
  P.u_res = a.u_res;
  P.accepted = a.accepted;
  P.tokens = a.tokens;
  P.kld = a.kld;
  P.seq_err = a.seq_err;
  P.row_lse = a.row_lse;
  P.entropy = a.draft_entropy;
  P.part = part;
  P.gathered = gath;
  P.chunk_arg = cargs;
  const SignalArgs S = a.signal ? *a.signal : SignalArgs{};
  int st;
  if (a.dtype == DSDE_BF16)
    st = vec ? launch_seq<DSDE_BF16, true>(a, P, S) : launch_seq<DSDE_BF16, false>(a, P, S);
  else
    st = vec ? launch_seq<DSDE_FP32, true>(a, P, S) : launch_seq<DSDE_FP32, false>(a, P, S);
  if (st != DSDE_OK || hipGetLastError() != hipSuccess) return DSDE_DEVICE_ERROR;
  if (a.signal)
    return launch_next_sl(a.B, S.sf, S.wvir, S.sl_max, S.sl_min, S.sl_hi, S.budget, S.sl_hat, S.sl_cap, S.sl_next,
                          a.seq_err, true, a.stream);
  return DSDE_OK;
}

}  // namespace dsde
