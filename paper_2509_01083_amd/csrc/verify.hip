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
//                      totals in LDS, a fixed-order fp64 prefix to the chunk
//                      holding u' * Z, and a block-wide ordered scan inside it.
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
          const double f0t = exp2(d0t), f0d = exp2(d0d), f1t = exp2(d1t), f1d = exp2(d1d);
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
      const double ft = exp2(dt), fd = exp2(dd);
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

// Total of the residual weights max(0, p - q) over one chunk of the rejected
// pair, by one wavefront (lane l plays the chunk-layout threads l + 64 k):
// per-thread fp32 sums in slot order, one wave sum per k, then the four in
// order in fp64.
template <int DT, bool VEC>
__device__ inline double residual_chunk(const char *trow, const char *drow, int64_t V, int64_t ch,
                                        const DrawJob &job) {
  const int lane = threadIdx.x & 63;
  float sw[kVirt];
  if constexpr (DT == DSDE_BF16 && VEC) {
    // every load of the chunk (both rows, all four chunk-layout threads: 32 KiB
    // per wavefront) is issued before any value is used, then the same sums in
    // the same order as below
    RawBf16 rt[kVirt], rd[kVirt];
#pragma unroll
    for (int k = 0; k < kVirt; ++k) {
      rt[k] = issue_raw_bf16(trow, V, ch, lane + 64 * k);
      rd[k] = issue_raw_bf16(drow, V, ch, lane + 64 * k);
    }
#pragma unroll
    for (int k = 0; k < kVirt; ++k) {
      const RawBf16 t_ = pad_raw_bf16(rt[k], V, ch, lane + 64 * k), d_ = pad_raw_bf16(rd[k], V, ch, lane + 64 * k);
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) {
        const float p = fast_exp2(fmaf(pick_bf16(t_, i), job.scale, -job.mt)) * job.inv_sp;
        const float q = fast_exp2(fmaf(pick_bf16(d_, i), job.scale, -job.md)) * job.inv_sq;
        a += fmaxf(p - q, 0.0f);
      }
      sw[k] = wave_sum(a);
    }
    double w = 0.0;
#pragma unroll
    for (int k = 0; k < kVirt; ++k) w += double(sw[k]);
    return w;
  }
#pragma unroll kVirtUnroll<DT, VEC>
  for (int k = 0; k < kVirt; ++k) {
    float zt[kEltsPerThread], zd[kEltsPerThread];
    load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * k, zt);
    load_chunk_f32<DT, VEC>(drow, V, ch, lane + 64 * k, zd);
    float a = 0.f;
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) {
      // padding gives p = q = 0, hence zero weight
      const float p = fast_exp2(fmaf(zt[i], job.scale, -job.mt)) * job.inv_sp;
      const float q = fast_exp2(fmaf(zd[i], job.scale, -job.md)) * job.inv_sq;
      a += fmaxf(p - q, 0.0f);
    }
    sw[k] = wave_sum(a);
  }
  double w = 0.0;
#pragma unroll
  for (int k = 0; k < kVirt; ++k) w += double(sw[k]);
  return w;
}

// Total of p over one chunk of the rejected pair's target row (the draw's
// fallback when the residual has no mass), in the same order.
template <int DT, bool VEC>
__device__ inline double target_p_chunk(const char *trow, int64_t V, int64_t ch, const DrawJob &job) {
  const int lane = threadIdx.x & 63;
  float sp[kVirt];
#pragma unroll kVirtUnroll<DT, VEC>
  for (int k = 0; k < kVirt; ++k) {
    float zt[kEltsPerThread];
    load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * k, zt);
    float b = 0.f;
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) b += fast_exp2(fmaf(zt[i], job.scale, -job.mt)) * job.inv_sp;
    sp[k] = wave_sum(b);
  }
  double p = 0.0;
#pragma unroll
  for (int k = 0; k < kVirt; ++k) p += double(sp[k]);
  return p;
}

// Bonus row, one chunk, by one wavefront: the chunk reference ref = max(z) c,
// the total of 2^(z c - ref), and whether a NaN or +-inf logit was seen (+inf
// shows in the max, NaN in the sum, -inf in the min; padding is finite).
template <int DT, bool VEC>
__device__ inline void bonus_chunk(const char *trow, int64_t V, int64_t ch, float scale, double *w_out,
                                   float *ref_out, int *bad_out) {
  const int lane = threadIdx.x & 63;
  float m = -INFINITY, lo = INFINITY;
  float sum[kVirt];
  if constexpr (VEC && DT == DSDE_BF16) {
    // one load: the raw chunk stays in registers for both passes
    RawBf16 r[kVirt];
#pragma unroll
    for (int k = 0; k < kVirt; ++k) r[k] = load_raw_bf16(trow, V, ch, lane + 64 * k);
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
    for (int k = 0; k < kVirt; ++k) {
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) a += fast_exp2(fmaf(pick_bf16(r[k], i), scale, -ref));
      sum[k] = a;
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
#pragma unroll kVirtUnroll<DT, VEC>
    for (int k = 0; k < kVirt; ++k) {
      float z[kEltsPerThread];
      load_chunk_f32<DT, VEC>(trow, V, ch, lane + 64 * k, z);
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i) a += fast_exp2(fmaf(z[i], scale, -ref));
      sum[k] = a;
    }
    *ref_out = ref;
  }
  double w = 0.0;
#pragma unroll
  for (int k = 0; k < kVirt; ++k) w += double(wave_sum(sum[k]));
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
//      wavefront 0: input checks, KLD, acceptance u < p(x)/q(x) (fp64), the
//      accepted tokens and the draw job.
//   2. wavefront w: the draw-weight totals of chunks w, w + 8, ... (residual
//      max(0, p - q) of the first rejected pair, or the bonus row), into LDS.
//   3. wavefront 0: fixed-order fp64 prefix over the chunk totals to the chunk
//      holding u' * Z, then the ordered scan inside it.
//   Fused: the last wavefront runs the signal update of the sequence between
//   steps 1 and 2.
template <int DT, bool VEC, bool FUSED, int NT>
__global__ __launch_bounds__(NT) void seq_kernel(const StepParams P, const SignalArgs S) {
  constexpr int kSeqThreads = NT;
  constexpr int kSeqWaves = NT / 64;
  constexpr int kSignalWave = kSeqWaves - 1;  // wavefront that runs the fused signal update
  __shared__ float st_mt[DSDE_MAX_K + 1], st_md[DSDE_MAX_K + 1];
  __shared__ double st_sp[DSDE_MAX_K + 1], st_sq[DSDE_MAX_K + 1], st_a[DSDE_MAX_K + 1], st_h[DSDE_MAX_K + 1];
  __shared__ int st_bad[DSDE_MAX_K + 1], st_arg[DSDE_MAX_K + 1];
  __shared__ float s_kld[64];
  __shared__ double ch_w[kMaxChunks], ch_p[kMaxChunks];
  __shared__ float ch_ref[kMaxChunks];
  __shared__ int ch_bad[kMaxChunks];
  __shared__ int32_t ch_arg[kMaxChunks];
  __shared__ DrawJob s_job;
  __shared__ int32_t s_chunk, s_mode, s_bad;
  __shared__ double s_rem;
  __shared__ float s_ref;
  __shared__ double s_wave_total[kSeqWaves];
  __shared__ int s_wave_cand[kSeqWaves];
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int32_t b = blockIdx.x;
  const int32_t width = P.k_max + 1;
  int32_t *tok = P.tokens + int64_t(b) * width;
  // first round trip: everything whose address depends on the sequence index
  // alone - the ring state (signal wavefront), this sequence's chunk partials
  // and gathered logits (stored by slot b * k_max + j; positions past SL_b are
  // fetched and ignored), and the per-sequence inputs
  // (every wavefront fetches the ring, a few hundred bytes, so that no branch
  // separates these loads from the rest of the round trip; only the signal
  // wavefront uses it)
  RingPrefetch rp{};
  if constexpr (FUSED) rp = wave_ring_prefetch(S.hist + int64_t(b) * S.W, S.head + b, S.count + b, S.W);
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
  if constexpr (FUSED) {
    pin(rp.head);
    pin(rp.count);
#pragma unroll
    for (int k = 0; k < kRingRegs; ++k) pin(rp.slot[k]);
  }
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
    float my_kld = 0.f, my_h = 0.f;
    if (active) {
      bad = st_bad[lane] != 0;
      const double sp = st_sp[lane], sq = st_sq[lane];
      const double l2sp = log2(sp), l2sq = log2(sq);
      // KL in log2 units: E_p[(z_t c - mt) - (z_d c - md)] - log2 S_p + log2 S_q
      const double kl = (st_a[lane] / sp - l2sp + l2sq) * kLn2;
      my_kld = kl > 0.0 ? float(kl) : 0.0f;
      // draft entropy in log2 units: log2 S_q - E_q[z_d c - md]
      my_h = float((l2sq - st_h[lane] / sq) * kLn2);
      // log2 p(x) - log2 q(x); z * c is exact in double
      const double lr = (double(gz.zt) * double(c) - double(st_mt[lane]) - l2sp) -
                        (double(gz.zd) * double(c) - double(st_md[lane]) - l2sq);
      // greedy: accept iff the drafted token is the target row's argmax
      ok = greedy ? x == st_arg[lane] : double(u) < exp2(lr);
      if (!bad && P.row_lse) {
        P.row_lse[2 * (first + lane)] = (double(st_mt[lane]) + l2sp) * kLn2;
        P.row_lse[2 * (first + lane) + 1] = (double(st_md[lane]) + l2sq) * kLn2;
      }
    }
    if (__ballot(bad)) err |= DSDE_ERR_LOGIT;
    const uint64_t mask = __ballot(ok);
    int32_t a = int32_t(__builtin_ctzll(~mask));
    if (a > s) a = s;
    if (err) {
      a = 0;
      my_kld = NAN;
      my_h = NAN;
    }
    if (lane < s) P.kld[first + lane] = my_kld;
    if (lane < s && P.entropy) P.entropy[first + lane] = my_h;
    s_kld[lane] = my_kld;
    if (lane < width) tok[lane] = lane < a ? x : P.pad_id;
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
          j.token = st_arg[a];
          tok[a] = st_arg[a];
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
          j.mt = st_mt[a];
          j.md = st_md[a];
          j.inv_sp = float(1.0 / st_sp[a]);
          j.inv_sq = float(1.0 / st_sq[a]);
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
  const DrawJob job = s_job;

  if constexpr (FUSED) {
    if (wave == kSignalWave) {
      // the signal update of Sec. 3.1.2 on the KLD values just computed, before
      // this wavefront's share of the draw stream (the last wavefront has the
      // fewest chunks), so that it is off the path of the chunk search
      const uint32_t e = wave_signal_update(s, first, nullptr, s_kld[lane], rp, S.hist + int64_t(b) * S.W,
                                            S.head + b, S.count + b, S.W, S.n_short, S.n_long, S.delta, S.eps,
                                            S.mu_last + b, S.var_short + b, S.var_long + b, S.wvir + b, S.sf + b);
      if (e && lane == 0) atomicOr(&P.seq_err[b], e);
    }
  }

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
        const double w = residual_chunk<DT, VEC>(trow, drow, P.V, ch, job);
        if (lane == 0) ch_w[ch] = w;
      }
    } else {
      for (int32_t ch = wave; ch < nc; ch += kSeqWaves) {
        double w;
        float ref;
        int bad;
        bonus_chunk<DT, VEC>(trow, P.V, ch, job.scale, &w, &ref, &bad);
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
          const double p = target_p_chunk<DT, VEC>(trow, P.V, ch, job);
          if (lane == 0) ch_p[ch] = p;
        }
        __syncthreads();
      }
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

  // ---- 3. the chunk holding u' * Z (wavefront 0, lanes over chunks, fixed-order fp64)
  if (wave == 0) {
    int mode = job.kind == 0 ? 0 : 2;  // 0: residual weights, 1: p of the rejected pair, 2: bonus exponentials
    float ref_max = -INFINITY;
    int bad = 0;
    if (mode == 2) {
      for (int32_t ch = lane; ch < nc; ch += 64) {
        bad |= ch_bad[ch];
        ref_max = fmaxf(ref_max, ch_ref[ch]);
      }
      ref_max = wave_max(ref_max);
      bad = lanes::wave_or(bad);
    }
    auto weight = [&](int32_t ch, int m) -> double {
      return m == 0 ? ch_w[ch] : m == 1 ? ch_p[ch] : ch_w[ch] * exp2(double(ch_ref[ch]) - double(ref_max));
    };
    int32_t best = -1;
    double best_excl = 0.0, Z = 0.0;
    if (!bad) {
      double part = 0.0;
      for (int32_t ch = lane; ch < nc; ch += 64) part += weight(ch, mode);
      Z = wave_sum_f64(part);
      if (mode == 0 && !(Z > 0.0)) {  // no residual mass: p of the same target row
        mode = 1;
        part = 0.0;
        for (int32_t ch = lane; ch < nc; ch += 64) part += weight(ch, 1);
        Z = wave_sum_f64(part);
      }
      const double target_mass = double(job.u) * Z;
      // inclusive scan 64 chunks at a time; the chunk holding the target is
      // the last one with positive weight whose exclusive prefix is <= the
      // target (prefixes tile exactly: each chunk's start is the previous
      // chunk's end), which also covers rounding past the total
      double base = 0.0;
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
      if (lane == 0) {
        const int32_t chunk = best >= 0 ? best : 0;
        double rem = target_mass - best_excl;
        if (rem < 0.0) rem = 0.0;
        float ref = 0.f;
        if (mode == 2) {
          ref = ch_ref[chunk];
          rem *= exp2(double(ref_max) - double(ref));  // into the chunk's own scale
        }
        s_chunk = chunk;
        s_rem = rem;
        s_ref = ref;
      }
    }
    if (lane == 0) {
      s_mode = mode;
      s_bad = bad;
    }
  }
  __syncthreads();
  if (s_bad) {
    // a NaN or infinite logit in the bonus row: no token is emitted
    if (wave == 0) {
      if (lane < width) tok[lane] = P.pad_id;
      if (lane == 0) {
        P.accepted[b] = 0;
        atomicOr(&P.seq_err[b], err | DSDE_ERR_LOGIT);
      }
    }
    return;
  }

  // ---- 4. the ordered scan inside that chunk: thread t holds the 16
  // consecutive logits from chunk * 8192 + 16 t; per-thread totals in token
  // order, a block-wide inclusive scan, and the thread holding the target
  // walks its own weights
  const int mode = s_mode;
  const int64_t chunk = s_chunk;
  const double rem = s_rem;
  const float ref = s_ref;
  const char *trow = (const char *)P.target + size_t(job.target_row) * size_t(P.V) * esz;
  constexpr int kRun = kChunk / kSeqThreads;  // 16 or 32
  const int64_t run0 = chunk * kChunk + int64_t(kRun) * t;
  float w[kRun];
  {
    float zt[kRun];
    load_run<DT, VEC, kRun>(trow, P.V, run0, zt);
    if (mode == 0) {
      float zd[kRun];
      const char *drow = (const char *)P.draft + size_t(job.draft_row) * size_t(P.V) * esz;
      load_run<DT, VEC, kRun>(drow, P.V, run0, zd);
#pragma unroll
      for (int i = 0; i < kRun; ++i) {
        const float p = fast_exp2(fmaf(zt[i], job.scale, -job.mt)) * job.inv_sp;
        const float q = fast_exp2(fmaf(zd[i], job.scale, -job.md)) * job.inv_sq;
        w[i] = fmaxf(p - q, 0.0f);
      }
    } else if (mode == 1) {
#pragma unroll
      for (int i = 0; i < kRun; ++i) w[i] = fast_exp2(fmaf(zt[i], job.scale, -job.mt)) * job.inv_sp;
    } else {
#pragma unroll
      for (int i = 0; i < kRun; ++i) w[i] = fast_exp2(fmaf(zt[i], job.scale, -ref));
    }
  }
  double run_total = 0.0;
  int last = -1;  // this thread's last positive weight
#pragma unroll
  for (int i = 0; i < kRun; ++i) {
    run_total += double(w[i]);
    if (w[i] > 0.0f) last = i;
  }
  const lanes::Scan<double> sc = lanes::wave_scan(run_total);
  if (lane == 63) s_wave_total[wave] = sc.incl;
  __syncthreads();
  double base = 0.0;
  for (int v = 0; v < wave; ++v) base += s_wave_total[v];
  const double excl = lane == 0 ? base : base + sc.excl;
  // the thread holding the target: the last one with positive weight whose
  // exclusive prefix is <= the target (rounding past the chunk's total lands
  // on its last positive weight)
  const uint64_t cand = __ballot(last >= 0 && excl <= rem);
  if (lane == 0) s_wave_cand[wave] = cand ? 64 * wave + 63 - __builtin_clzll(cand) : -1;
  __syncthreads();
  int winner = -1;
#pragma unroll
  for (int v = 0; v < kSeqWaves; ++v) winner = max(winner, s_wave_cand[v]);
  if (t == (winner >= 0 ? winner : 0)) {
    int pick = last >= 0 ? last : 0;
    double acc = excl;
#pragma unroll
    for (int i = 0; i < kRun; ++i) {
      acc += double(w[i]);
      if (acc > rem) {
        pick = i;
        break;
      }
    }
    tok[job.accepted] = int32_t(run0 + pick);
    if (err) atomicOr(&P.seq_err[b], err);
  }
}

}  // namespace

// Dynamic LDS of more than half a CU's LDS (see launch_seq); 0 when the
// runtime does not allow it.  Set up once per kernel.
template <typename K>
static size_t spread_lds(K kernel) {
  int dev = 0, lds = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) != hipSuccess ||
      lds <= 0) {
    (void)hipGetLastError();
    return 0;
  }
  const size_t bytes = size_t(lds) / 2 + 1;
  if (hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                          int(bytes)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return bytes;
}

template <int DT, bool VEC>
static void launch_seq(const VerifyArgs &a, const StepParams &P, const SignalArgs &S) {
  // With no more sequences than CUs: 512 threads per sequence, one sequence
  // per CU.  Two such workgroups would fit on one CU, and the dispatcher could
  // pair them up on half of the CUs, each pair then sharing one CU's load
  // bandwidth; reserving more than half of the CU's LDS per workgroup (unused)
  // places one sequence per CU.  With more sequences: 256 threads per sequence
  // and no reservation, so that several share a CU.
  static const size_t spread_fused = spread_lds(seq_kernel<DT, VEC, true, kSeqThreadsWide>);
  static const size_t spread_plain = spread_lds(seq_kernel<DT, VEC, false, kSeqThreadsWide>);
  int dev = 0, ncu = 0;
  const bool few = hipGetDevice(&dev) == hipSuccess &&
                   hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                   a.B <= ncu;
  (void)hipGetLastError();
  const dim3 grid(unsigned(a.B));
  if (few) {
    const dim3 block(kSeqThreadsWide);
    if (a.signal)
      seq_kernel<DT, VEC, true, kSeqThreadsWide><<<grid, block, spread_fused, a.stream>>>(P, S);
    else
      seq_kernel<DT, VEC, false, kSeqThreadsWide><<<grid, block, spread_plain, a.stream>>>(P, S);
  } else {
    const dim3 block(kSeqThreadsNarrow);
    if (a.signal)
      seq_kernel<DT, VEC, true, kSeqThreadsNarrow><<<grid, block, 0, a.stream>>>(P, S);
    else
      seq_kernel<DT, VEC, false, kSeqThreadsNarrow><<<grid, block, 0, a.stream>>>(P, S);
  }
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
  if (a.dtype == DSDE_BF16) {
    if (vec)
      launch_seq<DSDE_BF16, true>(a, P, S);
    else
      launch_seq<DSDE_BF16, false>(a, P, S);
  } else {
    if (vec)
      launch_seq<DSDE_FP32, true>(a, P, S);
    else
      launch_seq<DSDE_FP32, false>(a, P, S);
  }
  if (hipGetLastError() != hipSuccess) return DSDE_DEVICE_ERROR;
  if (a.signal)
    return launch_next_sl(a.B, S.sf, S.wvir, S.sl_max, S.sl_min, S.sl_hi, S.budget, S.sl_hat, S.sl_cap, S.sl_next,
                          a.seq_err, true, a.stream);
  return DSDE_OK;
}

}  // namespace dsde
