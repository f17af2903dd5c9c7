// Batched speculative verification with ragged per-sequence speculation
// lengths on gfx950: row statistics + per-token KLD, acceptance scan, and the
// inverse-CDF draw from the residual max(0, p - q) or the bonus row.
//
// Kernels, in launch order on the caller's stream:
//   setup_kernel        one workgroup: validates the packed layout and the
//                       per-sequence inputs, writes seq_err and the per-pair
//                       (target row, scale) table.
//   pair_stats_kernel   one workgroup per (drafted pair, 8192-logit chunk):
//                       reads the chunk of the target and the draft row once
//                       and writes the chunk's max-shifted exponential sums of
//                       p and q and the KL accumulator.  Carries almost all HBM
//                       bytes of the step; bound by HBM bandwidth.
//   accept_kernel       one wavefront per sequence, one lane per drafted
//                       position: combines the chunk partials (fp64), writes
//                       the KLD, evaluates u < p(x)/q(x) for every position in
//                       fp64, and finds the first rejection with a ballot.
//   draw_chunk_kernel   one workgroup per (sequence, chunk) of the row the draw
//                       uses: chunk totals of max(0, p - q) (re-reading the
//                       rejected pair) or of the bonus row's exponentials.
//   draw_kernel         one workgroup per sequence: prefix over the chunk
//                       totals (fp64), then an ordered scan inside the one chunk
//                       that holds u' * Z.
//
// All reductions run in a fixed order, so results are bitwise reproducible.
#include <math.h>

#include "common.hpp"

namespace dsde {
namespace {

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// 2^x on the transcendental unit (about 1 ulp; results below 2^-126 flush to 0).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float load_logit(const void *base, int dtype, int64_t idx) {
  if (dtype == DSDE_BF16) return __uint_as_float(uint32_t(((const uint16_t *)base)[idx]) << 16);
  return ((const float *)base)[idx];
}

// One row chunk held in registers: z[0..n) are the chunk's logits owned by
// this thread, the rest are -inf.  Element i of the thread lives at
//   VEC bf16 : 8 * (chunk*1024 + (i/8)*256 + t) + i%8
//   VEC fp32 : 4 * (chunk*2048 + (i/4)*256 + t) + i%4
//   scalar   : chunk*8192 + i*256 + t
// so every wavefront load is contiguous (16 B per lane, or 2/4 B per lane in
// the scalar layout) and a thread's valid elements are a prefix of z.
template <int DT, bool VEC>
struct Layout;

template <>
struct Layout<DSDE_BF16, true> {
  static constexpr int kVecElts = 8;
  __device__ static int64_t index(int64_t chunk, int i, int t) {
    return 8 * (chunk * 1024 + (i / 8) * 256 + t) + (i % 8);
  }
};
template <>
struct Layout<DSDE_FP32, true> {
  static constexpr int kVecElts = 4;
  __device__ static int64_t index(int64_t chunk, int i, int t) {
    return 4 * (chunk * 2048 + (i / 4) * 256 + t) + (i % 4);
  }
};
template <int DT>
struct Layout<DT, false> {
  static constexpr int kVecElts = 1;
  __device__ static int64_t index(int64_t chunk, int i, int t) { return chunk * kChunk + int64_t(i) * 256 + t; }
};

template <int DT, bool VEC>
__device__ __forceinline__ int load_chunk(const void *row, int64_t V, int64_t chunk, int t, float (&z)[kEltsPerThread]) {
  int n = 0;
  if constexpr (VEC && DT == DSDE_BF16) {
    const uint4 *p = (const uint4 *)row;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int64_t vi = chunk * 1024 + g * 256 + t;
      if (vi * 8 < V) {
        const uint4 w = p[vi];
        z[g * 8 + 0] = bf_lo(w.x);
        z[g * 8 + 1] = bf_hi(w.x);
        z[g * 8 + 2] = bf_lo(w.y);
        z[g * 8 + 3] = bf_hi(w.y);
        z[g * 8 + 4] = bf_lo(w.z);
        z[g * 8 + 5] = bf_hi(w.z);
        z[g * 8 + 6] = bf_lo(w.w);
        z[g * 8 + 7] = bf_hi(w.w);
        n += 8;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) z[g * 8 + e] = -INFINITY;
      }
    }
  } else if constexpr (VEC) {
    const float4 *p = (const float4 *)row;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int64_t vi = chunk * 2048 + g * 256 + t;
      if (vi * 4 < V) {
        const float4 w = p[vi];
        z[g * 4 + 0] = w.x;
        z[g * 4 + 1] = w.y;
        z[g * 4 + 2] = w.z;
        z[g * 4 + 3] = w.w;
        n += 4;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) z[g * 4 + e] = -INFINITY;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) {
      const int64_t v = chunk * kChunk + int64_t(i) * 256 + t;
      if (v < V) {
        z[i] = load_logit(row, DT, v);
        ++n;
      } else {
        z[i] = -INFINITY;
      }
    }
  }
  return n;
}

// Block-wide max of one value per thread (all threads receive it).
__device__ __forceinline__ float block_max(float v, float *lds) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  v = wave_max(v);
  if (lane == 0) lds[wave] = v;
  __syncthreads();
  float m = lds[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) m = fmaxf(m, lds[w]);
  __syncthreads();
  return m;
}

// ---------------------------------------------------------------------------
// set-up
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(1024) void setup_kernel(int64_t V, int32_t B, int64_t N, int32_t k_max,
                                                     const int32_t *__restrict__ sl,
                                                     const int32_t *__restrict__ cu_sl,
                                                     const int32_t *__restrict__ draft_tokens,
                                                     const float *__restrict__ temperature,
                                                     const float *__restrict__ u_acc,
                                                     const float *__restrict__ u_res, uint32_t *__restrict__ seq_err,
                                                     PairInfo *__restrict__ pinfo) {
  int bad = 0;
  for (int32_t b = threadIdx.x; b < B; b += blockDim.x) {
    const int64_t s = sl[b];
    if (s < 0 || s > k_max || int64_t(cu_sl[b + 1]) - int64_t(cu_sl[b]) != s) bad = 1;
  }
  bad = __syncthreads_or(bad);
  if (cu_sl[0] != 0 || int64_t(cu_sl[B]) != N) bad = 1;

  if (bad) {
    for (int32_t b = threadIdx.x; b < B; b += blockDim.x) seq_err[b] = DSDE_ERR_LAYOUT;
    for (int64_t i = threadIdx.x; i < N; i += blockDim.x) pinfo[i] = PairInfo{-1, 0};
    return;
  }
  for (int32_t b = threadIdx.x; b < B; b += blockDim.x) {
    const int32_t first = cu_sl[b], s = sl[b];
    uint32_t e = 0;
    const float T = temperature[b];
    if (!(isfinite(T) && T > 0.0f)) e |= DSDE_ERR_TEMP;
    const float ur = u_res[b];
    if (!(ur >= 0.0f && ur < 1.0f)) e |= DSDE_ERR_UNIFORM;
    for (int32_t j = 0; j < s; ++j) {
      const int32_t x = draft_tokens[first + j];
      if (x < 0 || int64_t(x) >= V) e |= DSDE_ERR_TOKEN;
      const float u = u_acc[first + j];
      if (!(u >= 0.0f && u < 1.0f)) e |= DSDE_ERR_UNIFORM;
    }
    seq_err[b] = e;
    const float c = e ? 0.0f : kLog2e / T;
    for (int32_t j = 0; j < s; ++j)
      pinfo[first + j] = PairInfo{e ? -1 : first + b + j, int32_t(__float_as_uint(c))};
  }
}

// ---------------------------------------------------------------------------
// row statistics of every drafted pair
// ---------------------------------------------------------------------------

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void pair_stats_kernel(const void *__restrict__ target,
                                                              const void *__restrict__ draft, int64_t V, int32_t nc,
                                                              const PairInfo *__restrict__ pinfo,
                                                              PairChunk *__restrict__ out) {
  __shared__ float red[5][kWaves];
  const int64_t unit = blockIdx.x;
  const int64_t pair = unit / nc;
  const int64_t chunk = unit - pair * nc;
  const PairInfo pi = pinfo[pair];
  if (pi.target_row < 0) return;
  const float c = __uint_as_float(uint32_t(pi.scale_bits));
  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const int t = threadIdx.x;
  const char *trow = (const char *)target + size_t(pi.target_row) * size_t(V) * esz;
  const char *drow = (const char *)draft + size_t(pair) * size_t(V) * esz;

  float zt[kEltsPerThread], zd[kEltsPerThread];
  const int n = load_chunk<DT, VEC>(trow, V, chunk, t, zt);
  load_chunk<DT, VEC>(drow, V, chunk, t, zd);

  // chunk maxima -> reference shifts used by every exponential of the chunk
  float mt = -INFINITY, md = -INFINITY;
#pragma unroll
  for (int i = 0; i < kEltsPerThread; ++i) {
    mt = fmaxf(mt, zt[i]);
    md = fmaxf(md, zd[i]);
  }
  const float Mt = block_max(mt, red[0]);
  const float Md = block_max(md, red[1]);
  const float rt = Mt * c, rd = Md * c;

  float sp0 = 0.f, sp1 = 0.f, sq0 = 0.f, sq1 = 0.f, a0 = 0.f, a1 = 0.f;
  if (n == kEltsPerThread) {
#pragma unroll
    for (int i = 0; i < kEltsPerThread; i += 2) {
      const float at0 = fmaf(zt[i], c, -rt), ad0 = fmaf(zd[i], c, -rd);
      const float at1 = fmaf(zt[i + 1], c, -rt), ad1 = fmaf(zd[i + 1], c, -rd);
      const float et0 = fast_exp2(at0), ed0 = fast_exp2(ad0);
      const float et1 = fast_exp2(at1), ed1 = fast_exp2(ad1);
      sp0 += et0;
      sq0 += ed0;
      a0 = fmaf(et0, at0 - ad0, a0);
      sp1 += et1;
      sq1 += ed1;
      a1 = fmaf(et1, at1 - ad1, a1);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) {
      if (i < n) {  // the padding must not reach the KL accumulator (0 * NaN)
        const float at = fmaf(zt[i], c, -rt), ad = fmaf(zd[i], c, -rd);
        const float et = fast_exp2(at), ed = fast_exp2(ad);
        sp0 += et;
        sq0 += ed;
        a0 = fmaf(et, at - ad, a0);
      }
    }
  }
  const float sp = wave_sum(sp0 + sp1), sq = wave_sum(sq0 + sq1), a = wave_sum(a0 + a1);
  const int wave = t >> 6, lane = t & 63;
  if (lane == 0) {
    red[2][wave] = sp;
    red[3][wave] = sq;
    red[4][wave] = a;
  }
  __syncthreads();
  if (t == 0) {
    double s_p = 0.0, s_q = 0.0, s_a = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      s_p += double(red[2][w]);
      s_q += double(red[3][w]);
      s_a += double(red[4][w]);
    }
    PairChunk pc;
    pc.mt = rt;
    pc.md = rd;
    pc.pad0 = pc.pad1 = 0.f;
    pc.sp = s_p;
    pc.sq = s_q;
    pc.a = s_a;
    pc.pad2 = 0.0;
    out[unit] = pc;
  }
}

// ---------------------------------------------------------------------------
// acceptance scan
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void accept_kernel(const void *__restrict__ target, const void *__restrict__ draft,
                                                     int32_t dtype, int64_t V, int32_t B, int32_t k_max, int32_t nc,
                                                     const int32_t *__restrict__ sl, const int32_t *__restrict__ cu_sl,
                                                     const int32_t *__restrict__ draft_tokens,
                                                     const float *__restrict__ temperature,
                                                     const float *__restrict__ u_acc, const float *__restrict__ u_res,
                                                     int32_t pad_id, const PairInfo *__restrict__ pinfo,
                                                     const PairChunk *__restrict__ part, int32_t *__restrict__ accepted,
                                                     int32_t *__restrict__ tokens, float *__restrict__ kld,
                                                     uint32_t *__restrict__ seq_err, double *__restrict__ row_lse,
                                                     DrawJob *__restrict__ jobs) {
  const int lane = threadIdx.x & 63;
  const int32_t b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const int32_t width = k_max + 1;
  int32_t *tok = tokens + int64_t(b) * width;
  uint32_t err = seq_err[b];
  DrawJob none{};
  none.kind = -1;
  if (err & DSDE_ERR_LAYOUT) {
    if (lane < width) tok[lane] = pad_id;
    if (lane == 0) {
      accepted[b] = 0;
      jobs[b] = none;
    }
    return;
  }
  const int32_t s = sl[b], first = cu_sl[b];
  const bool active = lane < s;
  const int64_t i = first + lane;

  float mt = -INFINITY, md = -INFINITY;
  double sp = 0.0, sq = 0.0, acc_a = 0.0;
  bool bad = false;
  if (active && !err) {
    const PairChunk *pc = part + i * nc;
    for (int32_t ch = 0; ch < nc; ++ch) {
      mt = fmaxf(mt, pc[ch].mt);
      md = fmaxf(md, pc[ch].md);
    }
    for (int32_t ch = 0; ch < nc; ++ch) {
      const PairChunk q = pc[ch];
      const double dt = double(q.mt) - double(mt), dd = double(q.md) - double(md);
      const double ft = exp2(dt), fd = exp2(dd);
      sp += q.sp * ft;
      sq += q.sq * fd;
      acc_a += ft * (q.a + q.sp * (dt - dd));
    }
    bad = !(isfinite(mt) && isfinite(md) && isfinite(sp) && isfinite(sq) && isfinite(acc_a));
  }
  if (__ballot(bad)) err |= DSDE_ERR_LOGIT;

  if (err) {
    if (lane < width) tok[lane] = pad_id;
    if (active) kld[i] = NAN;
    if (lane == 0) {
      accepted[b] = 0;
      seq_err[b] = err;
      jobs[b] = none;
    }
    return;
  }

  const float c = active ? __uint_as_float(uint32_t(pinfo[i].scale_bits)) : 0.f;
  bool ok = false;
  int32_t x = 0;
  if (active) {
    const double l2sp = log2(sp), l2sq = log2(sq);
    // KL in log2 units: E_p[(z_t c - mt) - (z_d c - md)] - log2 S_p + log2 S_q
    const double kl2 = acc_a / sp - l2sp + l2sq;
    const double kl = kl2 * kLn2;
    kld[i] = kl > 0.0 ? float(kl) : 0.0f;
    if (row_lse) {
      row_lse[2 * i] = (double(mt) + l2sp) * kLn2;
      row_lse[2 * i + 1] = (double(md) + l2sq) * kLn2;
    }
    x = draft_tokens[i];
    const int64_t trow = first + b + lane;
    const double zt = load_logit(target, dtype, trow * V + x);
    const double zd = load_logit(draft, dtype, i * V + x);
    // log2 p(x) - log2 q(x), with z*c exact in double
    const double lr = (zt * double(c) - double(mt) - l2sp) - (zd * double(c) - double(md) - l2sq);
    ok = double(u_acc[i]) < exp2(lr);
  }
  const uint64_t mask = __ballot(ok);
  int32_t a = int32_t(__builtin_ctzll(~mask));
  if (a > s) a = s;
  if (lane < width) tok[lane] = lane < a ? x : pad_id;
  if (lane == 0) accepted[b] = a;
  if (a < s) {
    if (lane == a) {
      DrawJob j;
      j.kind = 0;
      j.accepted = a;
      j.target_row = first + b + a;
      j.draft_row = first + a;
      j.scale = c;
      j.mt = mt;
      j.md = md;
      j.inv_sp = float(1.0 / sp);
      j.inv_sq = float(1.0 / sq);
      j.u = u_res[b];
      j.pad0 = j.pad1 = 0;
      jobs[b] = j;
    }
  } else if (lane == 0) {
    DrawJob j;
    j.kind = 1;
    j.accepted = a;
    j.target_row = first + b + s;
    j.draft_row = -1;
    j.scale = kLog2e / temperature[b];  // the same expression as the pair scale of the set-up
    j.mt = j.md = 0.f;
    j.inv_sp = j.inv_sq = 0.f;
    j.u = u_res[b];
    j.pad0 = j.pad1 = 0;
    jobs[b] = j;
  }
}

// ---------------------------------------------------------------------------
// draw: chunk totals of the weights
// ---------------------------------------------------------------------------

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void draw_chunk_kernel(const void *__restrict__ target,
                                                              const void *__restrict__ draft, int64_t V, int32_t nc,
                                                              const DrawJob *__restrict__ jobs,
                                                              DrawChunk *__restrict__ out) {
  __shared__ float red[3][kWaves];
  const int64_t unit = blockIdx.x;
  const int64_t b = unit / nc;
  const int64_t chunk = unit - b * nc;
  const DrawJob job = jobs[b];
  if (job.kind < 0) return;
  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const float c = job.scale;
  const char *trow = (const char *)target + size_t(job.target_row) * size_t(V) * esz;
  float zt[kEltsPerThread];
  const int n = load_chunk<DT, VEC>(trow, V, chunk, t, zt);

  if (job.kind == 0) {
    float zd[kEltsPerThread];
    const char *drow = (const char *)draft + size_t(job.draft_row) * size_t(V) * esz;
    load_chunk<DT, VEC>(drow, V, chunk, t, zd);
    float sw = 0.f, spp = 0.f;
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) {
      // -inf padding gives p = q = 0, hence zero weight
      const float p = fast_exp2(fmaf(zt[i], c, -job.mt)) * job.inv_sp;
      const float q = fast_exp2(fmaf(zd[i], c, -job.md)) * job.inv_sq;
      sw += fmaxf(p - q, 0.0f);
      spp += p;
    }
    sw = wave_sum(sw);
    spp = wave_sum(spp);
    if (lane == 0) {
      red[0][wave] = sw;
      red[1][wave] = spp;
    }
    __syncthreads();
    if (t == 0) {
      DrawChunk dc{};
      for (int w = 0; w < kWaves; ++w) {
        dc.w += double(red[0][w]);
        dc.p += double(red[1][w]);
      }
      out[unit] = dc;
    }
    return;
  }

  // bonus row: chunk-local reference shift, plus detection of non-finite logits
  float m = -INFINITY, lo = INFINITY;
#pragma unroll
  for (int i = 0; i < kEltsPerThread; ++i) {
    m = fmaxf(m, zt[i]);
    if (i < n) lo = fminf(lo, zt[i]);
  }
  int bad = (n > 0 && (lo == -INFINITY || m == INFINITY)) ? 1 : 0;
  const float M = block_max(m, red[0]);
  const float ref = M * c;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kEltsPerThread; ++i) s += fast_exp2(fmaf(zt[i], c, -ref));
  s = wave_sum(s);
  bad = __syncthreads_or(bad);
  if (lane == 0) red[1][wave] = s;
  __syncthreads();
  if (t == 0) {
    DrawChunk dc{};
    for (int w = 0; w < kWaves; ++w) dc.w += double(red[1][w]);
    dc.ref = ref;
    dc.bad = bad || !isfinite(dc.w) || !isfinite(ref);
    out[unit] = dc;
  }
}

// ---------------------------------------------------------------------------
// draw: locate u' * Z
// ---------------------------------------------------------------------------

// Exclusive block scan of one double per thread (fixed order); returns the
// exclusive prefix and sets *total.
__device__ double block_exclusive_scan(double v, double *lds, double *total) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  double incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == 63) lds[wave] = incl;
  __syncthreads();
  double base = 0.0, all = 0.0;
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) base += lds[w];
    all += lds[w];
  }
  __syncthreads();
  *total = all;
  return base + incl - v;
}

template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void draw_kernel(const void *__restrict__ target, const void *__restrict__ draft,
                                                        int64_t V, int32_t nc, int32_t k_max, int32_t pad_id,
                                                        const int32_t *__restrict__ sl,
                                                        const int32_t *__restrict__ cu_sl,
                                                        const DrawJob *__restrict__ jobs,
                                                        const DrawChunk *__restrict__ chunks,
                                                        int32_t *__restrict__ accepted, int32_t *__restrict__ tokens,
                                                        float *__restrict__ kld, uint32_t *__restrict__ seq_err) {
  __shared__ double dsh[kWaves];
  __shared__ double s_rem;
  __shared__ int64_t s_chunk;
  __shared__ int s_mode, s_bad, s_found;
  __shared__ float s_ref;
  __shared__ int64_t s_y, s_last;
  const int32_t b = blockIdx.x;
  const DrawJob job = jobs[b];
  if (job.kind < 0) return;
  const int t = threadIdx.x;
  const DrawChunk *dc = chunks + int64_t(b) * nc;

  if (t == 0) {
    int mode = 0;  // 0: residual weights, 1: p of the rejected pair, 2: bonus exponentials
    int bad = 0;
    double Z = 0.0, fmax_ref = 0.0;
    float ref_max = -INFINITY;
    if (job.kind == 0) {
      for (int32_t ch = 0; ch < nc; ++ch) Z += dc[ch].w;
      if (!(Z > 0.0)) {
        mode = 1;
        Z = 0.0;
        for (int32_t ch = 0; ch < nc; ++ch) Z += dc[ch].p;
      }
    } else {
      mode = 2;
      for (int32_t ch = 0; ch < nc; ++ch) {
        bad |= dc[ch].bad;
        ref_max = fmaxf(ref_max, dc[ch].ref);
      }
      if (!bad)
        for (int32_t ch = 0; ch < nc; ++ch) Z += dc[ch].w * exp2(double(dc[ch].ref) - double(ref_max));
      fmax_ref = ref_max;
    }
    const double target_mass = double(job.u) * Z;
    int64_t found = nc - 1;
    double before = 0.0;
    if (!bad) {
      double C = 0.0;
      for (int32_t ch = 0; ch < nc; ++ch) {
        const double w = mode == 0 ? dc[ch].w
                         : mode == 1 ? dc[ch].p
                                     : dc[ch].w * exp2(double(dc[ch].ref) - fmax_ref);
        if (C + w > target_mass) {
          found = ch;
          break;
        }
        C += w;
      }
      before = C;
    }
    double rem = target_mass - before;
    if (rem < 0.0) rem = 0.0;
    if (mode == 2 && !bad) rem *= exp2(fmax_ref - double(dc[found].ref));  // into the chunk's own scale
    s_rem = rem;
    s_chunk = found;
    s_mode = mode;
    s_bad = bad;
    s_ref = mode == 2 && !bad ? dc[found].ref : 0.f;
    s_found = 0;
    s_y = INT64_MAX;
    s_last = 0;
  }
  __syncthreads();
  const int32_t width = k_max + 1;
  if (s_bad) {
    if (t < width) tokens[int64_t(b) * width + t] = pad_id;
    if (t < sl[b]) kld[cu_sl[b] + t] = NAN;
    if (t == 0) {
      accepted[b] = 0;
      seq_err[b] |= DSDE_ERR_LOGIT;
    }
    return;
  }

  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const int64_t chunk = s_chunk;
  const int mode = s_mode;
  const float c = job.scale, ref = s_ref;
  const char *trow = (const char *)target + size_t(job.target_row) * size_t(V) * esz;
  const char *drow = job.draft_row >= 0 ? (const char *)draft + size_t(job.draft_row) * size_t(V) * esz : nullptr;
  float zt[kEltsPerThread], zd[kEltsPerThread];
  load_chunk<DT, VEC>(trow, V, chunk, t, zt);
  if (mode != 2) load_chunk<DT, VEC>(drow, V, chunk, t, zd);

  // weights of this thread's elements, recomputed exactly as for the chunk totals
  float w[kEltsPerThread];
  int64_t last = -1;
#pragma unroll
  for (int i = 0; i < kEltsPerThread; ++i) {
    float wi;
    if (mode == 2) {
      wi = fast_exp2(fmaf(zt[i], c, -ref));
    } else {
      const float p = fast_exp2(fmaf(zt[i], c, -job.mt)) * job.inv_sp;
      const float q = fast_exp2(fmaf(zd[i], c, -job.md)) * job.inv_sq;
      wi = mode == 0 ? fmaxf(p - q, 0.0f) : p;
    }
    w[i] = wi;
    if (wi > 0.0f) {
      const int64_t idx = Layout<DT, VEC>::index(chunk, i, t);
      last = idx > last ? idx : last;
    }
  }
  // slabs in ascending token order: slab g holds elements [g*kv, (g+1)*kv) of every thread
  constexpr int kv = Layout<DT, VEC>::kVecElts;
  double rem = s_rem;
  for (int g = 0; g < kEltsPerThread / kv; ++g) {
    double tot = 0.0;
#pragma unroll
    for (int e = 0; e < kv; ++e) tot += double(w[g * kv + e]);
    double slab_total;
    const double excl = block_exclusive_scan(tot, dsh, &slab_total);
    if (rem >= excl && rem < excl + tot) {
      double acc = excl;
      int64_t y = -1;
#pragma unroll
      for (int e = 0; e < kv; ++e) {
        acc += double(w[g * kv + e]);
        if (y < 0 && acc > rem) y = Layout<DT, VEC>::index(chunk, g * kv + e, t);
      }
      if (y >= 0) {
        atomicMin((unsigned long long *)&s_y, (unsigned long long)y);
        s_found = 1;
      }
    }
    __syncthreads();
    if (s_found) break;
    rem -= slab_total;
    if (rem < 0.0) rem = 0.0;
  }
  if (!s_found) {
    // rounding left u' * Z past this chunk's total: the last positive weight
    for (int o = 32; o > 0; o >>= 1) {
      const int64_t other = __shfl_xor(last, o);
      last = other > last ? other : last;
    }
    if ((t & 63) == 0) atomicMax((unsigned long long *)&s_last, (unsigned long long)(last + 1));
    __syncthreads();
  }
  if (t == 0) {
    const int64_t y = s_found ? s_y : (s_last > 0 ? s_last - 1 : 0);
    tokens[int64_t(b) * width + job.accepted] = int32_t(y);
  }
}

}  // namespace

static inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <int DT, bool VEC>
static int launch_rows(const VerifyArgs &a, const WorkspaceLayout &L, int32_t nc) {
  char *ws = (char *)a.workspace;
  PairInfo *pinfo = (PairInfo *)(ws + L.pair_info);
  PairChunk *part = (PairChunk *)(ws + L.pair_chunk);
  DrawJob *jobs = (DrawJob *)(ws + L.draw_job);
  DrawChunk *dchunks = (DrawChunk *)(ws + L.draw_chunk);
  hipStream_t st = a.stream;

  if (a.N > 0) {
    if (a.prof_start) (void)hipEventRecord(a.prof_start, st);
    pair_stats_kernel<DT, VEC><<<dim3(unsigned(a.N * nc)), dim3(kThreads), 0, st>>>(a.target, a.draft, a.V, nc,
                                                                                   pinfo, part);
    if (a.prof_stop) (void)hipEventRecord(a.prof_stop, st);
  }
  accept_kernel<<<dim3(unsigned((a.B + 3) / 4)), dim3(256), 0, st>>>(
      a.target, a.draft, a.dtype, a.V, a.B, a.k_max, nc, a.sl, a.cu_sl, a.draft_tokens, a.temperature, a.u_acc,
      a.u_res, a.pad_id, pinfo, part, a.accepted, a.tokens, a.kld, a.seq_err, a.row_lse, jobs);
  draw_chunk_kernel<DT, VEC><<<dim3(unsigned(int64_t(a.B) * nc)), dim3(kThreads), 0, st>>>(a.target, a.draft, a.V,
                                                                                          nc, jobs, dchunks);
  draw_kernel<DT, VEC><<<dim3(unsigned(a.B)), dim3(kThreads), 0, st>>>(a.target, a.draft, a.V, nc, a.k_max,
                                                                      a.pad_id, a.sl, a.cu_sl, jobs, dchunks,
                                                                      a.accepted, a.tokens, a.kld, a.seq_err);
  return 0;
}

int launch_verify(const VerifyArgs &a) {
  const WorkspaceLayout L = workspace_layout(a.B, a.N, a.V);
  const int32_t nc = int32_t((a.V + kChunk - 1) / kChunk);
  char *ws = (char *)a.workspace;
  PairInfo *pinfo = (PairInfo *)(ws + L.pair_info);
  (void)hipGetLastError();
  setup_kernel<<<dim3(1), dim3(1024), 0, a.stream>>>(a.V, a.B, a.N, a.k_max, a.sl, a.cu_sl, a.draft_tokens,
                                                    a.temperature, a.u_acc, a.u_res, a.seq_err, pinfo);
  const bool vec = aligned16(a.target) && (a.N == 0 || aligned16(a.draft)) &&
                   (a.dtype == DSDE_BF16 ? a.V % 8 == 0 : a.V % 4 == 0);
  if (a.dtype == DSDE_BF16) {
    if (vec)
      launch_rows<DSDE_BF16, true>(a, L, nc);
    else
      launch_rows<DSDE_BF16, false>(a, L, nc);
  } else {
    if (vec)
      launch_rows<DSDE_FP32, true>(a, L, nc);
    else
      launch_rows<DSDE_FP32, false>(a, L, nc);
  }
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

}  // namespace dsde
