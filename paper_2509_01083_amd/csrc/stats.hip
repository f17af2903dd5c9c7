// The row-statistics pass of the verification step: one workgroup per
// (drafted row pair, 8192-logit chunk) reads the chunk of the target and
// draft rows once and writes max-shifted exponential sums of p and q and the
// KL accumulator (Sec. 3.1.2), and captures the two logits at the drafted
// token.  It carries almost all HBM bytes of the step.  A one-workgroup
// set-up kernel before it validates the packed layout (Sec. 3.2) and writes
// the work list (target row and scale of every drafted pair, in sequence
// order).
#include <hip/hip_ext.h>
#include <math.h>

#include "common.hpp"
#include "row_io.hpp"

namespace dsde {
namespace {

// ---------------------------------------------------------------------------
// set-up
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(1024) void setup_kernel(int32_t B, int64_t N, int32_t k_max,
                                                     const int32_t *__restrict__ sl,
                                                     const int32_t *__restrict__ cu_sl,
                                                     const float *__restrict__ temperature,
                                                     uint32_t *__restrict__ seq_err, WorkItem *__restrict__ work) {
  const int t = threadIdx.x;
  // a batch of at most blockDim sequences (thread t: sequence t) is checked and
  // listed from values loaded once; larger batches loop and load twice
  const bool one = B <= int32_t(blockDim.x);
  const int64_t c_first = cu_sl[0], c_last = cu_sl[B];
  int32_t s0 = 0, f0 = 0;
  float T0 = 1.0f;
  int bad = 0;
  if (one) {
    if (t < B) {
      s0 = sl[t];
      f0 = cu_sl[t];
      T0 = temperature[t];
      if (s0 < 0 || s0 > k_max || int64_t(cu_sl[t + 1]) - int64_t(f0) != s0) bad = 1;
    }
  } else {
    for (int32_t b = t; b < B; b += blockDim.x) {
      const int64_t s = sl[b];
      if (s < 0 || s > k_max || int64_t(cu_sl[b + 1]) - int64_t(cu_sl[b]) != s) bad = 1;
    }
  }
  bad = __syncthreads_or(bad);
  if (c_first != 0 || c_last != N) bad = 1;
  if (bad) {
    for (int32_t b = t; b < B; b += blockDim.x) seq_err[b] = DSDE_ERR_LAYOUT;
    for (int64_t k = t; k < N; k += blockDim.x) work[k] = WorkItem{int32_t(k), -1, 0u, -1};
    return;
  }
  // the same expression as every later kernel's scale; a temperature outside
  // the admissible range is flagged by the acceptance kernel.  T = 0 selects
  // greedy verification: statistics at T = 1, and the sign bit asks the
  // statistics kernel for the chunk argmax of the target row.
  auto list = [&](int32_t b, int32_t first, int32_t s, float T) {
    seq_err[b] = 0u;
    const uint32_t cbits = T == 0.0f ? (__float_as_uint(kLog2e) | kGreedyBit) : __float_as_uint(kLog2e / T);
    for (int32_t j = 0; j < s; ++j) work[first + j] = WorkItem{first + j, first + b + j, cbits, b * k_max + j};
  };
  if (one) {
    if (t < B) list(t, f0, s0, T0);
  } else {
    for (int32_t b = t; b < B; b += blockDim.x) list(b, cu_sl[b], sl[b], temperature[b]);
  }
}

// ---------------------------------------------------------------------------
// row statistics of every drafted pair
// ---------------------------------------------------------------------------

// Greedy pairs: each wavefront's smallest token id holding the chunk maximum
// M of the target row, into red[wave] (0xffffffff if none).  Only a thread
// whose own maximum `tmax` equals M holds it, so only those threads scan
// their slots and only wavefronts holding one reduce (in most chunks one
// wavefront of four).  A thread's slots ascend in token order in every
// layout, so its first slot equal to M is its smallest such token.  `z(i)` is
// slot i of this thread's logits.
template <int DT, bool VEC, typename Z>
__device__ __forceinline__ void wave_chunk_argmax(float M, float tmax, Z z, int64_t chunk, uint32_t *red) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  uint32_t best = 0xffffffffu;
  if (tmax == M) {
    int first = -1;
#pragma unroll
    for (int i = kEltsPerThread - 1; i >= 0; --i)
      if (z(i) == M) first = i;
    if (first >= 0) best = uint32_t(Layout<DT, VEC>::index(chunk, first, t));
  }
  if (__ballot(best != 0xffffffffu)) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint32_t y = __shfl_xor(best, o);
      best = y < best ? y : best;
    }
  }
  if (lane == 0) red[wave] = best;
}

// Sum over the 64 lanes of a wavefront of four fp64 values at once (a
// reduce-scatter): lanes whose bits 5 and 4 are (0, 0), (0, 1), (1, 0) and
// (1, 1) end up holding the totals of v0, v1, v2 and v3.  The first exchange
// (partner lane ^ 32) keeps v0, v1 in the lower half of the wavefront and
// v2, v3 in the upper half, the second (lane ^ 16) keeps one of the two, and
// four butterfly steps finish each group of 16 lanes; every step adds the
// same two partials on both partners, so a group's lanes agree bit for bit.
__device__ __forceinline__ double wave_sum4_scatter(double v0, double v1, double v2, double v3) {
  const int lane = threadIdx.x & 63;
  const bool up5 = (lane & 32) != 0, up4 = (lane & 16) != 0;
  const double k0 = up5 ? v2 : v0, k1 = up5 ? v3 : v1;
  const double g0 = up5 ? v0 : v2, g1 = up5 ? v1 : v3;
  const double a0 = k0 + __shfl_xor(g0, 32), a1 = k1 + __shfl_xor(g1, 32);
  const double k = up4 ? a1 : a0, g = up4 ? a0 : a1;
  double r = k + __shfl_xor(g, 16);
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) r += __shfl_xor(r, o);
  return r;
}

// Chunk sums of one workgroup -> one PairChunk.  Each thread's two
// accumulator sets (the p sum, the q sum, the KL and the entropy
// accumulators) are joined in fp64, summed over the wavefront in fp64 and
// over the wavefronts in fp64, in a fixed order.  The fp64 wavefront sums
// matter for the KLD: KL = A / S_p - log2 S_p + log2 S_q cancels terms of
// order one down to values of order 1e-4, so rounding the partial sums to
// fp32 on the way (six butterfly levels) would cost about 1e-7 of absolute
// KLD accuracy.  With `arg` set (greedy pairs), also the chunk maximum M of
// the target row and the smallest token holding it, from the per-wave
// candidates wave_chunk_argmax left in red_arg (the same barrier serves both).
__device__ __forceinline__ void write_pair_chunk(float rt, float rd, const PairAcc &s, double (*red)[kWaves],
                                                 PairChunk *out, float M, const uint32_t *red_arg, ChunkArg *arg) {
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const double tot = wave_sum4_scatter(s.sp[0] + s.sp[1], s.sq[0] + s.sq[1], double(s.a[0]) + double(s.a[1]),
                                       double(s.h[0]) + double(s.h[1]));
  if ((lane & 15) == 0) red[lane >> 4][wave] = tot;
  __syncthreads();
  if (t == 0) {
    PairChunk pc;
    pc.mt = rt;
    pc.md = rd;
    pc.sp = pc.sq = pc.a = pc.h = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      pc.sp += red[0][w];
      pc.sq += red[1][w];
      pc.a += red[2][w];
      pc.h += red[3][w];
    }
    *out = pc;
    if (arg) {
      uint32_t m = red_arg[0];
#pragma unroll
      for (int v = 1; v < kWaves; ++v) m = red_arg[v] < m ? red_arg[v] : m;
      *arg = ChunkArg{M, int32_t(m)};
    }
  }
}

// bf16 rows with 16-byte alignment: the hot kernel.  ENT: accumulate the
// draft entropy, only for callers that ask for it (one FMA of about twenty
// VALU instructions per logit pair).  Two kernels rather than a branch in
// one: with both forms in one body the compiler hoists their common
// arithmetic above the branch and nearly doubles the register footprint.
template <bool ENT>
__global__ __launch_bounds__(kThreads) void stats_kernel_bf16(const void *__restrict__ target,
                                                             const void *__restrict__ draft, int64_t V, int32_t nc,
                                                             const WorkItem *__restrict__ work,
                                                             const int32_t *__restrict__ draft_tokens,
                                                             int64_t token_base, PairChunk *__restrict__ out,
                                                             Gathered *__restrict__ gathered,
                                                             ChunkArg *__restrict__ chunk_arg) {
  __shared__ float red[2][kWaves];
  __shared__ double red_sum[4][kWaves];
  __shared__ uint32_t red_arg[kWaves];
  const int64_t unit = blockIdx.x;
  const int64_t k = unit / nc;
  const int64_t chunk = unit - k * nc;
  const WorkItem w = work[k];
  if (w.target_row < 0) return;
  const int t = threadIdx.x;
  const bool greedy = (w.scale_bits & kGreedyBit) != 0;
  const float c = __uint_as_float(w.scale_bits & ~kGreedyBit);
  const char *trow = (const char *)target + size_t(w.target_row) * size_t(V) * 2;
  const char *drow = (const char *)draft + size_t(w.pair) * size_t(V) * 2;
  const RawBf16 rt_ = load_raw_bf16(trow, V, chunk, t);
  const RawBf16 rd_ = load_raw_bf16(drow, V, chunk, t);

  // chunk maxima -> the reference shifts every exponential of the chunk uses
  const float tmt = raw_max(rt_);
  const float Mt = block_max(tmt, red[0]);
  const float Md = block_max(raw_max(rd_), red[1]);
  if (greedy)
    wave_chunk_argmax<DSDE_BF16, true>(Mt, tmt, [&](int i) { return pick_bf16(rt_, i); }, chunk, red_arg);
  const float rt = Mt * c, rd = Md * c;
  PairAcc s;
  zero(s);
  acc_vec<ENT>(rt_.v0, rd_.v0, c, rt, rd, s);
  acc_vec<ENT>(rt_.v1, rd_.v1, c, rt, rd, s);
  acc_vec<ENT>(rt_.v2, rd_.v2, c, rt, rd, s);
  acc_vec<ENT>(rt_.v3, rd_.v3, c, rt, rd, s);

  // the logits at the drafted token, from registers
  // a token outside [0, V) never matches (its sequence is flagged later)
  const int64_t local = int64_t(draft_tokens[w.pair]) - token_base - chunk * kChunk;
  if (local >= 0 && local < kChunk) {
    int ot, oi;
    Layout<DSDE_BF16, true>::owner(local, &ot, &oi);
    if (t == ot) {
      // select with compile-time slots only: a runtime index into the
      // register arrays would put them in scratch memory
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i)
        if (i == oi) {
          a = pick_bf16(rt_, i);
          b = pick_bf16(rd_, i);
        }
      gathered[w.slot] = Gathered{a, b};
    }
  }
  write_pair_chunk(rt, rd, s, red_sum, out + int64_t(w.slot) * nc + chunk, Mt, red_arg,
                   greedy ? chunk_arg + int64_t(w.slot) * nc + chunk : nullptr);
}

// fp32 rows, or rows without 16-byte alignment.
template <int DT, bool VEC>
__global__ __launch_bounds__(kThreads) void stats_kernel_generic(const void *__restrict__ target,
                                                                const void *__restrict__ draft, int64_t V,
                                                                int32_t nc, const WorkItem *__restrict__ work,
                                                                const int32_t *__restrict__ draft_tokens,
                                                                int64_t token_base, PairChunk *__restrict__ out,
                                                                Gathered *__restrict__ gathered,
                                                                ChunkArg *__restrict__ chunk_arg) {
  __shared__ float red[2][kWaves];
  __shared__ double red_sum[4][kWaves];
  __shared__ uint32_t red_arg[kWaves];
  const int64_t unit = blockIdx.x;
  const int64_t k = unit / nc;
  const int64_t chunk = unit - k * nc;
  const WorkItem w = work[k];
  if (w.target_row < 0) return;
  const int t = threadIdx.x;
  const bool greedy = (w.scale_bits & kGreedyBit) != 0;
  const float c = __uint_as_float(w.scale_bits & ~kGreedyBit);
  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const char *trow = (const char *)target + size_t(w.target_row) * size_t(V) * esz;
  const char *drow = (const char *)draft + size_t(w.pair) * size_t(V) * esz;
  float zt[kEltsPerThread], zd[kEltsPerThread];
  load_chunk_f32<DT, VEC>(trow, V, chunk, t, zt);
  load_chunk_f32<DT, VEC>(drow, V, chunk, t, zd);
  float mt = zt[0], md = zd[0];
#pragma unroll
  for (int i = 1; i < kEltsPerThread; ++i) {
    mt = max_nan(mt, zt[i]);
    md = max_nan(md, zd[i]);
  }
  const float Mt = block_max(mt, red[0]);
  const float Md = block_max(md, red[1]);
  if (greedy) wave_chunk_argmax<DT, VEC>(Mt, mt, [&](int i) { return zt[i]; }, chunk, red_arg);
  const float rt = Mt * c, rd = Md * c;
  PairAcc s;
  zero(s);
#pragma unroll
  for (int i = 0; i < kEltsPerThread; i += 4) {
    acc_two<true>(zt[i], zt[i + 1], zd[i], zd[i + 1], c, rt, rd, s, 0);
    acc_two<true>(zt[i + 2], zt[i + 3], zd[i + 2], zd[i + 3], c, rt, rd, s, 1);
  }
  // a token outside [0, V) never matches (its sequence is flagged later)
  const int64_t local = int64_t(draft_tokens[w.pair]) - token_base - chunk * kChunk;
  if (local >= 0 && local < kChunk) {
    int ot, oi;
    Layout<DT, VEC>::owner(local, &ot, &oi);
    if (t == ot) {
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int i = 0; i < kEltsPerThread; ++i)
        if (i == oi) {
          a = zt[i];
          b = zd[i];
        }
      gathered[w.slot] = Gathered{a, b};
    }
  }
  write_pair_chunk(rt, rd, s, red_sum, out + int64_t(w.slot) * nc + chunk, Mt, red_arg,
                   greedy ? chunk_arg + int64_t(w.slot) * nc + chunk : nullptr);
}

}  // namespace

static inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// With profiling events set, `stop` is attached to the completion of the
// statistics dispatch and `start` to the completion of the set-up dispatch
// just before it, so that the interval is the statistics kernel alone (a
// start event attached to a dispatch is stamped when the packet is
// processed, which can be while the previous kernel still runs).
template <typename K, typename... Args>
static void launch_timed(K kernel, dim3 grid, dim3 block, hipStream_t stream, hipEvent_t done, Args... args) {
  if (done)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, nullptr, done, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
}

bool rows_vectorizable(const VerifyArgs &a) {
  return aligned16(a.target) && (a.N == 0 || aligned16(a.draft)) &&
         (a.dtype == DSDE_BF16 ? a.V % 8 == 0 : a.V % 4 == 0);
}

void launch_stats_pass(const VerifyArgs &a, WorkItem *work, PairChunk *part, Gathered *gath, ChunkArg *chunk_arg,
                       bool entropy) {
  const int32_t nc = int32_t(num_chunks(a.V));
  const bool prof = a.prof_start && a.prof_stop && a.N > 0;
  launch_timed(setup_kernel, dim3(1), dim3(1024), a.stream, prof ? a.prof_start : nullptr, a.B, a.N, a.k_max,
               a.sl, a.cu_sl, a.temperature, a.seq_err, work);
  if (a.N == 0) return;
  const bool vec = rows_vectorizable(a);
  const dim3 grid(unsigned(a.N * nc)), block(kThreads);
  hipEvent_t done = prof ? a.prof_stop : nullptr;
  const void *T = a.target, *D = a.draft;
  const int64_t V = a.V;
  const int32_t *tokens = a.draft_tokens;
  const int64_t base = a.token_base;
  const WorkItem *w = work;
  if (a.dtype == DSDE_BF16 && vec && entropy)
    launch_timed(stats_kernel_bf16<true>, grid, block, a.stream, done, T, D, V, nc, w, tokens, base, part, gath,
                 chunk_arg);
  else if (a.dtype == DSDE_BF16 && vec)
    launch_timed(stats_kernel_bf16<false>, grid, block, a.stream, done, T, D, V, nc, w, tokens, base, part, gath,
                 chunk_arg);
  else if (a.dtype == DSDE_BF16)
    launch_timed(stats_kernel_generic<DSDE_BF16, false>, grid, block, a.stream, done, T, D, V, nc, w, tokens, base,
                 part, gath, chunk_arg);
  else if (vec)
    launch_timed(stats_kernel_generic<DSDE_FP32, true>, grid, block, a.stream, done, T, D, V, nc, w, tokens, base,
                 part, gath, chunk_arg);
  else
    launch_timed(stats_kernel_generic<DSDE_FP32, false>, grid, block, a.stream, done, T, D, V, nc, w, tokens, base,
                 part, gath, chunk_arg);
}

}  // namespace dsde
