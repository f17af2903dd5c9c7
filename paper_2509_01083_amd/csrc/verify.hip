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
#include "draw_device.hpp"
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
  launch_stats_pass(a, work, part, gath, cargs, a.draft_entropy != nullptr);
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
