// Vocabulary-sharded verification on gfx950: the kernels one shard runs when
// the logits of every row are split by vocabulary across G devices (the
// calls and the exchanges between them are described with dsde_shard_stats in
// dsde.h).  Each call is the matching part of dsde_verify restricted to the
// shard's slice:
//   call 1  the set-up and statistics kernels of dsde_verify on the slice
//           (stats.hip; drafted tokens are offset by the slice's first id,
//           so tokens outside it gather nothing), then shard_combine_kernel:
//           the chunk partials of each drafted pair folded into one slice
//           partial.
//   call 2  shard_accept_kernel: one wavefront per sequence folds the G slice
//           partials in shard order (fp64), then KLD, acceptance and the draw
//           job exactly as the per-sequence kernel of dsde_verify; fused
//           (dsde_shard_accept_step), the same wavefront then runs the signal
//           update on those KLD values, and the SL rule follows as in
//           dsde_step.
//   call 3  shard_mass_kernel: one workgroup per sequence streams the draw
//           row(s) of its slice once, keeps chunk and sub-block totals in the
//           workspace and reports the slice's mass.
//   call 4  shard_pick_kernel: every workgroup finds the slice holding the
//           inverse-CDF point (a fixed-order fp64 prefix over the slices);
//           the shard owning it draws inside its slice from the totals.
#include <math.h>
#include <stddef.h>

#include <type_traits>

#include "common.hpp"
#include "draw_device.hpp"
#include "lanes.hpp"
#include "row_io.hpp"
#include "shard.hpp"
#include "signal_device.hpp"

namespace dsde {
namespace {

// the public job record is the kernels' DrawJob
static_assert(sizeof(dsde_draw_job) == sizeof(DrawJob), "draw job layout");
static_assert(offsetof(dsde_draw_job, scale) == offsetof(DrawJob, scale), "draw job layout");
static_assert(offsetof(dsde_draw_job, token) == offsetof(DrawJob, token), "draw job layout");
static_assert(sizeof(dsde_shard_partial) == 64, "partial layout");
static_assert(sizeof(dsde_shard_mass) == 32, "mass layout");

constexpr int kShardThreads = 256;
constexpr int kShardWaves = kShardThreads / 64;

// ---- call 1 --------------------------------------------------------------

// One workgroup per sequence: the chunk partials of each drafted pair folded
// into the slice partial (the combine of the per-sequence kernel).
template <int GL>
__global__ __launch_bounds__(kShardThreads) void shard_combine_kernel(
    const PairChunk *__restrict__ part, const ChunkArg *__restrict__ chunk_arg, const Gathered *__restrict__ gath,
    const int32_t *__restrict__ sl, const int32_t *__restrict__ cu_sl, const int32_t *__restrict__ draft_tokens,
    const float *__restrict__ temperature, const uint32_t *__restrict__ seq_err, int32_t k_max, int32_t nc,
    int64_t v_begin, int64_t V_shard, dsde_shard_partial *__restrict__ out) {
  __shared__ float st_mt[DSDE_MAX_K + 1], st_md[DSDE_MAX_K + 1], st_zmax[DSDE_MAX_K + 1];
  __shared__ double st_sp[DSDE_MAX_K + 1], st_sq[DSDE_MAX_K + 1], st_a[DSDE_MAX_K + 1], st_h[DSDE_MAX_K + 1];
  __shared__ int st_bad[DSDE_MAX_K + 1], st_arg[DSDE_MAX_K + 1];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int32_t b = blockIdx.x;
  if (seq_err[b] & DSDE_ERR_LAYOUT) return;  // the layout is invalid: no position is indexed
  const int32_t s = sl[b], first = cu_sl[b];
  const bool greedy = temperature[b] == 0.0f;
  const int64_t slot0 = int64_t(b) * k_max;
  const int32_t j0 = wave * (64 / GL) + lane / GL, g0 = lane % GL;
  PairChunk q0{};
  ChunkArg arg0{0.f, 0};
  if (j0 < k_max && g0 < nc) {
    q0 = part[(slot0 + j0) * nc + g0];
    arg0 = chunk_arg[(slot0 + j0) * nc + g0];
  }
  if (s > 0)
    combine_pairs<GL, kShardWaves>(part, slot0, s, nc, q0, greedy ? chunk_arg : nullptr, arg0, st_mt, st_md, st_sp,
                                   st_sq, st_a, st_h, st_bad, st_arg, st_zmax);
  __syncthreads();
  if (t < s) {
    dsde_shard_partial r;
    r.mt = st_mt[t];
    r.md = st_md[t];
    r.sp = st_sp[t];
    r.sq = st_sq[t];
    r.a = st_a[t];
    r.h = st_h[t];
    const int64_t l = int64_t(draft_tokens[first + t]) - v_begin;  // the token's index in the slice
    r.has_token = l >= 0 && l < V_shard;
    const Gathered gz = r.has_token ? gath[slot0 + t] : Gathered{0.f, 0.f};
    r.zt = gz.zt;
    r.zd = gz.zd;
    r.zmax = greedy ? st_zmax[t] : -INFINITY;
    r.argmax = greedy ? int32_t(v_begin + st_arg[t]) : -1;
    r.bad = st_bad[t];
    out[first + t] = r;
  }
}

// ---- call 2 --------------------------------------------------------------

// One wavefront per sequence; lane j holds drafted position j.
template <bool FUSED>
__global__ __launch_bounds__(64) void shard_accept_kernel(
    int32_t G, const dsde_shard_partial *__restrict__ parts, int64_t N, int64_t V, int32_t k_max,
    const int32_t *__restrict__ sl, const int32_t *__restrict__ cu_sl, const int32_t *__restrict__ draft_tokens,
    const float *__restrict__ temperature, const float *__restrict__ u_acc, const float *__restrict__ u_res,
    int32_t pad_id, int32_t *__restrict__ accepted, int32_t *__restrict__ tokens, float *__restrict__ kld,
    double *__restrict__ row_lse, float *__restrict__ entropy, DrawJob *__restrict__ jobs,
    uint32_t *__restrict__ seq_err, const SignalArgs S) {
  const int lane = threadIdx.x;
  const int32_t b = blockIdx.x;
  const int32_t width = k_max + 1;
  int32_t *tok = tokens + int64_t(b) * width;
  uint32_t err = seq_err[b];
  if (err & DSDE_ERR_LAYOUT) {
    if (lane < width) tok[lane] = pad_id;
    if (lane == 0) {
      accepted[b] = 0;
      DrawJob j{};
      j.kind = -1;
      jobs[b] = j;
      if constexpr (FUSED) S.mu_last[b] = S.var_short[b] = S.var_long[b] = S.wvir[b] = S.sf[b] = NAN;
    }
    return;
  }
  const int32_t s = sl[b], first = cu_sl[b];
  const float T = temperature[b], ur = u_res[b];
  RingPrefetch rp{};  // the ring state, in flight while the slices are folded
  if constexpr (FUSED) rp = wave_ring_prefetch(S.hist + int64_t(b) * S.W, S.head + b, S.count + b, S.W);
  const bool greedy = T == 0.0f;
  int32_t x = 0;
  float u = 0.f;
  if (lane < s) {
    x = draft_tokens[first + lane];
    u = u_acc[first + lane];
  }
  // the slices in shard order: the statistics folded as the chunk partials are,
  // the drafted token's logits from the one slice holding it, and (greedy) the
  // row maximum of the first slice that reaches it
  float mt = -INFINITY, md = -INFINITY, zt = 0.f, zd = 0.f, zbest = -INFINITY;
  double sp = 0.0, sq = 0.0, a = 0.0, h = 0.0;
  int32_t owners = 0, abest = 0x7fffffff;
  int bad = 0;
  if (lane < s) {
    for (int32_t g = 0; g < G; ++g) {
      const dsde_shard_partial p = parts[int64_t(g) * N + first + lane];
      bad |= p.bad;
      if (p.has_token) {
        ++owners;
        zt = p.zt;
        zd = p.zd;
      }
      if (greedy && (abest == 0x7fffffff || p.zmax > zbest)) {
        zbest = p.zmax;
        abest = p.argmax;
      }
      if (g == 0) {
        mt = p.mt;
        md = p.md;
        sp = p.sp;
        sq = p.sq;
        a = p.a;
        h = p.h;
      } else {
        fold_pair_stats(mt, md, sp, sq, a, h, p.mt, p.md, p.sp, p.sq, p.a, p.h);
      }
    }
    bad |= !(isfinite(mt) && isfinite(md) && isfinite(sp) && isfinite(sq) && isfinite(a));
  }
  {  // per-sequence input checks, as in dsde_verify; a token held by no slice or by several
    uint32_t e = 0;
    if (lane < s) {
      if (x < 0 || int64_t(x) >= V || owners != 1) e |= DSDE_ERR_TOKEN;
      if (!greedy && !(u >= 0.0f && u < 1.0f)) e |= DSDE_ERR_UNIFORM;
    }
    if (lane == 0 && !greedy) {
      if (!(T >= kMinTemp && T <= kMaxTemp)) e |= DSDE_ERR_TEMP;
      if (!(ur >= 0.0f && ur < 1.0f)) e |= DSDE_ERR_UNIFORM;
    }
    err |= lanes::wave_or(e);
  }
  const uint32_t e_in = err;
  const float c = greedy ? kLog2e : kLog2e / T;  // the scale of the statistics pass
  bool ok = false;
  float my_kld = NAN, my_h = NAN, my_isp = 0.f, my_isq = 0.f;
  double l2sp = 0.0, l2sq = 0.0;
  if (lane < s && !e_in) {
    const double rsp = rcp_newton(sp), rsq = rcp_newton(sq);
    my_isp = float(rsp);
    my_isq = float(rsq);
    if (greedy) {
      ok = x == abest;
    } else {
      // u < p(x) / q(x), tested as u S_p < 2^D S_q (as in dsde_verify)
      const double D = (double(zt) * double(c) - double(mt)) - (double(zd) * double(c) - double(md));
      ok = double(u) * sp < exp2_taylor(D) * sq;
    }
    l2sp = log2_rowsum(sp);
    l2sq = log2_rowsum(sq);
    const double kl = (a * rsp - l2sp + l2sq) * kLn2;
    my_kld = kl > 0.0 ? float(kl) : 0.0f;
    my_h = float((l2sq - h * rsq) * kLn2);
  }
  if (__ballot(bad)) err |= DSDE_ERR_LOGIT;
  const uint64_t mask = __ballot(ok);
  int32_t acc = int32_t(__builtin_ctzll(~mask));
  if (acc > s) acc = s;
  if (err) {
    acc = 0;
    my_kld = NAN;
    my_h = NAN;
  }
  if (lane < s) {
    kld[first + lane] = my_kld;
    if (entropy) entropy[first + lane] = my_h;
    if (row_lse && !e_in && !bad) {
      row_lse[2 * (first + lane)] = (double(mt) + l2sp) * kLn2;
      row_lse[2 * (first + lane) + 1] = (double(md) + l2sq) * kLn2;
    }
  }
  // fused: the signal update of the sequence on the KLD values just formed;
  // its error bits join seq_err but, as in the separate calls, leave the
  // acceptance and the draw alone
  uint32_t e_sig = 0;
  if constexpr (FUSED)
    e_sig = wave_signal_update(s, first, nullptr, my_kld, rp, S.hist + int64_t(b) * S.W, S.head + b, S.count + b,
                               S.W, S.n_short, S.n_long, S.delta, S.eps, S.mu_last + b, S.var_short + b,
                               S.var_long + b, S.wvir + b, S.sf + b);
  if (lane < width) tok[lane] = lane < acc ? x : pad_id;
  const float a_mt = lanes::readlane(mt, acc), a_md = lanes::readlane(md, acc);
  const float a_isp = lanes::readlane(my_isp, acc), a_isq = lanes::readlane(my_isq, acc);
  const int32_t a_arg = lanes::readlane(abest, acc);
  if (lane == 0) {
    accepted[b] = acc;
    seq_err[b] = err | e_sig;
    DrawJob j{};
    j.kind = -1;
    j.accepted = acc;
    if (!err && greedy) {
      j.target_row = first + b + acc;
      j.draft_row = -1;
      if (acc < s) {  // the argmax of the first rejected row is known already
        j.kind = 2;
        j.token = a_arg;
        tok[acc] = a_arg;
      } else {
        j.kind = 3;
      }
    } else if (!err) {
      j.scale = c;
      j.u = ur;
      if (acc < s) {
        j.kind = 0;
        j.target_row = first + b + acc;
        j.draft_row = first + acc;
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
    jobs[b] = j;
  }
}

// ---- call 3 --------------------------------------------------------------

// One workgroup per sequence: the draw weight of the slice, wavefront w taking
// chunks w, w + 4, ...; chunk totals, references, flags and sub-block
// partials go to the workspace at cell b * nc + ch.
template <int DT, bool VEC>
__global__ __launch_bounds__(kShardThreads) void shard_mass_kernel(
    const void *__restrict__ target, const void *__restrict__ draft, int64_t V, int32_t nc, int64_t v_begin,
    const dsde_shard_partial *__restrict__ part, const DrawJob *__restrict__ jobs, dsde_shard_mass *__restrict__ mass,
    double *__restrict__ ch_w, float *__restrict__ ch_ref, int32_t *__restrict__ ch_bad, float *__restrict__ sub) {
  __shared__ float s_zmax[kMaxChunks];
  __shared__ int32_t s_idx[kMaxChunks], s_bad[kMaxChunks];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int32_t b = blockIdx.x;
  const DrawJob job = uniform_job(jobs[b]);
  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const int64_t cell0 = int64_t(b) * nc;
  dsde_shard_mass m;
  m.mass = 0.0;
  m.p_mass = 0.0;
  m.ref = 0.f;
  m.zmax = -INFINITY;
  m.argmax = -1;
  m.bad = 0;
  if (job.kind == 0) {
    const char *trow = (const char *)target + size_t(job.target_row) * size_t(V) * esz;
    const char *drow = (const char *)draft + size_t(job.draft_row) * size_t(V) * esz;
    for (int32_t ch = wave; ch < nc; ch += kShardWaves) {
      const double w = residual_chunk<DT, VEC>(trow, drow, V, ch, job, sub + (cell0 + ch) * 64);
      if (lane == 0) ch_w[cell0 + ch] = w;
    }
    __syncthreads();
    if (wave == 0) {
      double acc = 0.0;
      for (int32_t ch = lane; ch < nc; ch += 64) acc += ch_w[cell0 + ch];
      m.mass = wave_sum_f64(acc);
      // this slice's share of p for the rejected pair, from its call-1 partial
      const dsde_shard_partial pp = part[job.draft_row];
      m.p_mass = pp.sp * exp2_taylor(double(pp.mt) - double(job.mt)) * double(job.inv_sp);
      if (lane == 0) mass[b] = m;
    }
  } else if (job.kind == 1) {
    const char *trow = (const char *)target + size_t(job.target_row) * size_t(V) * esz;
    for (int32_t ch = wave; ch < nc; ch += kShardWaves) {
      double w;
      float ref;
      int bd;
      bonus_chunk<DT, VEC>(trow, V, ch, job.scale, &w, &ref, &bd, sub + (cell0 + ch) * 64);
      if (lane == 0) {
        ch_w[cell0 + ch] = w;
        ch_ref[cell0 + ch] = ref;
        ch_bad[cell0 + ch] = bd;
      }
    }
    __syncthreads();
    if (wave == 0) {
      float ref = -INFINITY;
      int bd = 0;
      for (int32_t ch = lane; ch < nc; ch += 64) {
        ref = fmaxf(ref, ch_ref[cell0 + ch]);
        bd |= ch_bad[cell0 + ch];
      }
      ref = wave_max(ref);
      bd = lanes::wave_or(bd);
      double acc = 0.0;
      if (!bd)
        for (int32_t ch = lane; ch < nc; ch += 64)
          acc += ch_w[cell0 + ch] * exp2_taylor(double(ch_ref[cell0 + ch]) - double(ref));
      m.mass = wave_sum_f64(acc);
      m.ref = ref;
      m.bad = bd;
      if (lane == 0) mass[b] = m;
    }
  } else if (job.kind == 3) {
    const char *trow = (const char *)target + size_t(job.target_row) * size_t(V) * esz;
    for (int32_t ch = wave; ch < nc; ch += kShardWaves) {
      float zmax;
      int32_t idx;
      int bd;
      bonus_argmax_chunk<DT, VEC>(trow, V, ch, &zmax, &idx, &bd);
      if (lane == 0) {
        s_zmax[ch] = zmax;
        s_idx[ch] = idx;
        s_bad[ch] = bd;
      }
    }
    __syncthreads();
    if (wave == 0) {
      // the chunk holding the slice maximum (the earliest on ties)
      float best = -INFINITY;
      int32_t bch = 0x7fffffff;
      int bd = 0;
      for (int32_t ch = lane; ch < nc; ch += 64) {
        bd |= s_bad[ch];
        if (bch == 0x7fffffff || s_zmax[ch] > best) {
          best = s_zmax[ch];
          bch = ch;
        }
      }
      bd = lanes::wave_or(bd);
      const float M = wave_max(best);
      int32_t cand = bch != 0x7fffffff && best == M ? bch : 0x7fffffff;
      cand = lanes::wave_min(cand);
      m.zmax = M;
      m.argmax = int32_t(v_begin + s_idx[cand]);
      m.bad = bd;
      if (lane == 0) mass[b] = m;
    }
  } else if (t == 0) {
    mass[b] = m;
  }
}

// ---- call 4 --------------------------------------------------------------

// One workgroup per sequence.  Every wavefront evaluates the slice-level
// search alike (no barrier needed); the shard whose slice holds the target
// finishes the draw on wavefront 0 (the fallback to p first computes that
// slice's p totals with all wavefronts).
template <int DT, bool VEC>
__global__ __launch_bounds__(kShardThreads) void shard_pick_kernel(
    int32_t G, int32_t gself, const dsde_shard_mass *__restrict__ masses, int32_t B, const void *__restrict__ target,
    const void *__restrict__ draft, int64_t V, int32_t nc, int64_t v_begin, int32_t k_max,
    const DrawJob *__restrict__ jobs, int32_t pad_id, int32_t *__restrict__ accepted, int32_t *__restrict__ tokens,
    int32_t *__restrict__ drawn, uint32_t *__restrict__ seq_err, double *__restrict__ ch_w,
    const float *__restrict__ ch_ref, float *__restrict__ sub) {
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int32_t b = blockIdx.x;
  const DrawJob job = uniform_job(jobs[b]);
  const int32_t width = k_max + 1;
  int32_t *tok = tokens + int64_t(b) * width;
  if (job.kind < 0 || job.kind == 2) {  // flagged, or a greedy token already emitted
    if (t == 0) drawn[b] = job.kind == 2 ? job.token : -1;
    return;
  }
  if (wave != 0 && job.kind == 3) return;
  // a NaN or infinite logit in a sampled bonus row: no token is emitted
  auto withhold = [&]() {
    if (lane < width) tok[lane] = pad_id;
    if (lane == 0) {
      accepted[b] = 0;
      seq_err[b] |= DSDE_ERR_LOGIT;
      drawn[b] = -1;
    }
  };
  if (job.kind == 3) {
    // greedy bonus: the first slice holding the row maximum, and its argmax
    float best = -INFINITY;
    int32_t bg = 0x7fffffff;
    int bd = 0;
    for (int32_t g = lane; g < G; g += 64) {
      const dsde_shard_mass q = masses[int64_t(g) * B + b];
      bd |= q.bad;
      if (bg == 0x7fffffff || q.zmax > best) {
        best = q.zmax;
        bg = g;
      }
    }
    bd = lanes::wave_or(bd);
    const float M = wave_max(best);
    int32_t cand = bg != 0x7fffffff && best == M ? bg : 0x7fffffff;
    cand = lanes::wave_min(cand);
    if (bd) {
      withhold();
    } else if (lane == 0) {
      const int32_t token = masses[int64_t(cand) * B + b].argmax;
      tok[job.accepted] = token;
      drawn[b] = token;
    }
    return;
  }
  // the slice weights in one scale: 0 residual masses, 1 p masses, 2 bonus masses
  int mode = job.kind == 0 ? 0 : 2;
  float ref_max = -INFINITY;
  if (mode == 2) {
    int bd = 0;
    for (int32_t g = lane; g < G; g += 64) {
      const dsde_shard_mass q = masses[int64_t(g) * B + b];
      bd |= q.bad;
      ref_max = fmaxf(ref_max, q.ref);
    }
    ref_max = wave_max(ref_max);
    if (lanes::wave_or(bd)) {
      if (wave == 0) withhold();
      return;
    }
  }
  auto weight = [&](int32_t g, int md) -> double {
    const dsde_shard_mass q = masses[int64_t(g) * B + b];
    return md == 0 ? q.mass : md == 1 ? q.p_mass : q.mass * exp2_taylor(double(q.ref) - double(ref_max));
  };
  double acc = 0.0;
  for (int32_t g = lane; g < G; g += 64) acc += weight(g, mode);
  double Z = wave_sum_f64(acc);
  if (mode == 0 && !(Z > 0.0)) {  // no residual mass anywhere: p of the same target row
    mode = 1;
    acc = 0.0;
    for (int32_t g = lane; g < G; g += 64) acc += weight(g, 1);
    Z = wave_sum_f64(acc);
  }
  const double target_mass = double(job.u) * Z;
  int32_t best = -1;
  double best_excl = 0.0, base = 0.0;
  for (int32_t g0 = 0; g0 < G; g0 += 64) {
    const int32_t g = g0 + lane;
    const double w = g < G ? weight(g, mode) : 0.0;
    const lanes::Scan<double> sc = lanes::wave_scan(w);
    const double incl = base + sc.incl;
    const double excl = lane == 0 ? base : base + sc.excl;
    const uint64_t cand = __ballot(g < G && w > 0.0 && excl <= target_mass);
    if (cand) {
      const int l = 63 - __builtin_clzll(cand);
      best = g0 + l;
      best_excl = lanes::readlane(excl, l);
    }
    base = lanes::readlane(incl, 63);
  }
  const int32_t owner = best >= 0 ? best : 0;
  if (owner != gself) {
    if (t == 0) drawn[b] = -1;
    return;
  }
  double rem = target_mass - best_excl;
  if (rem < 0.0) rem = 0.0;
  const float row_ref = mode == 2 ? masses[int64_t(gself) * B + b].ref : 0.f;
  if (mode == 2) rem *= exp2_taylor(double(ref_max) - double(row_ref));  // into this slice's scale
  const size_t esz = DT == DSDE_BF16 ? 2 : 4;
  const char *trow = (const char *)target + size_t(job.target_row) * size_t(V) * esz;
  const char *drow = job.draft_row >= 0 ? (const char *)draft + size_t(job.draft_row) * size_t(V) * esz : nullptr;
  const int64_t cell0 = int64_t(b) * nc;
  if (mode == 1) {  // the slice's p totals, which call 3 did not keep
    for (int32_t ch = wave; ch < nc; ch += kShardWaves) {
      const double p = target_p_chunk<DT, VEC>(trow, V, ch, job, sub + (cell0 + ch) * 64);
      if (lane == 0) ch_w[cell0 + ch] = p;
    }
    __syncthreads();
  }
  if (wave != 0) return;
  const int32_t local = draw_in_row<DT, VEC>(
      nc,
      [&](int32_t ch) -> double {
        return mode == 2 ? ch_w[cell0 + ch] * exp2_taylor(double(ch_ref[cell0 + ch]) - double(row_ref))
                         : ch_w[cell0 + ch];
      },
      [&](int32_t ch) -> float { return ch_ref[cell0 + ch]; }, row_ref, rem, sub + cell0 * 64, trow, drow, V, mode,
      job);
  if (lane == 0) {
    const int32_t token = int32_t(v_begin + local);
    tok[job.accepted] = token;
    drawn[b] = token;
  }
}

bool shard_rows_vectorizable(const ShardRows &r) {
  const auto aligned16 = [](const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  return aligned16(r.target) && (r.N == 0 || aligned16(r.draft)) &&
         (r.dtype == DSDE_BF16 ? r.V_shard % 8 == 0 : r.V_shard % 4 == 0);
}

template <typename F>
void by_layout(const ShardRows &r, F f) {
  const bool vec = shard_rows_vectorizable(r);
  if (r.dtype == DSDE_BF16) {
    if (vec)
      f(std::integral_constant<int, DSDE_BF16>{}, std::true_type{});
    else
      f(std::integral_constant<int, DSDE_BF16>{}, std::false_type{});
  } else {
    if (vec)
      f(std::integral_constant<int, DSDE_FP32>{}, std::true_type{});
    else
      f(std::integral_constant<int, DSDE_FP32>{}, std::false_type{});
  }
}

}  // namespace

int launch_shard_stats(const ShardRows &r, int64_t V, const int32_t *sl, const int32_t *cu_sl,
                       const int32_t *draft_tokens, const float *temperature, dsde_shard_partial *part,
                       uint32_t *seq_err) {
  (void)V;
  const ShardLayout L = shard_layout(r.B, r.N, r.V_shard, r.k_max);
  char *ws = (char *)r.workspace;
  (void)hipGetLastError();
  VerifyArgs a{};
  a.target = r.target;
  a.draft = r.draft;
  a.dtype = r.dtype;
  a.V = r.V_shard;
  a.B = r.B;
  a.N = r.N;
  a.k_max = r.k_max;
  a.sl = sl;
  a.cu_sl = cu_sl;
  a.draft_tokens = draft_tokens;
  a.token_base = r.v_begin;
  a.temperature = temperature;
  a.seq_err = seq_err;
  a.workspace = r.workspace;
  a.stream = r.stream;
  WorkItem *work = (WorkItem *)(ws + L.stats.work);
  PairChunk *pc = (PairChunk *)(ws + L.stats.pair_chunk);
  Gathered *gath = (Gathered *)(ws + L.stats.gathered);
  ChunkArg *cargs = (ChunkArg *)(ws + L.stats.chunk_arg);
  // the shard partial always carries the entropy accumulator: whether a
  // caller wants the entropy is known only when the partials are combined
  launch_stats_pass(a, work, pc, gath, cargs, true);
  if (r.N > 0) {
    const int32_t nc = int32_t(num_chunks(r.V_shard));
    const dim3 grid(unsigned(r.B)), block(kShardThreads);
    if (nc <= 16)
      shard_combine_kernel<16><<<grid, block, 0, r.stream>>>(pc, cargs, gath, sl, cu_sl, draft_tokens, temperature,
                                                             seq_err, r.k_max, nc, r.v_begin, r.V_shard, part);
    else if (nc <= 32)
      shard_combine_kernel<32><<<grid, block, 0, r.stream>>>(pc, cargs, gath, sl, cu_sl, draft_tokens, temperature,
                                                             seq_err, r.k_max, nc, r.v_begin, r.V_shard, part);
    else
      shard_combine_kernel<64><<<grid, block, 0, r.stream>>>(pc, cargs, gath, sl, cu_sl, draft_tokens, temperature,
                                                             seq_err, r.k_max, nc, r.v_begin, r.V_shard, part);
  }
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

int launch_shard_accept(int32_t G, const dsde_shard_partial *parts, int64_t V, int32_t B, int64_t N, int32_t k_max,
                        const int32_t *sl, const int32_t *cu_sl, const int32_t *draft_tokens,
                        const float *temperature, const float *u_acc, const float *u_res, int32_t pad_id,
                        int32_t *accepted, int32_t *tokens, float *kld, double *row_lse, float *draft_entropy,
                        dsde_draw_job *jobs, uint32_t *seq_err, const SignalArgs *signal, hipStream_t stream) {
  (void)hipGetLastError();
  DrawJob *dj = reinterpret_cast<DrawJob *>(jobs);
  if (!signal) {
    shard_accept_kernel<false><<<dim3(unsigned(B)), dim3(64), 0, stream>>>(
        G, parts, N, V, k_max, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, pad_id, accepted, tokens, kld,
        row_lse, draft_entropy, dj, seq_err, SignalArgs{});
    return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
  }
  const SignalArgs &S = *signal;
  shard_accept_kernel<true><<<dim3(unsigned(B)), dim3(64), 0, stream>>>(
      G, parts, N, V, k_max, sl, cu_sl, draft_tokens, temperature, u_acc, u_res, pad_id, accepted, tokens, kld,
      row_lse, draft_entropy, dj, seq_err, S);
  if (hipGetLastError() != hipSuccess) return DSDE_DEVICE_ERROR;
  return launch_next_sl(B, S.sf, S.wvir, S.sl_max, S.sl_min, S.sl_hi, S.budget, S.sl_hat, S.sl_cap, S.sl_next,
                        seq_err, true, stream);
}

int launch_shard_draw_mass(const ShardRows &r, const dsde_shard_partial *part, const dsde_draw_job *jobs,
                           dsde_shard_mass *mass) {
  const ShardLayout L = shard_layout(r.B, r.N, r.V_shard, r.k_max);
  char *ws = (char *)r.workspace;
  const int32_t nc = int32_t(num_chunks(r.V_shard));
  (void)hipGetLastError();
  by_layout(r, [&](auto dt, auto vec) {
    shard_mass_kernel<decltype(dt)::value, decltype(vec)::value><<<dim3(unsigned(r.B)), dim3(kShardThreads), 0,
                                                                   r.stream>>>(
        r.target, r.draft, r.V_shard, nc, r.v_begin, part, reinterpret_cast<const DrawJob *>(jobs), mass,
        (double *)(ws + L.ch_w), (float *)(ws + L.ch_ref), (int32_t *)(ws + L.ch_bad), (float *)(ws + L.sub));
  });
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

int launch_shard_draw_pick(const ShardRows &r, int32_t G, int32_t g, const dsde_shard_mass *masses,
                           const dsde_draw_job *jobs, int32_t pad_id, int32_t *accepted, int32_t *tokens,
                           int32_t *drawn, uint32_t *seq_err) {
  const ShardLayout L = shard_layout(r.B, r.N, r.V_shard, r.k_max);
  char *ws = (char *)r.workspace;
  const int32_t nc = int32_t(num_chunks(r.V_shard));
  (void)hipGetLastError();
  by_layout(r, [&](auto dt, auto vec) {
    shard_pick_kernel<decltype(dt)::value, decltype(vec)::value><<<dim3(unsigned(r.B)), dim3(kShardThreads), 0,
                                                                   r.stream>>>(
        G, g, masses, r.B, r.target, r.draft, r.V_shard, nc, r.v_begin, r.k_max,
        reinterpret_cast<const DrawJob *>(jobs), pad_id, accepted, tokens, drawn, seq_err, (double *)(ws + L.ch_w),
        (const float *)(ws + L.ch_ref), (float *)(ws + L.sub));
  });
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

}  // namespace dsde
