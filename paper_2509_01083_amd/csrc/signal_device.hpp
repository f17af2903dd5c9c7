// Device code of the KLD stability signal (Sec. 3.1.2, Eqs. 3-7) and of the
// SL rule with the batch cap (Eqs. 2, 8; Sec. 3.3, Eqs. 9-11).  Used by the
// standalone kernels and by the fused step, so both give identical bits.
#pragma once

#include <math.h>

#include "common.hpp"
#include "lanes.hpp"

namespace dsde {

__device__ __forceinline__ double wave_sum_f64(double v) { return lanes::wave_sum(v); }

// Ring slots one wavefront keeps in registers: with W <= 64 * kRingRegs every
// window entry is read from registers, larger rings are read from memory.
constexpr int kRingRegs = 4;

// The ring state of one sequence, fetched by one wavefront ahead of use:
// head, count, and ring slot l + 64 k in lane l, register k.
struct RingPrefetch {
  int32_t head, count;
  float slot[kRingRegs];
};

__device__ __forceinline__ RingPrefetch wave_ring_prefetch(const float *ring, const int32_t *head,
                                                           const int32_t *count, int32_t W) {
  const int lane = threadIdx.x & 63;
  // mbcnt over an empty mask is 0 in every lane, but the compiler treats it
  // as lane-varying: head and count become vector loads, issued with the ring
  // loads, instead of scalar loads competing for scalar registers
  const uint32_t zero = __builtin_amdgcn_mbcnt_lo(0u, 0u);
  RingPrefetch r;
  r.head = head[zero];
  r.count = count[zero];
#pragma unroll
  for (int k = 0; k < kRingRegs; ++k) {
    const int32_t i = lane + 64 * k;
    r.slot[k] = ring[i < W ? i : W - 1];  // clamped index: always in bounds (W >= 1)
  }
  return r;
}

// Value of ring slot `slot` (0 <= slot < W), in every lane that asks.  Must be
// reached by the whole wavefront (it shuffles when the ring is in registers).
__device__ __forceinline__ float ring_slot(const RingPrefetch &rp, const float *ring, int32_t W, int32_t slot) {
  if (W <= 64 * kRingRegs) {
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < kRingRegs; ++k) {
      if (64 * k >= W) break;  // uniform: registers past the ring hold nothing
      const float x = __shfl(rp.slot[k], slot & 63);
      if ((slot >> 6) == k) v = x;
    }
    return v;
  }
  return ring[slot];
}

// delta^n for n >= 0 by binary powering (a few multiplications, no pow()).
__device__ __forceinline__ double pow_int(double x, int32_t n) {
  double r = 1.0;
  while (n) {
    if (n & 1) r *= x;
    x *= x;
    n >>= 1;
  }
  return r;
}

// Recency-weighted means and population variances (Eqs. 6-7) of the ns and
// nl newest ring entries (ns <= nl), evaluated together by one wavefront:
// entry i (i = 0 newest, value h1 passed in registers) sits in ring slot
// (newest - i) mod W and has weight alpha = delta^i.  The sums take each
// entry less h1 (exact in double: both are floats), which leaves Eq. 7
// unchanged and gives a window of equal entries a variance of exactly 0.  The
// means returned are those of the entries less h1.  Lane l holds entries
// l, l + 64, ...; fixed-order sums, bitwise reproducible.
__device__ inline void wave_windows(const RingPrefetch &rp, const float *ring, int32_t W, int32_t newest, float h1,
                                    int32_t ns, int32_t nl, double delta, double *ms, double *vs, double *ml,
                                    double *vl) {
  const int lane = threadIdx.x & 63;
  const int32_t rounds = (nl + 63) / 64;
  double sa_s = 0.0, sah_s = 0.0, sa_l = 0.0, sah_l = 0.0;
  for (int32_t r = 0; r < rounds; ++r) {
    const int32_t i = lane + 64 * r;
    const int32_t slot = i < W ? (newest - i + W) % W : 0;
    const float raw = ring_slot(rp, ring, W, slot);
    if (i < nl) {
      const double h = i == 0 ? 0.0 : double(raw) - double(h1);
      const double a = pow_int(delta, i);
      sa_l += a;
      sah_l += a * h;
      if (i < ns) {
        sa_s += a;
        sah_s += a * h;
      }
    }
  }
  sa_s = wave_sum_f64(sa_s);
  sah_s = wave_sum_f64(sah_s);
  sa_l = wave_sum_f64(sa_l);
  sah_l = wave_sum_f64(sah_l);
  const double mu_s = ns > 0 ? sah_s / sa_s : 0.0, mu_l = nl > 0 ? sah_l / sa_l : 0.0;
  double sv_s = 0.0, sv_l = 0.0;
  for (int32_t r = 0; r < rounds; ++r) {
    const int32_t i = lane + 64 * r;
    const int32_t slot = i < W ? (newest - i + W) % W : 0;
    const float raw = ring_slot(rp, ring, W, slot);
    if (i < nl) {
      const double h = i == 0 ? 0.0 : double(raw) - double(h1);
      const double a = pow_int(delta, i);
      const double dl = h - mu_l;
      sv_l += a * dl * dl;
      if (i < ns) {
        const double ds = h - mu_s;
        sv_s += a * ds * ds;
      }
    }
  }
  sv_s = wave_sum_f64(sv_s);
  sv_l = wave_sum_f64(sv_l);
  *ms = mu_s;
  *ml = mu_l;
  *vs = ns > 0 ? sv_s / sa_s : 0.0;
  *vl = nl > 0 ? sv_l / sa_l : 0.0;
}

// Signal update of one sequence by one wavefront (Sec. 3.1.2).  The sequence's
// `s` KLD values are kld[first .. first + s) or, when kld is null (s <= 64),
// the per-lane values `lane_kld` (lane j holds position j).  `rp` is the ring
// state fetched by this wavefront; the ring is hist[0..W).  Returns the error
// bits (DSDE_ERR_STATE, DSDE_ERR_SIGNAL); on error nothing is pushed and every
// output is NaN.  Must be reached by the whole wavefront.
__device__ inline uint32_t wave_signal_update(int32_t s, int64_t first, const float *kld, float lane_kld,
                                              const RingPrefetch &rp, float *ring, int32_t *head, int32_t *count,
                                              int32_t W, int32_t n_short, int32_t n_long, float delta, float eps,
                                              float *mu_last, float *var_short, float *var_long, float *wvir,
                                              float *sf) {
  const int lane = threadIdx.x & 63;
  uint32_t err = 0;
  const int32_t hd = rp.head, cnt = rp.count;
  if (hd < 0 || hd >= W || cnt < 0 || cnt > W) err |= DSDE_ERR_STATE;
  double mu = 0.0;
  if (!err && s > 0) {
    double acc = 0.0;
    if (kld)
      for (int32_t j = lane; j < s; j += 64) acc += double(kld[first + j]);
    else if (lane < s)
      acc = double(lane_kld);
    acc = wave_sum_f64(acc);
    mu = acc / double(s);
    if (!isfinite(mu)) err |= DSDE_ERR_SIGNAL;
  }
  if (err) {
    if (lane == 0) *mu_last = *var_short = *var_long = *wvir = *sf = NAN;
    return err;
  }
  int32_t h = hd, c = cnt;
  float h1;
  if (s > 0) {  // push the step's mean KLD; i = 0 is the step just verified
    h1 = float(mu);
    // the older entries are read before lane 0 overwrites the slot below; the
    // pushed value itself is passed in registers
    h = (h + 1) % W;
    c = c < W ? c + 1 : W;
  } else {
    const float newest_old = ring_slot(rp, ring, W, (h - 1 + W) % W);
    h1 = c > 0 ? newest_old : 0.0f;
    mu = c > 0 ? double(h1) : 0.0;
  }
  const int32_t newest = (h - 1 + W) % W;
  double ms, vs, ml, vl;
  wave_windows(rp, ring, W, newest, h1, n_short < c ? n_short : c, n_long < c ? n_long : c, double(delta), &ms, &vs,
               &ml, &vl);
  if (s > 0 && lane == 0) {
    ring[newest] = h1;
    *head = h;
    *count = c;
  }
  if (lane == 0) {
    *mu_last = float(mu);
    *var_short = float(vs);
    *var_long = float(vl);
    // Eq. 4; eps stands in for the long-window variance only where that is 0
    // (equal entries, so the short window is constant too and WVIR = 0)
    *wvir = float(vs / (vl > 0.0 ? vl : double(eps)));
    *sf = float(expm1(2.0 * mu));
  }
  return 0;
}

// Eq. 2 with Eq. 8's lower bound, in double from the float inputs.
__device__ __forceinline__ double sl_hat_of(double sf, double wvir, double sl_max, double sl_min) {
  const double pen = sf * wvir;
  return pen <= 1.0 ? (1.0 - pen) * (sl_max - sl_min) + sl_min : sl_min;
}

// Sequences per thread whose inputs block_next_sl keeps in registers between
// its two passes (one memory round trip); larger batches load them twice.
constexpr int kNextSlRegs = 4;

// SL rule and batch cap by one workgroup (blockDim a multiple of 64, at most
// 1024; `red_s`, `red_n` are LDS arrays of blockDim / 64 entries), then the
// per-sequence token budget (optional) bounds each next length.  Per-thread
// fp64 partial sums, wavefront butterflies, then the wavefront totals in order:
// a fixed order, so the cap is bitwise reproducible.  seq_err bits are OR-ed
// into what earlier kernels wrote when `or_err` is set (fused step), else
// written.

__device__ inline void block_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max,
                                     float sl_min, int32_t sl_hi, const int32_t *budget, float *sl_hat,
                                     float *sl_cap, int32_t *sl_next, uint32_t *seq_err, bool or_err, double *red_s,
                                     int *red_n) {
  const int t = threadIdx.x, nt = blockDim.x, lane = t & 63, wave = t >> 6;
  const double lo_f = double(sl_min);
  const int32_t lo = int32_t(ceil(lo_f));
  const bool cached = B <= kNextSlRegs * nt;
  // pass 1: SL_hat of every sequence (thread t: sequences t, t + nt, ...);
  // with a small batch every input of both passes is loaded here at once
  float r_f[kNextSlRegs], r_w[kNextSlRegs], r_m[kNextSlRegs];
  int32_t r_bud[kNextSlRegs];
  uint32_t r_err[kNextSlRegs];
  if (cached) {
#pragma unroll
    for (int i = 0; i < kNextSlRegs; ++i) {
      const int32_t b = t + i * nt;
      r_f[i] = b < B ? sf[b] : 0.f;
      r_w[i] = b < B ? wvir[b] : 0.f;
      r_m[i] = b < B ? sl_max[b] : 0.f;
      r_bud[i] = b < B && budget ? budget[b] : 0;
      r_err[i] = b < B && or_err ? seq_err[b] : 0u;
    }
  }
  double part = 0.0;
  int cnt = 0;
  if (cached) {
#pragma unroll
    for (int i = 0; i < kNextSlRegs; ++i) {
      const int32_t b = t + i * nt;
      if (b >= B) continue;
      const double f = r_f[i], w = r_w[i], mx = r_m[i];
      const bool ok = isfinite(f) && isfinite(w) && isfinite(mx) && mx >= lo_f;
      const double hat = ok ? sl_hat_of(f, w, mx, lo_f) : 0.0;
      sl_hat[b] = ok ? float(hat) : NAN;
      part += hat;
      cnt += ok;
    }
  } else {
    for (int32_t b = t; b < B; b += nt) {
      const double f = sf[b], w = wvir[b], mx = sl_max[b];
      const bool ok = isfinite(f) && isfinite(w) && isfinite(mx) && mx >= lo_f;
      if (ok) {
        const double hat = sl_hat_of(f, w, mx, lo_f);
        sl_hat[b] = float(hat);
        part += hat;
        ++cnt;
      } else {
        sl_hat[b] = NAN;
      }
    }
  }
  part = wave_sum_f64(part);
  cnt = lanes::wave_sum(cnt);
  if (lane == 0) {
    red_s[wave] = part;
    red_n[wave] = cnt;
  }
  __syncthreads();
  double total = 0.0;
  int n = 0;
  for (int v = 0; v < nt / 64; ++v) {
    total += red_s[v];
    n += red_n[v];
  }
  const double cap = n > 0 ? total / double(n) : NAN;
  if (t == 0) sl_cap[0] = float(cap);
  // pass 2: the rounded, clamped next length under the cap
  auto next_of = [&](int32_t b, double f, double w, double mx, int32_t bud, uint32_t err) {
    const bool ok = isfinite(f) && isfinite(w) && isfinite(mx) && mx >= lo_f;
    // or_err: only this thread writes seq_err[b] in this kernel, so a plain
    // read-modify-write adds the signal bit to what earlier kernels set
    seq_err[b] = or_err ? (ok ? err : err | DSDE_ERR_SIGNAL) : (ok ? 0u : DSDE_ERR_SIGNAL);
    int32_t next = lo;
    if (ok) {
      const double hat = sl_hat_of(f, w, mx, lo_f);
      const double x = hat < cap ? hat : cap;
      double r = floor(x + 0.5);
      r = r < double(lo) ? double(lo) : r;
      r = r > double(sl_hi) ? double(sl_hi) : r;
      next = int32_t(r);
    }
    if (budget) {  // a step emits up to SL + 1 tokens (Sec. 3.2's budget clamp)
      const int32_t room = bud - 1 > 0 ? bud - 1 : 0;
      next = next < room ? next : room;
    }
    sl_next[b] = next;
  };
  if (cached) {
#pragma unroll
    for (int i = 0; i < kNextSlRegs; ++i) {
      const int32_t b = t + i * nt;
      if (b < B) next_of(b, r_f[i], r_w[i], r_m[i], r_bud[i], r_err[i]);
    }
  } else {
    for (int32_t b = t; b < B; b += nt)
      next_of(b, sf[b], wvir[b], sl_max[b], budget ? budget[b] : 0, or_err ? seq_err[b] : 0u);
  }
}

}  // namespace dsde
