// Device code of the KLD stability signal (Sec. 3.1.2, Eqs. 3-7) and of the
// SL rule with the batch cap (Eqs. 2, 8; Sec. 3.3, Eqs. 9-11).  Used by the
// standalone kernels and by the fused step, so both give identical bits.
#pragma once

#include <math.h>

#include "common.hpp"

namespace dsde {

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Recency-weighted mean and population variance of the n newest ring entries
// (h_1 newest, whose value is passed as `h1`), alpha_i = delta^(i-1),
// evaluated by one wavefront (lane i holds entries i, i + 64, ...).
// Fixed-order sums: bitwise reproducible.
__device__ inline void wave_window_stats(const float *ring, int32_t W, int32_t newest, float h1, int32_t n,
                                         double delta, double *mean, double *var) {
  const int lane = threadIdx.x & 63;
  if (n <= 0) {
    *mean = 0.0;
    *var = 0.0;
    return;
  }
  double sa = 0.0, sah = 0.0;
  for (int32_t i = lane; i < n; i += 64) {
    const double alpha = pow(delta, double(i));
    const double h = i == 0 ? double(h1) : double(ring[(newest - i + W) % W]);
    sa += alpha;
    sah += alpha * h;
  }
  sa = wave_sum_f64(sa);
  sah = wave_sum_f64(sah);
  const double mu = sah / sa;
  double sv = 0.0;
  for (int32_t i = lane; i < n; i += 64) {
    const double alpha = pow(delta, double(i));
    const double d = (i == 0 ? double(h1) : double(ring[(newest - i + W) % W])) - mu;
    sv += alpha * d * d;
  }
  sv = wave_sum_f64(sv);
  *mean = mu;
  *var = sv / sa;
}

// Signal update of one sequence by one wavefront.  The sequence's `s` KLD
// values are kld[first .. first + s) or, when kld is null (s <= 64), the
// per-lane values `lane_kld` (lane j holds position j).  Ring hist[0..W) with
// head/count.  Returns the error bits (DSDE_ERR_STATE, DSDE_ERR_SIGNAL); on
// error nothing is pushed and every output is NaN.
__device__ inline uint32_t wave_signal_update(int32_t s, int64_t first, const float *kld, float lane_kld, float *ring,
                                              int32_t *head, int32_t *count, int32_t W, int32_t n_short,
                                              int32_t n_long, float delta, float eps, float *mu_last,
                                              float *var_short, float *var_long, float *wvir, float *sf) {
  const int lane = threadIdx.x & 63;
  uint32_t err = 0;
  const int32_t hd = *head, cnt = *count;
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
  if (s > 0) {  // push the step's mean KLD; i = 1 is the step just verified
    h1 = float(mu);
    // every lane reads the older entries before lane 0 overwrites the slot
    // below; the pushed value itself is passed in registers
    h = (h + 1) % W;
    c = c < W ? c + 1 : W;
  } else {
    h1 = c > 0 ? ring[(h - 1 + W) % W] : 0.0f;
    mu = c > 0 ? double(h1) : 0.0;
  }
  const int32_t newest = (h - 1 + W) % W;
  double ms, vs, ml, vl;
  wave_window_stats(ring, W, newest, h1, n_short < c ? n_short : c, double(delta), &ms, &vs);
  wave_window_stats(ring, W, newest, h1, n_long < c ? n_long : c, double(delta), &ml, &vl);
  if (s > 0 && lane == 0) {
    ring[newest] = h1;
    *head = h;
    *count = c;
  }
  if (lane == 0) {
    *mu_last = float(mu);
    *var_short = float(vs);
    *var_long = float(vl);
    *wvir = float(vs / (vl + double(eps)));
    *sf = float(expm1(2.0 * mu));
  }
  return 0;
}

// Eq. 2 with Eq. 8's lower bound, in double from the float inputs.
__device__ __forceinline__ double sl_hat_of(double sf, double wvir, double sl_max, double sl_min) {
  const double pen = sf * wvir;
  return pen <= 1.0 ? (1.0 - pen) * (sl_max - sl_min) + sl_min : sl_min;
}

// SL rule and batch cap by one workgroup (any blockDim up to 1024; `red_s`,
// `red_n` are blockDim-sized LDS arrays).  seq_err bits are OR-ed atomically
// when `or_err` is set (fused step), else written.
__device__ inline void block_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max,
                                     float sl_min, int32_t sl_hi, float *sl_hat, float *sl_cap, int32_t *sl_next,
                                     uint32_t *seq_err, bool or_err, double *red_s, int *red_n) {
  const int t = threadIdx.x, nt = blockDim.x;
  const double lo_f = double(sl_min);
  const int32_t lo = int32_t(ceil(lo_f));
  double part = 0.0;
  int cnt = 0;
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
  red_s[t] = part;
  red_n[t] = cnt;
  __syncthreads();
  for (int o = nt / 2; o > 0; o >>= 1) {
    if (t < o) {
      red_s[t] += red_s[t + o];
      red_n[t] += red_n[t + o];
    }
    __syncthreads();
  }
  const double cap = red_n[0] > 0 ? red_s[0] / double(red_n[0]) : NAN;
  if (t == 0) sl_cap[0] = float(cap);
  for (int32_t b = t; b < B; b += nt) {
    const double f = sf[b], w = wvir[b], mx = sl_max[b];
    const bool ok = isfinite(f) && isfinite(w) && isfinite(mx) && mx >= lo_f;
    if (or_err) {
      if (!ok) atomicOr(&seq_err[b], DSDE_ERR_SIGNAL);
    } else {
      seq_err[b] = ok ? 0u : DSDE_ERR_SIGNAL;
    }
    if (!ok) {
      sl_next[b] = lo;
      continue;
    }
    const double hat = sl_hat_of(f, w, mx, lo_f);
    const double x = hat < cap ? hat : cap;
    double r = floor(x + 0.5);
    r = r < double(lo) ? double(lo) : r;
    r = r > double(sl_hi) ? double(sl_hi) : r;
    sl_next[b] = int32_t(r);
  }
}

}  // namespace dsde
