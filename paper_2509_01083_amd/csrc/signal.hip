// KLD stability signal (Sec. 3.1.2, Eqs. 3-7) and the next speculation length
// under the batch cap (Eqs. 2, 8 and Sec. 3.3, Eqs. 9-11).
//
// Both kernels are one workgroup of 1024 threads: the layout check and the cap
// are batch-wide, and the work per sequence is a few dozen flops, so these
// kernels cost their launch, not bytes.  Sums run in double precision in a
// fixed order (per-thread strided partial sums, then a fixed tree).
#include <math.h>

#include "common.hpp"

namespace dsde {
namespace {

constexpr int kSigThreads = 1024;

// Recency-weighted mean and population variance of the n newest ring entries
// (h_1 newest), alpha_i = delta^(i-1); an empty window gives (0, 0).
__device__ void window_stats(const float *ring, int32_t W, int32_t newest, int32_t n, double delta, double *mean,
                             double *var) {
  if (n <= 0) {
    *mean = 0.0;
    *var = 0.0;
    return;
  }
  double sa = 0.0, sah = 0.0, alpha = 1.0;
  for (int32_t i = 0; i < n; ++i) {
    const double h = ring[(newest - i + W) % W];
    sa += alpha;
    sah += alpha * h;
    alpha *= delta;
  }
  const double mu = sah / sa;
  double sv = 0.0;
  alpha = 1.0;
  for (int32_t i = 0; i < n; ++i) {
    const double d = double(ring[(newest - i + W) % W]) - mu;
    sv += alpha * d * d;
    alpha *= delta;
  }
  *mean = mu;
  *var = sv / sa;
}

__global__ __launch_bounds__(kSigThreads) void kld_signal_kernel(
    int32_t B, int64_t N, const int32_t *__restrict__ sl, const int32_t *__restrict__ cu_sl,
    const float *__restrict__ kld, float *__restrict__ hist, int32_t *__restrict__ head,
    int32_t *__restrict__ count, int32_t W, int32_t n_short, int32_t n_long, float delta, float eps,
    float *__restrict__ mu_last, float *__restrict__ var_short, float *__restrict__ var_long,
    float *__restrict__ wvir, float *__restrict__ sf, uint32_t *__restrict__ seq_err) {
  int bad = 0;
  for (int32_t b = threadIdx.x; b < B; b += blockDim.x)
    if (sl[b] < 0 || int64_t(cu_sl[b + 1]) - int64_t(cu_sl[b]) != int64_t(sl[b])) bad = 1;
  bad = __syncthreads_or(bad);
  if (cu_sl[0] != 0 || int64_t(cu_sl[B]) != N) bad = 1;

  for (int32_t b = threadIdx.x; b < B; b += blockDim.x) {
    uint32_t err = bad ? DSDE_ERR_LAYOUT : 0u;
    const int32_t hd = head[b], cnt = count[b];
    if (hd < 0 || hd >= W || cnt < 0 || cnt > W) err |= DSDE_ERR_STATE;
    const int32_t s = bad ? 0 : sl[b];
    double mu = 0.0;
    if (!err && s > 0) {
      double acc = 0.0;
      const int32_t first = cu_sl[b];
      for (int32_t j = 0; j < s; ++j) acc += double(kld[first + j]);
      mu = acc / double(s);
      if (!isfinite(mu)) err |= DSDE_ERR_SIGNAL;
    }
    seq_err[b] = err;
    if (err) {
      mu_last[b] = var_short[b] = var_long[b] = wvir[b] = sf[b] = NAN;
      continue;
    }
    float *ring = hist + int64_t(b) * W;
    int32_t h = hd, c = cnt;
    if (s > 0) {  // push the step's mean KLD; i = 1 is the step just verified
      ring[h] = float(mu);
      h = (h + 1) % W;
      c = c < W ? c + 1 : W;
      head[b] = h;
      count[b] = c;
    } else {
      mu = c > 0 ? double(ring[(h - 1 + W) % W]) : 0.0;
    }
    const int32_t newest = (h - 1 + W) % W;
    double ms, vs, ml, vl;
    window_stats(ring, W, newest, n_short < c ? n_short : c, double(delta), &ms, &vs);
    window_stats(ring, W, newest, n_long < c ? n_long : c, double(delta), &ml, &vl);
    mu_last[b] = float(mu);
    var_short[b] = float(vs);
    var_long[b] = float(vl);
    wvir[b] = float(vs / (vl + double(eps)));
    sf[b] = float(expm1(2.0 * mu));
  }
}

__global__ __launch_bounds__(kSigThreads) void next_sl_kernel(int32_t B, const float *__restrict__ sf,
                                                              const float *__restrict__ wvir,
                                                              const float *__restrict__ sl_max, float sl_min,
                                                              int32_t sl_hi, float *__restrict__ sl_hat,
                                                              float *__restrict__ sl_cap,
                                                              int32_t *__restrict__ sl_next,
                                                              uint32_t *__restrict__ seq_err) {
  __shared__ double red_s[kSigThreads];
  __shared__ int red_n[kSigThreads];
  const int t = threadIdx.x;
  const double lo_f = double(sl_min);
  double part = 0.0;
  int cnt = 0;
  for (int32_t b = t; b < B; b += blockDim.x) {
    const double f = sf[b], w = wvir[b], mx = sl_max[b];
    const bool ok = isfinite(f) && isfinite(w) && isfinite(mx) && mx >= lo_f;
    seq_err[b] = ok ? 0u : DSDE_ERR_SIGNAL;
    if (ok) {
      const double pen = f * w;
      const double hat = pen <= 1.0 ? (1.0 - pen) * (mx - lo_f) + lo_f : lo_f;
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
  for (int o = kSigThreads / 2; o > 0; o >>= 1) {
    if (t < o) {
      red_s[t] += red_s[t + o];
      red_n[t] += red_n[t + o];
    }
    __syncthreads();
  }
  const double cap = red_n[0] > 0 ? red_s[0] / double(red_n[0]) : NAN;
  if (t == 0) sl_cap[0] = float(cap);
  const int32_t lo = int32_t(ceil(lo_f));
  for (int32_t b = t; b < B; b += blockDim.x) {
    if (seq_err[b]) {
      sl_next[b] = lo;
      continue;
    }
    // recompute SL_hat in double rather than reading back its float copy
    const double f = sf[b], w = wvir[b], mx = sl_max[b];
    const double pen = f * w;
    const double hat = pen <= 1.0 ? (1.0 - pen) * (mx - lo_f) + lo_f : lo_f;
    const double x = hat < cap ? hat : cap;
    double r = floor(x + 0.5);
    r = r < double(lo) ? double(lo) : r;
    r = r > double(sl_hi) ? double(sl_hi) : r;
    sl_next[b] = int32_t(r);
  }
}

}  // namespace

int launch_kld_signal(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const float *kld, float *hist,
                      int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long, float delta,
                      float eps, float *mu_last, float *var_short, float *var_long, float *wvir, float *sf,
                      uint32_t *seq_err, hipStream_t stream) {
  (void)hipGetLastError();
  kld_signal_kernel<<<dim3(1), dim3(kSigThreads), 0, stream>>>(B, N, sl, cu_sl, kld, hist, head, count, W,
                                                               n_short, n_long, delta, eps, mu_last, var_short,
                                                               var_long, wvir, sf, seq_err);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

int launch_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max, float sl_min, int32_t sl_hi,
                   float *sl_hat, float *sl_cap, int32_t *sl_next, uint32_t *seq_err, hipStream_t stream) {
  (void)hipGetLastError();
  next_sl_kernel<<<dim3(1), dim3(kSigThreads), 0, stream>>>(B, sf, wvir, sl_max, sl_min, sl_hi, sl_hat, sl_cap,
                                                            sl_next, seq_err);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

}  // namespace dsde
