// Standalone kernels of the KLD stability signal (Sec. 3.1.2, Eqs. 3-7) and
// of the next speculation length under the batch cap (Eqs. 2, 8; Sec. 3.3,
// Eqs. 9-11).  The per-sequence and per-batch code is shared with the fused
// step (signal_device.hpp).
//
//   kld_signal_kernel  one wavefront per sequence (lanes over the window
//                      entries); every workgroup re-checks the batch layout.
//   calibration_update_kernel, calibrate_kernel
//                      the SL_max calibration of Eq. 1 (Sec. 3.1.1): per-sequence
//                      statistics folded over the calibration steps, then
//                      SL_max per sequence or pooled over the batch.
//   next_sl_kernel     one workgroup: SL_hat per sequence, the mean cap, the
//                      rounded and clamped next lengths (also the last kernel
//                      of the fused step, where it ORs its error bits).
// Both cost their launch, not bytes.
#include <math.h>

#include "common.hpp"
#include "signal_device.hpp"

namespace dsde {
namespace {

constexpr int kSigThreads = 256;  // 4 sequences per workgroup
constexpr int kCapThreads = 256;

__global__ __launch_bounds__(kSigThreads) void kld_signal_kernel(
    int32_t B, int64_t N, const int32_t *__restrict__ sl, const int32_t *__restrict__ cu_sl,
    const float *__restrict__ kld, float *__restrict__ hist, int32_t *__restrict__ head,
    int32_t *__restrict__ count, int32_t W, int32_t n_short, int32_t n_long, float delta, float eps,
    float *__restrict__ mu_last, float *__restrict__ var_short, float *__restrict__ var_long,
    float *__restrict__ wvir, float *__restrict__ sf, uint32_t *__restrict__ seq_err) {
  const int32_t b = int32_t(blockIdx.x) * (kSigThreads / 64) + int32_t(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  // the ring state does not depend on the layout: fetch it with the layout check
  RingPrefetch rp{};
  if (b < B) rp = wave_ring_prefetch(hist + int64_t(b) * W, head + b, count + b, W);
  int bad = 0;
  for (int32_t q = threadIdx.x; q < B; q += blockDim.x)
    if (sl[q] < 0 || int64_t(cu_sl[q + 1]) - int64_t(cu_sl[q]) != int64_t(sl[q])) bad = 1;
  bad = __syncthreads_or(bad);
  if (cu_sl[0] != 0 || int64_t(cu_sl[B]) != N) bad = 1;
  if (b >= B) return;
  if (bad) {
    if (lane == 0) {
      seq_err[b] = DSDE_ERR_LAYOUT;
      mu_last[b] = var_short[b] = var_long[b] = wvir[b] = sf[b] = NAN;
    }
    return;
  }
  const uint32_t e = wave_signal_update(sl[b], cu_sl[b], kld, 0.0f, rp, hist + int64_t(b) * W, head + b, count + b,
                                        W, n_short, n_long, delta, eps, mu_last + b, var_short + b, var_long + b,
                                        wvir + b, sf + b);
  if (lane == 0) seq_err[b] = e;
}

__global__ __launch_bounds__(kCapThreads) void next_sl_kernel(int32_t B, const float *__restrict__ sf,
                                                              const float *__restrict__ wvir,
                                                              const float *__restrict__ sl_max, float sl_min,
                                                              int32_t sl_hi, const int32_t *__restrict__ budget,
                                                              float *__restrict__ sl_hat,
                                                              float *__restrict__ sl_cap,
                                                              int32_t *__restrict__ sl_next,
                                                              uint32_t *__restrict__ seq_err, bool or_err) {
  __shared__ double red_s[kCapThreads / 64];
  __shared__ int red_n[kCapThreads / 64];
  block_next_sl(B, sf, wvir, sl_max, sl_min, sl_hi, budget, sl_hat, sl_cap, sl_next, seq_err, or_err, red_s, red_n);
}

__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Eq. 1's statistics of one verification step folded into the running ones,
// one wavefront per sequence: the largest accepted count, the sum (fp64, a
// fixed order) and number of KLD values, and the largest KLD.  Sequences with
// error bits are skipped; an invalid batch layout skips the whole step.
__global__ __launch_bounds__(kSigThreads) void calibration_update_kernel(
    int32_t B, int64_t N, const int32_t *__restrict__ sl, const int32_t *__restrict__ cu_sl,
    const int32_t *__restrict__ accepted, const float *__restrict__ kld, const uint32_t *__restrict__ seq_err,
    int32_t *__restrict__ a_max, double *__restrict__ kld_sum, int64_t *__restrict__ kld_count,
    float *__restrict__ kld_max) {
  int bad = 0;
  for (int32_t q = threadIdx.x; q < B; q += blockDim.x)
    if (sl[q] < 0 || int64_t(cu_sl[q + 1]) - int64_t(cu_sl[q]) != int64_t(sl[q])) bad = 1;
  bad = __syncthreads_or(bad);
  if (bad || cu_sl[0] != 0 || int64_t(cu_sl[B]) != N) return;
  const int32_t b = int32_t(blockIdx.x) * (kSigThreads / 64) + int32_t(threadIdx.x >> 6);
  if (b >= B || seq_err[b] != 0) return;
  const int lane = threadIdx.x & 63;
  const int32_t s = sl[b];
  const int64_t first = cu_sl[b];
  double acc = 0.0;
  float mx = 0.0f;
  for (int32_t j = lane; j < s; j += 64) {
    const float v = kld[first + j];
    acc += double(v);
    mx = fmaxf(mx, v);
  }
  acc = wave_sum_f64(acc);
  mx = wave_max_f32(mx);
  if (lane == 0) {
    a_max[b] = accepted[b] > a_max[b] ? accepted[b] : a_max[b];
    kld_sum[b] += acc;
    kld_count[b] += s;
    kld_max[b] = fmaxf(kld_max[b], mx);
  }
}

// Eq. 1: SL_max = SL_A,max (1 + mu_KLD,pre / (KLD_pre,max + eps)), per sequence
// or from the statistics pooled over the batch (fixed-order reductions).
__global__ __launch_bounds__(kCapThreads) void calibrate_kernel(int32_t B, const int32_t *__restrict__ a_max,
                                                                const double *__restrict__ kld_sum,
                                                                const int64_t *__restrict__ kld_count,
                                                                const float *__restrict__ kld_max, float eps,
                                                                bool pooled, float *__restrict__ sl_max) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  auto eq1 = [&](double amax, double sum, double cnt, double kmax) {
    const double mean = cnt > 0.0 ? sum / cnt : 0.0;
    return float(amax * (1.0 + mean / (kmax + double(eps))));
  };
  if (!pooled) {
    for (int32_t b = t; b < B; b += blockDim.x)
      sl_max[b] = eq1(double(a_max[b]), kld_sum[b], double(kld_count[b]), double(kld_max[b]));
    return;
  }
  __shared__ double r_sum[kCapThreads / 64];
  __shared__ int64_t r_cnt[kCapThreads / 64];
  __shared__ int32_t r_amax[kCapThreads / 64];
  __shared__ float r_kmax[kCapThreads / 64];
  double sum = 0.0;
  int64_t cnt = 0;
  int32_t amax = 0;
  float kmax = 0.0f;
  for (int32_t b = t; b < B; b += blockDim.x) {
    sum += kld_sum[b];
    cnt += kld_count[b];
    amax = a_max[b] > amax ? a_max[b] : amax;
    kmax = fmaxf(kmax, kld_max[b]);
  }
  sum = wave_sum_f64(sum);
  kmax = wave_max_f32(kmax);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    cnt += __shfl_xor(cnt, o);
    amax = max(amax, __shfl_xor(amax, o));
  }
  if (lane == 0) {
    r_sum[wave] = sum;
    r_cnt[wave] = cnt;
    r_amax[wave] = amax;
    r_kmax[wave] = kmax;
  }
  __syncthreads();
  double S = 0.0;
  int64_t C = 0;
  int32_t A = 0;
  float K = 0.0f;
  for (int v = 0; v < int(blockDim.x) / 64; ++v) {
    S += r_sum[v];
    C += r_cnt[v];
    A = r_amax[v] > A ? r_amax[v] : A;
    K = fmaxf(K, r_kmax[v]);
  }
  const float value = eq1(double(A), S, double(C), double(K));
  for (int32_t b = t; b < B; b += blockDim.x) sl_max[b] = value;
}

}  // namespace

int launch_kld_signal(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const float *kld, float *hist,
                      int32_t *head, int32_t *count, int32_t W, int32_t n_short, int32_t n_long, float delta,
                      float eps, float *mu_last, float *var_short, float *var_long, float *wvir, float *sf,
                      uint32_t *seq_err, hipStream_t stream) {
  (void)hipGetLastError();
  const unsigned blocks = unsigned((B + kSigThreads / 64 - 1) / (kSigThreads / 64));
  kld_signal_kernel<<<dim3(blocks), dim3(kSigThreads), 0, stream>>>(B, N, sl, cu_sl, kld, hist, head, count, W,
                                                                    n_short, n_long, delta, eps, mu_last, var_short,
                                                                    var_long, wvir, sf, seq_err);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

int launch_next_sl(int32_t B, const float *sf, const float *wvir, const float *sl_max, float sl_min, int32_t sl_hi,
                   const int32_t *budget, float *sl_hat, float *sl_cap, int32_t *sl_next, uint32_t *seq_err,
                   bool or_err, hipStream_t stream) {
  (void)hipGetLastError();
  next_sl_kernel<<<dim3(1), dim3(kCapThreads), 0, stream>>>(B, sf, wvir, sl_max, sl_min, sl_hi, budget, sl_hat,
                                                            sl_cap, sl_next, seq_err, or_err);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

int launch_calibration_update(int32_t B, int64_t N, const int32_t *sl, const int32_t *cu_sl, const int32_t *accepted,
                              const float *kld, const uint32_t *seq_err, int32_t *a_max, double *kld_sum,
                              int64_t *kld_count, float *kld_max, hipStream_t stream) {
  (void)hipGetLastError();
  const unsigned blocks = unsigned((B + kSigThreads / 64 - 1) / (kSigThreads / 64));
  calibration_update_kernel<<<dim3(blocks), dim3(kSigThreads), 0, stream>>>(B, N, sl, cu_sl, accepted, kld, seq_err,
                                                                            a_max, kld_sum, kld_count, kld_max);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

int launch_calibrate_sl_max(int32_t B, const int32_t *a_max, const double *kld_sum, const int64_t *kld_count,
                            const float *kld_max, float eps, bool pooled, float *sl_max, hipStream_t stream) {
  (void)hipGetLastError();
  calibrate_kernel<<<dim3(1), dim3(kCapThreads), 0, stream>>>(B, a_max, kld_sum, kld_count, kld_max, eps, pooled,
                                                              sl_max);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

}  // namespace dsde
