// Standalone kernels of the KLD stability signal (Sec. 3.1.2, Eqs. 3-7) and
// of the next speculation length under the batch cap (Eqs. 2, 8; Sec. 3.3,
// Eqs. 9-11).  The per-sequence and per-batch code is shared with the fused
// step (signal_device.hpp).
//
//   kld_signal_kernel  one wavefront per sequence (lanes over the window
//                      entries); every workgroup re-checks the batch layout.
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
                                                              int32_t sl_hi, float *__restrict__ sl_hat,
                                                              float *__restrict__ sl_cap,
                                                              int32_t *__restrict__ sl_next,
                                                              uint32_t *__restrict__ seq_err, bool or_err) {
  __shared__ double red_s[kCapThreads / 64];
  __shared__ int red_n[kCapThreads / 64];
  block_next_sl(B, sf, wvir, sl_max, sl_min, sl_hi, sl_hat, sl_cap, sl_next, seq_err, or_err, red_s, red_n);
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
                   float *sl_hat, float *sl_cap, int32_t *sl_next, uint32_t *seq_err, bool or_err,
                   hipStream_t stream) {
  (void)hipGetLastError();
  next_sl_kernel<<<dim3(1), dim3(kCapThreads), 0, stream>>>(B, sf, wvir, sl_max, sl_min, sl_hi, sl_hat, sl_cap,
                                                            sl_next, seq_err, or_err);
  return hipGetLastError() == hipSuccess ? DSDE_OK : DSDE_DEVICE_ERROR;
}

}  // namespace dsde
