// Device helpers shared by the row kernels: bf16/fp32 logit loads in the
// chunk layouts, padding, and wavefront/workgroup reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace dsde {

// bf16 -2^96: padding for logits past V.  It is below every admissible logit
// (|z| <= 2^64), its exponential is exactly 0, and differences of two padding
// values stay finite, so padding adds exactly nothing to any sum.
constexpr uint32_t kPadBf16x2 = 0xef80ef80u;
constexpr float kPadF32 = -7.9228162514264337593543950336e28f;  // -2^96

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Streaming 16-byte loads (the nontemporal hint): logit rows are read once per
// pass, and with the hint a plain read of a buffer far larger than the caches
// runs about 10% faster on this part than with ordinary loads.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 stream_load(const uint4 *p) {
  const u32x4_t w = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(w.x, w.y, w.z, w.w);
}
__device__ __forceinline__ float4 stream_load(const float4 *p) {
  const f32x4_t w = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(p));
  return make_float4(w.x, w.y, w.z, w.w);
}

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
// chunk of a row held by one workgroup
// ---------------------------------------------------------------------------
//
// The 8192 logits of chunk k of a row are spread over the 256 threads so that
// each wavefront load is contiguous.  Thread t owns slots i = 0..31:
//   bf16, 16-byte rows : logit 8 * (1024 k + 256 (i / 8) + t) + i % 8  (4 x uint4)
//   fp32, 16-byte rows : logit 4 * (2048 k + 256 (i / 4) + t) + i % 4  (8 x float4)
//   any other row      : logit 8192 k + 256 i + t                       (32 scalars)
// Every load uses an in-bounds (clamped) index and the value is replaced by
// padding past V, so the loads never branch.

template <int DT, bool VEC>
struct Layout;
template <>
struct Layout<DSDE_BF16, true> {
  __device__ static int64_t index(int64_t chunk, int i, int t) {
    return 8 * (chunk * 1024 + (i / 8) * 256 + t) + (i % 8);
  }
  __device__ static void owner(int64_t local, int *t, int *i) {
    *t = int((local >> 3) & 255);
    *i = int((local >> 11) * 8 + (local & 7));
  }
};
template <>
struct Layout<DSDE_FP32, true> {
  __device__ static int64_t index(int64_t chunk, int i, int t) {
    return 4 * (chunk * 2048 + (i / 4) * 256 + t) + (i % 4);
  }
  __device__ static void owner(int64_t local, int *t, int *i) {
    *t = int((local >> 2) & 255);
    *i = int((local >> 10) * 4 + (local & 3));
  }
};
template <int DT>
struct Layout<DT, false> {
  __device__ static int64_t index(int64_t chunk, int i, int t) { return chunk * kChunk + int64_t(i) * 256 + t; }
  __device__ static void owner(int64_t local, int *t, int *i) {
    *t = int(local & 255);
    *i = int(local >> 8);
  }
};

// Raw bf16 chunk of one row: 4 x uint4 per thread.
struct RawBf16 {
  uint4 v0, v1, v2, v3;
};

// The same loads without the padding (indices clamped into the row), and the
// padding applied afterwards: callers that issue many loads up front pad only
// where the values are used, so that no load waits for another.
__device__ __forceinline__ RawBf16 issue_raw_bf16(const void *row, int64_t V, int64_t chunk, int t) {
  const uint4 *p = (const uint4 *)row;
  const int64_t last = V / 8 - 1;
  const int64_t i0 = chunk * 1024 + t;
  RawBf16 r;
  r.v0 = stream_load(p + min(i0, last));
  r.v1 = stream_load(p + min(i0 + 256, last));
  r.v2 = stream_load(p + min(i0 + 512, last));
  r.v3 = stream_load(p + min(i0 + 768, last));
  return r;
}
__device__ __forceinline__ RawBf16 pad_raw_bf16(const RawBf16 &a, int64_t V, int64_t chunk, int t) {
  const int64_t last = V / 8 - 1;
  const int64_t i0 = chunk * 1024 + t;
  const uint4 pad = make_uint4(kPadBf16x2, kPadBf16x2, kPadBf16x2, kPadBf16x2);
  RawBf16 r;
  r.v0 = i0 <= last ? a.v0 : pad;
  r.v1 = i0 + 256 <= last ? a.v1 : pad;
  r.v2 = i0 + 512 <= last ? a.v2 : pad;
  r.v3 = i0 + 768 <= last ? a.v3 : pad;
  return r;
}

__device__ __forceinline__ RawBf16 load_raw_bf16(const void *row, int64_t V, int64_t chunk, int t) {
  const uint4 *p = (const uint4 *)row;
  const int64_t last = V / 8 - 1;
  const int64_t i0 = chunk * 1024 + t;
  const uint4 pad = make_uint4(kPadBf16x2, kPadBf16x2, kPadBf16x2, kPadBf16x2);
  const uint4 a0 = stream_load(p + min(i0, last)), a1 = stream_load(p + min(i0 + 256, last));
  const uint4 a2 = stream_load(p + min(i0 + 512, last)), a3 = stream_load(p + min(i0 + 768, last));
  RawBf16 r;
  r.v0 = i0 <= last ? a0 : pad;
  r.v1 = i0 + 256 <= last ? a1 : pad;
  r.v2 = i0 + 512 <= last ? a2 : pad;
  r.v3 = i0 + 768 <= last ? a3 : pad;
  return r;
}

// Larger of two floats, NaN if either is NaN (the IEEE 754-2019 maximum:
// v_maximum3_f32 on gfx950).  fmaxf would first quiet every loaded value
// (one v_max_f32 x, x, x per logit in IEEE mode).  A NaN logit makes its
// thread's maximum NaN (the cross-lane fmaxf steps of block_max may drop
// it), and its exponential makes every sum of the chunk NaN, so the row is
// flagged as with fmaxf.
__device__ __forceinline__ float max_nan(float a, float b) { return __builtin_elementwise_maximum(a, b); }
__device__ __forceinline__ float max2(uint32_t w) { return max_nan(bf_lo(w), bf_hi(w)); }
__device__ __forceinline__ float vmax(uint4 v) {
  return max_nan(max_nan(max2(v.x), max2(v.y)), max_nan(max2(v.z), max2(v.w)));
}
__device__ __forceinline__ float raw_max(const RawBf16 &r) {
  return max_nan(max_nan(vmax(r.v0), vmax(r.v1)), max_nan(vmax(r.v2), vmax(r.v3)));
}
__device__ __forceinline__ float pick_bf16(const RawBf16 &r, int i) {
  const uint4 v = (i >> 3) == 0 ? r.v0 : (i >> 3) == 1 ? r.v1 : (i >> 3) == 2 ? r.v2 : r.v3;
  const int w = (i >> 1) & 3;
  const uint32_t x = w == 0 ? v.x : w == 1 ? v.y : w == 2 ? v.z : v.w;
  return (i & 1) ? bf_hi(x) : bf_lo(x);
}

// Per-thread accumulators of the statistics pass, two interleaved sets
// (index 0 and 1).  The exponential sums are fp64: near-identical target and
// draft rows make KL = A / S_p - log S_p + log S_q cancel to values of order
// 1e-4 and below, and a thread's fp32 running sum near 1 (its largest
// exponential is 1 at the chunk maximum) would round each later term to
// about 6e-8 of it, leaving ~1e-7 of uncorrelated relative error in S_p and
// S_q.  The two exponentials of one bf16 word are added in fp32 (one
// rounding) and the pair is added in fp64: half the conversions of per-term
// fp64 sums, and as accurate for the KLD (groups of four were not, on
// sharply peaked rows).  The KL and entropy accumulators enter the results
// through ratios to the sums and stay fp32.
struct PairAcc {
  double sp[2], sq[2];  // sum 2^at, sum 2^ad
  float a[2], h[2];     // sum 2^at (at - ad), sum 2^ad ad
};
__device__ __forceinline__ void zero(PairAcc &s) {
  s.sp[0] = s.sp[1] = s.sq[0] = s.sq[1] = 0.0;
  s.a[0] = s.a[1] = s.h[0] = s.h[1] = 0.0f;
}

// Statistics of two logit pairs (target zt0, zt1; draft zd0, zd1) with
// references rt, rd (log2 domain) into accumulator set k: the two
// exponential sums, the KL accumulator sum 2^at (at - ad), and, with ENT, the
// draft entropy accumulator sum 2^ad ad (left at zero without it).
template <bool ENT>
__device__ __forceinline__ void acc_two(float zt0, float zt1, float zd0, float zd1, float c, float rt, float rd,
                                        PairAcc &s, int k) {
  const float at0 = fmaf(zt0, c, -rt), ad0 = fmaf(zd0, c, -rd);
  const float at1 = fmaf(zt1, c, -rt), ad1 = fmaf(zd1, c, -rd);
  const float et0 = fast_exp2(at0), ed0 = fast_exp2(ad0);
  const float et1 = fast_exp2(at1), ed1 = fast_exp2(ad1);
  s.sp[k] += double(et0 + et1);
  s.sq[k] += double(ed0 + ed1);
  s.a[k] = fmaf(et1, at1 - ad1, fmaf(et0, at0 - ad0, s.a[k]));
  if constexpr (ENT) s.h[k] = fmaf(ed1, ad1, fmaf(ed0, ad0, s.h[k]));
}
// The 8 bf16 pairs of one 16-byte load of each row, one word at a time,
// words alternating between the two sets.
template <bool ENT>
__device__ __forceinline__ void acc_vec(uint4 t, uint4 d, float c, float rt, float rd, PairAcc &s) {
  acc_two<ENT>(bf_lo(t.x), bf_hi(t.x), bf_lo(d.x), bf_hi(d.x), c, rt, rd, s, 0);
  acc_two<ENT>(bf_lo(t.y), bf_hi(t.y), bf_lo(d.y), bf_hi(d.y), c, rt, rd, s, 1);
  acc_two<ENT>(bf_lo(t.z), bf_hi(t.z), bf_lo(d.z), bf_hi(d.z), c, rt, rd, s, 0);
  acc_two<ENT>(bf_lo(t.w), bf_hi(t.w), bf_lo(d.w), bf_hi(d.w), c, rt, rd, s, 1);
}

// Generic chunk of one row as 32 floats (fp32 rows, or rows without 16-byte alignment).
template <int DT, bool VEC>
__device__ __forceinline__ void load_chunk_f32(const void *row, int64_t V, int64_t chunk, int t,
                                               float (&z)[kEltsPerThread]) {
  if constexpr (VEC && DT == DSDE_FP32) {
    const float4 *p = (const float4 *)row;
    const int64_t last = V / 4 - 1;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      const int64_t i = chunk * 2048 + g * 256 + t;
      const float4 w = stream_load(p + min(i, last));
      const bool ok = i <= last;
      z[g * 4 + 0] = ok ? w.x : kPadF32;
      z[g * 4 + 1] = ok ? w.y : kPadF32;
      z[g * 4 + 2] = ok ? w.z : kPadF32;
      z[g * 4 + 3] = ok ? w.w : kPadF32;
    }
  } else if constexpr (VEC && DT == DSDE_BF16) {
    const RawBf16 r = load_raw_bf16(row, V, chunk, t);
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) z[i] = pick_bf16(r, i);
  } else {
#pragma unroll
    for (int i = 0; i < kEltsPerThread; ++i) {
      const int64_t v = chunk * kChunk + int64_t(i) * 256 + t;
      const float x = load_logit(row, DT, v < V ? v : V - 1);
      z[i] = v < V ? x : kPadF32;
    }
  }
}

// R consecutive logits of a row, from `start` (a multiple of R, R a multiple
// of 8), padded past V.
template <int DT, bool VEC, int R>
__device__ __forceinline__ void load_run(const void *row, int64_t V, int64_t start, float (&z)[R]) {
  if constexpr (VEC && DT == DSDE_BF16) {
    const uint4 *p = (const uint4 *)row;
    const int64_t last = V / 8 - 1;
#pragma unroll
    for (int q = 0; q < R / 8; ++q) {
      const int64_t i = start / 8 + q;
      const uint4 a = p[min(i, last)];
      const uint4 v = i <= last ? a : make_uint4(kPadBf16x2, kPadBf16x2, kPadBf16x2, kPadBf16x2);
      z[8 * q + 0] = bf_lo(v.x);
      z[8 * q + 1] = bf_hi(v.x);
      z[8 * q + 2] = bf_lo(v.y);
      z[8 * q + 3] = bf_hi(v.y);
      z[8 * q + 4] = bf_lo(v.z);
      z[8 * q + 5] = bf_hi(v.z);
      z[8 * q + 6] = bf_lo(v.w);
      z[8 * q + 7] = bf_hi(v.w);
    }
  } else if constexpr (VEC && DT == DSDE_FP32) {
    const float4 *p = (const float4 *)row;
    const int64_t last = V / 4 - 1;
#pragma unroll
    for (int q = 0; q < R / 4; ++q) {
      const int64_t i = start / 4 + q;
      const float4 a = p[min(i, last)];
      const bool ok = i <= last;
      z[4 * q + 0] = ok ? a.x : kPadF32;
      z[4 * q + 1] = ok ? a.y : kPadF32;
      z[4 * q + 2] = ok ? a.z : kPadF32;
      z[4 * q + 3] = ok ? a.w : kPadF32;
    }
  } else {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int64_t v = start + i;
      const float x = load_logit(row, DT, v < V ? v : V - 1);
      z[i] = v < V ? x : kPadF32;
    }
  }
}

// Keeps a prefetched value where it was loaded: an empty asm statement that
// takes it as an operand (it emits no instruction).  Without it the compiler
// may sink a load to its first use, past the branches and barriers the
// prefetch is meant to overlap with.
__device__ __forceinline__ void pin(float v) { asm volatile("" ::"v"(v)); }
__device__ __forceinline__ void pin(double v) { asm volatile("" ::"v"(v)); }
__device__ __forceinline__ void pin(int32_t v) { asm volatile("" ::"v"(v)); }

}  // namespace dsde
