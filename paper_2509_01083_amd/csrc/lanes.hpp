// Cross-lane reductions and scans of one 64-lane wavefront on gfx950, built
// from DPP moves inside rows of 16 lanes and v_readlane across the four rows.
// A ds_bpermute-based shuffle takes a round trip through the LDS unit per
// step; these take a few VALU cycles per step, which matters where a
// reduction or scan sits on a latency-bound path (the per-sequence kernel).
// The bandwidth-bound row passes keep their ds_bpermute butterflies: there the
// LDS unit runs them beside the VALU work, and the DPP forms measured slower.
//
// Every reduction leaves the same bits in every lane (of the group), and each
// one evaluates in a fixed order, so results are reproducible run to run.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dsde {
namespace lanes {

// DPP controls of the gfx9 family
constexpr int kQuadSwap1 = 0xB1;       // quad_perm [1,0,3,2]: lane i reads lane i ^ 1
constexpr int kQuadSwap2 = 0x4E;       // quad_perm [2,3,0,1]: lane i reads lane i ^ 2
constexpr int kRowHalfMirror = 0x141;  // lane i reads lane 7 - i of its group of 8
constexpr int kRowMirror = 0x140;      // lane i reads lane 15 - i of its row
constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;  // i reads i - n (row)
constexpr int kRowRor4 = 0x124, kRowRor8 = 0x128;  // i reads (i - n) mod 16 (row rotation)

// A DPP move of 32 bits; lanes whose source lies outside the row read 0.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ int32_t dpp(int32_t v) {
  return int32_t(dpp<CTRL>(uint32_t(v)));
}
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __uint_as_float(dpp<CTRL>(__float_as_uint(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp(double v) {
  const uint64_t b = uint64_t(__double_as_longlong(v));
  const uint64_t lo = dpp<CTRL>(uint32_t(b)), hi = dpp<CTRL>(uint32_t(b >> 32));
  return __longlong_as_double(int64_t((hi << 32) | lo));
}

// The value of `lane` (wave-uniform) in every lane.
__device__ __forceinline__ uint32_t readlane(uint32_t v, int lane) {
  return uint32_t(__builtin_amdgcn_readlane(int(v), lane));
}
__device__ __forceinline__ int32_t readlane(int32_t v, int lane) { return __builtin_amdgcn_readlane(v, lane); }
__device__ __forceinline__ float readlane(float v, int lane) {
  return __uint_as_float(readlane(__float_as_uint(v), lane));
}
__device__ __forceinline__ double readlane(double v, int lane) {
  const uint64_t b = uint64_t(__double_as_longlong(v));
  const uint64_t lo = readlane(uint32_t(b), lane), hi = readlane(uint32_t(b >> 32), lane);
  return __longlong_as_double(int64_t((hi << 32) | lo));
}

struct Add {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a + b; }
};
struct Max {
  __device__ float operator()(float a, float b) const { return fmaxf(a, b); }
};
struct Min {
  template <typename T>
  __device__ T operator()(T a, T b) const { return b < a ? b : a; }
};
struct Or {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a | b; }
};

// The combination of the 16 lanes of each row, in every lane of the row.
// Each step combines a lane with a partner holding the same partial, so the
// (commutative) operation gives equal bits on both sides.
template <typename T, typename OP>
__device__ __forceinline__ T row_reduce(T v, OP op) {
  v = op(v, dpp<kQuadSwap1>(v));
  v = op(v, dpp<kQuadSwap2>(v));
  v = op(v, dpp<kRowHalfMirror>(v));
  v = op(v, dpp<kRowMirror>(v));
  return v;
}

// The combination over aligned groups of G lanes (G = 16, 32 or 64), in every
// lane of the group.
template <int G, typename T, typename OP>
__device__ __forceinline__ T group_reduce(T v, OP op) {
  static_assert(G == 16 || G == 32 || G == 64, "groups of 16, 32 or 64 lanes");
  v = row_reduce(v, op);
  if constexpr (G == 16) return v;
  const T r0 = readlane(v, 0), r1 = readlane(v, 16), r2 = readlane(v, 32), r3 = readlane(v, 48);
  const T lo = op(r0, r1), hi = op(r2, r3);
  if constexpr (G == 32) return (threadIdx.x & 63) < 32 ? lo : hi;
  return op(lo, hi);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) { return group_reduce<64>(v, Add{}); }

// Sixteen sums at once (a reduce-scatter): on return lane i of each row of 16
// holds the sum over the 16 lanes of its row of a[i % 16].  Each step halves
// the entries a lane keeps and adds the partner's copy of the kept half:
// partners differ in lane bit 0, 1, 2, 3 in turn (a rotation by 4 or 8 pairs
// lanes that agree in the bits already used and differ in the next one), so
// 15 DPP additions do the work of 16 row sums.
__device__ __forceinline__ float row_transpose_sum16(const float (&a)[16]) {
  const int l = threadIdx.x & 15;
  const bool b0 = l & 1, b1 = l & 2, b2 = l & 4, b3 = l & 8;
  float s8[8], s4[4], s2[2];
#pragma unroll
  for (int i = 0; i < 8; ++i) {  // entry 2i + b0
    const float keep = b0 ? a[2 * i + 1] : a[2 * i], send = b0 ? a[2 * i] : a[2 * i + 1];
    s8[i] = keep + dpp<kQuadSwap1>(send);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {  // entry 4i + 2 b1 + b0
    const float keep = b1 ? s8[2 * i + 1] : s8[2 * i], send = b1 ? s8[2 * i] : s8[2 * i + 1];
    s4[i] = keep + dpp<kQuadSwap2>(send);
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {  // entry 8i + 4 b2 + 2 b1 + b0
    const float keep = b2 ? s4[2 * i + 1] : s4[2 * i], send = b2 ? s4[2 * i] : s4[2 * i + 1];
    s2[i] = keep + dpp<kRowRor4>(send);
  }
  const float keep = b3 ? s2[1] : s2[0], send = b3 ? s2[0] : s2[1];
  return keep + dpp<kRowRor8>(send);
}
__device__ __forceinline__ float wave_max(float v) { return group_reduce<64>(v, Max{}); }
template <typename T>
__device__ __forceinline__ T wave_min(T v) { return group_reduce<64>(v, Min{}); }
template <typename T>
__device__ __forceinline__ T wave_or(T v) { return group_reduce<64>(v, Or{}); }

// Inclusive prefix sums over the 64 lanes in lane order (Hillis-Steele inside
// each row, then the row totals carried across), and the exclusive ones
// derived from them: excl of lane i is exactly incl of lane i - 1 (0 in lane
// 0), so consecutive intervals [excl, incl) tile without gaps or overlaps.
template <typename T>
struct Scan {
  T incl, excl;
};
template <typename T>
__device__ __forceinline__ Scan<T> wave_scan(T x) {
  const int lane = threadIdx.x & 63, row = lane >> 4;
  x += dpp<kRowShr1>(x);
  x += dpp<kRowShr2>(x);
  x += dpp<kRowShr4>(x);
  x += dpp<kRowShr8>(x);
  const T t0 = readlane(x, 15), t1 = readlane(x, 31), t2 = readlane(x, 47);
  const T b1 = t0, b2 = b1 + t1, b3 = b2 + t2;  // equal to incl of lanes 15, 31, 47 below
  const T base = row == 0 ? T(0) : row == 1 ? b1 : row == 2 ? b2 : b3;
  Scan<T> s;
  s.incl = row == 0 ? x : base + x;
  const T prev = dpp<kRowShr1>(s.incl);  // incl of lane i - 1 inside the row
  s.excl = (lane & 15) == 0 ? base : prev;
  return s;
}

}  // namespace lanes
}  // namespace dsde
