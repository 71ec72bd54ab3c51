// Device helpers shared by the HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mkv_internal.h"

namespace mkv {

#define MKV_DEV __device__ __forceinline__

constexpr float kLog2e = 1.4426950408889634f;

MKV_DEV float h2f(uint32_t bits16) {
  return (float)__builtin_bit_cast(_Float16, (unsigned short)(bits16 & 0xFFFFu));
}

MKV_DEV uint16_t f2h_bits(float x) {
  return __builtin_bit_cast(unsigned short, (_Float16)x);
}

// 8 fp16 values packed in a uint4 -> float[8]
MKV_DEV void unpack8(const uint4 &u, float *f) {
  f[0] = h2f(u.x); f[1] = h2f(u.x >> 16);
  f[2] = h2f(u.y); f[3] = h2f(u.y >> 16);
  f[4] = h2f(u.z); f[5] = h2f(u.z >> 16);
  f[6] = h2f(u.w); f[7] = h2f(u.w >> 16);
}

// Loads and stores through pointers known to be in global memory.  Region pointers come from
// the descriptor table, so without the address-space cast the compiler emits flat accesses,
// which share the LDS wait counter and serialise against LDS traffic.
#define MKV_GLOBAL __attribute__((address_space(1)))
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <typename T>
MKV_DEV T gld(const T *p) { return *(const MKV_GLOBAL T *)p; }
template <typename T>
MKV_DEV void gst(T *p, T v) { *(MKV_GLOBAL T *)p = v; }
MKV_DEV uint4 gld16(const void *p) {
  const u32x4 v = *(const MKV_GLOBAL u32x4 *)p;
  // element subscripts, not .x/.y: with hipcc 7.2, __builtin_bit_cast of an ext_vector_type
  // swizzle element (e.g. .y) has been seen to read element 0 instead
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// 16 bytes as four scalars (the backend merges the four loads into one 16-byte load); loader
// state holds plain scalars rather than vector types
struct U4 {
  uint32_t x, y, z, w;
};
MKV_DEV U4 gld16u(const void *p) {
  const uint32_t *q = reinterpret_cast<const uint32_t *>(p);
  return U4{gld(q), gld(q + 1), gld(q + 2), gld(q + 3)};
}
MKV_DEV void unpack8(const U4 &u, float *f) {
  f[0] = h2f(u.x); f[1] = h2f(u.x >> 16);
  f[2] = h2f(u.y); f[3] = h2f(u.y >> 16);
  f[4] = h2f(u.z); f[5] = h2f(u.z >> 16);
  f[6] = h2f(u.w); f[7] = h2f(u.w >> 16);
}

// 2^x on the hardware exponential unit (inputs here are <= 0; -inf gives 0)
MKV_DEV float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---- DPP row reductions ---------------------------------------------------------------------
template <int CTRL>
MKV_DEV float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL,
                                                               0xF, 0xF, false));
}

// Sum over aligned groups of L lanes (L in {8, 16}); every lane of a group gets the total.
template <int L>
MKV_DEV float group_sum(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  if constexpr (L == 16) x += dpp<0x140>(x);  // row_mirror
  return x;
}

// Reductions over the wave (all lanes active), without LDS traffic: four DPP steps give every lane
// its row's result, row_bcast:15 and row_bcast:31 carry rows 0 and 2 into rows 1 and 3 and rows
// 0-1 into rows 2-3, and lane 63's total is read back as a wave-uniform value.
template <typename Op>
MKV_DEV float wave_reduce(float x, float identity, Op op) {
  x = op(x, dpp<0xB1>(x));   // quad_perm [1,0,3,2]
  x = op(x, dpp<0x4E>(x));   // quad_perm [2,3,0,1]
  x = op(x, dpp<0x141>(x));  // row_half_mirror
  x = op(x, dpp<0x140>(x));  // row_mirror
  const int id = __builtin_bit_cast(int, identity);
  x = op(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(id, __builtin_bit_cast(int, x), 0x142, 0xA, 0xF, false)));
  x = op(x, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(id, __builtin_bit_cast(int, x), 0x143, 0xC, 0xF, false)));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), 63));
}
MKV_DEV float wave_max(float x) {
  return wave_reduce(x, -INFINITY, [](float a, float b) { return fmaxf(a, b); });
}
MKV_DEV float wave_min(float x) {
  return wave_reduce(x, INFINITY, [](float a, float b) { return fminf(a, b); });
}
// Sum over the wave: rows first, then rows 0 + 1 and 2 + 3, then the two halves (an association
// other than wave_sum's, so it is used only where that order is free).
MKV_DEV float wave_sum_rows(float x) {
  return wave_reduce(x, 0.f, [](float a, float b) { return a + b; });
}
// Minimum of a 64-bit key over the wave, in every lane.
MKV_DEV unsigned long long wave_min_u64(unsigned long long x) {
  auto step = [&](auto ctrl) {
    constexpr int C = decltype(ctrl)::value;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, C, 0xF, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), C, 0xF, 0xF, false);
    const unsigned long long y = ((unsigned long long)hi << 32) | lo;
    x = y < x ? y : x;
  };
  step(std::integral_constant<int, 0xB1>{});
  step(std::integral_constant<int, 0x4E>{});
  step(std::integral_constant<int, 0x141>{});
  step(std::integral_constant<int, 0x140>{});
  unsigned long long y = __shfl_xor(x, 16);
  x = y < x ? y : x;
  y = __shfl_xor(x, 32);
  return y < x ? y : x;
}
MKV_DEV float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}
MKV_DEV int wave_sum_i(int x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}

// Order-preserving unsigned key of a float (-0 treated as +0).
MKV_DEV uint32_t float_key(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if (u == 0x80000000u) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Inclusive prefix sum over the wave (all lanes active) by DPP: four row shifts give every row of
// 16 lanes its own prefix sums (lanes whose source lies before the row add 0), then row_bcast:15
// adds row 0's and row 2's totals to rows 1 and 3, and row_bcast:31 the total of rows 0-1 to
// rows 2 and 3.
MKV_DEV int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// Exclusive prefix sum over a block of NT threads (NT multiple of 64).  `tmp` is NT/64 ints of LDS.
template <int NT>
MKV_DEV int block_exclusive_scan(int x, int *tmp, int *total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int inc = wave_incl_scan(x);
  if (lane == 63) tmp[wid] = inc;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    int t = tmp[w];
    if (w < wid) base += t;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return base + inc - x;
}

}  // namespace mkv
