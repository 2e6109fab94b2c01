// Device-side helpers shared by the routine kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace sn {
namespace k {

typedef __bf16 bf16;
typedef _Float16 f16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// layouts (same values as sn_layout)
constexpr int NCHW = 0, NHWC = 1, NC8 = 2;
// activations (same values as sn_act)
constexpr int ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2;

__device__ __forceinline__ float act_f(float v, int act) {
  if (act == ACT_RELU) return fmaxf(v, 0.f);
  if (act == ACT_RELU6) return fminf(fmaxf(v, 0.f), 6.f);
  return v;
}

template <typename T>
__device__ __forceinline__ float to_f(T v) {
  return (float)v;
}
template <typename T>
__device__ __forceinline__ T from_f(float v) {
  return (T)v;  // float -> f16 / bf16 rounds to nearest even
}

// Element offset of logical (n, c, h, w) in a tensor of layout L with
// stored channel count cs (cs = C for NCHW/NHWC, round8(C) for NC8).
template <int L>
__device__ __forceinline__ int64_t toff(int cs, int H, int W, int n, int c, int h, int w) {
  if constexpr (L == NCHW) return (((int64_t)n * cs + c) * H + h) * W + w;
  if constexpr (L == NHWC) return (((int64_t)n * H + h) * W + w) * cs + c;
  return ((((int64_t)n * (cs >> 3) + (c >> 3)) * H + h) * W + w) * 8 + (c & 7);
}

// 8 consecutive elements as a register bundle (16 B for 16-bit types, 32 B for float).
template <typename T>
struct V8 {
  T v[8];
};

template <typename T>
__device__ __forceinline__ V8<T> ld8(const T* p) {
  V8<T> r;
  if constexpr (sizeof(T) == 2) {
    uint4 u = *reinterpret_cast<const uint4*>(p);
    __builtin_memcpy(&r, &u, 16);
  } else {
    float4 a = reinterpret_cast<const float4*>(p)[0];
    float4 b = reinterpret_cast<const float4*>(p)[1];
    __builtin_memcpy(&r, &a, 16);
    __builtin_memcpy(reinterpret_cast<char*>(&r) + 16, &b, 16);
  }
  return r;
}

template <typename T>
__device__ __forceinline__ void st8(T* p, const V8<T>& r) {
  if constexpr (sizeof(T) == 2) {
    uint4 u;
    __builtin_memcpy(&u, &r, 16);
    *reinterpret_cast<uint4*>(p) = u;
  } else {
    float4 a, b;
    __builtin_memcpy(&a, &r, 16);
    __builtin_memcpy(&b, reinterpret_cast<const char*>(&r) + 16, 16);
    reinterpret_cast<float4*>(p)[0] = a;
    reinterpret_cast<float4*>(p)[1] = b;
  }
}

template <typename T>
__device__ __forceinline__ V8<T> zero8() {
  V8<T> r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r.v[i] = (T)0.f;
  return r;
}

// Sum over the 64 lanes of a wave, in every lane.  Within each row of 16
// lanes the partial sums move by DPP (data-parallel primitives: the operand
// of a VALU op read from another lane of the row): XOR 1 and XOR 2 as quad
// permutations, then the half-row mirror (lane i takes lane 7 - i of its
// 8-lane half, which holds the other quad's sum) and the row mirror (lane i
// takes lane 15 - i, the other half's sum).  The two rows of each 32-lane
// half combine through a swizzle with XOR 16, and the halves through two
// scalar lane reads.
template <int CTRL>
__device__ __forceinline__ float dpp_take(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_take<0xB1>(v);   // quad_perm [1, 0, 3, 2]: XOR 1
  v += dpp_take<0x4E>(v);   // quad_perm [2, 3, 0, 1]: XOR 2
  v += dpp_take<0x141>(v);  // row_half_mirror
  v += dpp_take<0x140>(v);  // row_mirror
  v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));  // XOR 16
  const int b = __builtin_bit_cast(int, v);
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0)) +
         __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32));
}

}  // namespace k
}  // namespace sn
