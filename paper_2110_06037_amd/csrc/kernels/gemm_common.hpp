// Device helpers shared by the MFMA convolution kernels (gfx950 / CDNA4):
// MFMA traits, buffer resources with hardware range checks, LDS direct
// loads, pipeline barriers and the workgroup-to-tile order.
#pragma once

#include <stdexcept>
#include <string>

#include "kcommon.hpp"

namespace sn {
namespace k {

inline void check(bool ok, const char* what) {
  if (!ok) throw std::invalid_argument(std::string("kernel launch: ") + what);
}

// ------------------------------------------------------------------ MFMA
template <typename T>
struct Mfma;
template <>
struct Mfma<bf16> {
  static constexpr int KSTEP = 32;  // reduction elements per instruction
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<f16> {
  static constexpr int KSTEP = 32;
  typedef f16x8 frag;
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mfma<float> {
  static constexpr int KSTEP = 4;
  typedef float frag;
  static __device__ __forceinline__ f32x4 run(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// Raw buffer access: an SGPR resource (base, byte range) plus a 32-bit
// offset; loads at offsets beyond the range return zero, which implements
// the zero padding and the ragged tile edges without branches.
constexpr unsigned kOOB = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

// epilogue modes
constexpr int EPI_LAYOUT = 0;  // bias + activation, store in the tensor layout
constexpr int EPI_RAW = 1;     // raw float32 [M][Ng] (Winograd tile GEMMs)
constexpr int EPI_SPLIT = 2;   // raw float32 partial tile of one reduction split
constexpr int EPI_FIXUP = 3;   // reduction split whose last finishing workgroup sums the
                               // partial tiles and runs the layout epilogue

// Map the linear workgroup id to (m-tile, n-tile): consecutive ids are
// dispatched round-robin over the 8 XCDs, so first regroup them into one
// contiguous range per XCD, then walk groups of 8 m-tiles across all
// n-tiles (tiles of a group share A rows in that XCD's L2).
__device__ __forceinline__ void tile_of(int pid, int tiles_m, int tiles_n, int& mt, int& nt) {
  const int nb = tiles_m * tiles_n;
  const int q = nb >> 3, r = nb & 7;
  const int xcd = pid & 7, slot = pid >> 3;
  const int v = xcd * q + min(xcd, r) + slot;
  constexpr int GM = 8;
  const int group = v / (GM * tiles_n);
  const int first = group * GM;
  const int gsize = min(tiles_m - first, GM);
  const int in = v - group * GM * tiles_n;
  mt = first + in % gsize;
  nt = in / gsize;
}

// Workgroup barrier for the LDS pipeline: waits only for this wave's LDS
// operations (the tile stores), not for its in-flight global loads, which
// target registers and belong to the next step.  (__syncthreads() also
// drains all global loads, which would serialise the prefetch.)  The memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Division by a kernel-invariant positive divisor d as a multiply-high and a
// shift (numerators below 2^31): with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1, n / d = (mulhi(n, m) + n) >> l.
// Integer division on the GPU is a ~40-instruction sequence; kernels that
// split pixel indices into (image, row, column) take these from the host.
struct FastDiv {
  unsigned mul = 1, shift = 0;
};
inline FastDiv make_fastdiv(int d) {
  unsigned l = 0;
  while ((1ull << l) < (unsigned long long)d) ++l;
  FastDiv f;
  f.mul = (unsigned)((((1ull << 32) * ((1ull << l) - (unsigned long long)d)) / (unsigned long long)d) + 1);
  f.shift = l;
  return f;
}
__device__ __forceinline__ int fdiv(int n, FastDiv f) {
  const unsigned t = __umulhi((unsigned)n, f.mul);
  return (int)((t + (unsigned)n) >> f.shift);
}

// Small-integer division n / d for 0 <= n and n + d < 2^21 through fp32:
// floor((n + 0.5) * (1/d)).  The rounding error of the two fp32 operations
// stays below (n/d + 1) * 2^-22, less than the 0.5/d gap between (n + 0.5)/d
// and the nearest integer, so the floor is exact.  Full-rate VALU, unlike
// the quarter-rate 32-bit integer multiplies of an integer division.
__device__ __forceinline__ int sdiv(int n, float inv_d) { return (int)(((float)n + 0.5f) * inv_d); }

// Activation as a clamp to [lo, hi] (uniform bounds, no branches).
struct ActClamp {
  float lo, hi;
};
__device__ __forceinline__ ActClamp act_clamp(int act) {
  return ActClamp{act == ACT_NONE ? -__builtin_huge_valf() : 0.f, act == ACT_RELU6 ? 6.f : __builtin_huge_valf()};
}
__device__ __forceinline__ float act_apply(float v, ActClamp c) { return fminf(fmaxf(v, c.lo), c.hi); }

// LDS direct loads (buffer loads whose destination is LDS; 64 lanes x 16
// bytes land in lane order at the wave-uniform LDS address) and the waits
// of their pipelines.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Waits for this wave's LDS reads, then for all waves: after it, every
// wave's earlier tile reads are done and (with the vmcnt wait before it)
// every wave's tile loads have landed in LDS.
__device__ __forceinline__ void dma_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

typedef __attribute__((address_space(3))) void* lds_void_ptr;
typedef __attribute__((address_space(3))) char lds_char;

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, char* lds_block, unsigned voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_ptr)lds_block, 16, (int)voff, soff, 0, 0);
}
// The same with a 32-bit LDS address (uniform offsets stay scalar).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, lds_char* lds_block, unsigned voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_ptr)lds_block, 16, (int)voff, soff, 0, 0);
}

}  // namespace k
}  // namespace sn
