// Adapt routines (Sec. III-C: converting between schemas is an adapt job).
//
// Layout converters for 16-bit tensors, moving 16-byte vectors on both
// sides (every load and store a whole 8-element chunk; 32-bit index math):
//  * NHWC <-> NC8HW8 with C % 8 == 0: a chunk is 8 channels of one pixel in
//    both layouts, so the conversion permutes whole chunks; a workgroup
//    takes 64 pixels of one image and every channel block of them, so the
//    NC8HW8 side is written in 1 KB runs and the NHWC pixels it reads stay
//    in L2 until every block of them is taken.
//  * NCHW <-> NC8HW8 with H*W % 4 == 0: a thread takes 8 channels x G
//    pixels (G = 8 or 4), reads G pixels of each channel plane, transposes
//    8 x G in registers and writes G consecutive chunks.
//  * NCHW <-> NHWC with C % 8 == 0 and H*W % 8 == 0: 64 channels x 64
//    pixels of one image through an LDS tile: 16-byte rows in, 16-byte
//    pixel vectors out (gathered from 8 tile rows).
// Other shapes take the element-wise converters (misc.hip).  Padded NC8HW8
// channels are written as zero.
//
// Casts (precision-hybrid schemas): a value is widened exactly to float32
// and rounded once to the destination type (nearest-even), so a chain of
// casts rounds like the one cast from the stored value.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

// Same layout, other type: 8 consecutive stored elements per thread (the
// padded channels of NC8HW8 are zero on both sides, and zero casts to zero).
template <typename S, typename D>
__global__ __launch_bounds__(256) void cast_kernel(const S* __restrict__ x, D* __restrict__ y, long long n) {
  const long long i = ((long long)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i + 8 <= n) {
    const V8<S> a = ld8(x + i);
    V8<D> b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b.v[e] = from_f<D>(to_f(a.v[e]));
    st8(y + i, b);
  } else {
    for (long long j = i; j < n; ++j) y[j] = from_f<D>(to_f(x[j]));
  }
}

// Any layout to any other with a type change: one destination element per
// thread, the index split by multiply-high divisions (32-bit indices).
template <typename S, typename D, int LI, int LO>
__global__ __launch_bounds__(256) void cast_convert_kernel(const S* __restrict__ x, D* __restrict__ y, int C,
                                                           int H, int W, int csi, int cso, int total,
                                                           FastDiv fd_w, FastDiv fd_h, FastDiv fd_c, FastDiv fd_8,
                                                           FastDiv fd_cb) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  int n, c, h, w, r = idx;
  if constexpr (LO == NCHW) {
    int q = fdiv(r, fd_w); w = r - q * W; r = q;
    q = fdiv(r, fd_h); h = r - q * H; r = q;
    n = fdiv(r, fd_c); c = r - n * cso;
  } else if constexpr (LO == NHWC) {
    int q = fdiv(r, fd_c); c = r - q * cso; r = q;
    q = fdiv(r, fd_w); w = r - q * W; r = q;
    n = fdiv(r, fd_h); h = r - n * H;
  } else {
    const int e = r & 7; r >>= 3;
    int q = fdiv(r, fd_w); w = r - q * W; r = q;
    q = fdiv(r, fd_h); h = r - q * H; r = q;
    n = fdiv(r, fd_cb); c = (r - n * (cso >> 3)) * 8 + e;
  }
  D v = from_f<D>(0.f);
  if (c < C) v = from_f<D>(to_f(x[toff<LI>(csi, H, W, n, c, h, w)]));
  y[idx] = v;
}

template <typename S, typename D>
static void cast_t(const void* xv, const TDesc& xd, void* yv, const TDesc& yd, hipStream_t st) {
  const S* x = reinterpret_cast<const S*>(xv);
  D* y = reinterpret_cast<D*>(yv);
  if (xd.layout == yd.layout) {
    const long long n = (long long)xd.n * xd.cs * xd.h * xd.w;
    const long long threads = (n + 7) / 8;
    SN_LAUNCH((cast_kernel<S, D>), dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, x, y, n);
    return;
  }
  const long long total = (long long)yd.n * yd.cs * yd.h * yd.w;
  check(total < (1ll << 31) && (long long)xd.n * xd.cs * xd.h * xd.w < (1ll << 31), "tensor too large");
  const FastDiv fw = make_fastdiv(xd.w), fh = make_fastdiv(xd.h), fc = make_fastdiv(yd.cs), f8 = make_fastdiv(8),
                fcb = make_fastdiv(std::max(1, yd.cs / 8));
  dim3 g((unsigned)((total + 255) / 256));
#define CC(A, B)                                                                                             \
  case A * 3 + B:                                                                                            \
    SN_LAUNCH((cast_convert_kernel<S, D, A, B>), g, dim3(256), 0, st, x, y, xd.c, xd.h, xd.w, xd.cs, yd.cs, \
              (int)total, fw, fh, fc, f8, fcb);                                                              \
    break;
  switch (xd.layout * 3 + yd.layout) {
    CC(NCHW, NHWC)
    CC(NCHW, NC8)
    CC(NHWC, NCHW)
    CC(NHWC, NC8)
    CC(NC8, NCHW)
    CC(NC8, NHWC)
    default: check(false, "layout pair");
  }
#undef CC
}

template <typename S>
static void cast_from(int ddt, const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t st) {
  if (ddt == 0) cast_t<S, float>(x, xd, y, yd, st);
  else if (ddt == 1) cast_t<S, f16>(x, xd, y, yd, st);
  else cast_t<S, bf16>(x, xd, y, yd, st);
}

// ------------------------------------------------------------------ 16-bit layout converters
typedef unsigned short u16;

// NHWC <-> NC8HW8, C % 8 == 0: chunk (n, cb, hw) of NC8HW8 is NHWC chunk
// (n, hw, cb).  Workgroup (pixel tile, image); thread k handles pixel
// k % 64 of channel block k / 64.
template <bool TO_NC8>
__global__ __launch_bounds__(256) void nhwc_nc8_kernel(const uint4* __restrict__ x, uint4* __restrict__ y, int HW,
                                                       int CB) {
  const int n = blockIdx.y, hw0 = blockIdx.x * 64;
  const int npx = min(64, HW - hw0);
  for (int k = threadIdx.x; k < 64 * CB; k += 256) {
    const int px = k & 63, cb = k >> 6;
    if (px >= npx) continue;
    const int hw = hw0 + px;
    const unsigned nhwc = (unsigned)(n * HW + hw) * (unsigned)CB + (unsigned)cb;
    const unsigned nc8 = (unsigned)(n * CB + cb) * (unsigned)HW + (unsigned)hw;
    if (TO_NC8) y[nc8] = x[nhwc];
    else y[nhwc] = x[nc8];
  }
}

// NCHW <-> NC8HW8 for H*W % G == 0: thread = (image, channel block, group of
// G pixels); 8 channel rows of G pixels <-> G chunks of 8 channels.
template <int G, bool TO_NC8>
__global__ __launch_bounds__(256) void nchw_nc8_kernel(const u16* __restrict__ x, u16* __restrict__ y, int C, int CB,
                                                       int HW, int groups_img, int total) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int per_img = CB * groups_img;
  const int n = t / per_img, r = t - n * per_img;
  const int cb = r / groups_img, hw = (r - cb * groups_img) * G;
  u16 v[8][G];  // [channel][pixel]
  const u16* plane = x + ((size_t)n * C + cb * 8) * HW + hw;     // NCHW side (TO_NC8 reads it)
  u16* chunk = y + ((size_t)(n * CB + cb) * HW + hw) * 8;        // NC8HW8 side (TO_NC8 writes it)
  if (TO_NC8) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (cb * 8 + e < C) {
        if constexpr (G == 8) {
          const uint4 q = *reinterpret_cast<const uint4*>(plane + (size_t)e * HW);
          __builtin_memcpy(v[e], &q, 16);
        } else {
          const uint2 q = *reinterpret_cast<const uint2*>(plane + (size_t)e * HW);
          __builtin_memcpy(v[e], &q, 8);
        }
      } else {
#pragma unroll
        for (int p = 0; p < G; ++p) v[e][p] = 0;
      }
    }
#pragma unroll
    for (int p = 0; p < G; ++p) {
      u16 o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = v[e][p];
      uint4 q;
      __builtin_memcpy(&q, o, 16);
      reinterpret_cast<uint4*>(chunk)[p] = q;
    }
  } else {
    const u16* src = x + ((size_t)(n * CB + cb) * HW + hw) * 8;
    u16* dst = y + ((size_t)n * C + cb * 8) * HW + hw;
#pragma unroll
    for (int p = 0; p < G; ++p) {
      const uint4 q = reinterpret_cast<const uint4*>(src)[p];
      u16 o[8];
      __builtin_memcpy(o, &q, 16);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e][p] = o[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (cb * 8 + e >= C) continue;
      if constexpr (G == 8) {
        uint4 q;
        __builtin_memcpy(&q, v[e], 16);
        *reinterpret_cast<uint4*>(dst + (size_t)e * HW) = q;
      } else {
        uint2 q;
        __builtin_memcpy(&q, v[e], 8);
        *reinterpret_cast<uint2*>(dst + (size_t)e * HW) = q;
      }
    }
  }
}

// NCHW <-> NHWC for C % 8 == 0 and H*W % 8 == 0: a 64-channel x 64-pixel
// tile of one image in LDS ([channel][pixel], rows padded to 72 elements so
// that the 8 rows one pixel vector gathers fall in different banks).
template <bool TO_NHWC>
__global__ __launch_bounds__(256) void nchw_nhwc_tile_kernel(const u16* __restrict__ x, u16* __restrict__ y, int C,
                                                             int HW) {
  constexpr int RP = 72;
  __shared__ __attribute__((aligned(16))) u16 tile[64 * RP];
  const int n = blockIdx.z, hw0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const int nc = min(64, C - c0), npx = min(64, HW - hw0);
  const size_t img = (size_t)n * C * HW;
  if (TO_NHWC) {
    // 16-byte rows: chunk j = (channel j / 8, pixels (j % 8) * 8 ..)
    for (int j = threadIdx.x; j < 512; j += 256) {
      const int c = j >> 3, p8 = (j & 7) * 8;
      if (c < nc && p8 < npx) {
        const uint4 q = *reinterpret_cast<const uint4*>(x + img + (size_t)(c0 + c) * HW + hw0 + p8);
        *reinterpret_cast<uint4*>(tile + c * RP + p8) = q;
      }
    }
    __syncthreads();
    // pixel vectors: chunk j = (pixel j / 8, channels (j % 8) * 8 ..)
    for (int j = threadIdx.x; j < 512; j += 256) {
      const int px = j >> 3, c8 = (j & 7) * 8;
      if (px < npx && c8 < nc) {
        u16 o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = tile[(c8 + e) * RP + px];
        uint4 q;
        __builtin_memcpy(&q, o, 16);
        *reinterpret_cast<uint4*>(y + img + (size_t)(hw0 + px) * C + c0 + c8) = q;
      }
    }
  } else {
    for (int j = threadIdx.x; j < 512; j += 256) {
      const int px = j >> 3, c8 = (j & 7) * 8;
      if (px < npx && c8 < nc) {
        const uint4 q = *reinterpret_cast<const uint4*>(x + img + (size_t)(hw0 + px) * C + c0 + c8);
        u16 o[8];
        __builtin_memcpy(o, &q, 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[(c8 + e) * RP + px] = o[e];
      }
    }
    __syncthreads();
    for (int j = threadIdx.x; j < 512; j += 256) {
      const int c = j >> 3, p8 = (j & 7) * 8;
      if (c < nc && p8 < npx)
        *reinterpret_cast<uint4*>(y + img + (size_t)(c0 + c) * HW + hw0 + p8) =
            *reinterpret_cast<const uint4*>(tile + c * RP + p8);
    }
  }
}

// The vector converters above for a 16-bit tensor, when the shape allows
// one; returns whether it launched.
bool convert_vec16(const void* xv, const TDesc& xd, void* yv, const TDesc& yd, hipStream_t st) {
  const int C = xd.c, HW = xd.h * xd.w, N = xd.n;
  if ((long long)N * ((C + 7) / 8 * 8) * HW >= (1ll << 31) || N > 65535) return false;
  const int a = xd.layout, b = yd.layout;
  const u16* x = reinterpret_cast<const u16*>(xv);
  u16* y = reinterpret_cast<u16*>(yv);
  if ((a == NHWC && b == NC8) || (a == NC8 && b == NHWC)) {
    if (C % 8 != 0) return false;
    const dim3 g((HW + 63) / 64, N);
    if (b == NC8)
      SN_LAUNCH((nhwc_nc8_kernel<true>), g, dim3(256), 0, st, (const uint4*)x, (uint4*)y, HW, C / 8);
    else
      SN_LAUNCH((nhwc_nc8_kernel<false>), g, dim3(256), 0, st, (const uint4*)x, (uint4*)y, HW, C / 8);
    return true;
  }
  if ((a == NCHW && b == NC8) || (a == NC8 && b == NCHW)) {
    const int CB = (C + 7) / 8;
    const int G = HW % 8 == 0 ? 8 : HW % 4 == 0 ? 4 : 0;
    if (!G) return false;
    const int groups = HW / G, total = N * CB * groups;
    const dim3 g((total + 255) / 256);
#define NC8K(GG, T)                                                                                       \
  SN_LAUNCH((nchw_nc8_kernel<GG, T>), g, dim3(256), 0, st, x, y, C, CB, HW, groups, total)
    if (G == 8) {
      if (b == NC8) NC8K(8, true);
      else NC8K(8, false);
    } else {
      if (b == NC8) NC8K(4, true);
      else NC8K(4, false);
    }
#undef NC8K
    return true;
  }
  if ((a == NCHW && b == NHWC) || (a == NHWC && b == NCHW)) {
    if (C % 8 != 0 || HW % 8 != 0 || C <= 8) return false;
    const dim3 g((HW + 63) / 64, (C + 63) / 64, N);
    if (b == NHWC) SN_LAUNCH((nchw_nhwc_tile_kernel<true>), g, dim3(256), 0, st, x, y, C, HW);
    else SN_LAUNCH((nchw_nhwc_tile_kernel<false>), g, dim3(256), 0, st, x, y, C, HW);
    return true;
  }
  return false;
}

void convert_cast(int sdt, const void* x, const TDesc& xd, int ddt, void* y, const TDesc& yd, hipStream_t st) {
  check(xd.n == yd.n && xd.c == yd.c && xd.h == yd.h && xd.w == yd.w, "converter keeps the shape");
  check(sdt >= 0 && sdt <= 2 && ddt >= 0 && ddt <= 2, "dtype");
  if (sdt == ddt) {
    convert(sdt, x, xd, y, yd, st);
    return;
  }
  if (sdt == 0) cast_from<float>(ddt, x, xd, y, yd, st);
  else if (sdt == 1) cast_from<f16>(ddt, x, xd, y, yd, st);
  else cast_from<bf16>(ddt, x, xd, y, yd, st);
}

}  // namespace k
}  // namespace sn
