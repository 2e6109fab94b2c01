// Adapt routines (Sec. III-C: converting between schemas is an adapt job).
//
// Layout converters for 16-bit tensors, moving 16-byte vectors on both
// sides (every load and store a whole 8-element chunk; 32-bit index math):
//  * NHWC <-> NC8HW8 with C % 8 == 0: a chunk is 8 channels of one pixel in
//    both layouts, so the conversion permutes whole chunks, a wave taking 8
//    pixels x 8 channel blocks (128-byte runs on both sides).
//  * NCHW <-> NC8HW8: a thread takes 8 channels x G pixels (G = 8, 4 or 1,
//    the largest dividing H*W), reads G pixels of each channel plane,
//    transposes 8 x G in registers and writes G consecutive chunks.
//  * NCHW <-> NHWC with C % 8 == 0: 64 channels x 64 pixels of one image
//    through an LDS tile: 16-byte rows (elements when H*W % 8 != 0) on the
//    NCHW side, 16-byte pixel vectors (gathered from 8 tile rows) on the
//    NHWC side.
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
// (n, hw, cb).  A wave takes 8 channel blocks x 8 pixels of one image (lane
// = block * 8 + pixel), so each load and store instruction covers 8 runs of
// 128 contiguous bytes on either side; the grid has one wave per such tile,
// whatever the split between pixels and channel blocks.
template <bool TO_NC8>
__global__ __launch_bounds__(256) void nhwc_nc8_kernel(const uint4* __restrict__ x, uint4* __restrict__ y, int HW,
                                                       int CB, int HWT, int CBT, int tiles, FastDiv fd_hwt,
                                                       FastDiv fd_cbt) {
  const int tile = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tile >= tiles) return;
  const int lane = threadIdx.x & 63;
  // tile = (n * CBT + cbt) * HWT + hwt
  int r = fdiv(tile, fd_hwt);
  const int hwt = tile - r * HWT;
  const int n = fdiv(r, fd_cbt), cbt = r - n * CBT;
  const int hw = hwt * 8 + (lane & 7), cb = cbt * 8 + (lane >> 3);
  if (hw >= HW || cb >= CB) return;
  const unsigned nhwc = (unsigned)(n * HW + hw) * (unsigned)CB + (unsigned)cb;
  const unsigned nc8 = (unsigned)(n * CB + cb) * (unsigned)HW + (unsigned)hw;
  if (TO_NC8) y[nc8] = x[nhwc];
  else y[nhwc] = x[nc8];
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
    // every load is issued unconditionally (channels past C read the
    // block's first row and are zeroed afterwards), so all eight are in
    // flight together
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int er = cb * 8 + e < C ? e : 0;
      if constexpr (G == 8) {
        const uint4 q = *reinterpret_cast<const uint4*>(plane + (size_t)er * HW);
        __builtin_memcpy(v[e], &q, 16);
      } else if constexpr (G == 4) {
        const uint2 q = *reinterpret_cast<const uint2*>(plane + (size_t)er * HW);
        __builtin_memcpy(v[e], &q, 8);
      } else {
        v[e][0] = plane[(size_t)er * HW];
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int p = 0; p < G; ++p) v[e][p] = cb * 8 + e < C ? v[e][p] : (u16)0;
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
    // a channel row past C is not stored: its store goes to a channel row
    // that is stored anyway (row 0 of the block, with the same values), so
    // that no store sits behind a branch (a branch join would wait for the
    // stores before it to complete)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int er = cb * 8 + e < C ? e : 0;
      if constexpr (G == 8) {
        uint4 q;
        __builtin_memcpy(&q, v[er == e ? e : 0], 16);
        *reinterpret_cast<uint4*>(dst + (size_t)er * HW) = q;
      } else if constexpr (G == 4) {
        uint2 q;
        __builtin_memcpy(&q, v[er == e ? e : 0], 8);
        *reinterpret_cast<uint2*>(dst + (size_t)er * HW) = q;
      } else {
        dst[(size_t)er * HW] = v[er == e ? e : 0][0];
      }
    }
  }
}

// NCHW <-> NHWC for C % 8 == 0: a 64-channel x 64-pixel tile of one image
// in LDS ([channel][pixel], rows padded to 72 elements so that the 8 rows
// one pixel vector gathers fall in different banks); 16-byte pixel vectors
// on the NHWC side, and on the NCHW side 16-byte row pieces when H*W % 8 ==
// 0 (VEC), else single elements with consecutive lanes on consecutive
// pixels (the 14x14 and 7x7 planes of the late stages).
template <bool TO_NHWC, bool VEC>
__global__ __launch_bounds__(256) void nchw_nhwc_tile_kernel(const u16* __restrict__ x, u16* __restrict__ y, int C,
                                                             int HW) {
  constexpr int RP = 72;
  __shared__ __attribute__((aligned(16))) u16 tile[64 * RP];
  const int n = blockIdx.z, hw0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const int nc = min(64, C - c0), npx = min(64, HW - hw0);
  const size_t img = (size_t)n * C * HW;
  if (TO_NHWC) {
    // loads are issued unconditionally (outside the tile they read the
    // image's first element) so that all of a thread's are in flight
    // together; only the LDS writes are predicated
    if constexpr (VEC) {
      // 16-byte rows: chunk j = (channel j / 8, pixels (j % 8) * 8 ..)
      uint4 q[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int j = threadIdx.x + k * 256, c = j >> 3, p8 = (j & 7) * 8;
        const size_t o = c < nc && p8 < npx ? (size_t)(c0 + c) * HW + hw0 + p8 : 0;
        q[k] = *reinterpret_cast<const uint4*>(x + img + o);
      }
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int j = threadIdx.x + k * 256, c = j >> 3, p8 = (j & 7) * 8;
        if (c < nc && p8 < npx) *reinterpret_cast<uint4*>(tile + c * RP + p8) = q[k];
      }
    } else {
      u16 q[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int j = threadIdx.x + k * 256, c = j >> 6, px = j & 63;
        const size_t o = c < nc && px < npx ? (size_t)(c0 + c) * HW + hw0 + px : 0;
        q[k] = x[img + o];
      }
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int j = threadIdx.x + k * 256, c = j >> 6, px = j & 63;
        if (c < nc && px < npx) tile[c * RP + px] = q[k];
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
    uint4 q[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int j = threadIdx.x + k * 256, px = j >> 3, c8 = (j & 7) * 8;
      const size_t o = px < npx && c8 < nc ? (size_t)(hw0 + px) * C + c0 + c8 : 0;
      q[k] = *reinterpret_cast<const uint4*>(x + img + o);
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int j = threadIdx.x + k * 256, px = j >> 3, c8 = (j & 7) * 8;
      if (px < npx && c8 < nc) {
        u16 o[8];
        __builtin_memcpy(o, &q[k], 16);
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[(c8 + e) * RP + px] = o[e];
      }
    }
    __syncthreads();
    if constexpr (VEC) {
      for (int j = threadIdx.x; j < 512; j += 256) {
        const int c = j >> 3, p8 = (j & 7) * 8;
        if (c < nc && p8 < npx)
          *reinterpret_cast<uint4*>(y + img + (size_t)(c0 + c) * HW + hw0 + p8) =
              *reinterpret_cast<const uint4*>(tile + c * RP + p8);
      }
    } else {
      for (int j = threadIdx.x; j < 4096; j += 256) {
        const int c = j >> 6, px = j & 63;
        if (c < nc && px < npx) y[img + (size_t)(c0 + c) * HW + hw0 + px] = tile[c * RP + px];
      }
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
    const int CB = C / 8, HWT = (HW + 7) / 8, CBT = (CB + 7) / 8;
    const long long tiles = (long long)N * CBT * HWT;
    if (tiles >= (1ll << 31) - 4) return false;
    const dim3 g((unsigned)((tiles + 3) / 4));
    const FastDiv fh = make_fastdiv(HWT), fc = make_fastdiv(CBT);
    if (b == NC8)
      SN_LAUNCH((nhwc_nc8_kernel<true>), g, dim3(256), 0, st, (const uint4*)x, (uint4*)y, HW, CB, HWT, CBT,
                (int)tiles, fh, fc);
    else
      SN_LAUNCH((nhwc_nc8_kernel<false>), g, dim3(256), 0, st, (const uint4*)x, (uint4*)y, HW, CB, HWT, CBT,
                (int)tiles, fh, fc);
    return true;
  }
  if ((a == NCHW && b == NC8) || (a == NC8 && b == NCHW)) {
    const int CB = (C + 7) / 8;
    const int G = HW % 8 == 0 ? 8 : HW % 4 == 0 ? 4 : 1;
    const int groups = HW / G, total = N * CB * groups;
    const dim3 g((total + 255) / 256);
#define NC8K(GG, T)                                                                                       \
  SN_LAUNCH((nchw_nc8_kernel<GG, T>), g, dim3(256), 0, st, x, y, C, CB, HW, groups, total)
    if (G == 8) {
      if (b == NC8) NC8K(8, true);
      else NC8K(8, false);
    } else if (G == 4) {
      if (b == NC8) NC8K(4, true);
      else NC8K(4, false);
    } else {
      if (b == NC8) NC8K(1, true);
      else NC8K(1, false);
    }
#undef NC8K
    return true;
  }
  if ((a == NCHW && b == NHWC) || (a == NHWC && b == NCHW)) {
    if (C % 8 != 0 || C <= 8) return false;
    const dim3 g((HW + 63) / 64, (C + 63) / 64, N);
    const bool vec = HW % 8 == 0;
    if (b == NHWC) {
      if (vec) SN_LAUNCH((nchw_nhwc_tile_kernel<true, true>), g, dim3(256), 0, st, x, y, C, HW);
      else SN_LAUNCH((nchw_nhwc_tile_kernel<true, false>), g, dim3(256), 0, st, x, y, C, HW);
    } else {
      if (vec) SN_LAUNCH((nchw_nhwc_tile_kernel<false, true>), g, dim3(256), 0, st, x, y, C, HW);
      else SN_LAUNCH((nchw_nhwc_tile_kernel<false, false>), g, dim3(256), 0, st, x, y, C, HW);
    }
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
