// Adapt routines that change the element type (casts), with or without a
// layout change: the schema conversions of precision-hybrid tuning.  A
// value is widened exactly to float32 and rounded once to the destination
// type (nearest-even), so a chain of casts rounds like the one cast from the
// stored value.  Padded NC8HW8 channels are written as zero.
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
