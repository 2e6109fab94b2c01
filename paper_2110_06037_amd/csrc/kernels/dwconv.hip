// Depthwise 3x3 convolution (stride 1 or 2) of 16-bit NHWC (C % 8 == 0) or
// NC8HW8 tensors: the inverted-residual middle layer, bound by memory.
//
// A thread computes a strip of QS consecutive output pixels of one row for
// one block of 8 channels: it reads the three input rows under the strip
// once, as 16-byte channel vectors ((QS - 1) * stride + 3 of them per row;
// for QS = 4 at stride 1, 6 instead of 12), keeps the filter vectors in
// registers and accumulates in float32.  Longer strips read less but leave
// fewer threads: at stride 1 QS is the longest of 4, 2, 1 that still gives
// 64 K threads, enough to keep every CU's loads in flight; at stride 2 a
// strip saves little (27 loads for 4 outputs against 36) and QS is 1.
// Consecutive lanes take consecutive channel blocks (NHWC: one pixel's
// channels are contiguous) or consecutive strips (NC8HW8: a channel block's
// row is contiguous), so every load and store instruction of a wave covers
// contiguous memory.  Index arithmetic is 32-bit with multiply-high
// divisions.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

struct Dw3Args {
  const void* x;
  const void* w;      // [3][3][C8]
  const float* bias;  // [C8]
  void* y;
  int H, W, P, Q, CB, Cs, stride, pad, act;
  int strips, total;  // strips per output row, threads
  FastDiv fd_cb, fd_strips, fd_p;
};

template <typename T, int L, int ST, int QS>
__global__ __launch_bounds__(256) void dw3x3_kernel(Dw3Args a) {
  constexpr int IW = (QS - 1) * ST + 3;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= a.total) return;
  // NHWC: t = ((n * P + p) * strips + s) * CB + cb; NC8: t = ((n * CB + cb) * P + p) * strips + s
  int n, p, s, cb, r = t;
  if constexpr (L == NHWC) {
    int q = fdiv(r, a.fd_cb); cb = r - q * a.CB; r = q;
    q = fdiv(r, a.fd_strips); s = r - q * a.strips; r = q;
    n = fdiv(r, a.fd_p); p = r - n * a.P;
  } else {
    int q = fdiv(r, a.fd_strips); s = r - q * a.strips; r = q;
    q = fdiv(r, a.fd_p); p = r - q * a.P; r = q;
    n = fdiv(r, a.fd_cb); cb = r - n * a.CB;
  }
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x);
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w);
  const int q0 = s * QS;
  // element offset of input pixel (h, ww) of this image and channel block
  auto xoff = [&](int h, int ww) -> unsigned {
    if constexpr (L == NHWC) return ((unsigned)(n * a.H + h) * (unsigned)a.W + (unsigned)ww) * (unsigned)a.Cs + cb * 8;
    return (((unsigned)(n * a.CB + cb) * (unsigned)a.H + (unsigned)h) * (unsigned)a.W + (unsigned)ww) * 8u;
  };
  float acc[QS][8];
  {
    const float* b = a.bias + cb * 8;
#pragma unroll
    for (int j = 0; j < QS; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j][e] = b[e];
  }
  const int w0 = q0 * ST - a.pad;
#pragma unroll
  for (int rr = 0; rr < 3; ++rr) {
    const int h = p * ST - a.pad + rr;
    if ((unsigned)h >= (unsigned)a.H) continue;
    V8<T> row[IW];
#pragma unroll
    for (int i = 0; i < IW; ++i) {
      const int ww = w0 + i;
      row[i] = (unsigned)ww < (unsigned)a.W ? ld8(x + xoff(h, ww)) : zero8<T>();
    }
#pragma unroll
    for (int ss = 0; ss < 3; ++ss) {
      const V8<T> f = ld8(w + (rr * 3 + ss) * (a.CB * 8) + cb * 8);
#pragma unroll
      for (int j = 0; j < QS; ++j)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[j][e] = fmaf(to_f(f.v[e]), to_f(row[j * ST + ss].v[e]), acc[j][e]);
    }
  }
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
#pragma unroll
  for (int j = 0; j < QS; ++j) {
    const int q = q0 + j;
    if (q >= a.Q) break;
    V8<T> o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.v[e] = from_f<T>(act_f(acc[j][e], a.act));
    unsigned off;
    if constexpr (L == NHWC) off = ((unsigned)(n * a.P + p) * (unsigned)a.Q + (unsigned)q) * (unsigned)a.Cs + cb * 8;
    else off = (((unsigned)(n * a.CB + cb) * (unsigned)a.P + (unsigned)p) * (unsigned)a.Q + (unsigned)q) * 8u;
    st8(y + off, o);
  }
}

template <typename T>
static void dw3_t(const ConvArgs& c, hipStream_t st) {
  Dw3Args a{};
  a.x = c.x;
  a.w = c.w;
  a.bias = c.bias;
  a.y = c.y;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.P = c.yd.h;
  a.Q = c.yd.w;
  a.CB = (c.xd.c + 7) / 8;
  a.Cs = c.xd.cs;
  a.stride = c.stride;
  a.pad = c.pad;
  a.act = c.act;
  const long long rows = (long long)c.xd.n * a.P * a.CB;
  const int qs = c.stride != 1 ? 1 : rows * ((a.Q + 3) / 4) >= 65536 ? 4 : rows * ((a.Q + 1) / 2) >= 65536 ? 2 : 1;
  a.strips = (a.Q + qs - 1) / qs;
  const long long total = rows * a.strips;
  check(total < (1ll << 31), "depthwise grid");
  a.total = (int)total;
  a.fd_cb = make_fastdiv(a.CB);
  a.fd_strips = make_fastdiv(a.strips);
  a.fd_p = make_fastdiv(a.P);
  const dim3 g((unsigned)((total + 255) / 256));
#define DW3(LL, SS, QQ) \
  if (c.xd.layout == LL && c.stride == SS && qs == QQ) {                                                   \
    SN_LAUNCH((dw3x3_kernel<T, LL, SS, QQ>), g, dim3(256), 0, st, a);                                       \
    return;                                                                                                \
  }
  DW3(NHWC, 1, 4) DW3(NHWC, 1, 2) DW3(NHWC, 1, 1) DW3(NHWC, 2, 1)
  DW3(NC8, 1, 4) DW3(NC8, 1, 2) DW3(NC8, 1, 1) DW3(NC8, 2, 1)
#undef DW3
}

// Takes the layer when it fits the strip kernel; false otherwise (the
// general depthwise kernel of conv.hip runs it).
bool dwconv3x3_vec(int dtype, const ConvArgs& c, hipStream_t st) {
  if (dtype == 0 || c.r != 3 || c.s != 3 || (c.stride != 1 && c.stride != 2)) return false;
  if (!(c.xd.layout == NC8 || (c.xd.layout == NHWC && c.xd.c % 8 == 0)) || c.yd.layout != c.xd.layout) return false;
  const long long xe = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w, ye = (long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w;
  if (xe >= (1ll << 31) || ye >= (1ll << 31)) return false;
  if (dtype == 1) dw3_t<f16>(c, st);
  else dw3_t<bf16>(c, st);
  return true;
}

}  // namespace k
}  // namespace sn
