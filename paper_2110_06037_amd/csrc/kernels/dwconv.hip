// Depthwise 3x3 convolution (stride 1 or 2) of 16-bit NHWC (C % 8 == 0) or
// NC8HW8 tensors: the inverted-residual middle layer, bound by memory.
//
// A thread computes a vertical strip of QS output pixels (rows p0 .. p0 +
// QS - 1 of one column q) for one block of 8 channels.  It walks the
// (QS - 1) * stride + 3 input rows under the strip once, reading the three
// 16-byte channel vectors of each row at columns q * stride - 1 .. + 1, and
// adds each row into every output of the strip that covers it; the nine
// filter vectors stay in registers and the sums are float32.  At stride 1
// QS = 4 reads 18 vectors for 4 outputs instead of 36.  Consecutive lanes
// take consecutive channel blocks of one pixel and then consecutive columns
// (NHWC) or consecutive columns of one channel block (NC8HW8), so every load
// and store instruction of a wave covers one contiguous run of memory (at
// stride 2 the loads cover every other vector of a run, and the three
// horizontal taps together fill it).  QS is the longest of 4, 2, 1 (stride
// 1) or 2, 1 (stride 2) that still leaves 64 K threads, enough to keep every
// CU's loads in flight.  Index arithmetic is 32-bit with multiply-high
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
  int strips, total;  // vertical strips per output column, threads
  long long x_bytes;  // input tensor bytes (< 2 GiB)
  FastDiv fd_cb, fd_strips, fd_q;
};

template <typename T, int L, int ST, int QS>
__global__ __launch_bounds__(256) void dw3x3_kernel(Dw3Args a) {
  constexpr int IH = (QS - 1) * ST + 3;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= a.total) return;
  // NHWC: t = ((n * strips + ps) * Q + q) * CB + cb; NC8: t = ((n * CB + cb) * strips + ps) * Q + q
  int n, ps, q, cb, r = t;
  if constexpr (L == NHWC) {
    int d = fdiv(r, a.fd_cb); cb = r - d * a.CB; r = d;
    d = fdiv(r, a.fd_q); q = r - d * a.Q; r = d;
    n = fdiv(r, a.fd_strips); ps = r - n * a.strips;
  } else {
    int d = fdiv(r, a.fd_q); q = r - d * a.Q; r = d;
    d = fdiv(r, a.fd_strips); ps = r - d * a.strips; r = d;
    n = fdiv(r, a.fd_cb); cb = r - n * a.CB;
  }
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_bytes);
  const int p0 = ps * QS;
  // byte offset of input pixel (h, ww) of this image and channel block;
  // padding pixels take an offset past the buffer, which loads as zero, so
  // every load is issued without a branch and all of them are in flight
  // together
  auto xoff = [&](int h, int ww) -> unsigned {
    if ((unsigned)h >= (unsigned)a.H || (unsigned)ww >= (unsigned)a.W) return kOOB;
    if constexpr (L == NHWC)
      return (((unsigned)(n * a.H + h) * (unsigned)a.W + (unsigned)ww) * (unsigned)a.Cs + cb * 8) * sizeof(T);
    return ((((unsigned)(n * a.CB + cb) * (unsigned)a.H + (unsigned)h) * (unsigned)a.W + (unsigned)ww) * 8u) *
           sizeof(T);
  };
  V8<T> f[9];
#pragma unroll
  for (int k2 = 0; k2 < 9; ++k2) f[k2] = ld8(w + k2 * (a.CB * 8) + cb * 8);
  float acc[QS][8];
  {
    const float* b = a.bias + cb * 8;
#pragma unroll
    for (int j = 0; j < QS; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j][e] = b[e];
  }
  const int w0 = q * ST - a.pad, h0 = p0 * ST - a.pad;
  u32x4 raw[IH][3];
#pragma unroll
  for (int i = 0; i < IH; ++i)
#pragma unroll
    for (int dx = 0; dx < 3; ++dx)
      raw[i][dx] = __builtin_amdgcn_raw_buffer_load_b128(rx, (int)xoff(h0 + i, w0 + dx), 0, 0);
#pragma unroll
  for (int i = 0; i < IH; ++i) {
    V8<T> row[3];
#pragma unroll
    for (int dx = 0; dx < 3; ++dx) row[dx] = __builtin_bit_cast(V8<T>, raw[i][dx]);
    // output j of the strip takes this row as its filter row i - j * ST
#pragma unroll
    for (int j = 0; j < QS; ++j) {
      const int rr = i - j * ST;
      if (rr < 0 || rr > 2) continue;
#pragma unroll
      for (int dx = 0; dx < 3; ++dx)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          acc[j][e] = fmaf(to_f(f[rr * 3 + dx].v[e]), to_f(row[dx].v[e]), acc[j][e]);
    }
  }
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
#pragma unroll
  for (int j = 0; j < QS; ++j) {
    const int p = p0 + j;
    if (p >= a.P) break;
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
static void dw3_t(const ConvArgs& c, int qs_req, hipStream_t st) {
  Dw3Args a{};
  a.x = c.x;
  a.x_bytes = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w * (long long)sizeof(T);
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
  const long long cols = (long long)c.xd.n * a.Q * a.CB;
  auto enough = [&](int qs) { return cols * ((a.P + qs - 1) / qs) >= 65536; };
  const int qs = qs_req > 0 ? qs_req : c.stride == 1 ? (enough(4) ? 4 : enough(2) ? 2 : 1) : (enough(2) ? 2 : 1);
  check(qs == 1 || qs == 2 || (qs == 4 && c.stride == 1), "depthwise strip length");
  a.strips = (a.P + qs - 1) / qs;
  const long long total = cols * a.strips;
  check(total < (1ll << 31), "depthwise grid");
  a.total = (int)total;
  a.fd_cb = make_fastdiv(a.CB);
  a.fd_strips = make_fastdiv(a.strips);
  a.fd_q = make_fastdiv(a.Q);
  const dim3 g((unsigned)((total + 255) / 256));
#define DW3(LL, SS, QQ) \
  if (c.xd.layout == LL && c.stride == SS && qs == QQ) {                                                   \
    SN_LAUNCH((dw3x3_kernel<T, LL, SS, QQ>), g, dim3(256), 0, st, a);                                       \
    return;                                                                                                \
  }
  DW3(NHWC, 1, 4) DW3(NHWC, 1, 2) DW3(NHWC, 1, 1) DW3(NHWC, 2, 2) DW3(NHWC, 2, 1)
  DW3(NC8, 1, 4) DW3(NC8, 1, 2) DW3(NC8, 1, 1) DW3(NC8, 2, 2) DW3(NC8, 2, 1)
#undef DW3
}

static bool strip_kernel_fits(int dtype, int layout, int c, int r, int s, int stride) {
  return dtype != 0 && r == 3 && s == 3 && (stride == 1 || stride == 2) &&
         (layout == NC8 || (layout == NHWC && c % 8 == 0));
}

// Strip lengths of routine parameters 1, 2, 3 (3 only at stride 1).
int dw_strip_len(int param) { return param == 1 ? 1 : param == 2 ? 2 : 4; }

int dw_num_strip_params(int dtype, int layout, int c, int r, int s, int stride) {
  if (!strip_kernel_fits(dtype, layout, c, r, s, stride)) return 0;
  return stride == 1 ? 3 : 2;
}

// Takes the layer when it fits the strip kernel (qs = strip length, 0 =
// by the thread count); false otherwise (the general depthwise kernel of
// conv.hip runs it).
bool dwconv3x3_vec(int dtype, const ConvArgs& c, int qs, hipStream_t st) {
  if (!strip_kernel_fits(dtype, c.xd.layout, c.xd.c, c.r, c.s, c.stride) || c.yd.layout != c.xd.layout)
    return false;
  const long long xe = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w, ye = (long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w;
  if (xe >= (1ll << 31) || ye >= (1ll << 31)) return false;
  if (dtype == 1) dw3_t<f16>(c, qs, st);
  else dw3_t<bf16>(c, qs, st);
  return true;
}

}  // namespace k
}  // namespace sn
