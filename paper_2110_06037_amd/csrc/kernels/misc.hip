// Bandwidth-bound routines for gfx950: max pooling, global average pooling,
// residual add (+ activation), FC as a dot-product kernel (large batches and
// float32; small 16-bit batches go to the MFMA kernel), layout converters
// (the adapt routines of the paper, Sec. III-C, job 3: changing data layout)
// and the profiler's scratch fill.
#include <stdexcept>
#include <string>

#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

thread_local LaunchTiming g_timing;
thread_local long long g_launches = 0;
thread_local int g_count_only = 0;


static unsigned blocks(long long n, int per = 256) { return (unsigned)((n + per - 1) / per); }

// ------------------------------------------------------------------ max pooling
template <typename T, int L>
__global__ __launch_bounds__(256) void maxpool_kernel(const T* __restrict__ x, T* __restrict__ y,
                                                      int N, int C, int H, int W, int Cs, int P,
                                                      int Q, int k, int st, int pad) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const int PQ = P * Q;
  if constexpr (L == NCHW) {
    if (idx >= (long long)N * C * PQ) return;
    const int pq = (int)(idx % PQ);
    const long long nc = idx / PQ;
    const int p = pq / Q, q = pq - p * Q;
    const T* xp = x + nc * H * W;
    float m = -INFINITY;
    for (int r = 0; r < k; ++r) {
      const int h = p * st - pad + r;
      if ((unsigned)h >= (unsigned)H) continue;
      for (int s = 0; s < k; ++s) {
        const int w = q * st - pad + s;
        if ((unsigned)w >= (unsigned)W) continue;
        m = fmaxf(m, to_f(xp[h * W + w]));
      }
    }
    y[idx] = from_f<T>(m);
  } else {
    // 32-bit index arithmetic (the host checks N * P * Q * CB < 2^31): the
    // 64-bit divisions it replaces cost more than the nine 16-byte loads
    // Consecutive workgroups are dispatched round-robin over the 8 XCDs;
    // renumber them so each XCD takes one contiguous range of output rows,
    // and the input row shared by vertically adjacent windows is read into
    // that XCD's L2 once.
    const unsigned nb = gridDim.x, b = blockIdx.x;
    const unsigned xq = nb >> 3, xr = nb & 7, xcd = b & 7;
    const unsigned vb = xcd * xq + min(xcd, xr) + (b >> 3);
    const int CB = (Cs + 7) / 8;
    const bool vec = L == NC8 || C % 8 == 0;
    const unsigned total = (unsigned)N * (unsigned)PQ * (unsigned)CB;
    const unsigned id = vb * 256u + threadIdx.x;
    if (id >= total) return;
    int cb;
    unsigned mm;
    if constexpr (L == NC8) {
      const unsigned npq = (unsigned)N * (unsigned)PQ;
      cb = (int)(id / npq);
      mm = id - (unsigned)cb * npq;
    } else {
      mm = id / (unsigned)CB;
      cb = (int)(id - mm * (unsigned)CB);
    }
    const int n = (int)(mm / (unsigned)PQ), pq = (int)(mm - (unsigned)n * (unsigned)PQ);
    const int p = (int)((unsigned)pq / (unsigned)Q), q = pq - p * Q;
    float m[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) m[e] = -INFINITY;
    const bool fast = sizeof(T) == 2 && vec && k == 3;
    if constexpr (sizeof(T) == 2) if (fast) {
      // the 3x3 window (every pooling layer of the nets here): all nine
      // 16-byte loads are issued at once through a buffer resource (taps
      // outside the image read zero past its end and are masked out of the
      // maximum), instead of one load round trip per tap
      const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (long long)N * H * W * ((Cs + 7) / 8 * 8) * sizeof(T));
      u32x4 raw[9];
      bool ok[9];
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int h = p * st - pad + t / 3, w = q * st - pad + t % 3;
        ok[t] = (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
        unsigned off;
        if constexpr (L == NC8) off = (((unsigned)(n * CB + cb) * (unsigned)H + (unsigned)h) * (unsigned)W + (unsigned)w) * 8u;
        else off = ((unsigned)(n * H + h) * (unsigned)W + (unsigned)w) * (unsigned)Cs + (unsigned)cb * 8u;
        raw[t] = __builtin_amdgcn_raw_buffer_load_b128(rx, ok[t] ? (int)(off * sizeof(T)) : (int)kOOB, 0, 0);
      }
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const V8<T> v = __builtin_bit_cast(V8<T>, raw[t]);
#pragma unroll
        for (int e = 0; e < 8; ++e) m[e] = ok[t] ? fmaxf(m[e], to_f(v.v[e])) : m[e];
      }
    }
    for (int r = 0; r < (fast ? 0 : k); ++r) {
      const int h = p * st - pad + r;
      if ((unsigned)h >= (unsigned)H) continue;
      for (int s = 0; s < k; ++s) {
        const int w = q * st - pad + s;
        if ((unsigned)w >= (unsigned)W) continue;
        if (vec) {
          V8<T> v;
          if constexpr (L == NC8)
            v = ld8(x + ((((long long)n * CB + cb) * H + h) * W + w) * 8);
          else
            v = ld8(x + (((long long)n * H + h) * W + w) * Cs + cb * 8);
#pragma unroll
          for (int e = 0; e < 8; ++e) m[e] = fmaxf(m[e], to_f(v.v[e]));
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (cb * 8 + e < C) m[e] = fmaxf(m[e], to_f(x[(((long long)n * H + h) * W + w) * Cs + cb * 8 + e]));
        }
      }
    }
    V8<T> o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.v[e] = from_f<T>(m[e]);
    if constexpr (L == NC8) {
      st8(y + ((((long long)n * CB + cb) * P + p) * Q + q) * 8, o);
    } else if (vec) {
      st8(y + (((long long)n * P + p) * Q + q) * Cs + cb * 8, o);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (cb * 8 + e < C) y[(((long long)n * P + p) * Q + q) * Cs + cb * 8 + e] = o.v[e];
    }
  }
}

template <typename T>
static void maxpool_t(const void* x, const TDesc& xd, void* y, const TDesc& yd, int k, int st,
                      int pad, hipStream_t s) {
  check(xd.layout == yd.layout && xd.cs == yd.cs, "pooling keeps the layout");
  long long total = xd.layout == NCHW ? (long long)xd.n * xd.c * yd.h * yd.w
                                      : (long long)xd.n * yd.h * yd.w * ((xd.cs + 7) / 8);
  check(total < (1ll << 31), "pooling output too large for 32-bit indices");
  const T* xp = reinterpret_cast<const T*>(x);
  T* yp = reinterpret_cast<T*>(y);
#define MP(LL)                                                                                   \
  SN_LAUNCH((maxpool_kernel<T, LL>), dim3(blocks(total)), dim3(256), 0, s, xp, yp, xd.n, \
                     xd.c, xd.h, xd.w, xd.cs, yd.h, yd.w, k, st, pad)
  switch (xd.layout) {
    case NCHW: MP(NCHW); break;
    case NHWC: MP(NHWC); break;
    case NC8: MP(NC8); break;
  }
#undef MP
}

void maxpool(int dtype, const void* x, const TDesc& xd, void* y, const TDesc& yd, int k, int st,
             int pad, hipStream_t s) {
  if (dtype == 0) maxpool_t<float>(x, xd, y, yd, k, st, pad, s);
  else if (dtype == 1) maxpool_t<f16>(x, xd, y, yd, k, st, pad, s);
  else maxpool_t<bf16>(x, xd, y, yd, k, st, pad, s);
}

// ------------------------------------------------------------------ global average pooling
// NCHW: one wave reduces one (n, c) plane; the lanes' partial sums meet in a
// DPP reduction (wave_sum).
// NHWC / NC8: a workgroup takes 64 stored channels of one image; its 4 waves
// sum interleaved quarters of the pixels with lanes along channels
// (coalesced), and the 4 partial sums meet in LDS.
template <typename T, int L>
__global__ __launch_bounds__(256) void gap_kernel(const T* __restrict__ x, T* __restrict__ y, int N,
                                                  int C, int HW, int Cs) {
  const float inv = 1.f / (float)HW;
  if constexpr (L == NCHW) {
    const long long plane = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (plane >= (long long)N * C) return;  // wave-uniform
    const T* xp = x + plane * HW;
    float s = 0.f;
    for (int i = lane; i < HW; i += 64) s += to_f(xp[i]);
    s = wave_sum(s);
    if (lane == 0) y[plane] = from_f<T>(s * inv);
  } else {
    __shared__ float part[4][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int n = blockIdx.y, c = blockIdx.x * 64 + lane;
    float s = 0.f;
    if (c < Cs) {
      if constexpr (L == NC8) {
        const T* xp = x + ((size_t)n * (Cs >> 3) + (c >> 3)) * HW * 8 + (c & 7);
#pragma unroll 4
        for (int i = wv; i < HW; i += 4) s += to_f(xp[(size_t)i * 8]);
      } else {
        const T* xp = x + (size_t)n * HW * Cs + c;
#pragma unroll 4
        for (int i = wv; i < HW; i += 4) s += to_f(xp[(size_t)i * Cs]);
      }
    }
    part[wv][lane] = s;
    __syncthreads();
    if (wv == 0 && c < Cs)
      y[(size_t)n * Cs + c] = from_f<T>(((part[0][lane] + part[1][lane]) + (part[2][lane] + part[3][lane])) * inv);
  }
}

template <typename T>
static void gap_t(const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t s) {
  check(xd.layout == yd.layout && yd.h == 1 && yd.w == 1, "gap output is N x C x 1 x 1");
  check(xd.n <= 65535 && (long long)xd.n * xd.cs * xd.h * xd.w < (1ll << 40), "gap grid");
  const int HW = xd.h * xd.w;
  const T* xp = reinterpret_cast<const T*>(x);
  T* yp = reinterpret_cast<T*>(y);
  switch (xd.layout) {
    case NCHW:
      SN_LAUNCH((gap_kernel<T, NCHW>), dim3(blocks((long long)xd.n * xd.c, 4)), dim3(256), 0, s,
                         xp, yp, xd.n, xd.c, HW, xd.cs);
      break;
    case NHWC:
      SN_LAUNCH((gap_kernel<T, NHWC>), dim3((xd.cs + 63) / 64, xd.n), dim3(256), 0, s,
                         xp, yp, xd.n, xd.c, HW, xd.cs);
      break;
    case NC8:
      SN_LAUNCH((gap_kernel<T, NC8>), dim3((xd.cs + 63) / 64, xd.n), dim3(256), 0, s,
                         xp, yp, xd.n, xd.c, HW, xd.cs);
      break;
  }
}

void gap(int dtype, const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t s) {
  if (dtype == 0) gap_t<float>(x, xd, y, yd, s);
  else if (dtype == 1) gap_t<f16>(x, xd, y, yd, s);
  else gap_t<bf16>(x, xd, y, yd, s);
}

// ------------------------------------------------------------------ residual add
// Both inputs share the layout, so the sum is elementwise over the stored
// elements (padded channels are 0 + 0).
template <typename T>
__global__ __launch_bounds__(256) void add_kernel(const T* __restrict__ a, const T* __restrict__ b,
                                                  T* __restrict__ y, long long n, int act) {
  const long long i8 = ((long long)blockIdx.x * 256 + threadIdx.x) * 8;
  if (i8 + 8 <= n) {
    V8<T> va = ld8(a + i8), vb = ld8(b + i8), o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.v[e] = from_f<T>(act_f(to_f(va.v[e]) + to_f(vb.v[e]), act));
    st8(y + i8, o);
  } else {
    for (long long i = i8; i < n; ++i) y[i] = from_f<T>(act_f(to_f(a[i]) + to_f(b[i]), act));
  }
}

void add_act(int dtype, const void* a, const void* b, void* y, int64_t n, int act, hipStream_t s) {
  dim3 g(blocks((n + 7) / 8));
  if (dtype == 0)
    SN_LAUNCH(add_kernel<float>, g, dim3(256), 0, s, (const float*)a, (const float*)b, (float*)y, (long long)n, act);
  else if (dtype == 1)
    SN_LAUNCH(add_kernel<f16>, g, dim3(256), 0, s, (const f16*)a, (const f16*)b, (f16*)y, (long long)n, act);
  else
    SN_LAUNCH(add_kernel<bf16>, g, dim3(256), 0, s, (const bf16*)a, (const bf16*)b, (bf16*)y, (long long)n, act);
}

// ------------------------------------------------------------------ FC (dot products)
// One wave per output feature k: lanes stride the input features with 8-wide
// loads, the batch is processed in groups of 4 sharing each weight load, and
// each dot product finishes with a DPP reduction (wave_sum).
template <typename T>
__global__ __launch_bounds__(256) void fc_kernel(const T* __restrict__ x, int N, int cin, int cin_s,
                                                 const T* __restrict__ w, int c8,
                                                 const float* __restrict__ bias, T* __restrict__ y,
                                                 int kout_s, int act) {
  const int k = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (k >= kout_s) return;
  const T* wr = w + (long long)k * c8;
  const bool vec = (cin % 8 == 0) && (cin_s % 8 == 0);
  for (int n0 = 0; n0 < N; n0 += 4) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (vec) {
      for (int c = lane * 8; c < cin; c += 512) {
        V8<T> wv = ld8(wr + c);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (n0 + j >= N) break;
          V8<T> xv = ld8(x + (long long)(n0 + j) * cin_s + c);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[j] = fmaf(to_f(wv.v[e]), to_f(xv.v[e]), acc[j]);
        }
      }
    } else {
      for (int c = lane; c < cin; c += 64) {
        const float wv = to_f(wr[c]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (n0 + j < N) acc[j] = fmaf(wv, to_f(x[(long long)(n0 + j) * cin_s + c]), acc[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float s = wave_sum(acc[j]);
      if (lane == 0 && n0 + j < N) y[(long long)(n0 + j) * kout_s + k] = from_f<T>(act_f(s + bias[k], act));
    }
  }
}

// the MFMA kernel for small 16-bit batches (fc.hip)
bool fc_mfma_applicable(int dtype, int n, int cin, int cin_s);
void fc_mfma(int dtype, const void* x, int n, int cin, int cin_s, const void* w, int c8,
             const float* bias, void* y, int kout, int kout_s, int act, hipStream_t st);

void fc_direct(int dtype, const void* x, int n, int cin, int cin_s, const void* w, int c8,
               const float* bias, void* y, int kout, int kout_s, int act, hipStream_t s) {
  check(kout_s >= kout && c8 >= cin, "fc shapes");
  if (fc_mfma_applicable(dtype, n, cin, cin_s)) {
    fc_mfma(dtype, x, n, cin, cin_s, w, c8, bias, y, kout, kout_s, act, s);
    return;
  }
  dim3 g(blocks(kout_s, 4));
  if (dtype == 0)
    SN_LAUNCH(fc_kernel<float>, g, dim3(256), 0, s, (const float*)x, n, cin, cin_s, (const float*)w, c8, bias, (float*)y, kout_s, act);
  else if (dtype == 1)
    SN_LAUNCH(fc_kernel<f16>, g, dim3(256), 0, s, (const f16*)x, n, cin, cin_s, (const f16*)w, c8, bias, (f16*)y, kout_s, act);
  else
    SN_LAUNCH(fc_kernel<bf16>, g, dim3(256), 0, s, (const bf16*)x, n, cin, cin_s, (const bf16*)w, c8, bias, (bf16*)y, kout_s, act);
}

// ------------------------------------------------------------------ layout converters
// Bit-exact permutations; padded channels of NC8HW8 are written as zero.
// E is the element's storage type (the converter moves bits).

// NCHW <-> NHWC: per image a [C][HW] <-> [HW][C] transpose through a
// 64 x 64 LDS tile (padded row to avoid bank conflicts), both sides coalesced.
template <typename E, bool TO_NHWC>
__global__ __launch_bounds__(256) void transpose_kernel(const E* __restrict__ x, E* __restrict__ y,
                                                        int C, int HW) {
  __shared__ E tile[64][65];
  const int n = blockIdx.z;
  const int hw0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4
  const long long base = (long long)n * C * HW;
  if (TO_NHWC) {
    // read rows of [C][HW] (hw contiguous), write rows of [HW][C] (c contiguous)
    for (int i = ty; i < 64; i += 4) {
      const int c = c0 + i, hw = hw0 + tx;
      if (c < C && hw < HW) tile[i][tx] = x[base + (long long)c * HW + hw];
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
      const int hw = hw0 + i, c = c0 + tx;
      if (c < C && hw < HW) y[base + (long long)hw * C + c] = tile[tx][i];
    }
  } else {
    for (int i = ty; i < 64; i += 4) {
      const int hw = hw0 + i, c = c0 + tx;
      if (c < C && hw < HW) tile[tx][i] = x[base + (long long)hw * C + c];
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
      const int c = c0 + i, hw = hw0 + tx;
      if (c < C && hw < HW) y[base + (long long)c * HW + hw] = tile[i][tx];
    }
  }
}

// NCHW <-> NHWC for few channels (C <= 8): one pixel per thread, its C
// values read from (or written to) C planes; both sides stay coalesced
// across the threads, where the 64 x 64 tile of the general transpose
// would be almost empty.
template <typename E, bool TO_NHWC>
__global__ __launch_bounds__(256) void transpose_smallc_kernel(const E* __restrict__ x, E* __restrict__ y,
                                                               int C, long long HW, long long pixels) {
  const long long p = (long long)blockIdx.x * 256 + threadIdx.x;
  if (p >= pixels) return;
  const long long n = p / HW, hw = p - n * HW;
  const long long plane = n * C * HW + hw;
  for (int c = 0; c < C; ++c) {
    if (TO_NHWC)
      y[p * C + c] = x[plane + c * HW];
    else
      y[plane + c * HW] = x[p * C + c];
  }
}

// NCHW -> NHWC for C <= 8 with 16-bit elements and H * W % 8 == 0: a
// thread reads 8 consecutive pixels of one image from each of the C planes
// (16-byte loads) and interleaves them into the workgroup's LDS copy of its
// output run (256 * 8 pixels, contiguous in NHWC); the run then goes out in
// 16-byte stores with consecutive lanes on consecutive addresses.  C is a
// template constant so the shuffle stays in registers.
template <typename E, int C>
__global__ __launch_bounds__(256) void transpose_smallc8_kernel(const E* __restrict__ x, E* __restrict__ y,
                                                                int HW, int groups) {
  static_assert(sizeof(E) == 2 && C >= 1 && C <= 8, "16-bit elements, C <= 8");
  __shared__ __attribute__((aligned(16))) E run[256 * 8 * C];
  const int g0 = blockIdx.x * 256;
  const int g = g0 + threadIdx.x;  // group of 8 pixels
  if (g < groups) {
    const int gpi = HW >> 3;       // groups per image
    const int n = g / gpi, hw = (g - n * gpi) * 8;
    const E* xp = x + ((long long)n * C) * HW + hw;
    E o[8 * C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const V8<E> t = ld8(xp + (long long)c * HW);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e * C + c] = t.v[e];
    }
#pragma unroll
    for (int k = 0; k < C; ++k) {
      V8<E> w;
#pragma unroll
      for (int e = 0; e < 8; ++e) w.v[e] = o[k * 8 + e];
      *reinterpret_cast<V8<E>*>(run + (threadIdx.x * C + k) * 8) = w;
    }
  }
  __syncthreads();
  const int chunks = min(256, groups - g0) * C;  // 16-byte chunks of this run
  E* yp = y + (long long)g0 * 8 * C;
#pragma unroll
  for (int k = 0; k < C; ++k) {
    const int i = k * 256 + threadIdx.x;
    if (i < chunks) st8(yp + i * 8, *reinterpret_cast<const V8<E>*>(run + i * 8));
  }
}

// Any layout -> any layout, one destination element per thread (padded
// channels get zero).  Used for the pairs without a specialised kernel.
template <typename E, int LI, int LO>
__global__ __launch_bounds__(256) void convert_kernel(const E* __restrict__ x, E* __restrict__ y,
                                                      int N, int C, int H, int W, int csi, int cso) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long total = (long long)N * cso * H * W;
  if (idx >= total) return;
  int n, c, h, w;
  long long r = idx;
  if constexpr (LO == NCHW) {
    w = (int)(r % W); r /= W;
    h = (int)(r % H); r /= H;
    c = (int)(r % cso); n = (int)(r / cso);
  } else if constexpr (LO == NHWC) {
    c = (int)(r % cso); r /= cso;
    w = (int)(r % W); r /= W;
    h = (int)(r % H); n = (int)(r / H);
  } else {
    const int e = (int)(r % 8); r /= 8;
    w = (int)(r % W); r /= W;
    h = (int)(r % H); r /= H;
    const int cb = (int)(r % (cso >> 3)); n = (int)(r / (cso >> 3));
    c = cb * 8 + e;
  }
  E v = (E)0;
  if (c < C) v = x[toff<LI>(csi, H, W, n, c, h, w)];
  y[idx] = v;
}

template <typename E>
static void convert_e(const void* xv, const TDesc& xd, void* yv, const TDesc& yd, hipStream_t s) {
  const E* x = reinterpret_cast<const E*>(xv);
  E* y = reinterpret_cast<E*>(yv);
  const int HW = xd.h * xd.w;
  if constexpr (sizeof(E) == 2) {
    // C <= 8 into NHWC keeps its 8-pixel kernel below; the rest of the
    // 16-bit pairs take the vector converters when the shape allows
    const bool smallc_nhwc = xd.c <= 8 && yd.layout == NHWC && xd.layout == NCHW;
    if (!smallc_nhwc && convert_vec16(xv, xd, yv, yd, s)) return;
  }
  if ((xd.layout == NCHW && yd.layout == NHWC) || (xd.layout == NHWC && yd.layout == NCHW)) {
    if constexpr (sizeof(E) == 2) {
      if (xd.c <= 8 && yd.layout == NHWC && HW % 8 == 0 && (long long)xd.n * HW < (1ll << 31)) {
        const int groups = xd.n * HW / 8;
#define T8(CC)                                                                                       \
  case CC:                                                                                           \
    SN_LAUNCH((transpose_smallc8_kernel<E, CC>), dim3(blocks(groups)), dim3(256), 0, s, x, y, HW, groups); \
    return;
        switch (xd.c) { T8(1) T8(2) T8(3) T8(4) T8(5) T8(6) T8(7) T8(8) }
#undef T8
      }
    }
    if (xd.c <= 8) {
      const long long pixels = (long long)xd.n * HW;
      if (yd.layout == NHWC)
        SN_LAUNCH((transpose_smallc_kernel<E, true>), dim3(blocks(pixels)), dim3(256), 0, s, x, y, xd.c,
                  (long long)HW, pixels);
      else
        SN_LAUNCH((transpose_smallc_kernel<E, false>), dim3(blocks(pixels)), dim3(256), 0, s, x, y, xd.c,
                  (long long)HW, pixels);
      return;
    }
    dim3 g((HW + 63) / 64, (xd.c + 63) / 64, xd.n);
    check(xd.n <= 65535, "batch too large for the transpose grid");
    if (yd.layout == NHWC)
      SN_LAUNCH((transpose_kernel<E, true>), g, dim3(256), 0, s, x, y, xd.c, HW);
    else
      SN_LAUNCH((transpose_kernel<E, false>), g, dim3(256), 0, s, x, y, xd.c, HW);
    return;
  }
  const long long total = (long long)yd.n * yd.cs * yd.h * yd.w;
  dim3 g(blocks(total));
#define CV(A, B)                                                                              \
  SN_LAUNCH((convert_kernel<E, A, B>), g, dim3(256), 0, s, x, y, xd.n, xd.c, xd.h, xd.w, \
                     xd.cs, yd.cs)
  const int key = xd.layout * 3 + yd.layout;
  switch (key) {
    case NCHW * 3 + NC8: CV(NCHW, NC8); break;
    case NHWC * 3 + NC8: CV(NHWC, NC8); break;
    case NC8 * 3 + NCHW: CV(NC8, NCHW); break;
    case NC8 * 3 + NHWC: CV(NC8, NHWC); break;
    case NCHW * 3 + NHWC: CV(NCHW, NHWC); break;
    case NHWC * 3 + NCHW: CV(NHWC, NCHW); break;
    default: check(false, "converter between equal layouts");
  }
#undef CV
}

void convert(int dtype, const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t s) {
  check(xd.n == yd.n && xd.c == yd.c && xd.h == yd.h && xd.w == yd.w, "converter keeps the shape");
  if (dtype == 0) convert_e<uint32_t>(x, xd, y, yd, s);
  else convert_e<uint16_t>(x, xd, y, yd, s);
}

// ------------------------------------------------------------------ scratch fill
// Uniform values in [-1, 1) from a 64-bit mix of (seed, index); only used to
// give profiled routines realistic operands.
template <typename T>
__global__ __launch_bounds__(256) void fill_kernel(T* __restrict__ p, long long n, unsigned long long seed) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  unsigned long long z = seed + 0x9E3779B97F4A7C15ull * (unsigned long long)(i + 1);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  const float u = (float)(z >> 40) * (1.0f / 16777216.0f);
  p[i] = from_f<T>(2.f * u - 1.f);
}

void fill_random(int dtype, void* p, int64_t n, uint64_t seed, hipStream_t s) {
  dim3 g(blocks(n));
  if (dtype == 0) SN_LAUNCH(fill_kernel<float>, g, dim3(256), 0, s, (float*)p, (long long)n, (unsigned long long)seed);
  else if (dtype == 1) SN_LAUNCH(fill_kernel<f16>, g, dim3(256), 0, s, (f16*)p, (long long)n, (unsigned long long)seed);
  else SN_LAUNCH(fill_kernel<bf16>, g, dim3(256), 0, s, (bf16*)p, (long long)n, (unsigned long long)seed);
}

}  // namespace k
}  // namespace sn
