// Convolution routines for gfx950: implicit GEMM on MFMA, direct VALU,
// Winograd F(2x2, 3x3) (input transform -> batched MFMA GEMM -> output
// transform, the three sub-layers of the paper's Winograd childnet,
// Sec. III-D), and depthwise 3x3.
//
// All routines compute the cross-correlation
//   y[n,k,p,q] = act(b[k] + sum_{c,r,s} w[k,c,r,s] x[n,c,p*st-pad+r,q*st-pad+s])
// with zero padding, accumulating in float32.  Weights arrive prepared:
// dense [Kp][R][S][C8] (C8 = C rounded up to 8, Kp = K rounded up to 8,
// zero-filled), so the reduction index runs over (r, s, 8-channel chunk,
// lane-in-chunk) for every layout.
#include "igemm.hpp"
#include "wino.hpp"

namespace sn {
namespace k {

int igemm_num_params(int dtype) {
  return dtype == 0 ? (int)(sizeof(kIg32) / sizeof(kIg32[0])) : (int)(sizeof(kIg16) / sizeof(kIg16[0]));
}

// A configuration whose tile rows do not divide the 256 threads needs the
// 8-channel vector loader (NHWC with C % 8 == 0, or NC8HW8).
bool igemm_param_valid(int dtype, int param, int layout, int n, int c, int h, int w, int r, int s,
                       int stride, int pad, int k) {
  if (param < 0 || param >= igemm_num_params(dtype)) return false;
  const IgCfg& g = dtype == 0 ? kIg32[param] : kIg16[param];
  const bool vec = layout == NC8 || (layout == NHWC && c % 8 == 0);
  if (g.dma == 2)
    return patch_applicable(layout, c, h, w, r, s, stride, pad, n, g.pc.fmt, g.pc.pwt, g.pc.prows, g.pc.sd,
                            g.pc.ra);
  if (g.dma == 3) return smallc_applicable(layout, c, h, w, r, s, stride, pad, n, k, g.bm / 16, g.ppx, g.gmax);
  if (g.dma == 4) return stream1x1_applicable(layout, c, c, n, h, w, r, s, stride, pad, k, g.bk);
  if (g.dma) {
    // fp32 index division and 32-bit byte offsets bound the output size
    const long long p = (h + 2 * pad - r) / stride + 1, q = (w + 2 * pad - s) / stride + 1;
    const long long m = (long long)n * p * q;
    return vec && ((c + 7) / 8) % (g.bk / 8) == 0 && r * s <= 32 && m + p * q < (1 << 21);
  }
  return vec || 256 % g.bm == 0;
}

bool igemm_param_takes_residual(int dtype, int param, int layout, int k) {
  if (param < 0 || param >= igemm_num_params(dtype)) return false;
  const IgCfg& g = dtype == 0 ? kIg32[param] : kIg16[param];
  return g.dma == 0 || (g.dma == 1 && (layout == NC8 || k % 8 == 0)) || (g.dma == 4 && layout == NHWC && k % 8 == 0);
}

bool igemm_param_takes_projection(int dtype, int param, int layout, int n, int c, int h, int w, int r, int s,
                                  int stride, int pad, int k, int c2) {
  if (dtype == 0 || param < 0 || param >= igemm_num_params(dtype)) return false;
  if (kIg16[param].dma == 4)  // the streaming 1x1 kernel: both inputs' slabs in one reduction
    return stream1x1_takes_projection(layout, c, c, n, h, w, r, s, stride, pad, k, c2, kIg16[param].bk);
  if (!igemm_param_valid(dtype, param, layout, n, c, h, w, r, s, stride, pad, k)) return false;
  const IgCfg& g = kIg16[param];
  // the LDS-DMA tiles (summed in one kernel: no separate reduction pass)
  return g.dma == 1 && g.split != 1 && c2 % 8 == 0 && (c2 / 8) % (g.bk / 8) == 0;
}

size_t igemm_ws_bytes(int dtype, int param, const TDesc& xd, const TDesc& yd, int r, int s, int c2) {
  const IgCfg c = ig_cfg(dtype, param);
  if (!c.split) return 0;
  ConvArgs cv{};
  cv.xd = xd;
  cv.yd = yd;
  cv.r = r;
  cv.s = s;
  cv.stride = 1;
  IgArgs a = make_ig(cv);
  a.M = xd.n * yd.h * yd.w;
  a.KC2 = (c2 + 7) / 8;
  ig_decompose(a, c);
  if (a.splits <= 1) return 0;
  if (c.split == 2) return (size_t)a.splits * a.tiles_m * a.tiles_n * c.bm * c.bn * sizeof(float);
  return (size_t)a.splits * a.M * a.Ng * sizeof(float);
}

void conv_igemm(int dtype, int param, const ConvArgs& c, hipStream_t st) {
  if (dtype == 0) igemm_dispatch<float>(dtype, param, c, st);
  else if (dtype == 1) conv_igemm_f16(param, c, st);
  else conv_igemm_bf16(param, c, st);
}

// ------------------------------------------------------------------ direct (VALU)
// One thread computes 8 output channels of one output pixel, looping over
// the taps and input channels; the weights of the workgroup's 8 channels are
// uniform across it.
template <typename T, int L>
__global__ __launch_bounds__(256) void direct_kernel(IgArgs a) {
  const int m = blockIdx.x * 256 + threadIdx.x;
  const int n0 = blockIdx.y * 8;
  if (m >= a.M) return;
  const int img = m / a.PQ, pq = m - img * a.PQ;
  const int p = pq / a.Q, q = pq - p * a.Q;
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x);
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w);
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  const bool vec = (L == NC8) || (L == NHWC && a.vec);
  for (int r = 0; r < a.R; ++r) {
    const int h = p * a.stride - a.pad + r;
    const bool hv = (unsigned)h < (unsigned)a.H;
    for (int s = 0; s < a.S; ++s) {
      const int ww = q * a.stride - a.pad + s;
      const bool ok = hv && (unsigned)ww < (unsigned)a.W;
      for (int cb = 0; cb < a.CB; ++cb) {
        float xv[8];
        if (vec) {
          V8<T> t = zero8<T>();
          if (ok) {
            if constexpr (L == NC8)
              t = ld8(x + ((((long long)img * a.CB + cb) * a.H + h) * a.W + ww) * 8);
            else
              t = ld8(x + (((long long)img * a.H + h) * a.W + ww) * a.Cs + cb * 8);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) xv[e] = to_f(t.v[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int c = cb * 8 + e;
            float v = 0.f;
            if (ok && c < a.C) {
              if constexpr (L == NCHW)
                v = to_f(x[(((long long)img * a.Cs + c) * a.H + h) * a.W + ww]);
              else
                v = to_f(x[(((long long)img * a.H + h) * a.W + ww) * a.Cs + c]);
            }
            xv[e] = v;
          }
        }
        const int tap = (r * a.S + s) * a.CB + cb;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const T* wp = w + (long long)(n0 + j) * a.Kred + tap * 8;
          V8<T> wt = ld8(wp);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[j] = fmaf(to_f(wt.v[e]), xv[e], acc[j]);
        }
      }
    }
  }
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
  T out[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int n = n0 + j;
    float rv = 0.f;
    if (a.res && n < a.Ng) rv = to_f(reinterpret_cast<const T*>(a.res)[out_index<L>(a, m, n)]);
    out[j] = from_f<T>(act_f(acc[j] + (n < a.Ng ? a.bias[n] : 0.f) + rv, a.act));
  }
  if constexpr (L == NCHW) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (n0 + j < a.Ng) y[((long long)img * a.Ks + n0 + j) * a.PQ + pq] = out[j];
  } else if constexpr (L == NC8) {
    V8<T> v;
#pragma unroll
    for (int j = 0; j < 8; ++j) v.v[j] = out[j];
    st8(y + (((long long)img * (a.Ks >> 3) + (n0 >> 3)) * a.PQ + pq) * 8, v);
  } else {
    if (a.Ks % 8 == 0) {
      V8<T> v;
#pragma unroll
      for (int j = 0; j < 8; ++j) v.v[j] = out[j];
      st8(y + (long long)m * a.Ks + n0, v);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (n0 + j < a.Ng) y[(long long)m * a.Ks + n0 + j] = out[j];
    }
  }
}

template <typename T>
static void direct_dispatch(const ConvArgs& c, hipStream_t st) {
  IgArgs a = make_ig(c);
  check(c.xd.layout == c.yd.layout, "direct convolution reads and writes one layout");
  dim3 grid((a.M + 255) / 256, (a.Ng + 7) / 8);
  switch (c.xd.layout) {
    case NCHW: SN_LAUNCH((direct_kernel<T, NCHW>), grid, dim3(256), 0, st, a); break;
    case NHWC: SN_LAUNCH((direct_kernel<T, NHWC>), grid, dim3(256), 0, st, a); break;
    case NC8: SN_LAUNCH((direct_kernel<T, NC8>), grid, dim3(256), 0, st, a); break;
  }
}

void conv_direct(int dtype, const ConvArgs& c, hipStream_t st) {
  if (dtype == 0) direct_dispatch<float>(c, st);
  else if (dtype == 1) direct_dispatch<f16>(c, st);
  else direct_dispatch<bf16>(c, st);
}

// ------------------------------------------------------------------ Winograd F(2x2, 3x3)
// Input transform V = B^T d B of every 4x4 input tile (stride 2, the input
// zero-extended beyond the padding), computed in float32 and stored in the
// run dtype as V[16][T][C8] (T = N * ceil(H/2) * ceil(W/2) tiles).  The
// 16 products M_xi = V_xi U_xi^T run as one batched MFMA GEMM with float32
// output M[16][T][Ng]; the output transform Y = A^T M A adds the bias and
// the activation.  Matrices are those of the minimal filtering algorithm
// F(2, 3) nested with itself.
struct WinoArgs {
  const void* x;
  void* v;
  const float* m;
  const float* bias;
  void* y;
  int N, C, H, W, Cs, C8, TH, TW, T;
  int Ng, Ks, act;
};

template <typename T, int L>
__global__ __launch_bounds__(256) void wino_in_kernel(WinoArgs a) {
  const int CB = a.C8 >> 3;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  int t, cb;
  if constexpr (L == NCHW) {  // tile index fastest: consecutive lanes read along w
    t = (int)(idx % a.T);
    cb = (int)(idx / a.T);
  } else {
    cb = (int)(idx % CB);
    t = (int)(idx / CB);
  }
  if (t >= a.T || cb >= CB) return;
  const int per = a.TH * a.TW;
  const int n = t / per, tt = t - n * per;
  const int ty = tt / a.TW, tx = tt - ty * a.TW;
  const int h0 = ty * 2 - 1, w0 = tx * 2 - 1;
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x);
  float d[4][4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int h = h0 + i, w = w0 + j;
      const bool ok = (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
      if (L == NC8 || (L == NHWC && a.C % 8 == 0)) {
        V8<T> v = zero8<T>();
        if (ok) {
          if constexpr (L == NC8)
            v = ld8(x + ((((long long)n * CB + cb) * a.H + h) * a.W + w) * 8);
          else
            v = ld8(x + (((long long)n * a.H + h) * a.W + w) * a.Cs + cb * 8);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) d[i][j][e] = to_f(v.v[e]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int c = cb * 8 + e;
          float v = 0.f;
          if (ok && c < a.C) {
            if constexpr (L == NCHW)
              v = to_f(x[(((long long)n * a.Cs + c) * a.H + h) * a.W + w]);
            else
              v = to_f(x[(((long long)n * a.H + h) * a.W + w) * a.Cs + c]);
          }
          d[i][j][e] = v;
        }
      }
    }
  T* __restrict__ vout = reinterpret_cast<T*>(a.v);
  const long long plane = (long long)a.T * a.C8;
  {
    float u[4][4][8];
    // rows: B^T d
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        u[0][j][e] = d[0][j][e] - d[2][j][e];
        u[1][j][e] = d[1][j][e] + d[2][j][e];
        u[2][j][e] = d[2][j][e] - d[1][j][e];
        u[3][j][e] = d[1][j][e] - d[3][j][e];
      }
    // columns: (B^T d) B
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      V8<T> c0, c1, c2, c3;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        c0.v[e] = from_f<T>(u[i][0][e] - u[i][2][e]);
        c1.v[e] = from_f<T>(u[i][1][e] + u[i][2][e]);
        c2.v[e] = from_f<T>(u[i][2][e] - u[i][1][e]);
        c3.v[e] = from_f<T>(u[i][1][e] - u[i][3][e]);
      }
      T* base = vout + (long long)t * a.C8 + cb * 8;
      st8(base + (i * 4 + 0) * plane, c0);
      st8(base + (i * 4 + 1) * plane, c1);
      st8(base + (i * 4 + 2) * plane, c2);
      st8(base + (i * 4 + 3) * plane, c3);
    }
  }
}

template <typename T, int L>
__global__ __launch_bounds__(256) void wino_out_kernel(WinoArgs a) {
  const int NB = (a.Ng + 7) / 8;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  int t, kb;
  if constexpr (L == NCHW) {
    t = (int)(idx % a.T);
    kb = (int)(idx / a.T);
  } else {
    kb = (int)(idx % NB);
    t = (int)(idx / NB);
  }
  if (t >= a.T || kb >= NB) return;
  const int per = a.TH * a.TW;
  const int n = t / per, tt = t - n * per;
  const int ty = tt / a.TW, tx = tt - ty * a.TW;
  const long long plane = (long long)a.T * a.Ng;
  const float* __restrict__ mp = a.m + (long long)t * a.Ng + kb * 8;
  const bool full = kb * 8 + 8 <= a.Ng;
  float mm[4][4][8];
#pragma unroll
  for (int xi = 0; xi < 16; ++xi) {
    const float* q = mp + xi * plane;
#pragma unroll
    for (int e = 0; e < 8; ++e) mm[xi >> 2][xi & 3][e] = (full || kb * 8 + e < a.Ng) ? q[e] : 0.f;
  }
  float tmp[2][4][8];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      tmp[0][j][e] = mm[0][j][e] + mm[1][j][e] + mm[2][j][e];
      tmp[1][j][e] = mm[1][j][e] - mm[2][j][e] - mm[3][j][e];
    }
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int p = ty * 2 + i, q = tx * 2 + j;
      if (p >= a.H || q >= a.W) continue;  // output size equals input size
      V8<T> o;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int k = kb * 8 + e;
        float v = j == 0 ? tmp[i][0][e] + tmp[i][1][e] + tmp[i][2][e]
                         : tmp[i][1][e] - tmp[i][2][e] - tmp[i][3][e];
        o.v[e] = from_f<T>(act_f(v + (k < a.Ng ? a.bias[k] : 0.f), a.act));
      }
      if constexpr (L == NC8) {
        st8(y + ((((long long)n * (a.Ks >> 3) + kb) * a.H + p) * a.W + q) * 8, o);
      } else if constexpr (L == NHWC) {
        if (a.Ks % 8 == 0) {
          st8(y + (((long long)n * a.H + p) * a.W + q) * a.Ks + kb * 8, o);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (kb * 8 + e < a.Ng) y[(((long long)n * a.H + p) * a.W + q) * a.Ks + kb * 8 + e] = o.v[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (kb * 8 + e < a.Ng) y[(((long long)n * a.Ks + kb * 8 + e) * a.H + p) * a.W + q] = o.v[e];
      }
    }
}

// ------------------------------------------------------------------ Winograd F(4x4, 3x3)
// The same three steps with 4x4 output tiles: a 6x6 input patch per tile
// (stride 4), V = B^T d B with 36 positions, 36 batched GEMMs, Y = A^T M A.
// The matrices are those of the Toom-Cook construction of F(4, 3) on the
// points 0, 1, -1, 2, -2 and infinity, nested with themselves.  A thread
// transforms one tile for 4 channels (the 6x6x4 patch in registers).
template <typename T>
__device__ __forceinline__ void ld4f(const T* p, float* v) {
  if constexpr (sizeof(T) == 2) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
    T e[4];
    __builtin_memcpy(e, &w, 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = to_f(e[i]);
  } else {
    const f32x4 w = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = w[i];
  }
}
template <typename T>
__device__ __forceinline__ void st4f(T* p, const float* v) {
  if constexpr (sizeof(T) == 2) {
    T e[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) e[i] = from_f<T>(v[i]);
    u32x2 w;
    __builtin_memcpy(&w, e, 8);
    *reinterpret_cast<u32x2*>(p) = w;
  } else {
    *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
  }
}
// B^T applied to six values (rows of the patch, then columns of the result)
__device__ __forceinline__ void bt6(const float* x, float* r) {
  r[0] = 4.f * x[0] - 5.f * x[2] + x[4];
  r[1] = -4.f * x[1] - 4.f * x[2] + x[3] + x[4];
  r[2] = 4.f * x[1] - 4.f * x[2] - x[3] + x[4];
  r[3] = -2.f * x[1] - x[2] + 2.f * x[3] + x[4];
  r[4] = 2.f * x[1] - x[2] - 2.f * x[3] + x[4];
  r[5] = 4.f * x[1] - 5.f * x[3] + x[5];
}
// A^T applied to six values
__device__ __forceinline__ void at6(const float* m, float* o) {
  o[0] = m[0] + m[1] + m[2] + m[3] + m[4];
  o[1] = m[1] - m[2] + 2.f * (m[3] - m[4]);
  o[2] = m[1] + m[2] + 4.f * (m[3] + m[4]);
  o[3] = m[1] - m[2] + 8.f * (m[3] - m[4]) + m[5];
}

template <typename T, int L>
__global__ __launch_bounds__(256) void wino4_in_kernel(WinoArgs a) {
  const int CQ = a.C8 >> 2;  // channel quads
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  int t, cq;
  if constexpr (L == NCHW) {
    t = (int)(idx % a.T);
    cq = (int)(idx / a.T);
  } else {
    cq = (int)(idx % CQ);
    t = (int)(idx / CQ);
  }
  if (t >= a.T || cq >= CQ) return;
  const int per = a.TH * a.TW;
  const int n = t / per, tt = t - n * per;
  const int ty = tt / a.TW, tx = tt - ty * a.TW;
  const int h0 = ty * 4 - 1, w0 = tx * 4 - 1;
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x);
  // whole 4-channel vectors: NC8HW8 (padded channels are stored), or NHWC
  // quads inside the real channels with aligned pixel rows
  const bool vec = L == NC8 || (L == NHWC && a.Cs % 4 == 0 && cq * 4 + 4 <= a.C);
  float d[6][6][4];
#pragma unroll
  for (int i = 0; i < 6; ++i)
#pragma unroll
    for (int j = 0; j < 6; ++j) {
      const int h = h0 + i, w = w0 + j;
      const bool ok = (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W;
#pragma unroll
      for (int e = 0; e < 4; ++e) d[i][j][e] = 0.f;
      if (!ok) continue;
      if (vec) {
        if constexpr (L == NC8)
          ld4f(x + ((((long long)n * (a.C8 >> 3) + (cq >> 1)) * a.H + h) * a.W + w) * 8 + (cq & 1) * 4, d[i][j]);
        else
          ld4f(x + (((long long)n * a.H + h) * a.W + w) * a.Cs + cq * 4, d[i][j]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int c = cq * 4 + e;
          if (c >= a.C) continue;
          if constexpr (L == NCHW)
            d[i][j][e] = to_f(x[(((long long)n * a.Cs + c) * a.H + h) * a.W + w]);
          else
            d[i][j][e] = to_f(x[(((long long)n * a.H + h) * a.W + w) * a.Cs + c]);
        }
      }
    }
  // columns: B^T d, in place
#pragma unroll
  for (int j = 0; j < 6; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float col[6], r[6];
#pragma unroll
      for (int i = 0; i < 6; ++i) col[i] = d[i][j][e];
      bt6(col, r);
#pragma unroll
      for (int i = 0; i < 6; ++i) d[i][j][e] = r[i];
    }
  // rows: (B^T d) B, stored as position xi = 6 i + j
  T* __restrict__ vout = reinterpret_cast<T*>(a.v);
  const long long plane = (long long)a.T * a.C8;
  T* base = vout + (long long)t * a.C8 + cq * 4;
#pragma unroll
  for (int i = 0; i < 6; ++i) {
    float r[6][4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float row[6], o[6];
#pragma unroll
      for (int j = 0; j < 6; ++j) row[j] = d[i][j][e];
      bt6(row, o);
#pragma unroll
      for (int j = 0; j < 6; ++j) r[j][e] = o[j];
    }
#pragma unroll
    for (int j = 0; j < 6; ++j) st4f(base + (i * 6 + j) * plane, r[j]);
  }
}

template <typename T, int L>
__global__ __launch_bounds__(256) void wino4_out_kernel(WinoArgs a) {
  const int NQ = (a.Ng + 3) / 4;
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  int t, kq;
  if constexpr (L == NCHW) {
    t = (int)(idx % a.T);
    kq = (int)(idx / a.T);
  } else {
    kq = (int)(idx % NQ);
    t = (int)(idx / NQ);
  }
  if (t >= a.T || kq >= NQ) return;
  const int per = a.TH * a.TW;
  const int n = t / per, tt = t - n * per;
  const int ty = tt / a.TW, tx = tt - ty * a.TW;
  const long long plane = (long long)a.T * a.Ng;
  const float* __restrict__ mp = a.m + (long long)t * a.Ng + kq * 4;
  const bool full = kq * 4 + 4 <= a.Ng && a.Ng % 4 == 0;
  // rows of M: A^T M, four output rows of six
  float tmp[4][6][4];
#pragma unroll
  for (int j = 0; j < 6; ++j) {
    float col[6][4];
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      const float* q = mp + (i * 6 + j) * plane;
      if (full) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(q);
#pragma unroll
        for (int e = 0; e < 4; ++e) col[i][e] = v[e];
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) col[i][e] = kq * 4 + e < a.Ng ? q[e] : 0.f;
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float m6[6], o4[4];
#pragma unroll
      for (int i = 0; i < 6; ++i) m6[i] = col[i][e];
      at6(m6, o4);
#pragma unroll
      for (int i = 0; i < 4; ++i) tmp[i][j][e] = o4[i];
    }
  }
  float bias[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) bias[e] = kq * 4 + e < a.Ng ? a.bias[kq * 4 + e] : 0.f;
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float out[4][4];  // [column][channel]
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float m6[6], o4[4];
#pragma unroll
      for (int j = 0; j < 6; ++j) m6[j] = tmp[i][j][e];
      at6(m6, o4);
#pragma unroll
      for (int j = 0; j < 4; ++j) out[j][e] = act_f(o4[j] + bias[e], a.act);
    }
    const int p = ty * 4 + i;
    if (p >= a.H) continue;  // output size equals input size
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int q = tx * 4 + j;
      if (q >= a.W) continue;
      if constexpr (L == NC8) {
        st4f(y + ((((long long)n * (a.Ks >> 3) + (kq >> 1)) * a.H + p) * a.W + q) * 8 + (kq & 1) * 4, out[j]);
      } else if constexpr (L == NHWC) {
        if (full && a.Ks % 4 == 0) {
          st4f(y + (((long long)n * a.H + p) * a.W + q) * a.Ks + kq * 4, out[j]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (kq * 4 + e < a.Ng) y[(((long long)n * a.H + p) * a.W + q) * a.Ks + kq * 4 + e] = from_f<T>(out[j][e]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (kq * 4 + e < a.Ng) y[(((long long)n * a.Ks + kq * 4 + e) * a.H + p) * a.W + q] = from_f<T>(out[j][e]);
      }
    }
  }
}

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t winograd_ws_bytes(int dtype, const TDesc& xd, int k, int tile) {
  const long long T = (long long)xd.n * ((xd.h + tile - 1) / tile) * ((xd.w + tile - 1) / tile);
  const long long C8 = (xd.c + 7) / 8 * 8;
  const long long Kp = (k + 7) / 8 * 8;
  const long long np = (long long)(tile + 2) * (tile + 2);  // positions
  const size_t es = dtype == 0 ? 4 : 2;
  return align256(np * T * C8 * es) + align256(np * T * Kp * 4);
}

// The routine is a childnet of three sub-layers, each launched on its own:
// the input transform (wgenc), the 16 batched GEMMs (wgconv, whose tile is
// the sub-routine: index into kWinoGemm), the output transform (wgdec).
// V and M live in the workspace between them.
static const IgCfg kWinoGemm16[] = {{64, 64, 64, 0, 4}, {128, 64, 64, 0, 4}, {128, 128, 64, 0, 2}};
static const IgCfg kWinoGemm32[] = {{64, 64, 32, 0, 2}};

int winograd_gemm_num_configs(int dtype) {
  return dtype == 0 ? (int)(sizeof(kWinoGemm32) / sizeof(kWinoGemm32[0]))
                    : (int)(sizeof(kWinoGemm16) / sizeof(kWinoGemm16[0]));
}

template <typename T>
static WinoArgs wino_args(int dtype, int tile, const ConvArgs& c) {
  check(tile == 2 || tile == 4, "Winograd output tile 2x2 or 4x4");
  check(c.r == 3 && c.s == 3 && c.stride == 1 && c.pad == 1, "Winograd F(mxm,3x3) needs 3x3/1 pad 1");
  check(c.xd.layout == c.yd.layout, "Winograd reads and writes one layout");
  check(!c.res, "Winograd routine takes no residual");
  WinoArgs a{};
  a.x = c.x;
  a.bias = c.bias;
  a.y = c.y;
  a.N = c.xd.n;
  a.C = c.xd.c;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.Cs = c.xd.cs;
  a.C8 = (a.C + 7) / 8 * 8;
  a.TH = (a.H + tile - 1) / tile;
  a.TW = (a.W + tile - 1) / tile;
  a.T = a.N * a.TH * a.TW;
  a.Ng = c.yd.layout == NC8 ? c.yd.cs : c.yd.c;
  a.Ks = c.yd.cs;
  a.act = c.act;
  const int Kp = (c.yd.c + 7) / 8 * 8;
  const long long np = (long long)(tile + 2) * (tile + 2);
  const size_t vbytes = align256((size_t)np * a.T * a.C8 * sizeof(T));
  check(c.ws && c.ws_bytes >= winograd_ws_bytes(dtype, c.xd, c.yd.c, tile), "Winograd workspace too small");
  check(np * a.T * std::max(a.C8, Kp) < (1ll << 31), "tensor too large");
  a.v = c.ws;
  a.m = reinterpret_cast<float*>(reinterpret_cast<char*>(c.ws) + vbytes);
  return a;
}

template <typename T>
static void wino_enc_t(int dtype, int tile, const ConvArgs& c, hipStream_t st) {
  const WinoArgs a = wino_args<T>(dtype, tile, c);
  if (tile == 4) {
    dim3 g((unsigned)(((long long)a.T * (a.C8 / 4) + 255) / 256));
    switch (c.xd.layout) {
      case NCHW: SN_LAUNCH((wino4_in_kernel<T, NCHW>), g, dim3(256), 0, st, a); break;
      case NHWC: SN_LAUNCH((wino4_in_kernel<T, NHWC>), g, dim3(256), 0, st, a); break;
      case NC8: SN_LAUNCH((wino4_in_kernel<T, NC8>), g, dim3(256), 0, st, a); break;
    }
    return;
  }
  dim3 g((unsigned)(((long long)a.T * (a.C8 / 8) + 255) / 256));
  switch (c.xd.layout) {
    case NCHW: SN_LAUNCH((wino_in_kernel<T, NCHW>), g, dim3(256), 0, st, a); break;
    case NHWC: SN_LAUNCH((wino_in_kernel<T, NHWC>), g, dim3(256), 0, st, a); break;
    case NC8: SN_LAUNCH((wino_in_kernel<T, NC8>), g, dim3(256), 0, st, a); break;
  }
}

template <typename T>
static void wino_gemm_t(int dtype, int tile, const ConvArgs& c, int cfg, hipStream_t st) {
  const WinoArgs a = wino_args<T>(dtype, tile, c);
  check(cfg >= 0 && cfg < winograd_gemm_num_configs(dtype), "unknown Winograd GEMM tile");
  const int Kp = (c.yd.c + 7) / 8 * 8;
  // batched GEMM: A = V_xi as a [T][C8] matrix (1x1 "NHWC" convolution), B = U_xi [Kp][C8]
  IgArgs g{};
  g.x = a.v;
  g.w = c.w;
  g.bias = c.bias;
  g.y = const_cast<float*>(a.m);
  g.C = a.C8;
  g.H = 1;
  g.W = a.T;
  g.Cs = a.C8;
  g.K = a.Ng;
  g.P = 1;
  g.Q = a.T;
  g.Ks = a.Ng;
  g.R = g.S = 1;
  g.stride = 1;
  g.pad = 0;
  g.act = 0;
  g.PQ = a.T;
  g.M = a.T;
  g.Ng = a.Ng;
  g.CB = a.C8 / 8;
  g.KC = a.C8 / 8;
  g.Kred = a.C8;
  g.x_bs = (long long)a.T * a.C8;
  g.w_bs = (long long)Kp * a.C8;
  g.y_bs = (long long)a.T * a.Ng;
  g.vec = 1;
  g.x_elems = (long long)a.T * a.C8;
  g.w_elems = (long long)Kp * a.C8;
  const IgCfg gc = std::is_same<T, float>::value ? kWinoGemm32[cfg] : kWinoGemm16[cfg];
  ig_decompose(g, gc);
  igemm_cfg<T, NHWC, true, EPI_RAW>(gc, g, (tile + 2) * (tile + 2), st);
}

template <typename T>
static void wino_dec_t(int dtype, int tile, const ConvArgs& c, hipStream_t st) {
  const WinoArgs a = wino_args<T>(dtype, tile, c);
  if (tile == 4) {
    dim3 g((unsigned)(((long long)a.T * ((a.Ng + 3) / 4) + 255) / 256));
    switch (c.xd.layout) {
      case NCHW: SN_LAUNCH((wino4_out_kernel<T, NCHW>), g, dim3(256), 0, st, a); break;
      case NHWC: SN_LAUNCH((wino4_out_kernel<T, NHWC>), g, dim3(256), 0, st, a); break;
      case NC8: SN_LAUNCH((wino4_out_kernel<T, NC8>), g, dim3(256), 0, st, a); break;
    }
    return;
  }
  dim3 g((unsigned)(((long long)a.T * ((a.Ng + 7) / 8) + 255) / 256));
  switch (c.xd.layout) {
    case NCHW: SN_LAUNCH((wino_out_kernel<T, NCHW>), g, dim3(256), 0, st, a); break;
    case NHWC: SN_LAUNCH((wino_out_kernel<T, NHWC>), g, dim3(256), 0, st, a); break;
    case NC8: SN_LAUNCH((wino_out_kernel<T, NC8>), g, dim3(256), 0, st, a); break;
  }
}

void winograd_sub(int dtype, int tile, int sub, int cfg, const ConvArgs& c, hipStream_t st) {
  check(sub >= 0 && sub <= 2, "Winograd sub-layer is 0 (wgenc), 1 (wgconv) or 2 (wgdec)");
#define WSUB(T_)                                            \
  if (sub == 0) wino_enc_t<T_>(dtype, tile, c, st);         \
  else if (sub == 1) wino_gemm_t<T_>(dtype, tile, c, cfg, st); \
  else wino_dec_t<T_>(dtype, tile, c, st);
  if (dtype == 0) { WSUB(float) }
  else if (dtype == 1) { WSUB(f16) }
  else { WSUB(bf16) }
#undef WSUB
}

void conv_winograd(int dtype, int tile, const ConvArgs& c, int gemm_cfg, hipStream_t st) {
  for (int sub = 0; sub < 3; ++sub) winograd_sub(dtype, tile, sub, gemm_cfg, c, st);
}

int winograd_f4_param() { return 1 + wino_fused_num_configs(); }

// ------------------------------------------------------------------ depthwise
// Per-channel R x S convolution; weights [R][S][C8].  Channel-vector layouts
// process 8 channels per thread with 16-byte accesses; NCHW one element.
struct DwArgs {
  const void* x;
  const void* w;
  const float* bias;
  void* y;
  int N, C, H, W, Cs, P, Q, R, S, stride, pad, act, C8;
};

template <typename T, int L>
__global__ __launch_bounds__(256) void dw_kernel(DwArgs a) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x);
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w);
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
  const int PQ = a.P * a.Q;
  if constexpr (L == NCHW) {
    const long long total = (long long)a.N * a.C * PQ;
    if (idx >= total) return;
    const int pq = (int)(idx % PQ);
    const long long nc = idx / PQ;
    const int c = (int)(nc % a.C);
    const int p = pq / a.Q, q = pq - p * a.Q;
    const T* xp = x + nc * a.H * a.W;
    float acc = a.bias[c];
    for (int r = 0; r < a.R; ++r) {
      const int h = p * a.stride - a.pad + r;
      if ((unsigned)h >= (unsigned)a.H) continue;
      for (int s = 0; s < a.S; ++s) {
        const int ww = q * a.stride - a.pad + s;
        if ((unsigned)ww >= (unsigned)a.W) continue;
        acc = fmaf(to_f(w[(r * a.S + s) * a.C8 + c]), to_f(xp[h * a.W + ww]), acc);
      }
    }
    y[idx] = from_f<T>(act_f(acc, a.act));
  } else {
    const int CB = a.C8 >> 3;
    const long long total = (long long)a.N * PQ * CB;
    if (idx >= total) return;
    int cb;
    long long m;
    if constexpr (L == NC8) {  // pixel fastest: contiguous within a channel-block plane
      m = idx % ((long long)a.N * PQ);
      cb = (int)(idx / ((long long)a.N * PQ));
    } else {
      cb = (int)(idx % CB);
      m = idx / CB;
    }
    const int n = (int)(m / PQ), pq = (int)(m % PQ);
    const int p = pq / a.Q, q = pq - p * a.Q;
    const bool vec = L == NC8 || a.C % 8 == 0;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = a.bias[cb * 8 + e];
    for (int r = 0; r < a.R; ++r) {
      const int h = p * a.stride - a.pad + r;
      if ((unsigned)h >= (unsigned)a.H) continue;
      for (int s = 0; s < a.S; ++s) {
        const int ww = q * a.stride - a.pad + s;
        if ((unsigned)ww >= (unsigned)a.W) continue;
        V8<T> wt = ld8(w + (r * a.S + s) * a.C8 + cb * 8);
        if (vec) {
          V8<T> xv;
          if constexpr (L == NC8)
            xv = ld8(x + ((((long long)n * CB + cb) * a.H + h) * a.W + ww) * 8);
          else
            xv = ld8(x + (((long long)n * a.H + h) * a.W + ww) * a.Cs + cb * 8);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] = fmaf(to_f(wt.v[e]), to_f(xv.v[e]), acc[e]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int c = cb * 8 + e;
            if (c < a.C)
              acc[e] = fmaf(to_f(wt.v[e]), to_f(x[(((long long)n * a.H + h) * a.W + ww) * a.Cs + c]), acc[e]);
          }
        }
      }
    }
    V8<T> o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.v[e] = from_f<T>(act_f(acc[e], a.act));
    if constexpr (L == NC8) {
      st8(y + ((((long long)n * CB + cb) * a.P + p) * a.Q + q) * 8, o);
    } else if (vec) {
      st8(y + (((long long)n * a.P + p) * a.Q + q) * a.Cs + cb * 8, o);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (cb * 8 + e < a.C) y[(((long long)n * a.P + p) * a.Q + q) * a.Cs + cb * 8 + e] = o.v[e];
    }
  }
}

template <typename T>
static void dw_dispatch(const ConvArgs& c, hipStream_t st) {
  check(c.xd.layout == c.yd.layout, "depthwise reads and writes one layout");
  check(c.xd.c == c.yd.c, "depthwise keeps the channel count");
  DwArgs a{};
  a.x = c.x;
  a.w = c.w;
  a.bias = c.bias;
  a.y = c.y;
  a.N = c.xd.n;
  a.C = c.xd.c;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.Cs = c.xd.cs;
  a.P = c.yd.h;
  a.Q = c.yd.w;
  a.R = c.r;
  a.S = c.s;
  a.stride = c.stride;
  a.pad = c.pad;
  a.act = c.act;
  a.C8 = (a.C + 7) / 8 * 8;
  long long total = c.xd.layout == NCHW ? (long long)a.N * a.C * a.P * a.Q
                                        : (long long)a.N * a.P * a.Q * (a.C8 / 8);
  dim3 grid((unsigned)((total + 255) / 256));
  switch (c.xd.layout) {
    case NCHW: SN_LAUNCH((dw_kernel<T, NCHW>), grid, dim3(256), 0, st, a); break;
    case NHWC: SN_LAUNCH((dw_kernel<T, NHWC>), grid, dim3(256), 0, st, a); break;
    case NC8: SN_LAUNCH((dw_kernel<T, NC8>), grid, dim3(256), 0, st, a); break;
  }
}

bool dwconv3x3_vec(int dtype, const ConvArgs& c, int qs, hipStream_t st);  // dwconv.hip

void dwconv(int dtype, const ConvArgs& c, int param, hipStream_t st) {
  check(!c.res, "depthwise routine takes no residual");
  if (dwconv3x3_vec(dtype, c, param > 0 ? dw_strip_len(param) : 0, st)) return;
  check(param == 0, "depthwise strip parameter needs the strip kernel");
  if (dtype == 0) dw_dispatch<float>(c, st);
  else if (dtype == 1) dw_dispatch<f16>(c, st);
  else dw_dispatch<bf16>(c, st);
}

}  // namespace k
}  // namespace sn
