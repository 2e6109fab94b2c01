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
#include <algorithm>
#include <stdexcept>
#include <string>

#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

static void check(bool ok, const char* what) {
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

// ------------------------------------------------------------------ implicit GEMM
// GEMM view: rows m = (n, p, q) output pixels, columns = output channels,
// reduction = (r, s, c).  One workgroup (4 waves, 2 x 2) computes a BM x BN
// tile; each wave a (BM/2) x (BN/2) sub-tile of 16 x 16 MFMA blocks.  The
// reduction advances 32 elements (4 chunks of 8 channels) per step through
// double-buffered LDS tiles: A is gathered from the input (im2col on the
// fly), B streams from the prepared weights.
struct IgArgs {
  const void* x;
  const void* w;
  const float* bias;
  void* y;
  int C, H, W, Cs;     // input channels, spatial size, stored channels
  int K, P, Q, Ks;     // output channels (real), spatial size, stored channels
  int R, S, stride, pad, act;
  int M, Ng, CB, KC, Kred;  // rows, GEMM columns, chunks/tap, chunks total, weight row length
  int PQ;
  long long x_bs, w_bs, y_bs;  // per-blockIdx.z offsets (batched GEMM), elements
  int vec;                     // A chunks are aligned 8-element vectors (NHWC, C % 8 == 0)
};

struct ChunkPos {
  int r, s, cb;
};
__device__ __forceinline__ void chunk_set(ChunkPos& p, int g, int CB, int S) {
  p.cb = g % CB;
  int rs = g / CB;
  p.r = rs / S;
  p.s = rs - p.r * S;
}
__device__ __forceinline__ void chunk_adv4(ChunkPos& p, int CB, int S) {
  p.cb += 4;
  while (p.cb >= CB) {
    p.cb -= CB;
    if (++p.s == S) {
      p.s = 0;
      ++p.r;
    }
  }
}

template <typename T, int L, int BM, int BN, bool RAW>
__global__ __launch_bounds__(256) void igemm_kernel(IgArgs a) {
  constexpr int BK = 32;
  constexpr bool F32 = std::is_same<T, float>::value;
  constexpr int LDK = BK + (F32 ? 4 : 8);
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int NSA = BM / 64, NSB = BN / 64;  // 8-element chunks per thread
  constexpr int CPAD = F32 ? 4 : 8;
  constexpr int SM_AB = 2 * (BM + BN) * LDK * (int)sizeof(T);
  constexpr int SM_C = BM * (BN + CPAD) * (int)sizeof(T);
  constexpr int SM = SM_AB > SM_C ? SM_AB : SM_C;
  __shared__ __attribute__((aligned(16))) char smem[SM];
  T(*As)[BM][LDK] = reinterpret_cast<T(*)[BM][LDK]>(smem);
  T(*Bs)[BN][LDK] = reinterpret_cast<T(*)[BN][LDK]>(smem + 2 * BM * LDK * sizeof(T));

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x) + blockIdx.z * a.x_bs;
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w) + blockIdx.z * a.w_bs;

  constexpr bool VEC_L = (L == NC8);
  const bool vec = VEC_L || (L == NHWC && a.vec);

  // per-slot A state: row decode and reduction position
  int arow[NSA], aj[NSA], aimg[NSA], ah0[NSA], aw0[NSA];
  bool arv[NSA];
  ChunkPos apos[NSA];
#pragma unroll
  for (int i = 0; i < NSA; ++i) {
    if (vec) {
      arow[i] = (tid >> 2) + 64 * i;
      aj[i] = tid & 3;
    } else {
      arow[i] = tid % BM;
      aj[i] = (tid / BM) * NSA + i;
    }
    int m = m0 + arow[i];
    arv[i] = m < a.M;
    int mm = arv[i] ? m : 0;
    int img = mm / a.PQ, pq = mm - img * a.PQ;
    int p = pq / a.Q, q = pq - p * a.Q;
    aimg[i] = img;
    ah0[i] = p * a.stride - a.pad;
    aw0[i] = q * a.stride - a.pad;
    chunk_set(apos[i], aj[i], a.CB, a.S);
  }

  V8<T> ra[NSA], rb[NSB];
  auto load_a = [&](int kt) {
#pragma unroll
    for (int i = 0; i < NSA; ++i) {
      const int g = kt * 4 + aj[i];
      const int h = ah0[i] + apos[i].r, ww = aw0[i] + apos[i].s;
      const bool ok = arv[i] && g < a.KC && (unsigned)h < (unsigned)a.H && (unsigned)ww < (unsigned)a.W;
      if (vec) {
        if (ok) {
          const T* p;
          if constexpr (L == NC8)
            p = x + ((((long long)aimg[i] * a.CB + apos[i].cb) * a.H + h) * a.W + ww) * 8;
          else
            p = x + (((long long)aimg[i] * a.H + h) * a.W + ww) * a.Cs + apos[i].cb * 8;
          ra[i] = ld8(p);
        } else {
          ra[i] = zero8<T>();
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int c = apos[i].cb * 8 + e;
          T v = (T)0.f;
          if (ok && c < a.C) {
            if constexpr (L == NCHW)
              v = x[(((long long)aimg[i] * a.Cs + c) * a.H + h) * a.W + ww];
            else
              v = x[(((long long)aimg[i] * a.H + h) * a.W + ww) * a.Cs + c];
          }
          ra[i].v[e] = v;
        }
      }
    }
  };
  auto load_b = [&](int kt) {
#pragma unroll
    for (int i = 0; i < NSB; ++i) {
      const int row = (tid >> 2) + 64 * i, j = tid & 3;
      const int g = kt * 4 + j, n = n0 + row;
      if (n < a.Ng && g < a.KC)
        rb[i] = ld8(w + (long long)n * a.Kred + g * 8);
      else
        rb[i] = zero8<T>();
    }
  };
  auto store_ab = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NSA; ++i) st8(&As[buf][arow[i]][aj[i] * 8], ra[i]);
#pragma unroll
    for (int i = 0; i < NSB; ++i) st8(&Bs[buf][(tid >> 2) + 64 * i][(tid & 3) * 8], rb[i]);
  };
  auto advance = [&]() {
#pragma unroll
    for (int i = 0; i < NSA; ++i) chunk_adv4(apos[i], a.CB, a.S);
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = (a.KC + 3) / 4;
  load_a(0);
  load_b(0);
  store_ab(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) {
      advance();
      load_a(kt + 1);
      load_b(kt + 1);
    }
#pragma unroll
    for (int ks = 0; ks < BK / Mfma<T>::KSTEP; ++ks) {
      typename Mfma<T>::frag fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int r = wm * WTM + i * 16 + (lane & 15);
        if constexpr (F32)
          fa[i] = As[buf][r][ks * 4 + (lane >> 4)];
        else
          fa[i] = *reinterpret_cast<const typename Mfma<T>::frag*>(&As[buf][r][ks * 32 + (lane >> 4) * 8]);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int r = wn * WTN + j * 16 + (lane & 15);
        if constexpr (F32)
          fb[j] = Bs[buf][r][ks * 4 + (lane >> 4)];
        else
          fb[j] = *reinterpret_cast<const typename Mfma<T>::frag*>(&Bs[buf][r][ks * 32 + (lane >> 4) * 8]);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(fa[i], fb[j], acc[i][j]);
    }
    if (kt + 1 < KT) store_ab(buf ^ 1);
    __syncthreads();
  }

  // accumulator element (i, j, v) is C[wm*WTM + i*16 + (lane>>4)*4 + v][wn*WTN + j*16 + (lane&15)]
  if constexpr (RAW) {
    float* __restrict__ y = reinterpret_cast<float*>(a.y) + blockIdx.z * a.y_bs;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int n = n0 + wn * WTN + j * 16 + (lane & 15);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = m0 + wm * WTM + i * 16 + (lane >> 4) * 4 + v;
          if (m < a.M && n < a.Ng) y[(long long)m * a.Ng + n] = acc[i][j][v];
        }
      }
    return;
  } else {
    T(*Cs)[BN + CPAD] = reinterpret_cast<T(*)[BN + CPAD]>(smem);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nl = wn * WTN + j * 16 + (lane & 15);
      const int n = n0 + nl;
      const float bv = n < a.Ng ? a.bias[n] : 0.f;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int ml = wm * WTM + i * 16 + (lane >> 4) * 4 + v;
          Cs[ml][nl] = from_f<T>(act_f(acc[i][j][v] + bv, a.act));
        }
    }
    __syncthreads();
    T* __restrict__ y = reinterpret_cast<T*>(a.y) + blockIdx.z * a.y_bs;
    if constexpr (L == NCHW) {
      const int row = tid % BM, m = m0 + row;
      if (m < a.M) {
        const int img = m / a.PQ, pq = m - img * a.PQ;
        T* yb = y + (long long)img * a.Ks * a.PQ + pq;
        for (int col = tid / BM; col < BN; col += 256 / BM) {
          const int n = n0 + col;
          if (n < a.Ng) yb[(long long)n * a.PQ] = Cs[row][col];
        }
      }
    } else if (L == NC8 || a.Ks % 8 == 0) {
      for (int idx = tid; idx < BM * BN / 8; idx += 256) {
        const int row = idx / (BN / 8), cj = idx % (BN / 8);
        const int m = m0 + row, n = n0 + cj * 8;
        if (m >= a.M || n >= a.Ng) continue;
        V8<T> v = ld8(&Cs[row][cj * 8]);
        if constexpr (L == NC8) {
          const int img = m / a.PQ, pq = m - img * a.PQ;
          st8(y + (((long long)img * (a.Ks >> 3) + (n >> 3)) * a.PQ + pq) * 8, v);
        } else {
          st8(y + (long long)m * a.Ks + n, v);
        }
      }
    } else {
      for (int idx = tid; idx < BM * BN; idx += 256) {
        const int row = idx / BN, col = idx % BN;
        const int m = m0 + row, n = n0 + col;
        if (m < a.M && n < a.Ng) y[(long long)m * a.Ks + n] = Cs[row][col];
      }
    }
  }
}

template <typename T, int L, int BM, int BN, bool RAW>
static void igemm_go(const IgArgs& a, int batch, hipStream_t st) {
  dim3 grid((a.M + BM - 1) / BM, (a.Ng + BN - 1) / BN, batch);
  hipLaunchKernelGGL((igemm_kernel<T, L, BM, BN, RAW>), grid, dim3(256), 0, st, a);
}

template <typename T, int L, bool RAW>
static void igemm_tiles(int bm, int bn, const IgArgs& a, int batch, hipStream_t st) {
  if constexpr (std::is_same<T, float>::value) {
    check(bm == 64 && bn == 64, "fp32 implicit GEMM has one 64x64 tile");
    igemm_go<T, L, 64, 64, RAW>(a, batch, st);
  } else {
    if (bm == 128 && bn == 128)
      igemm_go<T, L, 128, 128, RAW>(a, batch, st);
    else if (bm == 64 && bn == 64)
      igemm_go<T, L, 64, 64, RAW>(a, batch, st);
    else if (bm == 128 && bn == 64)
      igemm_go<T, L, 128, 64, RAW>(a, batch, st);
    else
      check(false, "unknown implicit-GEMM tile");
  }
}

static IgArgs make_ig(const ConvArgs& c) {
  IgArgs a{};
  a.x = c.x;
  a.w = c.w;
  a.bias = c.bias;
  a.y = c.y;
  a.C = c.xd.c;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.Cs = c.xd.cs;
  a.K = c.yd.c;
  a.P = c.yd.h;
  a.Q = c.yd.w;
  a.Ks = c.yd.cs;
  a.R = c.r;
  a.S = c.s;
  a.stride = c.stride;
  a.pad = c.pad;
  a.act = c.act;
  a.PQ = a.P * a.Q;
  a.M = c.xd.n * a.PQ;
  a.Ng = c.yd.layout == NC8 ? c.yd.cs : c.yd.c;
  a.CB = (a.C + 7) / 8;
  a.KC = a.R * a.S * a.CB;
  a.Kred = a.KC * 8;
  a.vec = (c.xd.layout == NHWC && a.C % 8 == 0) ? 1 : 0;
  return a;
}

template <typename T>
static void igemm_dispatch(int bm, int bn, const ConvArgs& c, hipStream_t st) {
  IgArgs a = make_ig(c);
  check(c.xd.layout == c.yd.layout, "implicit GEMM reads and writes one layout");
  check((long long)a.M * a.Ks < (1ll << 31) && (long long)c.xd.n * a.Cs * a.H * a.W < (1ll << 31),
        "tensor too large");
  switch (c.xd.layout) {
    case NCHW: igemm_tiles<T, NCHW, false>(bm, bn, a, 1, st); break;
    case NHWC: igemm_tiles<T, NHWC, false>(bm, bn, a, 1, st); break;
    case NC8: igemm_tiles<T, NC8, false>(bm, bn, a, 1, st); break;
    default: check(false, "layout");
  }
}

void conv_igemm(int dtype, int bm, int bn, const ConvArgs& c, hipStream_t st) {
  if (dtype == 0) igemm_dispatch<float>(bm, bn, c, st);
  else if (dtype == 1) igemm_dispatch<f16>(bm, bn, c, st);
  else igemm_dispatch<bf16>(bm, bn, c, st);
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
    out[j] = from_f<T>(act_f(acc[j] + (n < a.Ng ? a.bias[n] : 0.f), a.act));
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
    case NCHW: hipLaunchKernelGGL((direct_kernel<T, NCHW>), grid, dim3(256), 0, st, a); break;
    case NHWC: hipLaunchKernelGGL((direct_kernel<T, NHWC>), grid, dim3(256), 0, st, a); break;
    case NC8: hipLaunchKernelGGL((direct_kernel<T, NC8>), grid, dim3(256), 0, st, a); break;
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
#pragma unroll
  for (int e0 = 0; e0 < 1; ++e0) {
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

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t winograd_ws_bytes(int dtype, const TDesc& xd, int k) {
  const long long T = (long long)xd.n * ((xd.h + 1) / 2) * ((xd.w + 1) / 2);
  const long long C8 = (xd.c + 7) / 8 * 8;
  const long long Kp = (k + 7) / 8 * 8;
  const size_t es = dtype == 0 ? 4 : 2;
  return align256(16 * T * C8 * es) + align256(16 * T * Kp * 4);
}

template <typename T>
static void wino_dispatch(int dtype, const ConvArgs& c, hipStream_t st) {
  check(c.r == 3 && c.s == 3 && c.stride == 1 && c.pad == 1, "Winograd F(2x2,3x3) needs 3x3/1 pad 1");
  check(c.xd.layout == c.yd.layout, "Winograd reads and writes one layout");
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
  a.TH = (a.H + 1) / 2;
  a.TW = (a.W + 1) / 2;
  a.T = a.N * a.TH * a.TW;
  a.Ng = c.yd.layout == NC8 ? c.yd.cs : c.yd.c;
  a.Ks = c.yd.cs;
  a.act = c.act;
  const int Kp = (c.yd.c + 7) / 8 * 8;
  const size_t es = sizeof(T);
  const size_t vbytes = align256(16ull * a.T * a.C8 * es);
  check(c.ws && c.ws_bytes >= winograd_ws_bytes(dtype, c.xd, c.yd.c), "Winograd workspace too small");
  check(16ll * a.T * std::max(a.C8, Kp) < (1ll << 31), "tensor too large");
  a.v = c.ws;
  float* mbuf = reinterpret_cast<float*>(reinterpret_cast<char*>(c.ws) + vbytes);
  a.m = mbuf;
  const int CB = a.C8 / 8, NB = (a.Ng + 7) / 8;
  dim3 gin((unsigned)(((long long)a.T * CB + 255) / 256));
  dim3 gout((unsigned)(((long long)a.T * NB + 255) / 256));
  // batched GEMM: A = V_xi as a [T][C8] matrix (1x1 "NHWC" convolution), B = U_xi [Kp][C8]
  IgArgs g{};
  g.x = a.v;
  g.w = c.w;
  g.bias = c.bias;
  g.y = mbuf;
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
  g.CB = CB;
  g.KC = CB;
  g.Kred = a.C8;
  g.x_bs = (long long)a.T * a.C8;
  g.w_bs = (long long)Kp * a.C8;
  g.y_bs = (long long)a.T * a.Ng;
  g.vec = 1;
  switch (c.xd.layout) {
    case NCHW: hipLaunchKernelGGL((wino_in_kernel<T, NCHW>), gin, dim3(256), 0, st, a); break;
    case NHWC: hipLaunchKernelGGL((wino_in_kernel<T, NHWC>), gin, dim3(256), 0, st, a); break;
    case NC8: hipLaunchKernelGGL((wino_in_kernel<T, NC8>), gin, dim3(256), 0, st, a); break;
  }
  if constexpr (std::is_same<T, float>::value)
    igemm_tiles<T, NHWC, true>(64, 64, g, 16, st);
  else
    igemm_tiles<T, NHWC, true>(a.T >= 4096 ? 128 : 64, a.Ng >= 128 && a.T >= 4096 ? 128 : 64, g, 16, st);
  switch (c.xd.layout) {
    case NCHW: hipLaunchKernelGGL((wino_out_kernel<T, NCHW>), gout, dim3(256), 0, st, a); break;
    case NHWC: hipLaunchKernelGGL((wino_out_kernel<T, NHWC>), gout, dim3(256), 0, st, a); break;
    case NC8: hipLaunchKernelGGL((wino_out_kernel<T, NC8>), gout, dim3(256), 0, st, a); break;
  }
}

void conv_winograd(int dtype, const ConvArgs& c, hipStream_t st) {
  if (dtype == 0) wino_dispatch<float>(dtype, c, st);
  else if (dtype == 1) wino_dispatch<f16>(dtype, c, st);
  else wino_dispatch<bf16>(dtype, c, st);
}

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
    case NCHW: hipLaunchKernelGGL((dw_kernel<T, NCHW>), grid, dim3(256), 0, st, a); break;
    case NHWC: hipLaunchKernelGGL((dw_kernel<T, NHWC>), grid, dim3(256), 0, st, a); break;
    case NC8: hipLaunchKernelGGL((dw_kernel<T, NC8>), grid, dim3(256), 0, st, a); break;
  }
}

void dwconv(int dtype, const ConvArgs& c, hipStream_t st) {
  if (dtype == 0) dw_dispatch<float>(c, st);
  else if (dtype == 1) dw_dispatch<f16>(c, st);
  else dw_dispatch<bf16>(c, st);
}

}  // namespace k
}  // namespace sn
