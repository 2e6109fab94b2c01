// Implicit-GEMM convolution kernels (register-staged and LDS-DMA tiles),
// their routine-parameter table and the host-side dispatch templates.  The
// 16-bit instantiations are compiled in their own translation units
// (conv_igemm_f16.hip, conv_igemm_bf16.hip) so the largest kernel families
// build in parallel; conv.hip holds the public entry points.
#pragma once
#include <algorithm>
#include <stdexcept>
#include <string>
#include <type_traits>

#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

// ------------------------------------------------------------------ implicit GEMM
// GEMM view: rows m = (n, p, q) output pixels, columns = output channels,
// reduction = (r, s, c).  One workgroup (4 waves, 2 x 2) computes a BM x BN
// tile; each wave a (BM/2) x (BN/2) sub-tile of 16 x 16 MFMA blocks.  The
// reduction advances BK elements (BK/8 chunks of 8 channels) per step
// through double-buffered LDS tiles: A is gathered from the input (im2col on
// the fly), B streams from the prepared weights; the next step's global
// loads are issued before the current step's MFMAs.  Workgroups are ordered
// so that each XCD (L2 domain) works on a contiguous group of tiles that
// share input rows, and small problems split the reduction over several
// workgroups (fp32 partial tiles, summed by a second kernel).
struct IgArgs {
  const void* x;
  const void* w;
  const float* bias;
  void* y;
  float* part;         // split-K partial tiles [splits][M][Ng]
  int C, H, W, Cs;     // input channels, spatial size, stored channels
  int K, P, Q, Ks;     // output channels (real), spatial size, stored channels
  int R, S, stride, pad, act;
  int M, Ng, CB, KC, Kred;  // rows, GEMM columns, chunks/tap, chunks total, weight row length
  int PQ;
  int tiles_m, tiles_n, splits, kt_per;  // grid decomposition
  long long x_bs, w_bs, y_bs;  // per-blockIdx.z offsets (batched GEMM), elements
  int vec;                     // NHWC input with C % 8 == 0 (aligned 8-channel vectors)
  long long x_elems, w_elems;  // elements addressable per blockIdx.z (buffer ranges)
  long long y_elems;
  float inv_pq, inv_q;         // 1/(P*Q), 1/Q for sdiv
  const void* res;             // residual [M][Ng] in the output layout, or null
  unsigned* cnt;               // EPI_FIXUP: per-tile arrival counters (zero between launches)
  // projected shortcut (LDS-DMA kernel): x2 [N][H2][W2][Cs2] (or NC8HW8) read
  // at stride2 by a 1 x 1 convolution with weights w2 [Kp][C2_8], its KC2
  // chunks of 8 channels reduced after the KC chunks of the convolution
  const void* x2;
  const void* w2;
  int H2, W2, Cs2, CB2, stride2, KC2, Kred2;
  long long x2_elems, w2_elems;
};

// Element offset of GEMM position (m, n) in the output tensor's layout (the
// residual has the output's shape and layout).
template <int L>
__device__ __forceinline__ long long out_index(const IgArgs& a, int m, int n) {
  if constexpr (L == NHWC) {
    return (long long)m * a.Ks + n;
  } else {
    const int img = m / a.PQ, pq = m - img * a.PQ;
    if constexpr (L == NCHW) return ((long long)img * a.Ks + n) * a.PQ + pq;
    else return (((long long)img * (a.Ks >> 3) + (n >> 3)) * a.PQ + pq) * 8 + (n & 7);
  }
}

// Residual values of channels n..n+3 of row m (zero outside the tensor).
template <typename T, int L>
__device__ __forceinline__ void residual4(const IgArgs& a, int m, int n, float (&r)[4]) {
  const T* rp = reinterpret_cast<const T*>(a.res);
#pragma unroll
  for (int v = 0; v < 4; ++v) r[v] = 0.f;
  if (m >= a.M) return;
  if (L != NCHW && n + 4 <= a.Ng && (L == NC8 || (a.Ks & 3) == 0)) {
    // 4 consecutive channels: 8 bytes (16-bit types) or 16 bytes (fp32)
    T t[4];
    if constexpr (sizeof(T) == 2) {
      const u32x2 w = *reinterpret_cast<const u32x2*>(rp + out_index<L>(a, m, n));
      __builtin_memcpy(t, &w, 8);
    } else {
      const u32x4 w = *reinterpret_cast<const u32x4*>(rp + out_index<L>(a, m, n));
      __builtin_memcpy(t, &w, 16);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) r[v] = to_f(t[v]);
  } else {
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (n + v < a.Ng) r[v] = to_f(rp[out_index<L>(a, m, n + v)]);
  }
}

template <typename T>
__device__ __forceinline__ V8<T> bload8(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
  V8<T> out;
  auto v0 = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, soff, 0);
  __builtin_memcpy(&out, &v0, 16);
  if constexpr (sizeof(T) == 4) {
    auto v1 = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(voff + 16), soff, 0);
    __builtin_memcpy(reinterpret_cast<char*>(&out) + 16, &v1, 16);
  }
  return out;
}

struct ChunkPos {
  int r, s, cb;
};
__device__ __forceinline__ void chunk_set(ChunkPos& p, int g, int CB, int S) {
  p.cb = g % CB;
  int rs = g / CB;
  p.r = rs / S;
  p.s = rs - p.r * S;
}
__device__ __forceinline__ void chunk_adv(ChunkPos& p, int step, int CB, int S) {
  p.cb += step;
  while (p.cb >= CB) {
    p.cb -= CB;
    if (++p.s == S) {
      p.s = 0;
      ++p.r;
    }
  }
}

// Read-only zero page: masked-off lanes load from here, so every global load
// is unconditional (no divergent branches around loads, which would force
// the compiler to drain all outstanding loads).
__device__ __attribute__((aligned(256))) unsigned char g_zero_page[256];


template <typename T, int L, bool VEC, bool ALIGNED, int BM, int BN, int BK, int EPI, int PF>
__global__ __launch_bounds__(256) void igemm_kernel(IgArgs a) {
  constexpr bool F32 = std::is_same<T, float>::value;
  constexpr int CPR = BK / 8;                   // chunks per tile row
  // 16-bit tiles: unpadded rows of BK elements with the 16-byte chunk slot
  // XOR-swizzled by the row, so both the 16-byte stores (consecutive chunks
  // of a few rows) and the MFMA fragment reads (one chunk of 16 rows) hit
  // distinct LDS banks.  fp32 tiles use padded rows instead.
  constexpr int LDK = BK + (F32 ? 4 : 0);
  constexpr int RPR = F32 || BK > 64 ? 1 : 2;  // rows sharing one chunk XOR key
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int NA = BM * CPR / 256;            // A chunks per thread
  constexpr int NB = BN * CPR / 256;            // B chunks per thread
  constexpr int RS = VEC ? NA : 1;              // distinct A rows per thread
  constexpr int CS = VEC ? 1 : NA;              // distinct A chunks per thread
  static_assert(NA >= 1 && NB >= 1 && (VEC || 256 % BM == 0), "tile too small for 256 threads");
  static_assert(PF >= 2 && PF % 2 == 0, "prefetch depth must be even (LDS double buffer parity)");
  constexpr int CPAD = F32 ? 4 : 8;
  // SWAP: weights are the MFMA's first operand, so each lane's 4 accumulator
  // values are 4 consecutive output channels of one pixel (channel-vector
  // layouts); otherwise 4 consecutive pixels of one channel (NCHW).
  constexpr bool SWAP = L != NCHW;
  constexpr int SM_AB = 2 * (BM + BN) * LDK * (int)sizeof(T);
  constexpr int SM_C = EPI == EPI_LAYOUT ? BM * (BN + CPAD) * (int)sizeof(T) : 0;
  constexpr int SM = SM_AB > SM_C ? SM_AB : SM_C;
  __shared__ __attribute__((aligned(16))) char smem[SM];
  T(*As)[BM][LDK] = reinterpret_cast<T(*)[BM][LDK]>(smem);
  T(*Bs)[BN][LDK] = reinterpret_cast<T(*)[BN][LDK]>(smem + 2 * BM * LDK * sizeof(T));
  auto slot = [](int row, int chunk) { return F32 ? chunk : chunk ^ ((row / RPR) % CPR); };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int wm = wave >> 1, wn = wave & 1;
  int mt, nt;
  tile_of(blockIdx.x, a.tiles_m, a.tiles_n, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int split = blockIdx.y;
  const int KT_all = (a.KC + CPR - 1) / CPR;
  const int kt0 = split * a.kt_per;
  const int KT = min(KT_all - kt0, a.kt_per);
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x) + blockIdx.z * a.x_bs;
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w) + blockIdx.z * a.w_bs;

  // A: thread -> (rows, chunk columns) of the tile
  int arow[RS], aimg[RS], ah0[RS], aw0[RS];
  bool arv[RS];
  int aj[CS];
  ChunkPos apos[CS];
#pragma unroll
  for (int i = 0; i < RS; ++i) {
    arow[i] = VEC ? (tid / CPR + (256 / CPR) * i) : (tid % BM);
    const int m = m0 + arow[i];
    arv[i] = m < a.M;
    const int mm = arv[i] ? m : 0;
    const int img = mm / a.PQ, pq = mm - img * a.PQ;
    const int p = pq / a.Q, q = pq - p * a.Q;
    aimg[i] = img;
    ah0[i] = p * a.stride - a.pad;
    aw0[i] = q * a.stride - a.pad;
  }
#pragma unroll
  for (int c = 0; c < CS; ++c) {
    aj[c] = VEC ? tid % CPR : (tid / BM) * CS + c;
    if constexpr (!ALIGNED) chunk_set(apos[c], kt0 * CPR + aj[c], a.CB, a.S);
  }
  // ALIGNED (C % BK == 0, R*S <= 32): every reduction step lies inside one
  // filter tap, so the tap (r, s) and first channel block cb0 are uniform per
  // step; each A row keeps its byte offset and a bitmask of the taps that
  // fall inside the (unpadded) input.
  const T* zp = reinterpret_cast<const T*>(g_zero_page);
  constexpr int ES = (int)sizeof(T);
  unsigned rbyte[RS], tvm[RS];
  ChunkPos upos{0, 0, 0};
  __amdgpu_buffer_rsrc_t rx = make_rsrc(x, a.x_elems * ES);
  __amdgpu_buffer_rsrc_t rw = make_rsrc(w, a.w_elems * ES);
  if constexpr (ALIGNED) {
#pragma unroll
    for (int i = 0; i < RS; ++i) {
      int e;
      if constexpr (L == NC8)
        e = (aimg[i] * a.CB * a.H * a.W + ah0[i] * a.W + aw0[i]) * 8 + aj[0] * a.H * a.W * 8;
      else
        e = ((aimg[i] * a.H + ah0[i]) * a.W + aw0[i]) * a.Cs + aj[0] * 8;
      rbyte[i] = (unsigned)(e * ES);
      unsigned m = 0;
      for (int r = 0; r < a.R; ++r)
        for (int q = 0; q < a.S; ++q)
          if (arv[i] && (unsigned)(ah0[i] + r) < (unsigned)a.H && (unsigned)(aw0[i] + q) < (unsigned)a.W)
            m |= 1u << (r * a.S + q);
      tvm[i] = m;
    }
    chunk_set(upos, kt0 * CPR, a.CB, a.S);
  }
  unsigned bbyte[NB];
  int brow[NB];
  bool bv[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int row = tid / CPR + (256 / CPR) * i;
    bv[i] = n0 + row < a.Ng;
    brow[i] = (n0 + row) * a.Kred + (tid % CPR) * 8;
    bbyte[i] = bv[i] ? (unsigned)(brow[i] * ES) : kOOB;
  }

  // PF register staging sets: the loads of step t+1 are issued PF-1 steps
  // before they are stored to LDS (prefetch distance PF, LDS double buffer)
  V8<T> ra[PF][NA], rb[PF][NB];
  auto load_a = [&](V8<T>(&rs)[NA], int kt) {
    if constexpr (ALIGNED) {
      int tap;
      if constexpr (L == NC8)
        tap = upos.cb * a.H * a.W * 8 + (upos.r * a.W + upos.s) * 8;
      else
        tap = (upos.r * a.W + upos.s) * a.Cs + upos.cb * 8;
      const unsigned tb = (unsigned)(tap * ES);
      const int t = upos.r * a.S + upos.s;
#pragma unroll
      for (int i = 0; i < RS; ++i) {
        const unsigned off = ((tvm[i] >> t) & 1u) ? rbyte[i] + tb : kOOB;
        rs[i] = bload8<T>(rx, off, 0);
      }
      // next step: channel blocks advance by CPR; CB is a multiple of CPR
      upos.cb += CPR;
      if (upos.cb == a.CB) {
        upos.cb = 0;
        if (++upos.s == a.S) {
          upos.s = 0;
          ++upos.r;
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < RS; ++i)
#pragma unroll
      for (int c = 0; c < CS; ++c) {
        const int slot = i * CS + c;
        const int g = kt * CPR + aj[c];
        const int h = ah0[i] + apos[c].r, ww = aw0[i] + apos[c].s;
        const bool ok = arv[i] && g < a.KC && (unsigned)h < (unsigned)a.H && (unsigned)ww < (unsigned)a.W;
        if constexpr (VEC) {
          const T* p;
          if constexpr (L == NC8)
            p = x + ((((long long)aimg[i] * a.CB + apos[c].cb) * a.H + h) * a.W + ww) * 8;
          else
            p = x + (((long long)aimg[i] * a.H + h) * a.W + ww) * a.Cs + apos[c].cb * 8;
          rs[slot] = ld8(ok ? p : zp);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int ch = apos[c].cb * 8 + e;
            T v = (T)0.f;
            if (ok && ch < a.C) {
              if constexpr (L == NCHW)
                v = x[(((long long)aimg[i] * a.Cs + ch) * a.H + h) * a.W + ww];
              else if constexpr (L == NHWC)
                v = x[(((long long)aimg[i] * a.H + h) * a.W + ww) * a.Cs + ch];
              else
                v = x[((((long long)aimg[i] * a.CB + (ch >> 3)) * a.H + h) * a.W + ww) * 8 + (ch & 7)];
            }
            rs[slot].v[e] = v;
          }
        }
      }
#pragma unroll
    for (int c = 0; c < CS; ++c) chunk_adv(apos[c], CPR, a.CB, a.S);
  };
  auto load_b = [&](V8<T>(&rs)[NB], int kt) {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if constexpr (ALIGNED) {
        rs[i] = bload8<T>(rw, bbyte[i], kt * BK * ES);
      } else {
        const bool ok = bv[i] && kt * CPR + (tid % CPR) < a.KC;
        rs[i] = ld8(ok ? w + (brow[i] + kt * BK) : zp);
      }
    }
  };
  auto store_ab = [&](const V8<T>(&sa)[NA], const V8<T>(&sb)[NB], int buf) {
#pragma unroll
    for (int i = 0; i < RS; ++i)
#pragma unroll
      for (int c = 0; c < CS; ++c) st8(&As[buf][arow[i]][slot(arow[i], aj[c]) * 8], sa[i * CS + c]);
#pragma unroll
    for (int i = 0; i < NB; ++i)
      st8(&Bs[buf][tid / CPR + (256 / CPR) * i][slot(tid / CPR + (256 / CPR) * i, tid % CPR) * 8], sb[i]);
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < BK / Mfma<T>::KSTEP; ++ks) {
      typename Mfma<T>::frag fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int r = wm * WTM + i * 16 + (lane & 15);
        if constexpr (F32)
          fa[i] = As[buf][r][ks * 4 + (lane >> 4)];
        else
          fa[i] = *reinterpret_cast<const typename Mfma<T>::frag*>(&As[buf][r][slot(r, ks * 4 + (lane >> 4)) * 8]);
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int r = wn * WTN + j * 16 + (lane & 15);
        if constexpr (F32)
          fb[j] = Bs[buf][r][ks * 4 + (lane >> 4)];
        else
          fb[j] = *reinterpret_cast<const typename Mfma<T>::frag*>(&Bs[buf][r][slot(r, ks * 4 + (lane >> 4)) * 8]);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = SWAP ? Mfma<T>::run(fb[j], fa[i], acc[i][j]) : Mfma<T>::run(fa[i], fb[j], acc[i][j]);
    }
  };

  // step t: store tile t+1 (register set (t+1) % PF, loaded PF-1 steps
  // earlier) into LDS[(t+1)&1], issue the loads of tile t+PF into set t % PF
  // (tile t went to LDS at step t-1), compute LDS[t&1]; one barrier per step
#pragma unroll
  for (int u = 0; u < PF; ++u)
    if (u < KT) {
      load_a(ra[u], kt0 + u);
      load_b(rb[u], kt0 + u);
    }
  if (KT > 0) store_ab(ra[0], rb[0], 0);
  lds_barrier();
  for (int it0 = 0; it0 < KT; it0 += PF) {
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int t = it0 + u;
      if (t < KT) {
        if (t + 1 < KT) store_ab(ra[(u + 1) % PF], rb[(u + 1) % PF], (u + 1) & 1);
        if (t + PF < KT) {
          load_a(ra[u], kt0 + t + PF);
          load_b(rb[u], kt0 + t + PF);
        }
        compute(u & 1);
        lds_barrier();
      }
    }
  }

  // accumulator element (i, j, v):
  //   !SWAP: C[wm*WTM + i*16 + (lane>>4)*4 + v][wn*WTN + j*16 + (lane&15)]
  //    SWAP: C[wm*WTM + i*16 + (lane&15)][wn*WTN + j*16 + (lane>>4)*4 + v]
  if constexpr (EPI != EPI_LAYOUT) {
    float* __restrict__ y = EPI == EPI_RAW ? reinterpret_cast<float*>(a.y) + blockIdx.z * a.y_bs
                                           : a.part + (long long)split * a.M * a.Ng;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        if constexpr (SWAP) {
          const int m = m0 + wm * WTM + i * 16 + (lane & 15);
          const int n = n0 + wn * WTN + j * 16 + (lane >> 4) * 4;
          if (m < a.M) {
            if (n + 4 <= a.Ng && (a.Ng & 3) == 0) {
              *reinterpret_cast<f32x4*>(y + (long long)m * a.Ng + n) = acc[i][j];
            } else {
#pragma unroll
              for (int v = 0; v < 4; ++v)
                if (n + v < a.Ng) y[(long long)m * a.Ng + n + v] = acc[i][j][v];
            }
          }
        } else {
          const int n = n0 + wn * WTN + j * 16 + (lane & 15);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + wm * WTM + i * 16 + (lane >> 4) * 4 + v;
            if (m < a.M && n < a.Ng) y[(long long)m * a.Ng + n] = acc[i][j][v];
          }
        }
      }
    return;
  } else {
    T(*Cs)[BN + CPAD] = reinterpret_cast<T(*)[BN + CPAD]>(smem);
    if constexpr (SWAP) {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int nl = wn * WTN + j * 16 + (lane >> 4) * 4;
        float bv[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) bv[v] = n0 + nl + v < a.Ng ? a.bias[n0 + nl + v] : 0.f;
        if (a.res) {
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            const int ml = wm * WTM + i * 16 + (lane & 15);
            float rv[4];
            residual4<T, L>(a, m0 + ml, n0 + nl, rv);
            T o[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = from_f<T>(act_f(acc[i][j][v] + bv[v] + rv[v], a.act));
            __builtin_memcpy(&Cs[ml][nl], o, sizeof(o));
          }
        } else {
#pragma unroll
          for (int i = 0; i < FM; ++i) {
            const int ml = wm * WTM + i * 16 + (lane & 15);
            T o[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = from_f<T>(act_f(acc[i][j][v] + bv[v], a.act));
            __builtin_memcpy(&Cs[ml][nl], o, sizeof(o));
          }
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int nl = wn * WTN + j * 16 + (lane & 15);
        const int n = n0 + nl;
        const float bv = n < a.Ng ? a.bias[n] : 0.f;
        if (a.res) {
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int ml = wm * WTM + i * 16 + (lane >> 4) * 4 + v;
              float rv = 0.f;
              if (m0 + ml < a.M && n < a.Ng)
                rv = to_f(reinterpret_cast<const T*>(a.res)[out_index<L>(a, m0 + ml, n)]);
              Cs[ml][nl] = from_f<T>(act_f(acc[i][j][v] + bv + rv, a.act));
            }
        } else {
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int ml = wm * WTM + i * 16 + (lane >> 4) * 4 + v;
              Cs[ml][nl] = from_f<T>(act_f(acc[i][j][v] + bv, a.act));
            }
        }
      }
    }
    __syncthreads();
    T* __restrict__ y = reinterpret_cast<T*>(a.y) + blockIdx.z * a.y_bs;
    if constexpr (L == NCHW) {
      for (int row = tid % BM; row < BM; row += 256) {
        const int m = m0 + row;
        if (m >= a.M) continue;
        const int img = m / a.PQ, pq = m - img * a.PQ;
        T* yb = y + (long long)img * a.Ks * a.PQ + pq;
        for (int col = tid / BM; col < BN; col += (BM >= 256 ? 1 : 256 / BM)) {
          const int n = n0 + col;
          if (n < a.Ng) yb[(long long)n * a.PQ] = Cs[row][col];
        }
      }
    } else if (L == NC8 || a.Ks % 8 == 0) {
      for (int idx = tid; idx < BM * BN / 8; idx += 256) {
        // NC8HW8: consecutive threads take consecutive pixels of one channel block
        const int row = L == NC8 ? idx % BM : idx / (BN / 8), cj = L == NC8 ? idx / BM : idx % (BN / 8);
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

// ------------------------------------------------------------------ implicit GEMM, LDS DMA
// The same GEMM and routine semantics as igemm_kernel, for 16-bit types in
// the channel-vector layouts (NHWC with C % 8 == 0, NC8HW8) when the channel
// count is a multiple of BK, so every reduction step lies inside one filter
// tap.  The tiles travel from global memory straight into LDS: buffer loads
// with the LDS as destination (16 bytes per lane; offsets beyond the buffer
// range write zeros, which gives the padding halo and the ragged edges), ST
// stages deep.  No registers stage the tiles and no LDS store instructions
// are issued, so the vector-memory and LDS pipes carry only the tile bytes
// and the MFMA operand reads.  One such load fills 1 KB of LDS, the 64 lanes'
// 16 bytes in lane order; the XOR swizzle of the tile rows is therefore
// applied on the global side: the lane that fills LDS slot (row, c) fetches
// logical chunk c ^ swizzle(row).  Each of the 4 waves computes a
// (BM/WM) x (BN/(4/WM)) sub-tile with the weights as the MFMA's first
// operand (4 consecutive output channels of one pixel per lane).

// LDS bytes of an LDS-DMA tile configuration, and the workgroups per CU it
// allows (the occupancy the register allocation is sized for).
// (the epilogue tile: fp32 rows of BN + 4 values, which also hold the
// 16-bit rows of BN + 8 values)
template <int BM, int BN, int BK, int ST, int EPI>
constexpr int dma_lds_bytes() {
  constexpr bool LAYOUT_EPI = EPI == EPI_LAYOUT || EPI == EPI_FIXUP;
  return ST * (BM + BN) * BK * 2 > (LAYOUT_EPI ? BM * (BN + 4) * 4 : 0) ? ST * (BM + BN) * BK * 2
                                                                         : (LAYOUT_EPI ? BM * (BN + 4) * 4 : 0);
}
template <int BM, int BN, int BK, int ST, int EPI, int NWV = 4>
constexpr int dma_occ() {
  return 160 * 1024 / dma_lds_bytes<BM, BN, BK, ST, EPI>() > 16 / NWV ? 16 / NWV
                                                                        : 160 * 1024 / dma_lds_bytes<BM, BN, BK, ST, EPI>();
}

template <int V>
using IC = std::integral_constant<int, V>;

// NWV waves (4 or 8) as WM x (NWV / WM); with 8 waves two share each SIMD,
// so one wave's loads and epilogue overlap the other's MFMAs.
template <typename T, int L, int BM, int BN, int BK, int WM, int ST, int EPI, int NWV = 4>
__global__ __launch_bounds__(64 * NWV, (dma_occ<BM, BN, BK, ST, EPI, NWV>()))
void igemm_dma_kernel(IgArgs a) {
  static_assert(sizeof(T) == 2 && L != NCHW, "16-bit channel-vector layouts only");
  static_assert(NWV == 4 || NWV == 8, "4 or 8 waves");
  constexpr int NT = 64 * NWV;
  constexpr int WN = NWV / WM;
  constexpr int CPR = BK / 8;       // 16-byte chunks per tile row
  constexpr int RPB = 64 / CPR;     // tile rows filled by one load instruction (1 KB)
  // the chunk XOR key changes every 2 rows (64- and 128-byte rows) or every
  // row (256-byte rows): one chunk of 16 consecutive rows then covers the 64
  // banks once and is read in a single LDS pass on gfx950
  constexpr int RPR = CPR == 16 ? 1 : 2;
  constexpr int NA = BM / RPB / NWV;  // A load instructions per wave and stage
  constexpr int NB = BN / RPB / NWV;  // B load instructions per wave and stage
  static_assert(NA * RPB * NWV == BM && NB * RPB * NWV == BN && WM * WN == NWV, "tile shape");
  static_assert(ST >= 2 && ST <= 6 && (ST - 2) * (NA + NB) <= 63, "pipeline depth");
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int A_BYTES = BM * BK * 2, STAGE = (BM + BN) * BK * 2;
  constexpr int CPAD = 8;
  constexpr int SM_C = EPI == EPI_LAYOUT || EPI == EPI_FIXUP ? BM * (BN + 4) * 4 : 0;  // fp32 epilogue rows
  constexpr int SM = ST * STAGE > SM_C ? ST * STAGE : SM_C;
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  auto swz = [](int row) { return (row / RPR) % CPR; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  tile_of(blockIdx.x, a.tiles_m, a.tiles_n, mt, nt);
  const int m0 = mt * BM, n0 = nt * BN;
  const int split = blockIdx.y;
  const int kt0 = split * a.kt_per;
  const int KT1 = a.KC / CPR;  // steps of the convolution; a projected shortcut's follow
  const int KT = min(KT1 + a.KC2 / CPR - kt0, a.kt_per);
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x);
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(w, a.w_elems * 2);

  // accumulators start at the bias of the lane's output channels (at zero
  // for a partial sum of a split reduction); the bias is loaded before the
  // tiles so that waiting for it does not wait for them
  float bias[FN][4];
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) bias[j][v] = 0.f;
  // (a split reduction: split 0 starts at the bias, the others at zero)
  if (EPI == EPI_LAYOUT || (EPI == EPI_FIXUP && split == 0)) {
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.bias, (long long)a.Ng * 4);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int n = n0 + wn * WTN + j * 16 + (lane >> 4) * 4;
#pragma unroll
      for (int v = 0; v < 4; ++v)
        bias[j][v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rb, (n + v) * 4, 0, 0));
    }
  }

  // this lane's load slots: block b = wave + NWV i fills tile rows
  // [b * RPB, (b + 1) * RPB); the lane fills row b * RPB + lane / CPR,
  // physical chunk lane % CPR, i.e. logical chunk (lane % CPR) ^ swz(row)
  const int prow = lane / CPR, pch = lane % CPR;
  unsigned rbyte[NA], tvm[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int row = (wave + NWV * i) * RPB + prow;
    const int lc = pch ^ swz(row);
    const int m = m0 + row;
    const bool ok = m < a.M;
    const int mm = ok ? m : 0;
    // fp32 division and 24-bit multiplies: indices stay far below 2^21
    const int img = sdiv(mm, a.inv_pq), pq = mm - __mul24(img, a.PQ);
    const int p = sdiv(pq, a.inv_q), q = pq - __mul24(p, a.Q);
    const int h0 = __mul24(p, a.stride) - a.pad, w0 = __mul24(q, a.stride) - a.pad;
    int e;
    if constexpr (L == NC8)
      e = __mul24(img, a.CB * a.H * a.W * 8) + __mul24(__mul24(h0, a.W) + w0, 8) + __mul24(lc, a.H * a.W * 8);
    else
      e = __mul24(__mul24(__mul24(img, a.H) + h0, a.W) + w0, a.Cs) + lc * 8;
    rbyte[i] = (unsigned)e * 2u;  // may wrap for the halo; valid taps add back
    unsigned msk = 0;
    for (int r = 0; r < a.R; ++r)
      for (int c = 0; c < a.S; ++c)
        if (ok && (unsigned)(h0 + r) < (unsigned)a.H && (unsigned)(w0 + c) < (unsigned)a.W)
          msk |= 1u << (r * a.S + c);
    tvm[i] = msk;
  }
  unsigned bbyte[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int row = (wave + NWV * i) * RPB + prow;
    const int lc = pch ^ swz(row);
    const int k = n0 + row;
    bbyte[i] = k < a.Ng ? (unsigned)((__mul24(k, a.Kred) + lc * 8) * 2) : kOOB;
  }
  // the projected shortcut: output pixel (img, p, q) reads pixel (p, q) *
  // stride2 of x2 (no padding), and output channel k row k of w2
  unsigned rbyte2[NA], bbyte2[NB];
  const bool proj = a.x2 != nullptr;
  const __amdgpu_buffer_rsrc_t rx2 = make_rsrc(proj ? a.x2 : a.x, proj ? a.x2_elems * 2 : 0);
  const __amdgpu_buffer_rsrc_t rw2 = make_rsrc(proj ? a.w2 : a.w, proj ? a.w2_elems * 2 : 0);
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    rbyte2[i] = kOOB;
    if (!proj) continue;
    const int row = (wave + NWV * i) * RPB + prow;
    const int lc = pch ^ swz(row);
    const int m = m0 + row;
    if (m >= a.M) continue;
    const int img = sdiv(m, a.inv_pq), pq = m - __mul24(img, a.PQ);
    const int p = sdiv(pq, a.inv_q), q = pq - __mul24(p, a.Q);
    const int h = __mul24(p, a.stride2), w2 = __mul24(q, a.stride2);
    int e;
    if constexpr (L == NC8)
      e = __mul24(img, a.CB2 * a.H2 * a.W2 * 8) + __mul24(__mul24(h, a.W2) + w2, 8) + __mul24(lc, a.H2 * a.W2 * 8);
    else
      e = __mul24(__mul24(__mul24(img, a.H2) + h, a.W2) + w2, a.Cs2) + lc * 8;
    rbyte2[i] = (unsigned)e * 2u;
  }
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int row = (wave + NWV * i) * RPB + prow;
    const int lc = pch ^ swz(row);
    const int k = n0 + row;
    bbyte2[i] = proj && k < a.Ng ? (unsigned)((__mul24(k, a.Kred2) + lc * 8) * 2) : kOOB;
  }

  // reduction position of the next step to load: tap (r, s), channel block cb
  ChunkPos upos;
  chunk_set(upos, kt0 * CPR, a.CB, a.S);
  auto issue = [&](auto SC, int kt) {
    char* base = smem + decltype(SC)::value * STAGE;
    if (kt >= KT1) {
      // a step of the projected shortcut: channel block cb2 of x2 (8 CPR
      // channels per tile row), the matching columns of w2
      const int k2 = kt - KT1;
      const unsigned cb = (unsigned)k2 * (unsigned)CPR;
      const unsigned xo = L == NC8 ? cb * (unsigned)(a.H2 * a.W2 * 8) * 2u : cb * 16u;
#pragma unroll
      for (int i = 0; i < NA; ++i)
        dma16(rx2, base + (wave + NWV * i) * 1024, rbyte2[i] == kOOB ? kOOB : rbyte2[i] + xo, 0);
#pragma unroll
      for (int i = 0; i < NB; ++i) dma16(rw2, base + A_BYTES + (wave + NWV * i) * 1024, bbyte2[i], k2 * BK * 2);
      return;
    }
    const int t = upos.r * a.S + upos.s;
    int tap;
    if constexpr (L == NC8)
      tap = upos.cb * a.H * a.W * 8 + (upos.r * a.W + upos.s) * 8;
    else
      tap = (upos.r * a.W + upos.s) * a.Cs + upos.cb * 8;
    const unsigned tb = (unsigned)tap * 2u;
#pragma unroll
    for (int i = 0; i < NA; ++i)
      dma16(rx, base + (wave + NWV * i) * 1024, ((tvm[i] >> t) & 1u) ? rbyte[i] + tb : kOOB, 0);
#pragma unroll
    for (int i = 0; i < NB; ++i) dma16(rw, base + A_BYTES + (wave + NWV * i) * 1024, bbyte[i], kt * BK * 2);
    upos.cb += CPR;  // CB is a multiple of CPR
    if (upos.cb == a.CB) {
      upos.cb = 0;
      if (++upos.s == a.S) {
        upos.s = 0;
        ++upos.r;
      }
    }
  };

  typedef typename Mfma<T>::frag frag;
  f32x4 acc[FM][FN];
  // operand chunk offsets in a stage: a 16-row block starts at a multiple of
  // 16 rows, so the row swizzle is the lane's own; the chunk of k-slice ks is
  // fixed per lane and the block offset is an instruction immediate
  constexpr int KS = BK / 32;
  int aofs[KS], bofs[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int l = lane & 15, xo = (((ks * 4 + (lane >> 4)) ^ swz(l)) << 4);
    aofs[ks] = (wm * WTM + l) * (BK * 2) + xo;
    bofs[ks] = A_BYTES + (wn * WTN + l) * (BK * 2) + xo;
  }
  auto load_frags = [&](const char* S, int ks, frag(&fa)[FM], frag(&fb)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i) fa[i] = *reinterpret_cast<const frag*>(S + aofs[ks] + i * 16 * (BK * 2));
#pragma unroll
    for (int j = 0; j < FN; ++j) fb[j] = *reinterpret_cast<const frag*>(S + bofs[ks] + j * 16 * (BK * 2));
  };
  // the fragments of k-slice ks+1 are read while the MFMAs of ks run (the
  // stage index is a template constant, so every LDS offset is an immediate)
  auto compute = [&](auto SC) {
    const char* S = smem + decltype(SC)::value * STAGE;
    frag fa[2][FM], fb[2][FN];
    load_frags(S, 0, fa[0], fb[0]);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) load_frags(S, ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(fb[ks & 1][j], fa[ks & 1][i], acc[i][j]);
    }
  };

  // step t: wait for tile t (the ST-2 tiles after it may stay in flight),
  // barrier, issue tile t+ST-1 into the buffer read at step t-1, compute t;
  // the loop is unrolled by ST so that stage indices are constants
  issue(IC<0>{}, kt0);
  if constexpr (ST > 2) { if (1 < KT) issue(IC<1>{}, kt0 + 1); }
  if constexpr (ST > 3) { if (2 < KT) issue(IC<2>{}, kt0 + 2); }
  if constexpr (ST > 4) { if (3 < KT) issue(IC<3>{}, kt0 + 3); }
  if constexpr (ST > 5) { if (4 < KT) issue(IC<4>{}, kt0 + 4); }
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int i = 0; i < FM; ++i) acc[i][j] = f32x4{bias[j][0], bias[j][1], bias[j][2], bias[j][3]};
  auto step = [&](auto UC, int t) {
    constexpr int U = decltype(UC)::value;
    if (t >= KT) return;
    if (t + ST - 2 < KT)
      wait_vmcnt<(ST - 2) * (NA + NB)>();
    else
      wait_vmcnt<0>();
    dma_barrier();
    if (t + ST - 1 < KT) issue(IC<(U + ST - 1) % ST>{}, kt0 + t + ST - 1);
    compute(UC);
  };
  for (int t0 = 0; t0 < KT; t0 += ST) {
    step(IC<0>{}, t0);
    step(IC<1>{}, t0 + 1);
    if constexpr (ST > 2) step(IC<2>{}, t0 + 2);
    if constexpr (ST > 3) step(IC<3>{}, t0 + 3);
    if constexpr (ST > 4) step(IC<4>{}, t0 + 4);
    if constexpr (ST > 5) step(IC<5>{}, t0 + 5);
  }

  // split reduction summed in the kernel: every split stores its partial
  // tile (each lane its accumulators, in lane order, so the stores and the
  // loads that read them back are whole contiguous rows) and counts itself
  // in at the tile's counter; the last split to arrive sums the partial
  // tiles in split order, clears the counter for the next launch and runs
  // the layout epilogue; the others are done.  The partial tiles bypass the
  // per-XCD L2 caches (device-coherent accesses, cache policy sc1:
  // written through to memory and read from it), and a workgroup's stores
  // are complete before its count, so no cache-wide fence is needed; the
  // counters are device-scope atomics.
  if constexpr (EPI == EPI_FIXUP) {
    if (a.splits > 1) {
      constexpr int COHERENT = 16;      // sc1: coherent across the agent
      __shared__ int fix_last;
      constexpr int TILE = BM * BN;     // fp32 values of a partial tile
      const __amdgpu_buffer_rsrc_t rp =
          make_rsrc(a.part, (long long)a.splits * gridDim.x * TILE * (long long)sizeof(float));
      const unsigned slot0 = (unsigned)blockIdx.x * (unsigned)a.splits * (unsigned)(TILE * 4);
      auto lane_off = [&](int sp, int i, int j) {
        return slot0 + (unsigned)sp * (TILE * 4) + (unsigned)(((i * FN + j) * NT + tid) * 16);
      };
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[i][j]), rp,
                                                 (int)lane_off(split, i, j), 0, COHERENT);
      wait_vmcnt<0>();
      __syncthreads();
      if (tid == 0)
        fix_last = __hip_atomic_fetch_add(a.cnt + blockIdx.x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                   (unsigned)(a.splits - 1);
      __syncthreads();
      if (!fix_last) return;
      // the partial tiles are summed in split order whichever split is last,
      // so the result does not depend on the order the workgroups finish in;
      // the next split's loads are in flight while one is added
      f32x4 sum[FM][FN];
      u32x4 cur[FM][FN], nxt[FM][FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          sum[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
          cur[i][j] = __builtin_amdgcn_raw_buffer_load_b128(rp, (int)lane_off(0, i, j), 0, COHERENT);
        }
      for (int sp = 0; sp < a.splits; ++sp) {
        if (sp + 1 < a.splits) {
#pragma unroll
          for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
              nxt[i][j] = __builtin_amdgcn_raw_buffer_load_b128(rp, (int)lane_off(sp + 1, i, j), 0, COHERENT);
        }
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j) {
            sum[i][j] += sp == split ? acc[i][j] : __builtin_bit_cast(f32x4, cur[i][j]);
            cur[i][j] = nxt[i][j];
          }
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = sum[i][j];
      if (tid == 0) __hip_atomic_exchange(a.cnt + blockIdx.x, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // accumulator element (i, j, v) is C[wm*WTM + i*16 + (lane&15)][wn*WTN + j*16 + (lane>>4)*4 + v]
  if constexpr (EPI == EPI_SPLIT) {
    float* __restrict__ y = a.part + (long long)split * a.M * a.Ng;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int m = m0 + wm * WTM + i * 16 + (lane & 15);
        const int n = n0 + wn * WTN + j * 16 + (lane >> 4) * 4;
        if (m < a.M) {
          if (n + 4 <= a.Ng && (a.Ng & 3) == 0) {
            *reinterpret_cast<f32x4*>(y + (long long)m * a.Ng + n) = acc[i][j];
          } else {
#pragma unroll
            for (int v = 0; v < 4; ++v)
              if (n + v < a.Ng) y[(long long)m * a.Ng + n + v] = acc[i][j][v];
          }
        }
      }
  } else if (a.res) {
    // residual (output rows of whole 16-byte chunks: NC8HW8, or NHWC with
    // K % 8 == 0, which the routine's validity requires): the fp32 sums go
    // through LDS, and each thread adds the
    // residual to 8 channels of one output row as it stores them, reading
    // and writing whole 16-byte chunks of consecutive channels
    __syncthreads();  // every wave is done with the last tile
    float(*Cf)[BN + 4] = reinterpret_cast<float(*)[BN + 4]>(smem);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nl = wn * WTN + j * 16 + (lane >> 4) * 4;
#pragma unroll
      for (int i = 0; i < FM; ++i) *reinterpret_cast<f32x4*>(&Cf[wm * WTM + i * 16 + (lane & 15)][nl]) = acc[i][j];
    }
    __syncthreads();
    const ActClamp ac = act_clamp(a.act);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(a.y, a.y_elems * 2);
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(a.res, a.y_elems * 2);
    constexpr int IT = (BM * BN / 8 + NT - 1) / NT;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int idx = tid + it * NT;
      // NC8HW8: consecutive threads take consecutive pixels of one channel block
      const int row = L == NC8 ? idx % BM : idx / (BN / 8), cj = L == NC8 ? idx / BM : idx % (BN / 8);
      const int m = m0 + row, n = n0 + cj * 8;
      unsigned off = kOOB;
      if (idx < BM * BN / 8 && m < a.M && n < a.Ng) {
        if constexpr (L == NC8) {
          const int img = sdiv(m, a.inv_pq), pq = m - __mul24(img, a.PQ);
          off = (unsigned)(((img * (a.Ks >> 3) + (n >> 3)) * a.PQ + pq) * 8) * 2u;
        } else {
          off = (unsigned)(m * a.Ks + n) * 2u;
        }
      }
      const u32x4 rraw = __builtin_amdgcn_raw_buffer_load_b128(rr, (int)off, 0, 0);
      T rt[8], o[8];
      __builtin_memcpy(rt, &rraw, 16);
      const int rrow = idx < BM * BN / 8 ? row : 0, rcj = idx < BM * BN / 8 ? cj : 0;
      const f32x4 c0 = *reinterpret_cast<const f32x4*>(&Cf[rrow][rcj * 8]);
      const f32x4 c1 = *reinterpret_cast<const f32x4*>(&Cf[rrow][rcj * 8 + 4]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        o[e] = from_f<T>(__builtin_amdgcn_fmed3f(c0[e] + to_f(rt[e]), ac.lo, ac.hi));
        o[4 + e] = from_f<T>(__builtin_amdgcn_fmed3f(c1[e] + to_f(rt[4 + e]), ac.lo, ac.hi));
      }
      __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4*>(o), ry, (int)off, 0, 0);
    }
  } else {
    __syncthreads();  // every wave is done with the last tile
    T(*Cs)[BN + CPAD] = reinterpret_cast<T(*)[BN + CPAD]>(smem);
    const ActClamp ac = act_clamp(a.act);
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int nl = wn * WTN + j * 16 + (lane >> 4) * 4;
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int ml = wm * WTM + i * 16 + (lane & 15);
        T o[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = from_f<T>(__builtin_amdgcn_fmed3f(acc[i][j][v], ac.lo, ac.hi));
        __builtin_memcpy(&Cs[ml][nl], o, sizeof(o));
      }
    }
    __syncthreads();
    T* __restrict__ y = reinterpret_cast<T*>(a.y);
    if (L == NC8 || a.Ks % 8 == 0) {
      // 16-byte rows through a buffer resource (32-bit offsets)
      const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, a.y_elems * 2);
      for (int idx = tid; idx < BM * BN / 8; idx += NT) {
        // NC8HW8: consecutive threads take consecutive pixels of one channel block
        const int row = L == NC8 ? idx % BM : idx / (BN / 8), cj = L == NC8 ? idx / BM : idx % (BN / 8);
        const int m = m0 + row, n = n0 + cj * 8;
        if (m >= a.M || n >= a.Ng) continue;
        const u32x4 v = *reinterpret_cast<const u32x4*>(&Cs[row][cj * 8]);
        unsigned off;
        if constexpr (L == NC8) {
          const int img = sdiv(m, a.inv_pq), pq = m - __mul24(img, a.PQ);
          off = (unsigned)(((img * (a.Ks >> 3) + (n >> 3)) * a.PQ + pq) * 8) * 2u;
        } else {
          off = (unsigned)(m * a.Ks + n) * 2u;
        }
        __builtin_amdgcn_raw_buffer_store_b128(v, ry, (int)off, 0, 0);
      }
    } else {
      for (int idx = tid; idx < BM * BN; idx += NT) {
        const int row = idx / BN, col = idx % BN;
        const int m = m0 + row, n = n0 + col;
        if (m < a.M && n < a.Ng) y[(long long)m * a.Ks + n] = Cs[row][col];
      }
    }
  }
}

// Sum the split-K partial tiles, add the bias, apply the activation and
// store in the tensor layout.  One thread per (pixel, 8 output channels);
// NCHW: one thread per (channel, pixel), pixels fastest.
template <typename T, int L>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(IgArgs a) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long plane = (long long)a.M * a.Ng;
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
  if constexpr (L == NCHW) {
    if (idx >= plane) return;
    const int m = (int)(idx % a.M), n = (int)(idx / a.M);
    float s = a.bias[n];
    for (int k = 0; k < a.splits; ++k) s += a.part[k * plane + (long long)m * a.Ng + n];
    const int img = m / a.PQ, pq = m - img * a.PQ;
    const long long o = ((long long)img * a.Ks + n) * a.PQ + pq;
    if (a.res) s += to_f(reinterpret_cast<const T*>(a.res)[o]);
    y[o] = from_f<T>(act_f(s, a.act));
  } else {
    const int NB8 = (a.Ng + 7) / 8;
    if (idx >= (long long)a.M * NB8) return;
    const int nb = (int)(idx % NB8), m = (int)(idx / NB8);
    const int n0 = nb * 8;
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = n0 + e < a.Ng ? a.bias[n0 + e] : 0.f;
    for (int k = 0; k < a.splits; ++k) {
      const float* p = a.part + k * plane + (long long)m * a.Ng + n0;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (n0 + e < a.Ng) s[e] += p[e];
    }
    if (a.res) {
      const T* rp = reinterpret_cast<const T*>(a.res);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (n0 + e < a.Ng) s[e] += to_f(rp[out_index<L>(a, m, n0 + e)]);
    }
    V8<T> o;
#pragma unroll
    for (int e = 0; e < 8; ++e) o.v[e] = from_f<T>(act_f(s[e], a.act));
    if constexpr (L == NC8) {
      const int img = m / a.PQ, pq = m - img * a.PQ;
      st8(y + (((long long)img * (a.Ks >> 3) + nb) * a.PQ + pq) * 8, o);
    } else if (a.Ks % 8 == 0) {
      st8(y + (long long)m * a.Ks + n0, o);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (n0 + e < a.Ng) y[(long long)m * a.Ks + n0 + e] = o.v[e];
    }
  }
}

// Routine parameters of the implicit-GEMM routine (index = routine param).
struct IgCfg {
  int bm, bn, bk, split, pf;  // split: 0 = none, 1 = split the reduction when tiles are few
                              // (partials summed by a second kernel), 2 = likewise, summed by
                              // the last workgroup of each tile (LDS-DMA kernel only);
                              // pf: prefetch depth (register staging sets)
  int dma = 0, wm = 2, st = 2;  // 1: LDS-DMA kernel, 2: 3x3 patch kernel (bm = 16 * row blocks),
                                // 3: small-channel kernel, 4: streaming 1x1 kernel (C = bk);
                                // wave rows WM (of 4 waves), LDS stages ST
  int ppx = 0;                  // small-channel kernel: patch capacity in pixels
  PatchCfg pc{};                // patch kernel tile
  int nw = 4;                   // LDS-DMA kernel: waves per workgroup (4 or 8)
  int gmax = 0;                 // small-channel kernel: filter chunks held (R * ceil(S / 2) <= gmax)
};
static const IgCfg kIg16[] = {
    {64, 64, 32, 0, 2},   {128, 128, 64, 0, 2}, {256, 128, 32, 0, 2}, {128, 64, 64, 0, 2},
    {64, 128, 64, 0, 4},  {128, 128, 64, 1, 2}, {64, 64, 64, 1, 4},   {128, 64, 32, 0, 4},
    {64, 128, 64, 0, 2},  {96, 128, 64, 0, 2},  {64, 64, 64, 0, 4},   {128, 128, 32, 0, 4},
    {64, 128, 32, 0, 4},  {128, 64, 64, 0, 4},  {64, 128, 128, 0, 2}, {128, 64, 128, 0, 2},
    {128, 128, 128, 0, 2},
    // LDS-DMA kernel (channel counts that are multiples of BK)
    {128, 128, 64, 0, 0, 1, 2, 2}, {128, 128, 64, 0, 0, 1, 2, 3}, {256, 64, 64, 0, 0, 1, 4, 2},
    {256, 64, 64, 0, 0, 1, 4, 3},  {128, 64, 64, 0, 0, 1, 2, 3},  {64, 128, 64, 0, 0, 1, 1, 3},
    {256, 128, 64, 0, 0, 1, 2, 2}, {128, 128, 32, 0, 0, 1, 2, 3}, {64, 64, 64, 0, 0, 1, 2, 3},
    {128, 128, 64, 1, 0, 1, 2, 3}, {128, 64, 64, 1, 0, 1, 2, 3}, {64, 64, 64, 1, 0, 1, 2, 3},
    // deeper pipelines (short reduction steps, more in flight)
    {128, 128, 32, 0, 0, 1, 2, 4}, {128, 64, 32, 0, 0, 1, 2, 4}, {64, 128, 32, 0, 0, 1, 1, 4},
    {64, 64, 64, 0, 0, 1, 2, 4},   {64, 64, 32, 0, 0, 1, 2, 6},  {256, 64, 32, 0, 0, 1, 4, 4},
    // LDS-DMA kernel with 8 waves (two per SIMD)
    {128, 128, 64, 0, 0, 1, 4, 2, 0, {}, 8}, {128, 128, 64, 0, 0, 1, 4, 3, 0, {}, 8},
    {128, 128, 64, 0, 0, 1, 4, 4, 0, {}, 8}, {256, 128, 64, 0, 0, 1, 4, 3, 0, {}, 8},
    {128, 64, 64, 0, 0, 1, 4, 4, 0, {}, 8},  {256, 64, 64, 0, 0, 1, 8, 3, 0, {}, 8},
    {64, 128, 64, 0, 0, 1, 2, 4, 0, {}, 8},  {128, 256, 64, 0, 0, 1, 2, 3, 0, {}, 8},
    {128, 128, 32, 0, 0, 1, 4, 4, 0, {}, 8}, {256, 128, 32, 0, 0, 1, 4, 4, 0, {}, 8},
    // deep pipelines for the small-M layers (more bytes in flight per CU)
    {64, 128, 64, 0, 0, 1, 2, 6, 0, {}, 8},  {128, 64, 64, 0, 0, 1, 4, 6, 0, {}, 8},
    {128, 128, 32, 0, 0, 1, 4, 6, 0, {}, 8}, {64, 64, 64, 0, 0, 1, 2, 6, 0, {}, 8},
    // 3x3 stride-1 patch kernel
#define SN_PATCH_IG(FMT, BN, PWT, WM, WN, TG, ST, PROWS) \
  {16 * FMT, BN, 32, 0, 0, 2, WM, ST, 0, {FMT, BN, PWT, WM, WN, TG, ST, PROWS}},
    PATCH_CONFIGS(SN_PATCH_IG)
#undef SN_PATCH_IG
    // small-channel (stem) kernel: NHWC, C <= 4, stride 1 or 2; 7 x 7 and 3 x 3 filters
    // (wm: wave rows; st: workgroups per CU)
    {112, 64, 32, 0, 0, 3, 2, 2, 1664, {}, 4, 28}, {224, 64, 32, 0, 0, 3, 2, 2, 2112, {}, 4, 28},
    {112, 64, 32, 0, 0, 3, 2, 3, 704, {}, 4, 8},   {224, 64, 32, 0, 0, 3, 2, 2, 1152, {}, 4, 8},
    // streaming 1x1 kernel: NHWC, C = bk (BM pixels x BN channels per tile, WM wave rows,
    // loads pf tiles ahead; st: workgroups per CU)
#define SN_STREAM_IG(CC, BM, BN, WM, PD) {BM, BN, CC, 0, PD, 4, WM, 1},
    STREAM_CONFIGS(SN_STREAM_IG)
#undef SN_STREAM_IG
    // LDS-DMA kernel, 8 waves, reduction split over workgroups when the
    // tiles alone cannot fill the GPU (the last split of a tile sums them)
    {128, 128, 64, 2, 0, 1, 4, 3, 0, {}, 8}, {128, 64, 64, 2, 0, 1, 4, 4, 0, {}, 8},
    {64, 128, 64, 2, 0, 1, 2, 4, 0, {}, 8},  {64, 64, 64, 2, 0, 1, 2, 4, 0, {}, 8},
    {64, 64, 64, 2, 0, 1, 2, 6, 0, {}, 8},   {128, 128, 32, 2, 0, 1, 4, 4, 0, {}, 8},
    // 3x3 stride-2 patch kernel
#define SN_PATCH2_IG(FMT, BN, PWT, WM, WN, TG, ST, PROWS) \
  {16 * FMT, BN, 32, 0, 0, 2, WM, ST, 0, {FMT, BN, PWT, WM, WN, TG, ST, PROWS, 2}},
    PATCH2_CONFIGS(SN_PATCH2_IG)
#undef SN_PATCH2_IG
    // small-channel (stem) kernel, 7 x 7: two output rows per tile, four wave
    // rows, two workgroups per CU
    {224, 64, 32, 0, 0, 3, 4, 2, 2112, {}, 4, 28},
    // LDS-DMA kernel with 128-channel reduction steps (half the steps, and
    // barriers, of long reductions)
    {64, 64, 128, 0, 0, 1, 2, 3},  {64, 64, 128, 0, 0, 1, 2, 4},
    {64, 128, 128, 0, 0, 1, 2, 3, 0, {}, 8}, {128, 64, 128, 0, 0, 1, 4, 3, 0, {}, 8},
    {128, 128, 128, 0, 0, 1, 4, 2, 0, {}, 8},
    // 3x3 stride-1 patch kernel, two workgroups per CU
#define SN_PATCHO2_IG(FMT, BN, PWT, WM, WN, TG, ST, PROWS) \
  {16 * FMT, BN, 32, 0, 0, 2, WM, ST, 0, {FMT, BN, PWT, WM, WN, TG, ST, PROWS, 1, 2}},
    PATCH_OCC2_CONFIGS(SN_PATCHO2_IG)
#undef SN_PATCHO2_IG
    // streaming 1x1 kernel for 512-channel inputs
#define SN_STREAM_IG(CC, BM, BN, WM, PD) {BM, BN, CC, 0, PD, 4, WM, 1},
    STREAM512_CONFIGS(SN_STREAM_IG)
#undef SN_STREAM_IG
    // 3x3 stride-1 patch kernel with row-aligned row blocks
#define SN_PATCHRA_IG(FMT, BN, PWT, WM, WN, TG, ST, PROWS, OCC) \
  {16 * FMT, BN, 32, 0, 0, 2, WM, ST, 0, {FMT, BN, PWT, WM, WN, TG, ST, PROWS, 1, OCC, 1}},
    PATCH_RA_CONFIGS(SN_PATCHRA_IG)
#undef SN_PATCHRA_IG
    // streaming 1x1 kernel, two workgroups per CU
#define SN_STREAM_IG(CC, BM, BN, WM, PD) {BM, BN, CC, 0, PD, 4, WM, 2},
    STREAM_OCC2_CONFIGS(SN_STREAM_IG)
#undef SN_STREAM_IG
};
static const IgCfg kIg32[] = {{64, 64, 32, 0, 2}};




static IgCfg ig_cfg(int dtype, int param) {
  check(param >= 0 && param < igemm_num_params(dtype), "unknown implicit-GEMM parameter");
  return dtype == 0 ? kIg32[param] : kIg16[param];
}

// Fills the grid decomposition of `a` for configuration `c`.
static void ig_decompose(IgArgs& a, const IgCfg& c) {
  a.tiles_m = (a.M + c.bm - 1) / c.bm;
  a.tiles_n = (a.Ng + c.bn - 1) / c.bn;
  const int cpr = c.bk / 8;
  const int KT = (a.KC + a.KC2 + cpr - 1) / cpr;  // with a projected shortcut: both reductions
  int splits = 1;
  const int tiles = a.tiles_m * a.tiles_n;
  if (c.split == 1) {
    if (tiles < 384) splits = std::min(std::min((768 + tiles - 1) / tiles, 8), std::max(1, KT / 2));
  } else if (c.split == 2) {
    // as many splits as still run in one round of resident workgroups (the
    // LDS stages bound the workgroups per CU), each at least two reduction
    // steps long
    const int lds = std::max(c.st * (c.bm + c.bn) * c.bk * 2, c.bm * (c.bn + 4) * 4);
    const int resident = 256 * std::max(1, std::min(160 * 1024 / lds, 2));
    if (2 * tiles <= resident) splits = std::min(std::min(resident / tiles, 8), std::max(1, KT / 2));
  }
  a.kt_per = (KT + splits - 1) / splits;
  a.splits = (KT + a.kt_per - 1) / a.kt_per;
}

template <typename T, int L, bool VEC, int BM, int BN, int BK, int EPI, int PF>
static void igemm_go(const IgArgs& a, int batch, hipStream_t st) {
  check(a.x_elems * (long long)sizeof(T) < (long long)kOOB && a.w_elems * (long long)sizeof(T) < (long long)kOOB,
        "tensor too large for 32-bit buffer offsets");
  dim3 grid(a.tiles_m * a.tiles_n, a.splits, batch);
  if (VEC && a.CB % (BK / 8) == 0 && a.R * a.S <= 32)
    SN_LAUNCH((igemm_kernel<T, L, VEC, VEC, BM, BN, BK, EPI, PF>), grid, dim3(256), 0, st, a);
  else
    SN_LAUNCH((igemm_kernel<T, L, VEC, false, BM, BN, BK, EPI, PF>), grid, dim3(256), 0, st, a);
}

template <typename T, int L, int BM, int BN, int BK, int WM, int ST, int EPI, int NWV = 4>
static void igemm_dma_go(const IgArgs& a, hipStream_t st) {
  check(a.x_elems * 2 < (long long)kOOB && a.w_elems * 2 < (long long)kOOB,
        "tensor too large for 32-bit buffer offsets");
  check(a.CB % (BK / 8) == 0 && a.R * a.S <= 32, "LDS-DMA tile needs C % BK == 0 and R*S <= 32");
  check(a.y_elems * 2 < (long long)kOOB && (long long)a.M + a.PQ < (1 << 21),
        "tensor too large for 32-bit offsets / fp32 index division");
  dim3 grid(a.tiles_m * a.tiles_n, a.splits, 1);
  SN_LAUNCH((igemm_dma_kernel<T, L, BM, BN, BK, WM, ST, EPI, NWV>), grid, dim3(64 * NWV), 0, st, a);
}

template <typename T, int L, int EPI>
static void igemm_dma_cfg(const IgCfg& c, const IgArgs& a, hipStream_t st) {
  const long long key = ((((c.bm * 1000LL + c.bn) * 1000 + c.bk) * 10 + c.wm) * 10 + c.st) * 10 + c.nw;
#define IGD(BM_, BN_, BK_, WM_, ST_) IGDN(BM_, BN_, BK_, WM_, ST_, 4)
#define IGDN(BM_, BN_, BK_, WM_, ST_, NW_)                                       \
  case ((((BM_ * 1000LL + BN_) * 1000 + BK_) * 10 + WM_) * 10 + ST_) * 10 + NW_: \
    igemm_dma_go<T, L, BM_, BN_, BK_, WM_, ST_, EPI, NW_>(a, st);                \
    break;
  if constexpr (EPI == EPI_SPLIT) {
    switch (key) {
      IGD(128, 128, 64, 2, 3)
      IGD(128, 64, 64, 2, 3)
      IGD(64, 64, 64, 2, 3)
      default: check(false, "LDS-DMA tile not instantiated for split reduction");
    }
    return;
  }
  if constexpr (EPI == EPI_FIXUP) {
    switch (key) {
      IGDN(128, 128, 64, 4, 3, 8)
      IGDN(128, 64, 64, 4, 4, 8)
      IGDN(64, 128, 64, 2, 4, 8)
      IGDN(64, 64, 64, 2, 4, 8)
      IGDN(64, 64, 64, 2, 6, 8)
      IGDN(128, 128, 32, 4, 4, 8)
      default: check(false, "LDS-DMA tile not instantiated for split reduction");
    }
    return;
  } else if constexpr (EPI == EPI_LAYOUT) {
  switch (key) {
    IGD(128, 128, 64, 2, 2)
    IGD(128, 128, 64, 2, 3)
    IGD(256, 64, 64, 4, 2)
    IGD(256, 64, 64, 4, 3)
    IGD(128, 64, 64, 2, 3)
    IGD(64, 128, 64, 1, 3)
    IGD(256, 128, 64, 2, 2)
    IGD(128, 128, 32, 2, 3)
    IGD(64, 64, 64, 2, 3)
    IGD(128, 128, 32, 2, 4)
    IGD(128, 64, 32, 2, 4)
    IGD(64, 128, 32, 1, 4)
    IGD(64, 64, 64, 2, 4)
    IGD(64, 64, 32, 2, 6)
    IGD(256, 64, 32, 4, 4)
    IGDN(128, 128, 64, 4, 2, 8)
    IGDN(128, 128, 64, 4, 3, 8)
    IGDN(128, 128, 64, 4, 4, 8)
    IGDN(256, 128, 64, 4, 3, 8)
    IGDN(128, 64, 64, 4, 4, 8)
    IGDN(256, 64, 64, 8, 3, 8)
    IGDN(64, 128, 64, 2, 4, 8)
    IGDN(128, 256, 64, 2, 3, 8)
    IGDN(128, 128, 32, 4, 4, 8)
    IGDN(256, 128, 32, 4, 4, 8)
    IGDN(64, 128, 64, 2, 6, 8)
    IGDN(128, 64, 64, 4, 6, 8)
    IGDN(128, 128, 32, 4, 6, 8)
    IGDN(64, 64, 64, 2, 6, 8)
    IGD(64, 64, 128, 2, 3)
    IGD(64, 64, 128, 2, 4)
    IGDN(64, 128, 128, 2, 3, 8)
    IGDN(128, 64, 128, 4, 3, 8)
    IGDN(128, 128, 128, 4, 2, 8)
    default: check(false, "LDS-DMA tile not instantiated");
  }
  }
#undef IGD
#undef IGDN
}

template <typename T, int L, bool VEC, int EPI>
static void igemm_cfg(const IgCfg& c, const IgArgs& a, int batch, hipStream_t st) {
  if (c.dma) {
    if constexpr (sizeof(T) == 2 && VEC && L != NCHW && EPI != EPI_RAW) {
      check(batch == 1, "LDS-DMA tiles run unbatched GEMMs");
      igemm_dma_cfg<T, L, EPI>(c, a, st);
    } else {
      check(false, "LDS-DMA tiles need 16-bit channel-vector tensors");
    }
    return;
  }
  if constexpr (std::is_same<T, float>::value) {
    igemm_go<T, L, VEC, 64, 64, 32, EPI, 2>(a, batch, st);
  } else {
    const int key = ((c.bm * 1000 + c.bn) * 100 + c.bk) * 10 + c.pf;
#define IGC(BM_, BN_, BK_, PF_) \
  case ((BM_ * 1000 + BN_) * 100 + BK_) * 10 + PF_: igemm_go<T, L, VEC, BM_, BN_, BK_, EPI, PF_>(a, batch, st); break;
    if constexpr (EPI == EPI_RAW) {  // Winograd tile GEMMs
      switch (key) {
        IGC(64, 64, 64, 4)
        IGC(128, 64, 64, 4)
        IGC(128, 128, 64, 2)
        default: check(false, "tile not instantiated for the raw epilogue");
      }
      return;
    }
    if constexpr (EPI == EPI_SPLIT) {  // split-reduction configurations
      switch (key) {
        IGC(128, 128, 64, 2)
        IGC(64, 64, 64, 4)
        default: check(false, "tile not instantiated for split reduction");
      }
      return;
    }
    switch (key) {
      IGC(64, 64, 32, 2)
      IGC(128, 128, 64, 2)
      IGC(256, 128, 32, 2)
      IGC(128, 64, 64, 2)
      IGC(64, 128, 64, 4)
      IGC(64, 64, 64, 4)
      IGC(128, 64, 32, 4)
      IGC(64, 128, 64, 2)
      IGC(128, 128, 32, 4)
      IGC(64, 128, 32, 4)
      IGC(128, 64, 64, 4)
      IGC(64, 128, 128, 2)
      IGC(128, 64, 128, 2)
      IGC(128, 128, 128, 2)
      case ((96 * 1000 + 128) * 100 + 64) * 10 + 2:
        if constexpr (VEC) igemm_go<T, L, VEC, 96, 128, 64, EPI, 2>(a, batch, st);
        else check(false, "96-row tiles need the vector loader");
        break;
      default: check(false, "implicit-GEMM tile not instantiated");
    }
#undef IGC
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
  a.x_elems = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w;
  a.w_elems = (long long)((a.K + 7) / 8 * 8) * a.Kred;
  a.y_elems = (long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w;
  a.inv_pq = 1.f / (float)std::max(a.PQ, 1);
  a.inv_q = 1.f / (float)std::max(a.Q, 1);
  a.res = c.res;
  a.x2 = c.x2;
  a.w2 = c.w2;
  if (c.x2) {
    a.H2 = c.x2d.h;
    a.W2 = c.x2d.w;
    a.Cs2 = c.x2d.cs;
    a.CB2 = (c.x2d.c + 7) / 8;
    a.KC2 = a.CB2;
    a.Kred2 = a.CB2 * 8;
    a.stride2 = c.stride2;
    a.x2_elems = (long long)c.x2d.n * c.x2d.cs * c.x2d.h * c.x2d.w;
    a.w2_elems = (long long)((a.K + 7) / 8 * 8) * a.Kred2;
  }
  return a;
}


template <typename T, int L, bool VEC>
static void igemm_run(const IgCfg& cfg, IgArgs& a, const ConvArgs& c, hipStream_t st) {
  if (cfg.split == 2) {
    // one kernel: with a single split it is the plain layout epilogue
    if (a.splits > 1) {
      check(c.ws && c.ws_bytes >= (size_t)a.splits * a.tiles_m * a.tiles_n * cfg.bm * cfg.bn * sizeof(float),
            "split-K workspace too small");
      check(c.cnt && a.tiles_m * a.tiles_n <= kFixupMaxTiles, "split-K tile counters");
      a.part = reinterpret_cast<float*>(c.ws);
      a.cnt = c.cnt;
    }
    igemm_cfg<T, L, VEC, EPI_FIXUP>(cfg, a, 1, st);
    return;
  }
  if (a.splits > 1) {
    check(c.ws && c.ws_bytes >= (size_t)a.splits * a.M * a.Ng * sizeof(float), "split-K workspace too small");
    a.part = reinterpret_cast<float*>(c.ws);
    igemm_cfg<T, L, VEC, EPI_SPLIT>(cfg, a, 1, st);
    const long long n = L == NCHW ? (long long)a.M * a.Ng : (long long)a.M * ((a.Ng + 7) / 8);
    SN_LAUNCH((splitk_reduce_kernel<T, L>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, a);
  } else {
    igemm_cfg<T, L, VEC, EPI_LAYOUT>(cfg, a, 1, st);
  }
}

template <typename T>
static void igemm_dispatch(int dtype, int param, const ConvArgs& c, hipStream_t st) {
  const IgCfg cfg = ig_cfg(dtype, param);
  check(!c.res || cfg.dma == 0 || ((cfg.dma == 1 || cfg.dma == 4) && (c.yd.layout == NC8 || c.yd.cs % 8 == 0)),
        "this tile configuration takes no residual");
  check(!c.x2 || cfg.dma == 4 ||
            (cfg.dma == 1 && cfg.split != 1 && !c.res && c.x2d.layout == c.xd.layout &&
             (long long)c.x2d.n * c.x2d.cs * c.x2d.h * c.x2d.w * 2 < (long long)kOOB && c.x2d.c % cfg.bk == 0),
        "a projected shortcut runs on the LDS-DMA tiles or the streaming kernel, in the convolution's layout");
  if (cfg.dma == 2) {
    conv_patch(dtype, cfg.pc, c, st);
    return;
  }
  if (cfg.dma == 3) {
    conv_smallc(dtype, cfg.bm / 16, cfg.gmax, c, st, cfg.wm, cfg.st);
    return;
  }
  if (cfg.dma == 4) {
    conv1x1_stream(dtype, cfg.bk, cfg.bm, cfg.bn, cfg.pf, c, st, cfg.st);
    return;
  }
  IgArgs a = make_ig(c);
  check(c.xd.layout == c.yd.layout, "implicit GEMM reads and writes one layout");
  check((long long)a.M * a.Ks < (1ll << 31) && (long long)c.xd.n * a.Cs * a.H * a.W < (1ll << 31),
        "tensor too large");
  ig_decompose(a, cfg);
  switch (c.xd.layout) {
    case NCHW: igemm_run<T, NCHW, false>(cfg, a, c, st); break;
    case NHWC:
      if (a.C % 8 == 0)
        igemm_run<T, NHWC, true>(cfg, a, c, st);
      else
        igemm_run<T, NHWC, false>(cfg, a, c, st);
      break;
    case NC8: igemm_run<T, NC8, true>(cfg, a, c, st); break;
    default: check(false, "layout");
  }
}

// 16-bit implicit-GEMM dispatch (conv_igemm_f16.hip, conv_igemm_bf16.hip)
void conv_igemm_f16(int param, const ConvArgs& c, hipStream_t st);
void conv_igemm_bf16(int param, const ConvArgs& c, hipStream_t st);

}  // namespace k
}  // namespace sn
