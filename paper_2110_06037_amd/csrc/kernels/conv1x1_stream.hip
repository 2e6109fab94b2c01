// 1x1 convolution (stride 1 or 2, no padding) of an NHWC input with CC =
// 64, 128, 256, 384 or 512 channels (16-bit types), an implicit-GEMM routine for the pointwise layers
// of a bottleneck whose reduction is short.
//
// Such a layer reads each pixel once and writes K channels (plus a residual
// of K channels when an add is folded in), so memory traffic, not MFMA work,
// bounds it, and its reduction takes one to four 64-wide steps: a workgroup
// of the tiled implicit GEMM loads its tiles, waits, computes and stores with
// little to overlap.  Here workgroups are persistent: each keeps its BN
// filter rows in LDS and streams tiles of BM pixels, loading the pixels (LDS
// direct loads) and the residual (into registers) of the tile PD tiles ahead
// while the current tile's MFMAs and stores run, so PD tiles' loads are in
// flight per workgroup (the residual comes from HBM and a tile's own work is
// far shorter than a load's latency); each wave holds its filter
// fragments in registers, so LDS serves only pixel fragments.  The tile's fp32 sums go
// through LDS so that the residual add and the stores move whole 16-byte
// chunks of consecutive channels with consecutive lanes on consecutive
// addresses.  In LDS a tile is CC / 64 slabs of 64 channels, each with
// 128-byte rows (8 chunks); chunk c of row r sits at c ^ ((r >> 1) & 7),
// which serves an MFMA operand read of 16 consecutive rows in one pass.
//
// With a projected shortcut (PJ) the reduction runs over the main input's
// slabs and then the shortcut's (C1 + C2 = CC channels): the shortcut's slabs
// load pixel (img, p * stride2, q * stride2) of its own tensor, and the
// filter rows hold both weights ([Kp][C1 + C2]); nothing else changes.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

struct StreamArgs {
  const void* x;     // [N][H][W][CC] (with a projected shortcut: [N][H][W][C1])
  const void* w;     // [Kp][CC]
  const float* bias; // [Kp]
  const void* res;   // [M][Ks] or null
  void* y;           // [M][Ks], M = N * P * Q output pixels
  int M, K, Ks, act;
  int H, W, P, Q, stride;
  FastDiv fd_pq, fd_q;
  int tiles_m;
  long long x_elems, w_elems, y_elems;
  const void* x2;    // projected shortcut [N][H2][W2][C2], or null
  int H2, W2, stride2, C1, C2;
  long long x2_elems;
};

template <int V>
using SIC = std::integral_constant<int, V>;

// OCC: workgroups per CU (the launch bound counts waves per SIMD: 2 OCC)
template <typename T, int CC, int BM, int BN, int WM, bool RES, int PD, bool PJ = false, int OCC = 1>
__global__ __launch_bounds__(512, 2 * OCC) void conv1x1_stream_kernel(StreamArgs a) {
  static_assert(sizeof(T) == 2 && CC % 64 == 0, "16-bit types, 64-channel slabs");
  static_assert(!(PJ && RES), "a projected shortcut replaces the residual");
  static_assert(PD >= 1 && PD <= 3, "one to three tiles ahead");
  constexpr int NB = PD + 1;                   // pixel buffers and residual register sets
  constexpr int NWV = 8, NT = 512, WN = NWV / WM;
  constexpr int RB = 128;                      // LDS row of a slab: 64 channels
  constexpr int NSL = CC / 64;                 // slabs
  constexpr int WTM = BM / WM, WTN = BN / WN, FM = WTM / 16, FN = WTN / 16;
  constexpr int NA = NSL * BM * RB / 1024 / NWV;   // pixel-tile load instructions per wave
  constexpr int NBL = NSL * BN * RB / 1024 / NWV;  // filter load instructions per wave
  constexpr int NEC = BM * BN / 8;                 // 16-byte output chunks per tile
  // chunks per thread and tile; with fewer chunks than threads the rest
  // issue their stores (and residual loads) at out-of-range offsets, so every
  // wave counts the same memory instructions
  constexpr int NE = (NEC + NT - 1) / NT;
  static_assert(NA >= 1 && NBL >= 1 && NE >= 1 && NA * 1024 * NWV == NSL * BM * RB &&
                    NBL * 1024 * NWV == NSL * BN * RB && (NEC % NT == 0 || NE == 1) && FM >= 1 && FN >= 1,
                "tile shape");
  constexpr int YR = RES ? NE : 0;             // residual loads per thread and tile
  static_assert(PD * (NA + YR + NE) <= 63, "outstanding-load counter range");
  constexpr int A_BYTES = NSL * BM * RB, B_BYTES = NSL * BN * RB;
  constexpr int CP = BN + 4;                   // fp32 staging row pitch (floats)
  constexpr int CS_BYTES = BM * CP * 4;
  // when a staging buffer of its own does not fit, a tile's sums are staged
  // in the tile's own pixel buffer once every wave has read it (ALIAS); the
  // loads of a later tile into a buffer then wait for the barrier after
  // which no wave reads that buffer's staging any more
  constexpr int LDS_CAP = 160 * 1024 / OCC;
  constexpr bool ALIAS = B_BYTES + NB * A_BYTES + CS_BYTES + BN * 4 > LDS_CAP;
  static_assert(!ALIAS || A_BYTES >= CS_BYTES, "staging fits the pixel buffer");
  constexpr int SM = B_BYTES + NB * A_BYTES + (ALIAS ? 0 : CS_BYTES) + BN * 4;
  static_assert(SM <= LDS_CAP, "LDS capacity at the occupancy");
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  char* const Bs = smem;
  char* const As = smem + B_BYTES;
  float* const Cs0 = reinterpret_cast<float*>(As + NB * A_BYTES);  // the staging buffer (without ALIAS)
  float* const Bias = reinterpret_cast<float*>(As + NB * A_BYTES + (ALIAS ? 0 : CS_BYTES));
  auto swz = [](int row) { return (row >> 1) & 7; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int n0 = blockIdx.y * BN;
  const int G = gridDim.x;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, a.w_elems * 2);
  const __amdgpu_buffer_rsrc_t ry = make_rsrc(a.y, a.y_elems * 2);
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(RES ? a.res : a.y, a.y_elems * 2);
  const __amdgpu_buffer_rsrc_t rx2 = make_rsrc(PJ ? a.x2 : a.x, PJ ? a.x2_elems * 2 : 0);

  // bias of the workgroup's channels through LDS (no global load of it
  // stays outstanding in the tile loop)
  if (tid < BN) Bias[tid] = n0 + tid < a.K ? a.bias[n0 + tid] : 0.f;

  // load slots: instruction b = wave + 8 i fills rows [8 r, 8 r + 8) of
  // slab s (b = s * rows / 8 + r); this lane fills row 8 r + lane / 8,
  // physical chunk lane % 8 = logical chunk (lane % 8) ^ swz(row) of the slab
  const int prow = lane >> 3, pch = lane & 7;
#pragma unroll
  for (int i = 0; i < NBL; ++i) {
    const int b = wave + NWV * i, sl = b / (BN / 8), row = (b % (BN / 8)) * 8 + prow;
    const int k = n0 + row;
    const unsigned off = k < a.K ? (unsigned)(k * CC + sl * 64 + ((pch ^ swz(row)) << 3)) * 2u : kOOB;
    dma16(rw, Bs + b * 1024, off, 0);
  }
  unsigned achk[NA];  // the lane's chunk within a pixel's channels (bytes)
  int arow[NA];
  bool asc[NA];       // (PJ) the slab is the shortcut's (wave-uniform)
  const int nsl1 = PJ ? a.C1 / 64 : NSL;
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int b = wave + NWV * i, sl = b / (BM / 8), row = (b % (BM / 8)) * 8 + prow;
    arow[i] = row;
    asc[i] = PJ && sl >= nsl1;
    achk[i] = (unsigned)((asc[i] ? sl - nsl1 : sl) * 64 + ((pch ^ swz(row)) << 3)) * 2u;
  }
  const unsigned xpix = (unsigned)(PJ ? a.C1 : CC) * 2u, x2pix = (unsigned)(PJ ? a.C2 : 0) * 2u;
  // output pixel m reads input pixel m (stride 1) or (img, 2p, 2q) (stride
  // 2); a tile past the end loads nothing (out-of-range offsets) but still
  // counts its load instructions, so every wait below has a fixed count
  auto issue_a = [&](int mtile, int buf) {
    const int m0 = mtile * BM;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int m = m0 + arow[i];
      const bool ok = mtile < a.tiles_m && m < a.M;
      if (PJ && asc[i]) {
        const int img = fdiv(m, a.fd_pq), pq = m - img * (a.P * a.Q);
        const int p = fdiv(pq, a.fd_q), q = pq - p * a.Q;
        const int pix2 = (img * a.H2 + p * a.stride2) * a.W2 + q * a.stride2;
        dma16(rx2, As + buf * A_BYTES + (wave + NWV * i) * 1024, ok ? (unsigned)pix2 * x2pix + achk[i] : kOOB, 0);
        continue;
      }
      int pix = m;
      if (a.stride != 1) {
        const int img = fdiv(m, a.fd_pq), pq = m - img * (a.P * a.Q);
        const int p = fdiv(pq, a.fd_q), q = pq - p * a.Q;
        pix = (img * a.H + p * a.stride) * a.W + q * a.stride;
      }
      dma16(rx, As + buf * A_BYTES + (wave + NWV * i) * 1024, ok ? (unsigned)pix * xpix + achk[i] : kOOB, 0);
    }
  };
  u32x4 res[NB][NE];  // residual register sets, one per tile in flight
  auto load_res = [&](int mtile, u32x4 (&r)[NE]) {
    const int m0r = mtile * BM;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int q = tid + e * NT, qc = q < NEC ? q : 0, row = qc / (BN / 8), cj = qc % (BN / 8);
      const int m = m0r + row, n = n0 + cj * 8;
      const unsigned off =
          q < NEC && mtile < a.tiles_m && m < a.M && n < a.K ? (unsigned)(m * a.Ks + n) * 2u : kOOB;
      r[e] = __builtin_amdgcn_raw_buffer_load_b128(rr, (int)off, 0, 0);
    }
  };
  // the loads of one tile: residual first, then pixels
  auto issue_tile = [&](int mtile, auto BC) {
    constexpr int B = decltype(BC)::value;
    if constexpr (RES) load_res(mtile, res[B]);
    __builtin_amdgcn_sched_barrier(0);
    issue_a(mtile, B);
    __builtin_amdgcn_sched_barrier(0);
  };

  // operand chunk offsets of the 32-wide reduction steps ks (slab ks / 2;
  // 16-row blocks keep the lane's swizzle)
  constexpr int KS = CC / 32;
  int aofs[KS], bofs[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const int l = lane & 15, xo = (((ks % 2) * 4 + (lane >> 4)) ^ swz(l)) << 4;
    aofs[ks] = (ks / 2) * BM * RB + (wm * WTM + l) * RB + xo;
    bofs[ks] = (ks / 2) * BN * RB + (wn * WTN + l) * RB + xo;
  }
  typedef typename Mfma<T>::frag frag;
  const ActClamp ac = act_clamp(a.act);

  const int mt0 = blockIdx.x;
  // prologue: the first PD tiles' loads (tile j into buffer and set j)
  issue_tile(mt0, SIC<0>{});
  if constexpr (PD > 1) issue_tile(mt0 + G, SIC<1>{});
  if constexpr (PD > 2) issue_tile(mt0 + 2 * G, SIC<2>{});
  // the filter and the first tile have landed once only the later tiles'
  // loads remain outstanding
  wait_vmcnt<(PD - 1) * (YR + NA)>();
  __syncthreads();  // every wave's filter share, first pixel tile and the bias are in LDS
  // the wave's filter fragments stay in registers for the whole kernel, so
  // the tile loop reads only pixel fragments from LDS
  frag fbr[KS][FN];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
#pragma unroll
    for (int j = 0; j < FN; ++j) fbr[ks][j] = *reinterpret_cast<const frag*>(Bs + bofs[ks] + j * 16 * RB);
  float bias[FN][4];
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) bias[j][v] = Bias[wn * WTN + j * 16 + (lane >> 4) * 4 + v];

  // tile t (index mt0 + t * G) uses buffer and residual set U = t % NB; it
  // first issues the loads of tile t + PD into set (U + PD) % NB (the set
  // tile t - 1 used), then waits for its own: younger than them are the
  // loads of the PD later tiles and the stores of the last min(t, PD)
  // tiles.  Returns whether tile t + 1 exists.
  auto tile = [&](auto UC, int t) {
    constexpr int U = decltype(UC)::value;
    constexpr int NX = (U + PD) % NB;
    const int mt = mt0 + t * G;
    float* const Cs = ALIAS ? reinterpret_cast<float*>(As + U * A_BYTES) : Cs0;
    if constexpr (!ALIAS) {
      issue_tile(mt + PD * G, SIC<NX>{});
      if (t < PD) wait_vmcnt<PD * (YR + NA) + (U < PD ? U : PD) * NE>();
      else wait_vmcnt<PD * (YR + NA + NE)>();
      dma_barrier();  // every wave's share landed; every wave is done with the last tile's Cs
    } else {
      // younger than this tile's loads: the PD - 1 later tiles' loads and
      // the stores of the last min(t, PD) tiles
      if (t < PD) wait_vmcnt<(PD - 1) * (YR + NA) + (U < PD ? U : PD) * NE>();
      else wait_vmcnt<(PD - 1) * (YR + NA) + PD * NE>();
      dma_barrier();  // every wave's share landed; no wave reads the last tile's staging
      issue_tile(mt + PD * G, SIC<NX>{});
    }

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{bias[j][0], bias[j][1], bias[j][2], bias[j][3]};
    const char* A = As + U * A_BYTES;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      frag fa[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) fa[i] = *reinterpret_cast<const frag*>(A + aofs[ks] + i * 16 * RB);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(fbr[ks][j], fa[i], acc[i][j]);
    }
    if constexpr (ALIAS) lds_barrier();  // every wave has read the tile's pixels
    // sums (bias included) to LDS: element (i, j, v) is pixel
    // wm*WTM + i*16 + (lane&15), channel wn*WTN + j*16 + (lane>>4)*4 + v
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        *reinterpret_cast<f32x4*>(Cs + (wm * WTM + i * 16 + (lane & 15)) * CP + wn * WTN + j * 16 + (lane >> 4) * 4) =
            acc[i][j];
    lds_barrier();
    const int m0 = mt * BM;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int q = tid + e * NT, qc = q < NEC ? q : 0, row = qc / (BN / 8), cj = qc % (BN / 8);
      const int m = m0 + row, n = n0 + cj * 8;
      const unsigned off = q < NEC && m < a.M && n < a.K ? (unsigned)(m * a.Ks + n) * 2u : kOOB;
      const f32x4 c0 = *reinterpret_cast<const f32x4*>(Cs + row * CP + cj * 8);
      const f32x4 c1 = *reinterpret_cast<const f32x4*>(Cs + row * CP + cj * 8 + 4);
      float s[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
      if constexpr (RES) {
        T rt[8];
        __builtin_memcpy(rt, &res[U][e], 16);
#pragma unroll
        for (int v = 0; v < 8; ++v) s[v] += to_f(rt[v]);
      }
      T o[8];
#pragma unroll
      for (int v = 0; v < 8; ++v) o[v] = from_f<T>(__builtin_amdgcn_fmed3f(s[v], ac.lo, ac.hi));
      u32x4 pk;
      __builtin_memcpy(&pk, o, 16);
      __builtin_amdgcn_raw_buffer_store_b128(pk, ry, (int)off, 0, 0);
    }
    return mt + G < a.tiles_m;
  };
  // the loop is unrolled by NB so that buffers and residual sets are
  // compile-time indices
  for (int t = 0;; t += NB) {
    if (!tile(SIC<0>{}, t)) break;
    if (!tile(SIC<1>{}, t + 1)) break;
    if constexpr (NB > 2) {
      if (!tile(SIC<2>{}, t + 2)) break;
    }
    if constexpr (NB > 3) {
      if (!tile(SIC<3>{}, t + 3)) break;
    }
  }
  // the loads issued for tiles past the end target LDS: let them land
  // before the workgroup ends
  wait_vmcnt<0>();
}

bool stream1x1_takes_projection(int layout, int c, int cs, int n, int h, int w, int r, int s, int stride, int pad,
                                int k, int c2, int cc) {
  return layout == NHWC && c % 64 == 0 && cs == c && c2 % 64 == 0 && c + c2 == cc && r == 1 && s == 1 &&
         stride == 1 && pad == 0 && k % 8 == 0 && (long long)n * h * w * ((k + 7) / 8 * 8) * 2 < (long long)kOOB &&
         (long long)n * h * w * c * 2 < (long long)kOOB;
}

bool stream1x1_applicable(int layout, int c, int cs, int n, int h, int w, int r, int s, int stride, int pad,
                          int k, int cc) {
  const long long p = (h - 1) / stride + 1, q = (w - 1) / stride + 1;
  return layout == NHWC && c == cc && cs == cc && r == 1 && s == 1 && (stride == 1 || stride == 2) &&
         pad == 0 && k % 8 == 0 && (long long)n * h * w * cc * 2 < (long long)kOOB &&
         (long long)n * p * q * ((k + 7) / 8 * 8) * 2 < (long long)kOOB;
}

template <typename T, int CC, int BM, int BN, int WM, int PD, int OCC = 1>
static void stream_go(const StreamArgs& a, int tiles_n, hipStream_t st) {
  // persistent: about OCC workgroups per CU over all channel tiles
  const int gx = std::max(1, std::min(a.tiles_m, 256 * OCC / tiles_n));
  const dim3 grid(gx, tiles_n);
  if (a.x2) {
    if constexpr (CC >= 128)
      SN_LAUNCH((conv1x1_stream_kernel<T, CC, BM, BN, WM, false, PD, true, OCC>), grid, dim3(512), 0, st, a);
    else check(false, "a projected shortcut needs two slabs or more");
  } else if (a.res) {
    SN_LAUNCH((conv1x1_stream_kernel<T, CC, BM, BN, WM, true, PD, false, OCC>), grid, dim3(512), 0, st, a);
  } else {
    SN_LAUNCH((conv1x1_stream_kernel<T, CC, BM, BN, WM, false, PD, false, OCC>), grid, dim3(512), 0, st, a);
  }
}

void conv1x1_stream(int dtype, int cc, int bm, int bn, int pd, const ConvArgs& c, hipStream_t st, int occ) {
  check(dtype != 0, "streaming 1x1 kernel runs 16-bit types");
  const long long m = (long long)c.yd.n * c.yd.h * c.yd.w;
  if (c.x2) {
    check(c.x2d.layout == NHWC && c.wcat && !c.res && c.yd.h == (c.x2d.h - 1) / c.stride2 + 1 &&
              c.yd.w == (c.x2d.w - 1) / c.stride2 + 1 && c.x2d.cs == c.x2d.c &&
              (long long)c.x2d.n * c.x2d.h * c.x2d.w * c.x2d.c * 2 < (long long)kOOB &&
              stream1x1_takes_projection(c.xd.layout, c.xd.c, c.xd.cs, c.xd.n, c.xd.h, c.xd.w, c.r, c.s, c.stride,
                                         c.pad, c.yd.c, c.x2d.c, cc),
          "streaming 1x1 kernel with a projected shortcut: NHWC, C + C2 = CC, both multiples of 64");
  } else {
    check(c.xd.layout == NHWC && c.yd.layout == NHWC && c.stride >= 1 &&
              c.yd.h == (c.xd.h - 1) / c.stride + 1 && c.yd.w == (c.xd.w - 1) / c.stride + 1 &&
              stream1x1_applicable(c.xd.layout, c.xd.c, c.xd.cs, c.xd.n, c.xd.h, c.xd.w, c.r, c.s, c.stride,
                                   c.pad, c.yd.c, cc),
          "streaming 1x1 kernel: NHWC, C = CC, 1x1 stride 1 or 2 without padding, K % 8 == 0");
  }
  StreamArgs a{};
  a.x = c.x;
  a.w = c.x2 ? c.wcat : c.w;
  a.bias = c.bias;
  a.res = c.res;
  a.y = c.y;
  a.M = (int)m;
  a.K = c.yd.c;
  a.Ks = c.yd.cs;
  a.act = c.act;
  a.tiles_m = (int)((m + bm - 1) / bm);
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.P = c.yd.h;
  a.Q = c.yd.w;
  a.stride = c.stride;
  a.fd_pq = make_fastdiv(a.P * a.Q);
  a.fd_q = make_fastdiv(a.Q);
  a.x_elems = (long long)c.xd.n * c.xd.h * c.xd.w * (c.x2 ? c.xd.c : cc);
  if (c.x2) {
    a.x2 = c.x2;
    a.H2 = c.x2d.h;
    a.W2 = c.x2d.w;
    a.stride2 = c.stride2;
    a.C1 = c.xd.c;
    a.C2 = c.x2d.c;
    a.x2_elems = (long long)c.x2d.n * c.x2d.h * c.x2d.w * c.x2d.c;
  }
  a.w_elems = (long long)((a.K + 7) / 8 * 8) * cc;
  a.y_elems = m * a.Ks;
  const int tiles_n = (a.K + bn - 1) / bn;
#define SG(CC_, BM_, BN_, WM_, PD_)                                              \
  if (cc == CC_ && bm == BM_ && bn == BN_ && pd == PD_ && occ == 1) {            \
    if (dtype == 1) stream_go<f16, CC_, BM_, BN_, WM_, PD_>(a, tiles_n, st);     \
    else stream_go<bf16, CC_, BM_, BN_, WM_, PD_>(a, tiles_n, st);               \
    return;                                                                      \
  }
#define SG2(CC_, BM_, BN_, WM_, PD_)                                             \
  if (cc == CC_ && bm == BM_ && bn == BN_ && pd == PD_ && occ == 2) {            \
    if (dtype == 1) stream_go<f16, CC_, BM_, BN_, WM_, PD_, 2>(a, tiles_n, st);  \
    else stream_go<bf16, CC_, BM_, BN_, WM_, PD_, 2>(a, tiles_n, st);            \
    return;                                                                      \
  }
  STREAM_CONFIGS(SG)
  STREAM512_CONFIGS(SG)
  STREAM_OCC2_CONFIGS(SG2)
#undef SG
#undef SG2
  check(false, "streaming 1x1 tile not instantiated");
}

}  // namespace k
}  // namespace sn
