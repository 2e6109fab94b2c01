// 3x3 stride-1 convolution as an implicit GEMM whose input tile is a
// spatial patch kept in LDS.
//
// A workgroup computes the outputs of TI whole images, or of TR consecutive
// output rows of one image (all Q columns), for BN output channels.  For
// every step of BK input channels it loads the tile's input patch -- the
// (TR + 2) x (Q + 2) input pixels (one halo pixel on each side; the zero
// padding comes from out-of-range buffer offsets) -- and the filter taps of
// those channels for all 9 taps, then runs the 9 taps' MFMAs out of LDS: tap
// (r, s) of output pixel (p, q) is patch pixel (p + r, q + s), so the per-tap
// operand rows are the same patch rows shifted by the uniform offset
// r * (Q + 2) + s.  Each input element therefore crosses the memory system
// about (TR + 2) / TR times per workgroup instead of 9 times, which is what
// bounds the per-tap (im2col) implicit GEMM on this chip.
//
// Tiles move from global memory into LDS with direct loads (16 bytes per
// lane, 1 KB per wave instruction in lane order).  LDS rows are padded by one
// 16-byte chunk (the lanes that land on a pad chunk load zeros), so 16
// consecutive rows of one chunk hit distinct banks and every operand address
// is a per-lane base plus compile-time offsets: tap (r, s) adds r row-strides
// of the patch (one add per row block and r) and s padded rows (an
// instruction immediate).  The MFMA takes the filter as its first operand, so
// each lane's 4 accumulators are 4 consecutive output channels of one
// pixel; the epilogue adds the bias, applies the activation and stores
// through LDS as 16-byte rows.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

struct PatchArgs {
  const void* x;
  const void* w;  // [Kp][3][3][C8]
  const float* bias;
  void* y;
  int N, C, H, W, Cs;  // input (H = P, W = Q: stride 1, pad 1)
  int K, P, Q, Ks, Ng;
  int act;
  int CB, C8, Kred;      // channel blocks of 8, padded channels, weight row length 9 * C8
  int TI, TR, PH, PW;    // images / output rows per tile, patch rows / columns per image
  int tiles_img;         // row tiles per image
  int tiles_m, tiles_n;
  FastDiv fd_ti_tiles;                    // division by tiles_img
  float inv_pw, inv_ph, inv_trq, inv_q;   // 1/PW, 1/PH, 1/(TR*Q), 1/Q for sdiv
  int HW8, W8;                            // NC8HW8 strides: H*W*8, W*8
  int lpw;                                // log2 of the patch row pitch PW
  float inv_pq;                           // 1/(P*Q) for sdiv
  long long y_elems;
  long long x_elems, w_elems;
};

// FMT: MFMA row blocks (16 pixels) per tile; BN output channels; BK input
// channels per step; WM wave rows (of 4 waves); ST LDS stages; PPX patch
// capacity in pixels.
template <typename T, int L, int FMT, int BN, int BK, int WM, int ST, int PPX, int OCC>
__global__ __launch_bounds__(256, OCC) void conv3x3_patch_kernel(PatchArgs a) {
  static_assert(sizeof(T) == 2 && L != NCHW, "16-bit channel-vector layouts only");
  static_assert(BK == 32, "one 16x16x32 MFMA k-slice per step");
  static_assert(BN == 32 || BN == 64, "filter rows per load round must be whole taps");
  constexpr int WN = 4 / WM;
  constexpr int CPR = BK / 8;     // 16-byte chunks per 64-byte LDS row
  constexpr int RB = BK * 2;      // bytes per LDS row
  constexpr int PROWS = (PPX + 63) / 64 * 64;           // patch rows (whole load rounds)
  constexpr int WROWS = (9 * BN + 63) / 64 * 64;        // filter rows
  constexpr int NP = PROWS / 64, NW = WROWS / 64;       // load instructions per wave and step
  static_assert(ST == 1 || ST == 2, "one or two LDS stages");
  constexpr int FMW = (FMT + WM - 1) / WM;  // row blocks per wave
  constexpr int WTN = BN / WN, FNW = WTN / 16;
  static_assert(FNW * 16 * WN == BN, "BN must split over the wave columns");
  constexpr int P_BYTES = PROWS * RB, STAGE = (PROWS + WROWS) * RB;
  constexpr int CPAD = 8;
  constexpr int SM_C = FMT * 16 * (BN + CPAD) * 2;
  constexpr int SM = ST * STAGE > SM_C ? ST * STAGE : SM_C;
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  lds_char* const sl = (lds_char*)smem;
  // 16-byte chunk c of LDS row r sits at chunk c ^ swz(r): any 16 consecutive
  // rows of one chunk then cover all 16 chunk positions of a 256-byte bank line
  auto swz = [](int row) { return (row >> 2) & 3; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  tile_of(blockIdx.x, a.tiles_m, a.tiles_n, mt, nt);
  const int ig = fdiv(mt, a.fd_ti_tiles), rt = mt - ig * a.tiles_img;
  const int img0 = ig * a.TI;
  const int row0 = rt * a.TR;
  const int imgs = min(a.TI, a.N - img0);
  const int rows = min(a.TR, a.P - row0);
  const int n0 = nt * BN;
  const int KT = a.CB / CPR;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, a.w_elems * 2);

  // Patch rows are (image, ph, pw) with a row pitch PW (a multiple of 16
  // that divides 64, at least Q + 2; columns past Q + 2 load zeros).  Load
  // instruction q = wave + 4 i fills LDS rows [16 q, 16 q + 16): this lane
  // fills row 16 q + lane / 4, physical chunk lane % 4 (logical chunk
  // (lane % 4) ^ swz(row)).  Consecutive i add 64 rows, i.e. 64 / PW patch
  // rows at the same column.  (Index arithmetic: 24-bit multiplies and fp32
  // division; every value is far below 2^24.)
  const int r0 = wave * 16 + (lane >> 2);
  const int pw = r0 & (a.PW - 1), ww = pw - 1;
  const int prow0 = r0 >> a.lpw;
  const int lcp = (lane & 3) ^ swz(r0);  // row + 64 i keeps swz
  unsigned poff[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int prow = prow0 + (i << (6 - a.lpw));
    const int ii = sdiv(prow, a.inv_ph), ph = prow - __umul24(ii, a.PH);
    const int img = img0 + ii, h = row0 - 1 + ph;
    const bool ok = ii < a.TI && img < a.N && (unsigned)h < (unsigned)a.H && (unsigned)ww < (unsigned)a.W;
    unsigned e;
    if constexpr (L == NC8)
      e = __umul24(__umul24(img, a.CB) + lcp, a.HW8) + __umul24(h, a.W8) + ww * 8;
    else
      e = __umul24(__umul24(__umul24(img, a.H) + h, a.W) + ww, a.Cs) + lcp * 8;
    poff[i] = ok ? e * 2u : kOOB;
  }
  // filter rows (tap, channel): + 64 rows = + 64 / BN taps, same channel
  const int tap0 = r0 / BN, kch = n0 + r0 % BN;
  const unsigned wof0 = (__umul24(kch, a.Kred) + __umul24(tap0, a.C8) + lcp * 8) * 2u;
  unsigned woff[NW];
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int tap = tap0 + i * (64 / BN);
    woff[i] = tap < 9 && kch < a.Ng ? wof0 + (unsigned)(i * (64 / BN)) * (unsigned)a.C8 * 2u : kOOB;
  }
  // per-step uniform offsets of channel block kt * CPR
  const int xstep = L == NC8 ? CPR * a.HW8 * 2 : BK * 2;
  auto issue = [&](int buf, int kt) {
    lds_char* base = sl + buf * STAGE + wave * 1024;
#pragma unroll
    for (int i = 0; i < NP; ++i) dma16(rx, base + i * 4096, poff[i], kt * xstep);
#pragma unroll
    for (int i = 0; i < NW; ++i) dma16(rw, base + P_BYTES + i * 4096, woff[i], kt * BK * 2);
  };
  issue(0, 0);  // the first step's tiles travel while the offsets below are computed

  // accumulators start at the bias of the lane's output channels
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.bias, (long long)a.Ng * 4);
  typedef typename Mfma<T>::frag frag;
  f32x4 acc[FMW][FNW];
#pragma unroll
  for (int j = 0; j < FNW; ++j) {
    const int n = n0 + wn * WTN + j * 16 + (lane >> 4) * 4;
    f32x4 b;
#pragma unroll
    for (int v = 0; v < 4; ++v) b[v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rb, (n + v) * 4, 0, 0));
#pragma unroll
    for (int i = 0; i < FMW; ++i) acc[i][j] = b;
  }

  // LDS byte offsets (within a stage) of this lane's operand chunks for every
  // tap: the three column taps of a pixel row block computed, the tap rows
  // one pitch apart (a multiple of 16 rows, so the swizzle is unchanged)
  int aoff[FMW][9];
  const int rowpitch = a.PW * RB;
#pragma unroll
  for (int i = 0; i < FMW; ++i) {
    const int m = (wm * FMW + i) * 16 + (lane & 15);
    const int ii = sdiv(m, a.inv_trq), rem = m - __umul24(ii, a.TR * a.Q);
    const int pr = sdiv(rem, a.inv_q), pc = rem - __umul24(pr, a.Q);
    const int pb = ii < a.TI ? __umul24(ii, a.PH * a.PW) + __umul24(pr, a.PW) + pc : 0;
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const int r = pb + c;
      aoff[i][c] = (r << 6) | (((lane >> 4) ^ swz(r)) << 4);
      aoff[i][3 + c] = aoff[i][c] + rowpitch;
      aoff[i][6 + c] = aoff[i][c] + 2 * rowpitch;
    }
  }
  const int boff = P_BYTES + (wn * WTN + (lane & 15)) * RB + (((lane >> 4) ^ ((lane >> 2) & 3)) << 4);

  // the fragments of tap t+1 are read from LDS while tap t's MFMAs run
  auto load_frags = [&](const char* S, int tap, frag(&fa)[FMW], frag(&fb)[FNW]) {
#pragma unroll
    for (int i = 0; i < FMW; ++i)
      if (wm * FMW + i < FMT) fa[i] = *reinterpret_cast<const frag*>(S + aoff[i][tap]);
#pragma unroll
    for (int j = 0; j < FNW; ++j) fb[j] = *reinterpret_cast<const frag*>(S + boff + (tap * BN + j * 16) * RB);
  };
  auto compute = [&](int buf) {
    const char* S = smem + buf * STAGE;
    frag fa[2][FMW], fb[2][FNW];
    load_frags(S, 0, fa[0], fb[0]);
#pragma unroll
    for (int u = 0; u < 9; ++u) {
      if (u + 1 < 9) load_frags(S, u + 1, fa[(u + 1) & 1], fb[(u + 1) & 1]);
#pragma unroll
      for (int i = 0; i < FMW; ++i)
        if (wm * FMW + i < FMT)
#pragma unroll
          for (int j = 0; j < FNW; ++j) acc[i][j] = Mfma<T>::run(fb[u & 1][j], fa[u & 1][i], acc[i][j]);
    }
  };

  if constexpr (ST == 1) {
    // one LDS stage: load, compute, and only then load the next step (the
    // other workgroups on the CU keep its MFMAs busy meanwhile)
    for (int t = 0; t < KT; ++t) {
      if (t > 0) issue(0, t);
      wait_vmcnt<0>();
      dma_barrier();
      compute(0);
      dma_barrier();
    }
  } else {
    for (int t = 0; t < KT; ++t) {
      wait_vmcnt<0>();
      dma_barrier();
      if (t + 1 < KT) issue((t + 1) & 1, t + 1);
      compute(t & 1);
    }
  }

  // epilogue: accumulator (i, j, v) is output pixel (wm*FMW + i)*16 + (lane&15)
  // of the tile, channel wn*WTN + j*16 + (lane>>4)*4 + v
  __syncthreads();
  T(*Cs)[BN + CPAD] = reinterpret_cast<T(*)[BN + CPAD]>(smem);
  const ActClamp ac = act_clamp(a.act);
#pragma unroll
  for (int j = 0; j < FNW; ++j) {
    const int nl = wn * WTN + j * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int i = 0; i < FMW; ++i) {
      if (wm * FMW + i >= FMT) continue;
      const int ml = (wm * FMW + i) * 16 + (lane & 15);
      T o[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) o[v] = from_f<T>(__builtin_amdgcn_fmed3f(acc[i][j][v], ac.lo, ac.hi));
      __builtin_memcpy(&Cs[ml][nl], o, sizeof(o));
    }
  }
  __syncthreads();
  // the tile's valid pixels are consecutive rows of the GEMM: whole rows of
  // one image, or whole images
  const int valid = imgs * rows * a.Q;
  const int mbase = img0 * a.P * a.Q + row0 * a.Q;
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
  const int PQ = a.P * a.Q;
  if (L == NC8 || a.Ks % 8 == 0) {
    // 16-byte rows through a buffer resource (32-bit offsets)
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, a.y_elems * 2);
    for (int idx = tid; idx < FMT * 16 * BN / 8; idx += 256) {
      const int row = idx / (BN / 8), cj = idx % (BN / 8);
      const int n = n0 + cj * 8;
      if (row >= valid || n >= a.Ng) continue;
      const int m = mbase + row;
      unsigned off;
      if constexpr (L == NC8) {
        const int img = sdiv(m, a.inv_pq), pq = m - img * PQ;
        off = (unsigned)(((img * (a.Ks >> 3) + (n >> 3)) * PQ + pq) * 8) * 2u;
      } else {
        off = (unsigned)(m * a.Ks + n) * 2u;
      }
      __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4*>(&Cs[row][cj * 8]), ry, (int)off, 0, 0);
    }
  } else {
    for (int idx = tid; idx < FMT * 16 * BN; idx += 256) {
      const int row = idx / BN, col = idx % BN;
      const int n = n0 + col;
      if (row < valid && n < a.Ng) y[(long long)(mbase + row) * a.Ks + n] = Cs[row][col];
    }
  }
}

// ------------------------------------------------------------------ host
// Tiling of a P x Q output for a tile of FMT * 16 pixels: whole images when
// one fits, else as many whole output rows as fit, balanced over the rows.
static bool patch_tiling(PatchArgs& a, int fmt, int ppx) {
  const int maxpx = fmt * 16;
  if (a.Q > maxpx) return false;
  if (a.P * a.Q <= maxpx) {
    a.TI = std::min(a.N, maxpx / (a.P * a.Q));
    a.TR = a.P;
    a.tiles_img = 1;
    a.tiles_m = (a.N + a.TI - 1) / a.TI;
  } else {
    const int fit = maxpx / a.Q;
    a.TI = 1;
    a.tiles_img = (a.P + fit - 1) / fit;
    a.TR = (a.P + a.tiles_img - 1) / a.tiles_img;
    a.tiles_m = a.N * a.tiles_img;
  }
  a.PH = a.TR + 2;
  // row pitch: a multiple of 16 dividing 64, at least Q + 2
  a.PW = 16;
  while (a.PW < a.Q + 2) a.PW *= 2;
  if (a.PW > 64) return false;
  a.lpw = a.PW == 16 ? 4 : a.PW == 32 ? 5 : 6;
  a.fd_ti_tiles = make_fastdiv(a.tiles_img);
  a.inv_pw = 1.f / (float)a.PW;
  a.inv_ph = 1.f / (float)a.PH;
  a.HW8 = a.H * a.W * 8;
  a.inv_pq = 1.f / (float)(a.P * a.Q);
  a.W8 = a.W * 8;
  a.inv_trq = 1.f / (float)(a.TR * a.Q);
  a.inv_q = 1.f / (float)a.Q;
  return a.TI * a.PH * a.PW <= ppx;
}

static PatchArgs make_patch(const ConvArgs& c) {
  PatchArgs a{};
  a.x = c.x;
  a.w = c.w;
  a.bias = c.bias;
  a.y = c.y;
  a.N = c.xd.n;
  a.C = c.xd.c;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.Cs = c.xd.cs;
  a.K = c.yd.c;
  a.P = c.yd.h;
  a.Q = c.yd.w;
  a.Ks = c.yd.cs;
  a.Ng = c.yd.layout == NC8 ? c.yd.cs : c.yd.c;
  a.act = c.act;
  a.CB = (a.C + 7) / 8;
  a.C8 = a.CB * 8;
  a.Kred = 9 * a.C8;
  a.x_elems = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w;
  a.w_elems = (long long)((a.K + 7) / 8 * 8) * a.Kred;
  a.y_elems = (long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w;
  return a;
}

bool patch_applicable(int layout, int c, int h, int w, int r, int s, int stride, int pad, int n,
                      int fmt, int bn, int bk, int ppx) {
  (void)bn;
  if (r != 3 || s != 3 || stride != 1 || pad != 1) return false;
  const bool vec = layout == NC8 || (layout == NHWC && c % 8 == 0);
  if (!vec || ((c + 7) / 8) % (bk / 8) != 0) return false;
  if ((long long)n * h * w + h * w >= (1 << 21)) return false;  // fp32 index division
  PatchArgs a{};
  a.N = n;
  a.P = h;
  a.Q = w;
  return patch_tiling(a, fmt, ppx);
}

template <typename T, int L, int FMT, int BN, int BK, int WM, int ST, int PPX, int OCC>
static void patch_go(PatchArgs a, hipStream_t st) {
  check(patch_tiling(a, FMT, PPX), "output too wide for the patch tile");
  check(a.CB % (BK / 8) == 0, "patch kernel needs C % BK == 0");
  check(a.x_elems * 2 < (long long)kOOB && a.w_elems * 2 < (long long)kOOB,
        "tensor too large for 32-bit buffer offsets");
  a.tiles_n = (a.Ng + BN - 1) / BN;
  dim3 grid(a.tiles_m * a.tiles_n);
  SN_LAUNCH((conv3x3_patch_kernel<T, L, FMT, BN, BK, WM, ST, PPX, OCC>), grid, dim3(256), 0, st, a);
}

template <typename T, int L>
static void patch_layout(int fmt, int bn, int bk, int wm, int stg, int ppx, const PatchArgs& a,
                         hipStream_t st) {
  const long long key = ((((fmt * 1000LL + bn) * 1000 + bk) * 10 + wm) * 10 + stg) * 10000 + ppx;
#define PGO(FMT_, BN_, BK_, WM_, ST_, PPX_, OCC_)                                      \
  case ((((FMT_ * 1000LL + BN_) * 1000 + BK_) * 10 + WM_) * 10 + ST_) * 10000 + PPX_: \
    patch_go<T, L, FMT_, BN_, BK_, WM_, ST_, PPX_, OCC_>(a, st);                        \
    break;
  switch (key) {
    PGO(14, 64, 32, 2, 2, 384, 1)
    PGO(14, 64, 32, 2, 1, 384, 2)
    PGO(14, 32, 32, 4, 1, 384, 3)
    PGO(7, 64, 32, 1, 2, 320, 1)
    PGO(7, 64, 32, 2, 1, 320, 2)
    PGO(7, 32, 32, 4, 2, 320, 2)
    default: check(false, "patch tile not instantiated");
  }
#undef PGO
}

void conv_patch(int dtype, int fmt, int bn, int bk, int wm, int stg, int ppx, const ConvArgs& c,
                hipStream_t st) {
  check(dtype != 0, "patch kernel runs 16-bit types");
  check(c.xd.layout == c.yd.layout && c.r == 3 && c.s == 3 && c.stride == 1 && c.pad == 1,
        "patch kernel: 3x3 stride 1 pad 1, one layout");
  check(c.xd.layout == NC8 || (c.xd.layout == NHWC && c.xd.c % 8 == 0), "patch kernel: channel-vector layout");
  check((long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w * 2 < (long long)kOOB, "tensor too large");
  const PatchArgs a = make_patch(c);
  if (dtype == 1) {
    if (c.xd.layout == NC8) patch_layout<f16, NC8>(fmt, bn, bk, wm, stg, ppx, a, st);
    else patch_layout<f16, NHWC>(fmt, bn, bk, wm, stg, ppx, a, st);
  } else {
    if (c.xd.layout == NC8) patch_layout<bf16, NC8>(fmt, bn, bk, wm, stg, ppx, a, st);
    else patch_layout<bf16, NHWC>(fmt, bn, bk, wm, stg, ppx, a, st);
  }
}

}  // namespace k
}  // namespace sn
