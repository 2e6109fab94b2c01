// 3x3 convolution (stride SD = 1 or 2, padding 1) as an implicit GEMM whose
// input tile is a spatial patch kept in LDS.
//
// A workgroup computes the outputs of TI whole images, or of TR consecutive
// output rows of one image (all Q columns), for BN output channels.  For
// every step of 32 input channels it loads the tile's input patch -- the
// ((TR - 1) SD + 3) x ((Q - 1) SD + 3) input pixels (one halo pixel on each
// side; the zero padding comes from out-of-range buffer offsets) -- and the
// filter taps of those channels for all 9 taps, then runs the 9 taps' MFMAs
// out of LDS: tap (r, s) of output pixel (p, q) is patch pixel
// (SD p + r, SD q + s), so the per-tap operand rows are the same patch rows
// shifted by the uniform offset r * PWT + s (PWT = the patch row pitch, a
// power of two).  Each input element therefore crosses the memory system
// about once per workgroup (plus the halo rows) instead of 9 / SD^2 times,
// which is what bounds the per-tap (im2col) implicit GEMM.
//
// Tiles move from global memory into LDS with direct loads (16 bytes per
// lane, 1 KB per wave instruction in lane order) through ST stages, so up to
// ST - 1 channel steps are in flight while one is computed.  An LDS row holds
// the 32 channels of one pixel (64 bytes); 16-byte chunk c of row r sits at
// chunk c ^ ((r >> 1) & 3).  An MFMA operand read takes one chunk of 16
// consecutive rows, which this placement serves in a single LDS pass on
// gfx950 for any starting row (an XOR of (r >> 2) & 3 measures two passes).
// Operand rows that wrap to the next image row are not consecutive and may
// take two passes.  Tap row offsets r * PWT are multiples of 16 rows, so they
// keep the placement and become instruction immediates, as do the stage
// offsets (the step loop is unrolled by the stage count): an operand read
// costs no address arithmetic.
//
// Eight waves (two per SIMD, so one wave's loads and epilogue overlap the
// other's MFMAs) form TG tap groups: group g runs taps [9g/TG, 9(g+1)/TG) of
// every step on the whole tile, which keeps each wave's operand tile large
// when the workgroup tile is small; the groups' sums meet in LDS at the end.
// The MFMA takes the filter as its first operand, so each lane's 4
// accumulators are 4 consecutive output channels of one pixel; sums start at
// the bias, and the epilogue applies the activation, stages the tile in LDS
// and stores it as 16-byte chunks of consecutive addresses.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

#include <type_traits>

namespace sn {
namespace k {

struct PatchArgs {
  const void* x;
  const void* w;  // [Kp][3][3][C8]
  const float* bias;
  void* y;
  int N, C, H, W, Cs;  // input (pad 1)
  int K, P, Q, Ks, Ng;
  int act;
  int CB, C8, Kred;      // channel blocks of 8, padded channels, weight row length 9 * C8
  int TI, TR, PH, PW;    // images / output rows per tile, patch rows, patch row pitch
  int IP;                // patch image pitch (rows of LDS per image)
  int tiles_img;         // row tiles per image
  int tiles_m, tiles_n;
  FastDiv fd_ti_tiles;   // division by tiles_img
  float inv_pw, inv_ip, inv_trq, inv_q;   // 1/PW, 1/IP, 1/(TR*Q), 1/Q for sdiv
  int HW8, W8;                            // NC8HW8 strides: H*W*8, W*8
  float inv_pq;                           // 1/(P*Q) for sdiv
  float inv_tr;                           // 1/TR (row-aligned tiles)
  long long y_elems;
  long long x_elems, w_elems;
};

template <int V>
using IC = std::integral_constant<int, V>;

// FMT: MFMA row blocks (16 pixels) per tile; BN output channels; PWT patch
// row pitch (a power of two >= Q + 2); the 8 waves form TG tap groups of
// WM x WN waves (group g runs taps [9g/TG, 9(g+1)/TG) of every step on the
// whole tile; the groups' sums meet in LDS at the end); ST LDS stages;
// PROWS patch rows per stage; OCC workgroups per CU (the launch bound's
// second figure counts waves per SIMD: 2 OCC, 8 waves on 4 SIMDs each);
// RA: row-aligned row blocks.
template <typename T, int L, int FMT, int BN, int PWT, int WM, int WN, int TG, int ST, int PROWS, int SD, int OCC = 1,
          bool RA = false>
__global__ __launch_bounds__(512, 2 * OCC) void conv3x3_patch_kernel(PatchArgs a) {
  static_assert(sizeof(T) == 2 && L != NCHW, "16-bit channel-vector layouts only");
  static_assert(!RA || SD == 1, "row-aligned blocks at stride 1");
  constexpr int NWV = 8;
  static_assert(WM * WN * TG == NWV, "8 waves");
  static_assert(PWT == 16 || PWT == 32 || PWT == 64, "patch pitch: a multiple of 16 rows");
  constexpr int LPW = PWT == 16 ? 4 : PWT == 32 ? 5 : 6;
  constexpr int BK = 32, RB = 64;                    // channels per step, bytes per LDS row
  constexpr int FMW = (FMT + WM - 1) / WM;           // row blocks per wave
  constexpr int WTN = BN / WN, FNW = WTN / 16;
  static_assert(FNW >= 1 && FNW * 16 * WN == BN, "BN must split over the wave columns");
  static_assert(PROWS % 16 == 0, "patch rows in whole 16-row loads");
  constexpr int WR = 9 * BN;                         // filter rows
  constexpr int NINS = (PROWS + WR + 15) / 16;       // 16-row load instructions per stage
  constexpr int NL = (NINS + NWV - 1) / NWV;         // per wave
  constexpr int STAGE = NL * NWV * 16 * RB;
  static_assert(ST >= 2 && ST <= 4, "two to four LDS stages");
  constexpr int RPITCH = BN * 4 + 16;                // partial-sum row pitch (bytes)
  constexpr int RED = TG > 1 ? FMT * 16 * RPITCH : 0;
  constexpr int SM = ST * STAGE > RED ? ST * STAGE : RED;
  static_assert(SM * OCC <= 160 * 1024, "LDS capacity at the occupancy");
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  lds_char* const sl = (lds_char*)smem;
  auto swz = [](int row) { return (row >> 1) & 3; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int grp = wave / (WM * WN), wig = wave % (WM * WN);
  const int wm = wig / WN, wn = wig % WN;
  const int blk0 = wm * FMW;
  int mt, nt;
  tile_of(blockIdx.x, a.tiles_m, a.tiles_n, mt, nt);
  const int ig = fdiv(mt, a.fd_ti_tiles), rt = mt - ig * a.tiles_img;
  const int img0 = ig * a.TI;
  const int row0 = rt * a.TR;
  const int imgs = min(a.TI, a.N - img0);
  const int rows = min(a.TR, a.P - row0);
  const int n0 = nt * BN;
  const int KT = a.CB / 4;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, a.w_elems * 2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.bias, (long long)a.Ng * 4);

  // bias of the lane's output channels (tap group 0 starts its sums there)
  float bias[FNW][4];
#pragma unroll
  for (int j = 0; j < FNW; ++j) {
    const int n = n0 + wn * WTN + j * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int v = 0; v < 4; ++v)
      bias[j][v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rb, (n + v) * 4, 0, 0));
  }

  // A stage holds PROWS patch rows (image ii at ii * IP, patch row ph at
  // + ph * PWT, column pw; pitch padding loads zeros), then the 9 * BN
  // filter rows (tap, output channel), then rows no load fills.  Load
  // instruction q = wave + 8 i fills stage rows [16 q, 16 q + 16): this lane
  // fills row 16 q + lane / 4, physical chunk lane % 4 (logical chunk
  // (lane % 4) ^ swz(row)).  (Index arithmetic: 24-bit multiplies and fp32
  // division; every value is far below 2^21.)
  unsigned loff[NL];
  const int lrow = lane >> 2;
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int q = wave + NWV * i;
    const int row = 16 * q + lrow;
    const int lcp = (lane & 3) ^ swz(row);
    unsigned off = kOOB;
    if (16 * q < PROWS) {
      const int ii = sdiv(row, a.inv_ip), rem = row - __umul24(ii, a.IP);
      const int ph = rem >> LPW, pw = rem & (PWT - 1);
      const int img = img0 + ii, h = row0 * SD - 1 + ph, ww = pw - 1;
      const bool ok = ii < a.TI && img < a.N && ph < a.PH && (unsigned)h < (unsigned)a.H &&
                      (unsigned)ww < (unsigned)a.W;
      unsigned e;
      if constexpr (L == NC8)
        e = __umul24(__umul24(img, a.CB) + lcp, a.HW8) + __umul24(h, a.W8) + ww * 8;
      else
        e = __umul24(__umul24(__umul24(img, a.H) + h, a.W) + ww, a.Cs) + lcp * 8;
      if (ok) off = e * 2u;
    } else if (16 * q < PROWS + WR) {
      const int fr = row - PROWS, tap = fr / BN, kch = n0 + fr % BN;
      if (kch < a.Ng) off = (__umul24(kch, a.Kred) + __umul24(tap, a.C8) + lcp * 8) * 2u;
    }
    loff[i] = off;
  }
  const int xstep = L == NC8 ? 4 * a.HW8 * 2 : BK * 2;
  auto issue = [&](auto SC, int kt) {
    constexpr int SI = decltype(SC)::value;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int q = wave + NWV * i;
      const bool patch = 16 * q < PROWS;
      dma16(patch ? rx : rw, sl + SI * STAGE + q * 1024, loff[i], kt * (patch ? xstep : BK * 2));
    }
  };
  issue(IC<0>{}, 0);
  if constexpr (ST > 2) {
    if (1 < KT) issue(IC<1>{}, 1);
  }
  if constexpr (ST > 3) {
    if (2 < KT) issue(IC<2>{}, 2);
  }

  // LDS byte offsets of this lane's operand chunk for the three column taps
  // of each row block; tap (r, s) adds r * PWT rows (a multiple of 16, so the
  // swizzle is unchanged) as an instruction immediate
  int aoff[FMW][3];
#pragma unroll
  for (int i = 0; i < FMW; ++i) {
    const int m = (blk0 + i) * 16 + (lane & 15);
    int pb;
    if constexpr (RA) {
      // virtual pixel m: row vr = m / PWT of the tile (image ii, row pr),
      // column pc = m % PWT; columns past Q compute values nobody stores,
      // from rows of the same stage (at most one row past the patch)
      const int vr = m >> LPW, pc = m & (PWT - 1);
      const int ii = sdiv(vr, a.inv_tr), pr = vr - __umul24(ii, a.TR);
      pb = blk0 + i < FMT && ii < a.TI ? __umul24(ii, a.IP) + (pr << LPW) + pc : 0;
    } else {
      const int ii = sdiv(m, a.inv_trq), rem = m - __umul24(ii, a.TR * a.Q);
      const int pr = sdiv(rem, a.inv_q), pc = rem - __umul24(pr, a.Q);
      pb = blk0 + i < FMT && ii < a.TI ? __umul24(ii, a.IP) + ((pr * SD) << LPW) + pc * SD : 0;
    }
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const int r = pb + c;
      aoff[i][c] = (r << 6) | (((lane >> 4) ^ swz(r)) << 4);
    }
  }
  const int boff = PROWS * RB + (wn * WTN + (lane & 15)) * RB + (((lane >> 4) ^ ((lane >> 1) & 3)) << 4);

  typedef typename Mfma<T>::frag frag;
  f32x4 acc[FMW][FNW];
#pragma unroll
  for (int j = 0; j < FNW; ++j)
#pragma unroll
    for (int i = 0; i < FMW; ++i)
      acc[i][j] = grp == 0 ? f32x4{bias[j][0], bias[j][1], bias[j][2], bias[j][3]} : f32x4{0.f, 0.f, 0.f, 0.f};

  // taps [T0, T1) of the stage SI; the fragments of tap t+1 are read from LDS
  // while tap t's MFMAs run
  auto compute = [&](auto SC, auto T0C, auto T1C) {
    constexpr int SI = decltype(SC)::value, T0 = decltype(T0C)::value, T1 = decltype(T1C)::value;
    const char* S = smem + SI * STAGE;
    frag fa[2][FMW], fb[2][FNW];
    auto load = [&](int tap, int b) {
#pragma unroll
      for (int i = 0; i < FMW; ++i)
        fa[b][i] = *reinterpret_cast<const frag*>(S + aoff[i][tap % 3] + (tap / 3) * PWT * RB);
#pragma unroll
      for (int j = 0; j < FNW; ++j) fb[b][j] = *reinterpret_cast<const frag*>(S + boff + (tap * BN + j * 16) * RB);
    };
    load(T0, 0);
#pragma unroll
    for (int u = T0; u < T1; ++u) {
      const int b = (u - T0) & 1;
      if (u + 1 < T1) load(u + 1, b ^ 1);
      // keep the next tap's reads ahead of this tap's MFMAs
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FMW; ++i)
#pragma unroll
        for (int j = 0; j < FNW; ++j) acc[i][j] = Mfma<T>::run(fb[b][j], fa[b][i], acc[i][j]);
    }
  };
  // step t on stage t % ST: wait for its own tiles (the ST - 2 later steps may
  // still be in flight), barrier (which also ends every wave's reads of the
  // stage the next issue overwrites), issue step t + ST - 1, compute
  auto step = [&](auto UC, int t) {
    constexpr int U = decltype(UC)::value;
    if (t >= KT) return;
    if (t + ST - 2 < KT) wait_vmcnt<(ST - 2) * NL>();
    else wait_vmcnt<0>();
    dma_barrier();
    if (t + ST - 1 < KT) issue(IC<(U + ST - 1) % ST>{}, t + ST - 1);
    if constexpr (TG == 1) {
      compute(UC, IC<0>{}, IC<9>{});
    } else {
      if (grp == 0) compute(UC, IC<0>{}, IC<5>{});
      else compute(UC, IC<5>{}, IC<9>{});
    }
  };
  for (int t0 = 0; t0 < KT; t0 += ST) {
    step(IC<0>{}, t0);
    step(IC<1>{}, t0 + 1);
    if constexpr (ST > 2) step(IC<2>{}, t0 + 2);
    if constexpr (ST > 3) step(IC<3>{}, t0 + 3);
  }

  // tap group 1 hands its sums to group 0 through LDS
  if constexpr (TG > 1) {
    __syncthreads();
    if (grp == 1) {
#pragma unroll
      for (int i = 0; i < FMW; ++i)
#pragma unroll
        for (int j = 0; j < FNW; ++j) {
          const int ml = (blk0 + i) * 16 + (lane & 15);
          if (blk0 + i < FMT)
            *reinterpret_cast<f32x4*>(smem + ml * RPITCH + (wn * WTN + j * 16 + (lane >> 4) * 4) * 4) = acc[i][j];
        }
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int i = 0; i < FMW; ++i)
#pragma unroll
        for (int j = 0; j < FNW; ++j) {
          const int ml = (blk0 + i) * 16 + (lane & 15);
          if (blk0 + i < FMT)
            acc[i][j] += *reinterpret_cast<const f32x4*>(smem + ml * RPITCH + (wn * WTN + j * 16 + (lane >> 4) * 4) * 4);
        }
    }
  }

  // epilogue: accumulator (i, j, v) is output pixel (blk0 + i)*16 + (lane&15)
  // of the tile, channel wn*WTN + j*16 + (lane>>4)*4 + v.  Tap group 0 puts
  // the outputs (activation applied, 16-bit) into LDS rows of BN channels;
  // then all waves store them as 16-byte chunks of 8 channels, consecutive
  // threads on consecutive chunks (NHWC: the chunks of a pixel, then the
  // next pixel; NC8HW8: the pixels of one channel block), so a wave's
  // stores cover contiguous runs.  The tile's valid pixels are consecutive
  // rows of the GEMM (whole rows of one image, or whole images).
  constexpr int OP = BN * 2 + 16;  // staging row bytes
  static_assert(FMT * 16 * OP <= SM, "output staging fits the tile's LDS");
  const ActClamp ac = act_clamp(a.act);
  __syncthreads();  // every wave is done with the stages (and group 0 with group 1's sums)
  if (grp == 0) {
#pragma unroll
    for (int i = 0; i < FMW; ++i) {
      if (blk0 + i >= FMT) continue;
      int ml = (blk0 + i) * 16 + (lane & 15);
      if constexpr (RA) {
        // the valid virtual pixels move to their place among the tile's
        // output pixels; the others are dropped
        const int vr = ml >> LPW, pc = ml & (PWT - 1);
        const int ii = sdiv(vr, a.inv_tr), pr = vr - ii * a.TR;
        if (pc >= a.Q || pr >= rows || ii >= imgs) continue;
        ml = (ii * rows + pr) * a.Q + pc;
      }
#pragma unroll
      for (int j = 0; j < FNW; ++j) {
        const int nl = wn * WTN + j * 16 + (lane >> 4) * 4;
        T o[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = from_f<T>(__builtin_amdgcn_fmed3f(acc[i][j][v], ac.lo, ac.hi));
        __builtin_memcpy(smem + ml * OP + nl * 2, o, 8);
      }
    }
  }
  __syncthreads();
  const int valid = imgs * rows * a.Q;
  const int mbase = img0 * a.P * a.Q + row0 * a.Q;
  const int PQ = a.P * a.Q;
  T* __restrict__ y = reinterpret_cast<T*>(a.y);
  const __amdgpu_buffer_rsrc_t ry = make_rsrc(y, a.y_elems * 2);
  constexpr int CPX = BN / 8;  // 16-byte chunks per pixel
  const bool vec8 = L == NC8 || a.Ks % 8 == 0;
  for (int q = tid; q < valid * CPX; q += NWV * 64) {
    int ml, c8;
    if constexpr (L == NC8) {
      c8 = q / valid;
      ml = q - c8 * valid;
    } else {
      ml = q / CPX;
      c8 = q - ml * CPX;
    }
    const int n = n0 + c8 * 8;
    if (n >= a.Ng) continue;
    const u32x4 v = *reinterpret_cast<const u32x4*>(smem + ml * OP + c8 * 16);
    const int m = mbase + ml;
    unsigned e;
    if constexpr (L == NC8) {
      const int img = sdiv(m, a.inv_pq), pq = m - img * PQ;
      e = (unsigned)(((img * (a.Ks >> 3) + (n >> 3)) * PQ + pq) * 8);
    } else {
      e = (unsigned)(m * a.Ks + n);
    }
    if (vec8 && n + 8 <= a.Ng) {
      __builtin_amdgcn_raw_buffer_store_b128(v, ry, (int)(e * 2u), 0, 0);
    } else {
      T o[8];
      __builtin_memcpy(o, &v, 16);
      for (int t = 0; t < 8 && n + t < a.Ng; ++t) y[e + t] = o[t];
    }
  }
}

// ------------------------------------------------------------------ host
// Tiling of a P x Q output for a tile of FMT * 16 pixels: whole images when
// one fits, else as many whole output rows as fit, balanced over the rows.
// The patch row pitch is pwt and the image pitch PH * pwt.  Returns whether
// the patch fits `prows`.
static bool patch_tiling(PatchArgs& a, int fmt, int pwt, int prows, int sd, int ra = 0) {
  const int maxpx = fmt * 16;
  if (a.Q > maxpx || (a.Q - 1) * sd + 3 > pwt || (ra && sd != 1)) return false;
  if (ra && 2 * a.Q <= pwt) return false;  // most virtual columns would be dropped
  // row-aligned tiles count an output row as pwt (virtual) pixels
  const int rowpx = ra ? pwt : a.Q;
  if (rowpx > maxpx) return false;
  if (a.P * rowpx <= maxpx) {
    a.TI = std::min(a.N, maxpx / (a.P * rowpx));
    a.TR = a.P;
    a.tiles_img = 1;
    a.tiles_m = (a.N + a.TI - 1) / a.TI;
  } else {
    const int fit = maxpx / rowpx;
    a.TI = 1;
    a.tiles_img = (a.P + fit - 1) / fit;
    a.TR = (a.P + a.tiles_img - 1) / a.tiles_img;
    a.tiles_m = a.N * a.tiles_img;
  }
  a.PH = (a.TR - 1) * sd + 3;
  a.PW = pwt;
  a.IP = a.PH * pwt;
  a.fd_ti_tiles = make_fastdiv(a.tiles_img);
  a.inv_pw = 1.f / (float)a.PW;
  a.inv_ip = 1.f / (float)a.IP;
  a.HW8 = a.H * a.W * 8;
  a.inv_pq = 1.f / (float)(a.P * a.Q);
  a.W8 = a.W * 8;
  a.inv_trq = 1.f / (float)(a.TR * a.Q);
  a.inv_q = 1.f / (float)a.Q;
  a.inv_tr = 1.f / (float)a.TR;
  return (long long)a.TI * a.IP <= prows;
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
                      int fmt, int pwt, int prows, int sd, int ra) {
  if (r != 3 || s != 3 || stride != sd || pad != 1) return false;
  const bool vec = layout == NC8 || (layout == NHWC && c % 8 == 0);
  if (!vec || ((c + 7) / 8) % 4 != 0) return false;
  if ((long long)n * h * w + h * w >= (1 << 21)) return false;  // fp32 index division
  PatchArgs a{};
  a.N = n;
  a.P = (h - 1) / sd + 1;
  a.Q = (w - 1) / sd + 1;
  return patch_tiling(a, fmt, pwt, prows, sd, ra);
}

template <typename T, int L, int FMT, int BN, int PWT, int WM, int WN, int TG, int ST, int PROWS, int SD, int OCC = 1,
          bool RA = false>
static void patch_go(PatchArgs a, hipStream_t st) {
  check(patch_tiling(a, FMT, PWT, PROWS, SD, RA), "output too wide for the patch tile");
  check(a.CB % 4 == 0, "patch kernel needs C % 32 == 0");
  check(a.x_elems * 2 < (long long)kOOB && a.w_elems * 2 < (long long)kOOB,
        "tensor too large for 32-bit buffer offsets");
  a.tiles_n = (a.Ng + BN - 1) / BN;
  dim3 grid(a.tiles_m * a.tiles_n);
  SN_LAUNCH((conv3x3_patch_kernel<T, L, FMT, BN, PWT, WM, WN, TG, ST, PROWS, SD, OCC, RA>), grid, dim3(512), 0, st,
            a);
}

static long long patch_key(int fmt, int bn, int pwt, int wm, int wn, int tg, int stg, int prows, int sd, int occ,
                           int ra) {
  return (((((((((fmt * 1000LL + bn) * 100 + pwt) * 10 + wm) * 10 + wn) * 10 + tg) * 10 + stg) * 10000 + prows) * 10 +
           sd) * 10 + occ) * 2 + ra;
}

template <typename T, int L>
static void patch_layout(const PatchCfg& c, const PatchArgs& a, hipStream_t st) {
  const long long key = patch_key(c.fmt, c.bn, c.pwt, c.wm, c.wn, c.tg, c.st, c.prows, c.sd, c.occ, c.ra);
#define PGO(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_)                               \
  if (key == patch_key(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 1, 1, 0)) {         \
    patch_go<T, L, FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 1>(a, st);              \
    return;                                                                            \
  }
#define PGO2(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_)                              \
  if (key == patch_key(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 2, 1, 0)) {         \
    patch_go<T, L, FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 2>(a, st);              \
    return;                                                                            \
  }
#define PGOO2(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_)                             \
  if (key == patch_key(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 1, 2, 0)) {         \
    patch_go<T, L, FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 1, 2>(a, st);           \
    return;                                                                            \
  }
#define PGORA(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, OCC_)                       \
  if (key == patch_key(FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 1, OCC_, 1)) {      \
    patch_go<T, L, FMT_, BN_, PWT_, WM_, WN_, TG_, ST_, PROWS_, 1, OCC_, true>(a, st);  \
    return;                                                                            \
  }
  PATCH_CONFIGS(PGO)
  PATCH2_CONFIGS(PGO2)
  PATCH_OCC2_CONFIGS(PGOO2)
  PATCH_RA_CONFIGS(PGORA)
#undef PGO
#undef PGO2
#undef PGOO2
#undef PGORA
  check(false, "patch tile not instantiated");
}

void conv_patch(int dtype, const PatchCfg& cfg, const ConvArgs& c, hipStream_t st) {
  check(dtype != 0, "patch kernel runs 16-bit types");
  check(c.xd.layout == c.yd.layout && c.r == 3 && c.s == 3 && c.stride == cfg.sd && c.pad == 1,
        "patch kernel: 3x3 pad 1 at the tile's stride, one layout");
  check(c.xd.layout == NC8 || (c.xd.layout == NHWC && c.xd.c % 8 == 0), "patch kernel: channel-vector layout");
  check((long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w * 2 < (long long)kOOB, "tensor too large");
  const PatchArgs a = make_patch(c);
  if (dtype == 1) {
    if (c.xd.layout == NC8) patch_layout<f16, NC8>(cfg, a, st);
    else patch_layout<f16, NHWC>(cfg, a, st);
  } else {
    if (c.xd.layout == NC8) patch_layout<bf16, NC8>(cfg, a, st);
    else patch_layout<bf16, NHWC>(cfg, a, st);
  }
}

}  // namespace k
}  // namespace sn
