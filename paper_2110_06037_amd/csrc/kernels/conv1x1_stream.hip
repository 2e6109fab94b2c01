// 1x1 convolution (stride 1 or 2, no padding) of an NHWC input with CC =
// 64, 128 or 256 channels (16-bit types), an implicit-GEMM routine for the pointwise layers
// of a bottleneck whose reduction is short.
//
// Such a layer reads each pixel once and writes K channels (plus a residual
// of K channels when an add is folded in), so memory traffic, not MFMA work,
// bounds it, and its reduction takes one to four 64-wide steps: a workgroup
// of the tiled implicit GEMM loads its tiles, waits, computes and stores with
// little to overlap.  Here workgroups are persistent: each keeps its BN
// filter rows in LDS and streams tiles of BM pixels, loading the next tile's
// pixels (LDS direct loads) and its residual (into registers) while the
// current tile's MFMAs and stores run; each wave holds its filter
// fragments in registers, so LDS serves only pixel fragments.  The tile's fp32 sums go
// through LDS so that the residual add and the stores move whole 16-byte
// chunks of consecutive channels with consecutive lanes on consecutive
// addresses.  In LDS a tile is CC / 64 slabs of 64 channels, each with
// 128-byte rows (8 chunks); chunk c of row r sits at c ^ ((r >> 1) & 7),
// which serves an MFMA operand read of 16 consecutive rows in one pass.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

struct StreamArgs {
  const void* x;     // [N][H][W][CC]
  const void* w;     // [Kp][CC]
  const float* bias; // [Kp]
  const void* res;   // [M][Ks] or null
  void* y;           // [M][Ks], M = N * P * Q output pixels
  int M, K, Ks, act;
  int H, W, P, Q, stride;
  FastDiv fd_pq, fd_q;
  int tiles_m;
  long long x_elems, w_elems, y_elems;
};

template <typename T, int CC, int BM, int BN, int WM, bool RES>
__global__ __launch_bounds__(512, 1) void conv1x1_stream_kernel(StreamArgs a) {
  static_assert(sizeof(T) == 2 && CC % 64 == 0, "16-bit types, 64-channel slabs");
  constexpr int NWV = 8, NT = 512, WN = NWV / WM;
  constexpr int RB = 128;                      // LDS row of a slab: 64 channels
  constexpr int NSL = CC / 64;                 // slabs
  constexpr int WTM = BM / WM, WTN = BN / WN, FM = WTM / 16, FN = WTN / 16;
  constexpr int NA = NSL * BM * RB / 1024 / NWV;   // pixel-tile load instructions per wave
  constexpr int NBL = NSL * BN * RB / 1024 / NWV;  // filter load instructions per wave
  constexpr int NE = BM * BN / 8 / NT;             // 16-byte output chunks per thread and tile
  static_assert(NA >= 1 && NBL >= 1 && NE >= 1 && NA * 1024 * NWV == NSL * BM * RB &&
                    NBL * 1024 * NWV == NSL * BN * RB && NE * 8 * NT == BM * BN && FM >= 1 && FN >= 1,
                "tile shape");
  constexpr int A_BYTES = NSL * BM * RB, B_BYTES = NSL * BN * RB;
  constexpr int CP = BN + 4;                   // fp32 staging row pitch (floats)
  constexpr int SM = B_BYTES + 2 * A_BYTES + BM * CP * 4 + BN * 4;
  static_assert(SM <= 160 * 1024, "LDS capacity");
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  char* const Bs = smem;
  char* const As = smem + B_BYTES;
  float* const Cs = reinterpret_cast<float*>(As + 2 * A_BYTES);
  float* const Bias = Cs + BM * CP;
  auto swz = [](int row) { return (row >> 1) & 7; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int n0 = blockIdx.y * BN;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, a.w_elems * 2);
  const __amdgpu_buffer_rsrc_t ry = make_rsrc(a.y, a.y_elems * 2);
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(RES ? a.res : a.y, a.y_elems * 2);

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
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int b = wave + NWV * i, sl = b / (BM / 8), row = (b % (BM / 8)) * 8 + prow;
    arow[i] = row;
    achk[i] = (unsigned)(sl * 64 + ((pch ^ swz(row)) << 3)) * 2u;
  }
  // output pixel m reads input pixel m (stride 1) or (img, 2p, 2q) (stride 2)
  auto issue_a = [&](int mt, int buf) {
    const int m0 = mt * BM;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int m = m0 + arow[i];
      int pix = m;
      if (a.stride != 1) {
        const int img = fdiv(m, a.fd_pq), pq = m - img * (a.P * a.Q);
        const int p = fdiv(pq, a.fd_q), q = pq - p * a.Q;
        pix = (img * a.H + p * a.stride) * a.W + q * a.stride;
      }
      dma16(rx, As + buf * A_BYTES + (wave + NWV * i) * 1024,
            m < a.M ? (unsigned)pix * (unsigned)(CC * 2) + achk[i] : kOOB, 0);
    }
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

  int mt = blockIdx.x;
  issue_a(mt, 0);
  // the wave's filter fragments stay in registers for the whole kernel, so
  // the tile loop reads only pixel fragments from LDS
  wait_vmcnt<0>();  // this wave's filter and first-tile loads
  __syncthreads();  // every wave's filter share, first pixel tile and the bias are in LDS
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

  // the residual of a tile is loaded one tile ahead, like its pixels
  auto load_res = [&](int mtile, u32x4 (&r)[NE]) {
    const int m0r = mtile * BM;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int q = tid + e * NT, row = q / (BN / 8), cj = q % (BN / 8);
      const int m = m0r + row, n = n0 + cj * 8;
      const unsigned off = m < a.M && n < a.K ? (unsigned)(m * a.Ks + n) * 2u : kOOB;
      r[e] = __builtin_amdgcn_raw_buffer_load_b128(rr, (int)off, 0, 0);
    }
  };
  // two residual register sets alternate between tiles (a copy from the
  // set still being loaded would wait for every outstanding load)
  u32x4 ra[NE], rb[NE];
  if constexpr (RES) load_res(mt, ra);

  // one tile: its pixels are in LDS buffer t % 2 (the first tile's landed
  // before the barrier above) and its residual in cur; the next tile's
  // residual goes to nxt and its pixels to the other buffer; returns whether
  // another tile follows
  auto tile = [&](int t, u32x4 (&cur)[NE], u32x4 (&nxt)[NE]) {
    const int buf = t & 1;
    const int m0 = mt * BM;
    const bool next = mt + (int)gridDim.x < a.tiles_m;
    if constexpr (RES) {
      if (next) load_res(mt + gridDim.x, nxt);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (next) issue_a(mt + gridDim.x, buf ^ 1);
    __builtin_amdgcn_sched_barrier(0);
    // wait for this tile's pixels: younger are the previous tile's stores
    // (NE), the next tile's residual and the next tile's pixel loads; this
    // tile's residual is older, so it has arrived too
    constexpr int YR = RES ? NE : 0;
    if (t > 0) {
      if (next) wait_vmcnt<NE + YR + NA>();
      else wait_vmcnt<NE>();
    }
    dma_barrier();  // every wave's share landed; every wave is done with the last tile's Cs

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{bias[j][0], bias[j][1], bias[j][2], bias[j][3]};
    const char* A = As + buf * A_BYTES;
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
    // sums (bias included) to LDS: element (i, j, v) is pixel
    // wm*WTM + i*16 + (lane&15), channel wn*WTN + j*16 + (lane>>4)*4 + v
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        *reinterpret_cast<f32x4*>(Cs + (wm * WTM + i * 16 + (lane & 15)) * CP + wn * WTN + j * 16 + (lane >> 4) * 4) =
            acc[i][j];
    lds_barrier();
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      const int q = tid + e * NT, row = q / (BN / 8), cj = q % (BN / 8);
      const int m = m0 + row, n = n0 + cj * 8;
      const unsigned off = m < a.M && n < a.K ? (unsigned)(m * a.Ks + n) * 2u : kOOB;
      const f32x4 c0 = *reinterpret_cast<const f32x4*>(Cs + row * CP + cj * 8);
      const f32x4 c1 = *reinterpret_cast<const f32x4*>(Cs + row * CP + cj * 8 + 4);
      float s[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
      if constexpr (RES) {
        T rt[8];
        __builtin_memcpy(rt, &cur[e], 16);
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
    return next;
  };
  // tiles mt, mt + G, ... (G = grid size); the loop is unrolled by two so
  // that the residual sets swap roles without copies
  for (int t = 0;; t += 2) {
    if (!tile(t, ra, rb)) break;
    mt += gridDim.x;
    if (!tile(t + 1, rb, ra)) break;
    mt += gridDim.x;
  }
}

bool stream1x1_applicable(int layout, int c, int cs, int n, int h, int w, int r, int s, int stride, int pad,
                          int k, int cc) {
  const long long p = (h - 1) / stride + 1, q = (w - 1) / stride + 1;
  return layout == NHWC && c == cc && cs == cc && r == 1 && s == 1 && (stride == 1 || stride == 2) &&
         pad == 0 && k % 8 == 0 && (long long)n * h * w * cc * 2 < (long long)kOOB &&
         (long long)n * p * q * ((k + 7) / 8 * 8) * 2 < (long long)kOOB;
}

template <typename T, int CC, int BM, int BN, int WM>
static void stream_go(const StreamArgs& a, int tiles_n, hipStream_t st) {
  // persistent: about one workgroup per CU over all channel tiles
  const int gx = std::max(1, std::min(a.tiles_m, 256 / tiles_n));
  const dim3 grid(gx, tiles_n);
  if (a.res)
    SN_LAUNCH((conv1x1_stream_kernel<T, CC, BM, BN, WM, true>), grid, dim3(512), 0, st, a);
  else
    SN_LAUNCH((conv1x1_stream_kernel<T, CC, BM, BN, WM, false>), grid, dim3(512), 0, st, a);
}

void conv1x1_stream(int dtype, int cc, int bm, int bn, const ConvArgs& c, hipStream_t st) {
  check(dtype != 0, "streaming 1x1 kernel runs 16-bit types");
  const long long m = (long long)c.yd.n * c.yd.h * c.yd.w;
  check(c.xd.layout == NHWC && c.yd.layout == NHWC && c.stride >= 1 &&
            c.yd.h == (c.xd.h - 1) / c.stride + 1 && c.yd.w == (c.xd.w - 1) / c.stride + 1 &&
            stream1x1_applicable(c.xd.layout, c.xd.c, c.xd.cs, c.xd.n, c.xd.h, c.xd.w, c.r, c.s, c.stride,
                                 c.pad, c.yd.c, cc),
        "streaming 1x1 kernel: NHWC, C = CC, 1x1 stride 1 or 2 without padding, K % 8 == 0");
  StreamArgs a{};
  a.x = c.x;
  a.w = c.w;
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
  a.x_elems = (long long)c.xd.n * c.xd.h * c.xd.w * cc;
  a.w_elems = (long long)((a.K + 7) / 8 * 8) * cc;
  a.y_elems = m * a.Ks;
  const int tiles_n = (a.K + bn - 1) / bn;
#define SG(CC_, BM_, BN_, WM_)                                                \
  if (cc == CC_ && bm == BM_ && bn == BN_) {                                  \
    if (dtype == 1) stream_go<f16, CC_, BM_, BN_, WM_>(a, tiles_n, st);       \
    else stream_go<bf16, CC_, BM_, BN_, WM_>(a, tiles_n, st);                 \
    return;                                                                   \
  }
  SG(64, 64, 256, 2)
  SG(64, 128, 128, 4)
  SG(64, 128, 64, 4)
  SG(128, 64, 128, 2)
  SG(128, 32, 256, 1)
  SG(256, 64, 64, 4)
  SG(256, 32, 128, 2)
#undef SG
  check(false, "streaming 1x1 tile not instantiated");
}

}  // namespace k
}  // namespace sn
