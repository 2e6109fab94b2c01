// Convolution of an input with few channels (C <= 4; the RGB stem of a CNN)
// in NHWC, stride 1 or 2, any R x S filter, as an implicit GEMM on MFMA.
//
// Padding three channels to the 8 of a 16-byte vector would waste 5/8 of
// the MFMA work, so the reduction is packed differently: the input patch of
// a tile sits in LDS with 4 channels per pixel (8 bytes, the fourth zero),
// and one 8-element MFMA operand chunk is a pixel pair -- filter columns
// (s, s + 1) of filter row r, 4 channels each, 16 consecutive LDS bytes
// (16-byte aligned with stride 2, 8-byte aligned with stride 1).  The
// reduction has R * ceil(S / 2) such chunks (28 for a 7 x 7 filter: 224 MFMA
// elements for 147 real ones; 6 for a 3 x 3 filter).  The filter is
// repacked into the same chunks in LDS once per workgroup (all its loads in
// flight together); workgroups are persistent over output-row tiles and
// prefetch the next tile's input pixels into registers while the current
// tile's MFMAs run.  A tile's outputs are whole output rows of one image,
// contiguous in NHWC: they go through LDS and leave as 16-byte stores of
// consecutive addresses (a wave stores 1 KB runs).
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

struct SmallCArgs {
  const void* x;
  const void* w;  // prepared [Kp][R][S][C8]
  const float* bias;
  void* y;
  int N, C, H, W;
  int K, P, Q, Ks, Ng;
  int R, S, pad, act, stride;
  int C8, Kred;          // prepared filter: channels per tap, row length R * S * C8
  int G, SP;             // operand chunks R * SP, column pairs per filter row SP = ceil(S / 2)
  int TR, PH, PWP;       // output rows per tile, patch rows, patch pitch in pixels (even)
  int tiles_img, tiles;  // row tiles per image, tiles in all
  float inv_sp, inv_pwp2, inv_q;  // 1/SP, 1/(PWP/2), 1/Q for sdiv
  FastDiv fd_tiles_img;
  long long x_elems, w_elems, y_elems;
};

// FMT: MFMA row blocks (16 output pixels) per tile; 64 output channels per
// workgroup; WM wave rows (of 4 waves); PPX patch capacity in pixels; GMAX
// operand chunks of the filter (multiple of 4: one k-slice of 32 is 4).
template <typename T, int FMT, int WM, int PPX, int GMAX, int OCC>
__global__ __launch_bounds__(256, OCC) void conv_smallc_kernel(SmallCArgs a) {
  static_assert(sizeof(T) == 2, "16-bit types");
  static_assert(GMAX % 4 == 0 && PPX % 2 == 0, "shape");
  constexpr int BN = 64;
  constexpr int WN = 4 / WM;
  constexpr int FMW = (FMT + WM - 1) / WM;
  constexpr int WTN = BN / WN, FNW = WTN / 16;
  constexpr int WPITCH = GMAX * 16 + 16;  // filter row bytes (odd number of 16-byte units)
  constexpr int P_BYTES = PPX * 8;
  constexpr int PAIRS = PPX / 2;                 // patch pixel pairs (16 bytes each)
  constexpr int NPF = (PAIRS + 255) / 256;       // pairs per thread
  constexpr int OPITCH = BN * 2 + 16;            // output staging row bytes
  constexpr int SM = P_BYTES + BN * WPITCH + BN * 4 + FMT * 16 * OPITCH;
  static_assert(SM * OCC <= 160 * 1024, "LDS capacity at the occupancy");
  __shared__ __attribute__((aligned(1024))) char smem[SM];
  char* const Ws = smem + P_BYTES;
  char* const Os = smem + P_BYTES + BN * WPITCH + BN * 4;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int n0 = blockIdx.y * BN;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, a.w_elems * 2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(a.bias, (long long)a.Ng * 4);
  const __amdgpu_buffer_rsrc_t ry = make_rsrc(a.y, a.y_elems * 2);

  // filter chunks: row n, chunk g = (r, sp) holds taps (r, 2 sp) and
  // (r, 2 sp + 1), channels 0..3 each (zero past C, S, G); loaded here,
  // put into LDS once the first patch's loads are in flight too
  constexpr int NFC = BN * GMAX / 256;  // chunks per thread
  static_assert(NFC * 256 == BN * GMAX, "filter chunks per thread");
  u32x2 d[NFC][2];
  {
#pragma unroll
    for (int u = 0; u < NFC; ++u) {
      const int idx = tid + u * 256;
      const int n = idx / GMAX, g = idx - n * GMAX;
      const int r = sdiv(g, a.inv_sp), sp = g - __umul24(r, a.SP);
      const int s0 = 2 * sp, k = n0 + n;
      const bool ok = g < a.G && k < a.Ng;
      const unsigned base = (unsigned)(__umul24(k, a.Kred) + __umul24(__umul24(r, a.S) + s0, a.C8)) * 2u;
      const unsigned lo = ok && s0 < a.S ? base : kOOB, hi = ok && s0 + 1 < a.S ? base + (unsigned)a.C8 * 2u : kOOB;
      d[u][0] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rw, (int)lo, 0, 0));
      d[u][1] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rw, (int)hi, 0, 0));
    }
  }

  // patch pixels of a tile: pair j = (row, column pair), 16 bytes in LDS;
  // an input pixel is C <= 4 16-bit values at any 2-byte alignment: three
  // aligned dwords cover it, realigned by the byte offset (a funnel shift).
  // A thread's pairs j = tid + 256 u sit at the same patch row and columns
  // in every tile, so their row index and column byte offsets are set once.
  const int Cm = a.C;
  const unsigned cmask0 = Cm < 2 ? 0xFFFFu : 0xFFFFFFFFu;                      // channels 0, 1
  const unsigned cmask1 = Cm < 3 ? 0u : Cm < 4 ? 0xFFFFu : 0xFFFFFFFFu;        // channels 2, 3
  int fprw[NPF], fcb[NPF][2];
  bool fcok[NPF][2];
#pragma unroll
  for (int u = 0; u < NPF; ++u) {
    const int j = tid + u * 256;
    const int prw = sdiv(j, a.inv_pwp2), pc2 = j - __umul24(prw, a.PWP >> 1);
    fprw[u] = j < PAIRS && prw < a.PH ? prw : -(1 << 24);  // a row no tile has
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int w = 2 * pc2 + e - a.pad;
      fcok[u][e] = (unsigned)w < (unsigned)a.W;
      fcb[u][e] = (prw * a.W + w) * Cm * 2;
    }
  }
  auto fetch = [&](int tile, u32x4 (&raw)[NPF][2], unsigned (&shf)[NPF][2], unsigned (&okm)[NPF][2]) {
    const int img = fdiv(tile, a.fd_tiles_img), rt = tile - img * a.tiles_img;
    const int h0 = rt * a.TR * a.stride - a.pad;
    const int tb = (img * a.H + h0) * a.W * Cm * 2;  // byte offset of input row h0 (may be < 0)
#pragma unroll
    for (int u = 0; u < NPF; ++u) {
      const bool rok = (unsigned)(h0 + fprw[u]) < (unsigned)a.H;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const bool ok = rok && fcok[u][e];
        const int byte = tb + fcb[u][e];
        okm[u][e] = ok ? 0xFFFFFFFFu : 0u;
        shf[u][e] = (unsigned)(byte & 3) * 8u;
        const auto d = __builtin_amdgcn_raw_buffer_load_b96(rx, ok ? (byte & ~3) : (int)kOOB, 0, 0);
        raw[u][e] = u32x4{d[0], d[1], d[2], 0u};
      }
    }
  };
  auto store_patch = [&](const u32x4 (&raw)[NPF][2], const unsigned (&shf)[NPF][2], const unsigned (&okm)[NPF][2]) {
#pragma unroll
    for (int u = 0; u < NPF; ++u) {
      const int j = tid + u * 256;
      if (j >= PAIRS) continue;
      unsigned px[2][2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        // channels (0, 1) and (2, 3) of the pixel; channels >= C and
        // pixels outside the image are zero
        px[e][0] = __builtin_amdgcn_alignbit(raw[u][e][1], raw[u][e][0], shf[u][e]) & (cmask0 & okm[u][e]);
        px[e][1] = __builtin_amdgcn_alignbit(raw[u][e][2], raw[u][e][1], shf[u][e]) & (cmask1 & okm[u][e]);
      }
      *reinterpret_cast<u32x4*>(smem + j * 16) = u32x4{px[0][0], px[0][1], px[1][0], px[1][1]};
    }
  };

  // operand offsets: output pixel m of the tile -> patch pixel (stride pr, stride pc);
  // chunk g = (r, sp) adds r rows and 2 sp columns
  // (pixels past the tile's rows, and a wave row's blocks past FMT, read
  // patch offset 0 and compute values that are never stored, which keeps
  // the step loop free of branches and every read inside the patch)
  int abase[FMW];
#pragma unroll
  for (int i = 0; i < FMW; ++i) {
    const int m = (wm * FMW + i) * 16 + (lane & 15);
    const int pr = sdiv(m, a.inv_q), pc = m - __umul24(pr, a.Q);
    abase[i] = wm * FMW + i < FMT && m < a.TR * a.Q ? (a.stride * (pr * a.PWP + pc)) * 8 : 0;
  }
  const int bbase = (wn * WTN + (lane & 15)) * WPITCH + (lane >> 4) * 16;
  const ActClamp ac = act_clamp(a.act);
  typedef typename Mfma<T>::frag frag;

  // the bias of the lane's output channels, staged through LDS so that no
  // global load of it is outstanding inside the tile loop (the compiler
  // would otherwise wait for every load there, the prefetch included)
  float* const Bs = reinterpret_cast<float*>(smem + P_BYTES + BN * WPITCH);
  if (tid < BN)
    Bs[tid] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rb, (n0 + tid) * 4, 0, 0));

  u32x4 raw[NPF][2];
  unsigned shf[NPF][2];
  unsigned ok[NPF][2];
  int tile = blockIdx.x;
  if (tile >= a.tiles) return;
  fetch(tile, raw, shf, ok);
#pragma unroll
  for (int u = 0; u < NFC; ++u) {
    const int idx = tid + u * 256;
    const int n = idx / GMAX, g = idx - n * GMAX;
    // channels past C are zero in the prepared filter
    *reinterpret_cast<u32x4*>(Ws + n * WPITCH + g * 16) = u32x4{d[u][0][0], d[u][0][1], d[u][1][0], d[u][1][1]};
  }
  store_patch(raw, shf, ok);
  __syncthreads();  // filter, bias and the first patch are in LDS
  f32x4 bias[FNW];
#pragma unroll
  for (int j = 0; j < FNW; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) bias[j][v] = Bs[wn * WTN + j * 16 + (lane >> 4) * 4 + v];

  // The patch of tile t + G (G = grid size) is loaded into registers while
  // tile t's MFMAs and stores run, then written to LDS.  The barriers wait
  // for LDS operations only, and every store is issued unconditionally
  // (masked by an out-of-range offset), so the wait for the prefetched
  // registers leaves the preceding output stores in flight.
  for (;; tile += gridDim.x) {
    const bool more = tile + (int)gridDim.x < a.tiles;
    if (more) fetch(tile + gridDim.x, raw, shf, ok);

    f32x4 acc[FMW][FNW];
#pragma unroll
    for (int i = 0; i < FMW; ++i)
#pragma unroll
      for (int j = 0; j < FNW; ++j) acc[i][j] = bias[j];
    // k-slice st + 1's fragments are read while st's MFMAs run
    frag fa[2][FMW], fb[2][FNW];
    auto load = [&](int st, int b) {
      const int g = st * 4 + (lane >> 4);
      const int r = sdiv(g, a.inv_sp), sp = g - __umul24(r, a.SP);
      const int toff = g < a.G ? (r * a.PWP + 2 * sp) * 8 : 0;
#pragma unroll
      for (int i = 0; i < FMW; ++i) fa[b][i] = *reinterpret_cast<const frag*>(smem + abase[i] + toff);
#pragma unroll
      for (int j = 0; j < FNW; ++j) fb[b][j] = *reinterpret_cast<const frag*>(Ws + bbase + j * 16 * WPITCH + st * 64);
    };
    load(0, 0);
#pragma unroll
    for (int st = 0; st < GMAX / 4; ++st) {
      if (st + 1 < GMAX / 4) load(st + 1, (st + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FMW; ++i)
#pragma unroll
        for (int j = 0; j < FNW; ++j) acc[i][j] = Mfma<T>::run(fb[st & 1][j], fa[st & 1][i], acc[i][j]);
    }

    // epilogue: each lane puts its 4 consecutive channels of a pixel (8
    // bytes) into the tile's LDS rows; then 16-byte chunks of 8 channels go
    // out, consecutive threads on consecutive chunks of the tile's pixels
    const int img = fdiv(tile, a.fd_tiles_img), rt = tile - img * a.tiles_img;
    const int row0 = rt * a.TR;
    const int valid = min(a.TR, a.P - row0) * a.Q;
    const int mbase = (img * a.P + row0) * a.Q;
#pragma unroll
    for (int i = 0; i < FMW; ++i) {
      const int ml = (wm * FMW + i) * 16 + (lane & 15);
      if (wm * FMW + i >= FMT) continue;
#pragma unroll
      for (int j = 0; j < FNW; ++j) {
        const int nl = wn * WTN + j * 16 + (lane >> 4) * 4;
        T o[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = from_f<T>(__builtin_amdgcn_fmed3f(acc[i][j][v], ac.lo, ac.hi));
        __builtin_memcpy(Os + ml * OPITCH + nl * 2, o, 8);
      }
    }
    lds_barrier();  // the tile's outputs are in LDS
    {
      constexpr int CPX = BN / 8;  // 16-byte chunks per pixel
      const bool vec = a.Ks % 8 == 0;
      for (int q = tid; q < valid * CPX; q += 256) {
        const int ml = q / CPX, c8 = q - ml * CPX;
        const int n = n0 + c8 * 8;
        if (n >= a.Ng) continue;
        const u32x4 v = *reinterpret_cast<const u32x4*>(Os + ml * OPITCH + c8 * 16);
        const unsigned e = (unsigned)((mbase + ml) * a.Ks + n);
        if (vec && n + 8 <= a.Ng) {
          __builtin_amdgcn_raw_buffer_store_b128(v, ry, (int)(e * 2u), 0, 0);
        } else {
          T o[8];
          __builtin_memcpy(o, &v, 16);
          T* __restrict__ y = reinterpret_cast<T*>(a.y);
          for (int t = 0; t < 8 && n + t < a.Ng; ++t) y[e + t] = o[t];
        }
      }
    }
    if (!more) break;
    lds_barrier();  // every wave is done reading this tile's patch
    store_patch(raw, shf, ok);
    lds_barrier();  // the next patch is in LDS
  }
}

// ------------------------------------------------------------------ host
static bool smallc_tiling(SmallCArgs& a, int fmt, int ppx, int gmax) {
  const int maxpx = fmt * 16;
  if (a.Q > maxpx) return false;
  const int fit = maxpx / a.Q;
  a.tiles_img = (a.P + fit - 1) / fit;
  a.TR = (a.P + a.tiles_img - 1) / a.tiles_img;
  a.tiles = a.N * a.tiles_img;
  a.PH = (a.TR - 1) * a.stride + a.R;
  const int pw = (a.Q - 1) * a.stride + a.S;
  a.PWP = (pw + 1) / 2 * 2;
  a.SP = (a.S + 1) / 2;
  a.G = a.R * a.SP;
  a.inv_sp = 1.f / (float)a.SP;
  a.inv_pwp2 = 1.f / (float)(a.PWP / 2);
  a.inv_q = 1.f / (float)a.Q;
  a.fd_tiles_img = make_fastdiv(a.tiles_img);
  return a.PH * a.PWP <= ppx && a.G <= gmax;
}

bool smallc_applicable(int layout, int c, int h, int w, int r, int s, int stride, int pad, int n,
                       int k, int fmt, int ppx, int gmax) {
  if (layout != NHWC || c > 4 || k % 4 != 0 || (stride != 1 && stride != 2)) return false;
  SmallCArgs a{};
  a.N = n;
  a.stride = stride;
  a.P = (h + 2 * pad - r) / stride + 1;
  a.Q = (w + 2 * pad - s) / stride + 1;
  a.R = r;
  a.S = s;
  // 32-bit byte offsets of the input and of the output (channels padded to 8)
  if ((long long)n * h * w * c * 2 >= (long long)kOOB ||
      (long long)n * a.P * a.Q * ((k + 7) / 8 * 8) * 2 >= (long long)kOOB)
    return false;
  return smallc_tiling(a, fmt, ppx, gmax);
}

template <typename T, int FMT, int WM, int PPX, int GMAX, int OCC>
static void smallc_go(SmallCArgs a, hipStream_t st) {
  check(smallc_tiling(a, FMT, PPX, GMAX), "small-channel tile does not fit");
  const int tn = (a.Ng + 63) / 64;
  // persistent: OCC workgroups per CU over 256 CUs, split over the channel tiles
  const int per_n = std::max(1, std::min(a.tiles, 256 * OCC / tn));
  dim3 grid(per_n, tn);
  SN_LAUNCH((conv_smallc_kernel<T, FMT, WM, PPX, GMAX, OCC>), grid, dim3(256), 0, st, a);
}

void conv_smallc(int dtype, int fmt, int gmax, const ConvArgs& c, hipStream_t st, int wm, int occ) {
  check(dtype != 0, "small-channel kernel runs 16-bit types");
  check(c.xd.layout == NHWC && c.yd.layout == NHWC && c.xd.c <= 4 && (c.stride == 1 || c.stride == 2),
        "small-channel kernel: NHWC, C <= 4, stride 1 or 2");
  SmallCArgs a{};
  a.x = c.x;
  a.w = c.w;
  a.bias = c.bias;
  a.y = c.y;
  a.N = c.xd.n;
  a.C = c.xd.c;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.K = c.yd.c;
  a.P = c.yd.h;
  a.Q = c.yd.w;
  a.Ks = c.yd.cs;
  a.Ng = c.yd.c;
  a.R = c.r;
  a.S = c.s;
  a.pad = c.pad;
  a.act = c.act;
  a.stride = c.stride;
  a.C8 = (a.C + 7) / 8 * 8;
  a.Kred = a.R * a.S * a.C8;
  a.x_elems = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w;
  a.w_elems = (long long)((a.K + 7) / 8 * 8) * a.Kred;
  a.y_elems = (long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w;
  check(a.x_elems * 2 < (long long)kOOB && a.y_elems * 2 < (long long)kOOB && a.w_elems * 2 < (long long)kOOB,
        "tensor too large for 32-bit offsets");
  check(c.yd.cs % 4 == 0 && c.yd.c % 4 == 0, "small-channel kernel stores 4-channel groups");
#define SC(FMT, PPX, GMAX, WM, OCC)                                         \
  if (fmt == FMT && gmax == GMAX && wm == WM && occ == OCC) {               \
    if (dtype == 1) smallc_go<f16, FMT, WM, PPX, GMAX, OCC>(a, st);         \
    else smallc_go<bf16, FMT, WM, PPX, GMAX, OCC>(a, st);                   \
    return;                                                                 \
  }
  SC(7, 1664, 28, 2, 2)
  SC(14, 2112, 28, 2, 2)
  SC(7, 704, 8, 2, 3)
  SC(14, 1152, 8, 2, 2)
  SC(14, 2112, 28, 4, 2)
#undef SC
  check(false, "small-channel tile not instantiated");
}

}  // namespace k
}  // namespace sn
