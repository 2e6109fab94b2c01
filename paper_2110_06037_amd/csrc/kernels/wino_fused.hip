// Winograd F(2x2, 3x3) convolution (Sec. II-B of the paper; stride 1,
// padding 1) fused into one kernel for 16-bit NHWC / NC8HW8 tensors.
//
// An output tile is 2x2 pixels; its 4x4 input patch d gives V = B^T d B (16
// values per channel), the filter gives U = G g G^T (prepared once, [16][Kp]
// [C8]), M_xi = sum over input channels of U_xi V_xi for each of the 16
// positions xi, and the tile's outputs are Y = A^T M A.  The 16 products are
// GEMMs over the input channels, run on MFMA with U as the first operand
// (rows: output channels) and V as the second (columns: tiles).
//
// Layout of the work.  A workgroup of NW waves takes 16 * NW tiles and
// 16 * FN output channels; each wave owns 16 tiles and all the workgroup's
// channels, and holds the 16 x FN accumulator blocks of all 16 positions.
// Per step of 32 input channels:
//  * V never leaves registers: lane l of a wave loads the 4x4 patch of tile
//    l % 16 for the 8 channels (l / 16) * 8 .. + 8 (16 loads of 16 bytes,
//    zero outside the image from the buffer range check), and computes V in
//    float32 -- exactly the MFMA operand layout (column = tile, reduction
//    chunk = lane / 16), so its 16 rounded vectors are the 16 positions'
//    second operands.  The next step's patch loads are issued before this
//    step's products, into the registers just freed.
//  * U of the step ([16][16 * FN][32], 64-byte rows) goes to LDS by direct
//    loads, double-buffered, and every wave reads it as first operands.
// After the last step each lane holds, for its tile and 4 consecutive
// output channels of each block, all 16 positions of M: the output
// transform, bias, activation and the 8-byte stores of 4 channels per
// output pixel need no data from other lanes.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "wino.hpp"

namespace sn {
namespace k {

// Element c of 8 packed 16-bit values, widened exactly to float32.
template <typename T>
__device__ __forceinline__ float elem(const u32x4& v, int c) {
  const unsigned w = v[c >> 1];
  if constexpr (std::is_same<T, bf16>::value) return __builtin_bit_cast(float, (c & 1) ? (w & 0xffff0000u) : (w << 16));
  return (float)__builtin_bit_cast(f16, (unsigned short)((c & 1) ? (w >> 16) : (w & 0xffffu)));
}

// Two float32 values rounded (nearest-even) to T and packed low, high.
template <typename T>
__device__ __forceinline__ unsigned pack2(float lo, float hi) {
  typedef T T2 __attribute__((ext_vector_type(2)));
  const T2 v = {from_f<T>(lo), from_f<T>(hi)};
  return __builtin_bit_cast(unsigned, v);
}

struct WinoFArgs {
  const void* x;       // input, N x C x H x W in NHWC or NC8HW8
  const void* u;       // [16][Kp][C8]
  const float* bias;   // [Kp]
  void* y;             // output, N x K x H x W, same layout
  int H, W, Cs, C8, Kp, Ng, Ks, act;
  int TH, TW, T;       // tiles per column / row, total tiles
  FastDiv fd_thw, fd_tw;
  int HW8, W8, CB;     // NC8HW8 strides
  long long x_elems, u_elems, y_elems;
};

template <typename T, int L, int NW, int FN>
__global__ __launch_bounds__(64 * NW, 1) void wino_fused_kernel(WinoFArgs a) {
  static_assert(sizeof(T) == 2 && (L == NHWC || L == NC8), "16-bit channel-vector layouts");
  constexpr int BN = 16 * FN;              // output channels per workgroup
  constexpr int RB = 64;                   // LDS row: 32 input channels of one (xi, k)
  constexpr int STAGE = 16 * BN * RB;      // bytes of U per step
  constexpr int NU = STAGE / 1024 / NW;    // direct-load instructions per wave and step
  static_assert(NU * 1024 * NW == STAGE, "U stage splits over the waves");
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
  auto swz = [](int row) { return (row >> 1) & 3; };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = blockIdx.y * BN;
  const int KT = a.C8 / 32;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, a.x_elems * 2);
  const __amdgpu_buffer_rsrc_t ru = make_rsrc(a.u, a.u_elems * 2);
  const __amdgpu_buffer_rsrc_t ry = make_rsrc(a.y, a.y_elems * 2);

  // this lane's tile and channel chunk
  const int t = (blockIdx.x * NW + wave) * 16 + (lane & 15);
  const int chunk = lane >> 4;
  int img = 0, th = 0, tw = 0;
  const bool tile_ok = t < a.T;
  if (tile_ok) {
    img = fdiv(t, a.fd_thw);
    const int r = t - img * (a.TH * a.TW);
    th = fdiv(r, a.fd_tw);
    tw = r - th * a.TW;
  }
  // byte offsets of the 16 patch pixels at channel step 0 (kOOB outside the
  // image or past the last tile); a step adds 32 channels
  unsigned doff[16];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int h = 2 * th - 1 + i, w = 2 * tw - 1 + j;
      unsigned off = kOOB;
      if (tile_ok && (unsigned)h < (unsigned)a.H && (unsigned)w < (unsigned)a.W) {
        if constexpr (L == NHWC) off = (unsigned)(((img * a.H + h) * a.W + w) * a.Cs + chunk * 8) * 2u;
        else off = (unsigned)((img * a.CB + chunk) * a.HW8 + h * a.W8 + w * 8) * 2u;
      }
      doff[i * 4 + j] = off;
    }
  const unsigned dstep = L == NHWC ? 64u : (unsigned)(4 * a.HW8 * 2);  // bytes per 32-channel step
  u32x4 d[16];
  auto load_patch = [&](int kt) {
#pragma unroll
    for (int q = 0; q < 16; ++q)
      d[q] = __builtin_amdgcn_raw_buffer_load_b128(rx, doff[q] == kOOB ? (int)kOOB : (int)(doff[q] + kt * dstep), 0, 0);
  };

  // U direct loads: instruction b = wave + NW * i fills LDS rows [16 b, 16 b + 16)
  // of the stage (row = xi * BN + k); this lane row 16 b + lane / 4, chunk
  // lane % 4 (logical chunk (lane % 4) ^ swz(row))
  unsigned uoff[NU];
#pragma unroll
  for (int i = 0; i < NU; ++i) {
    const int b = wave + NW * i;
    const int row = 16 * b + (lane >> 2);
    const int xi = row / BN, k = n0 + row % BN;
    const int lc = (lane & 3) ^ swz(row);
    uoff[i] = k < a.Kp ? (unsigned)(((xi * a.Kp + k) * a.C8) + lc * 8) * 2u : kOOB;
  }
  auto issue_u = [&](int kt, int buf) {
#pragma unroll
    for (int i = 0; i < NU; ++i)
      dma16(ru, smem + buf * STAGE + (wave + NW * i) * 1024, uoff[i], kt * 64);
  };

  // LDS byte offset of this lane's first-operand chunk: row xi * BN + 16 j + lane % 16
  const int arow = lane & 15;
  const int achk = ((lane >> 4) ^ swz(arow)) << 4;  // rows 16 apart keep the swizzle

  typedef typename Mfma<T>::frag frag;
  f32x4 acc[16][FN];
#pragma unroll
  for (int xi = 0; xi < 16; ++xi)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[xi][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_patch(0);
  issue_u(0, 0);
  for (int kt = 0; kt < KT; ++kt) {
    // this step's patch (younger: this step's U loads)
    wait_vmcnt<NU>();
    // V = B^T d B in float32, 8 channels per lane, rounded to T
    // (two channels at a time, so only their 32 values are live, and each
    // pair of results rounds and packs into one 32-bit register at once)
    u32x4 vw[16];
#pragma unroll
    for (int c = 0; c < 8; c += 2) {
      float vv[2][16];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float dv[4][4];
#pragma unroll
        for (int q = 0; q < 16; ++q) dv[q / 4][q % 4] = elem<T>(d[q], c + h);
        float tt[4][4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          tt[0][j] = dv[0][j] - dv[2][j];
          tt[1][j] = dv[1][j] + dv[2][j];
          tt[2][j] = dv[2][j] - dv[1][j];
          tt[3][j] = dv[1][j] - dv[3][j];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          vv[h][i * 4 + 0] = tt[i][0] - tt[i][2];
          vv[h][i * 4 + 1] = tt[i][1] + tt[i][2];
          vv[h][i * 4 + 2] = tt[i][2] - tt[i][1];
          vv[h][i * 4 + 3] = tt[i][1] - tt[i][3];
        }
      }
#pragma unroll
      for (int xi = 0; xi < 16; ++xi) vw[xi][c >> 1] = pack2<T>(vv[0][xi], vv[1][xi]);
    }
    frag vb[16];
#pragma unroll
    for (int xi = 0; xi < 16; ++xi) vb[xi] = __builtin_bit_cast(frag, vw[xi]);
    // the next step's patch into the registers just freed
    if (kt + 1 < KT) load_patch(kt + 1);
    // this step's U (younger: the next patch's loads)
    if (kt + 1 < KT) wait_vmcnt<16>();
    else wait_vmcnt<0>();
    dma_barrier();  // every wave's U share landed; every wave is done with the other buffer
    if (kt + 1 < KT) issue_u(kt + 1, (kt + 1) & 1);
    const char* S = smem + (kt & 1) * STAGE;
    frag ua[2][FN];
    auto read_u = [&](int xi, int b) {
#pragma unroll
      for (int j = 0; j < FN; ++j)
        ua[b][j] = *reinterpret_cast<const frag*>(S + (xi * BN + 16 * j + arow) * RB + achk);
    };
    read_u(0, 0);
#pragma unroll
    for (int xi = 0; xi < 16; ++xi) {
      if (xi + 1 < 16) read_u(xi + 1, (xi + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[xi][j] = Mfma<T>::run(ua[xi & 1][j], vb[xi], acc[xi][j]);
    }
  }

  // output transform: Y = A^T M A per channel; accumulator (xi, j) element v
  // is output channel n0 + 16 j + 4 (lane / 16) + v of tile lane % 16
  if (!tile_ok) return;
  const ActClamp ac = act_clamp(a.act);
  const int P = a.H, Q = a.W;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const int n = n0 + 16 * j + 4 * chunk;
    T out[4][4];  // [pixel][channel]
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      float m[4][4];
#pragma unroll
      for (int xi = 0; xi < 16; ++xi) m[xi / 4][xi % 4] = acc[xi][j][v];
      float s0[4], s1[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        s0[c] = m[0][c] + m[1][c] + m[2][c];
        s1[c] = m[1][c] - m[2][c] - m[3][c];
      }
      const float b = n + v < a.Ng ? a.bias[n + v] : 0.f;
      const float y00 = s0[0] + s0[1] + s0[2], y01 = s0[1] - s0[2] - s0[3];
      const float y10 = s1[0] + s1[1] + s1[2], y11 = s1[1] - s1[2] - s1[3];
      out[0][v] = from_f<T>(act_apply(y00 + b, ac));
      out[1][v] = from_f<T>(act_apply(y01 + b, ac));
      out[2][v] = from_f<T>(act_apply(y10 + b, ac));
      out[3][v] = from_f<T>(act_apply(y11 + b, ac));
    }
    if (n >= a.Ng) continue;
    // 4 channels as one 8-byte store where they are whole and aligned
    const bool vec4 = L == NC8 || (a.Ks % 4 == 0 && n + 4 <= a.Ng);
#pragma unroll
    for (int px = 0; px < 4; ++px) {
      const int p = 2 * th + (px >> 1), q = 2 * tw + (px & 1);
      if (p >= P || q >= Q) continue;
      unsigned e;
      if constexpr (L == NHWC) e = (unsigned)(((img * P + p) * Q + q) * a.Ks + n);
      else e = (unsigned)(((img * (a.Ks >> 3) + (n >> 3)) * P + p) * Q + q) * 8u + (n & 7);
      if (vec4) {
        __builtin_amdgcn_raw_buffer_store_b64(*reinterpret_cast<const u32x2*>(out[px]), ry, (int)(e * 2u), 0, 0);
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (n + v < a.Ng)
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, out[px][v]), ry,
                                                  (int)((e + v) * 2u), 0, 0);
      }
    }
  }
}

int wino_fused_num_configs() {
#define WN_COUNT(NW_, FN_) +1
  return 0 WINO_CONFIGS(WN_COUNT);
#undef WN_COUNT
}

bool wino_fused_applicable(int dtype, int layout, int c) {
  if (dtype == 0) return false;
  if (layout == NHWC) return c % 32 == 0;
  if (layout == NC8) return ((c + 7) / 8 * 8) % 32 == 0;
  return false;
}

template <typename T, int L>
static void wino_fused_layout(int cfg, const WinoFArgs& a, hipStream_t st) {
  int idx = 0;
#define WN_GO(NW_, FN_)                                                                     \
  if (cfg == idx++) {                                                                       \
    const dim3 grid((a.T + 16 * NW_ - 1) / (16 * NW_), (a.Ng + 16 * FN_ - 1) / (16 * FN_)); \
    SN_LAUNCH((wino_fused_kernel<T, L, NW_, FN_>), grid, dim3(64 * NW_), 0, st, a);         \
    return;                                                                                 \
  }
  WINO_CONFIGS(WN_GO)
#undef WN_GO
  check(false, "fused Winograd configuration");
}

void conv_wino_fused(int dtype, int cfg, const ConvArgs& c, hipStream_t st) {
  check(c.r == 3 && c.s == 3 && c.stride == 1 && c.pad == 1 && c.xd.layout == c.yd.layout &&
            c.xd.h == c.yd.h && c.xd.w == c.yd.w && wino_fused_applicable(dtype, c.xd.layout, c.xd.c) && !c.res,
        "fused Winograd: 16-bit 3x3 stride 1 pad 1, channels in steps of 32, no residual");
  WinoFArgs a{};
  a.x = c.x;
  a.u = c.w;
  a.bias = c.bias;
  a.y = c.y;
  a.H = c.xd.h;
  a.W = c.xd.w;
  a.Cs = c.xd.cs;
  a.C8 = (c.xd.c + 7) / 8 * 8;
  a.Kp = (c.yd.c + 7) / 8 * 8;
  a.Ng = c.yd.layout == NC8 ? c.yd.cs : c.yd.c;
  a.Ks = c.yd.cs;
  a.act = c.act;
  a.TH = (a.H + 1) / 2;
  a.TW = (a.W + 1) / 2;
  const long long T = (long long)c.xd.n * a.TH * a.TW;
  a.T = (int)T;
  a.fd_thw = make_fastdiv(a.TH * a.TW);
  a.fd_tw = make_fastdiv(a.TW);
  a.HW8 = a.H * a.W * 8;
  a.W8 = a.W * 8;
  a.CB = a.C8 / 8;
  a.x_elems = (long long)c.xd.n * c.xd.cs * c.xd.h * c.xd.w;
  a.u_elems = 16LL * a.Kp * a.C8;
  a.y_elems = (long long)c.yd.n * c.yd.cs * c.yd.h * c.yd.w;
  check(T < (1 << 21) && a.x_elems * 2 < (long long)kOOB && a.u_elems * 2 < (long long)kOOB &&
            a.y_elems * 2 < (long long)kOOB,
        "fused Winograd: tensor too large for 32-bit offsets");
  if (dtype == 1) {
    if (c.xd.layout == NHWC) wino_fused_layout<f16, NHWC>(cfg, a, st);
    else wino_fused_layout<f16, NC8>(cfg, a, st);
  } else {
    if (c.xd.layout == NHWC) wino_fused_layout<bf16, NHWC>(cfg, a, st);
    else wino_fused_layout<bf16, NC8>(cfg, a, st);
  }
}

}  // namespace k
}  // namespace sn
