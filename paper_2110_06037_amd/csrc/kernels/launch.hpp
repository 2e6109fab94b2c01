// Host-callable launchers of the routine kernels.  Every launcher checks
// that its operands fit the kernel's assumptions and enqueues on the given
// stream; none allocates or synchronises.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

namespace sn {
namespace k {

// Kernel-execution timing.  While `start` or `stop` is set, launches go
// through hipExtLaunchKernelGGL with these events, which the runtime ties to
// the kernel dispatches themselves: `start` to the start of the next launch
// (then cleared), `stop` to the end of every launch while it stays set.
// Each such event adds a dispatch gap of a few microseconds, so timers set
// them only at the first and last launch of a long back-to-back sequence.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchTiming g_timing;
// Launch accounting: every launch adds one to g_launches; while
// g_count_only is set the launches are only counted, not enqueued (used to
// list a plan's kernel launches without running them).
extern thread_local long long g_launches;
extern thread_local int g_count_only;

#define SN_LAUNCH(K, G, B, S, ST, ...)                                                  \
  do {                                                                                  \
    ++::sn::k::g_launches;                                                              \
    if (::sn::k::g_count_only) break;                                                   \
    if (::sn::k::g_timing.start || ::sn::k::g_timing.stop) {                            \
      hipExtLaunchKernelGGL(K, G, B, S, ST, ::sn::k::g_timing.start, ::sn::k::g_timing.stop, 0, \
                            __VA_ARGS__);                                               \
      ::sn::k::g_timing.start = nullptr;                                                \
    } else {                                                                            \
      hipLaunchKernelGGL(K, G, B, S, ST, __VA_ARGS__);                                  \
    }                                                                                   \
  } while (0)

// Logical tensor N x C x H x W stored in `layout` with `cs` stored channels.
struct TDesc {
  int n, c, h, w, cs, layout;
};

// Tile counters of implicit-GEMM launches whose reduction is split across
// workgroups (the last workgroup of a tile to finish sums the partial
// tiles): tile ids stay below this bound, and a caller's counter array
// holds this many.
constexpr int kFixupMaxTiles = 1024;

struct ConvArgs {
  const void* x;
  TDesc xd;
  const void* w;      // dense: [Kp][R][S][C8]; winograd: U [16][Kp][C8]; depthwise: [R][S][C8]
  const float* bias;  // [Kp], zero-padded
  void* y;
  TDesc yd;
  int r, s, stride, pad, act;
  void* ws;           // workspace (winograd); ws_bytes its size
  size_t ws_bytes;
  const void* res = nullptr;  // residual of the output's shape and layout, added before the
                              // activation (direct and implicit-GEMM routines), or null
  unsigned* cnt = nullptr;    // kFixupMaxTiles tile counters for reductions split across
                              // workgroups: zero before a launch, zero again after it
  // projected shortcut (implicit GEMM on the LDS-DMA tiles): x2 read by a
  // 1 x 1 convolution without padding at stride2 with weights w2 (dense
  // [Kp][1][1][C2_8]), added to the sums before the activation; or null
  const void* x2 = nullptr;
  TDesc x2d{};
  const void* w2 = nullptr;
  int stride2 = 1;
  const void* wcat = nullptr;  // 1x1 convolution with a projected shortcut: both weights,
                               // rows [Kp][C8 + C2_8] (the streaming kernel's filter)
};

void conv_direct(int dtype, const ConvArgs& a, hipStream_t st);
// Implicit GEMM; `param` selects the tile configuration (routine parameter).
// Parameters that split the reduction need a workspace of igemm_ws_bytes.
void conv_igemm(int dtype, int param, const ConvArgs& a, hipStream_t st);
int igemm_num_params(int dtype);
// whether the tile configuration adds a residual in its epilogue (for an
// output of k channels in the layout)
bool igemm_param_takes_residual(int dtype, int param, int layout, int k);
bool igemm_param_valid(int dtype, int param, int layout, int n, int c, int h, int w, int r, int s,
                       int stride, int pad, int k);
// whether the tile configuration takes a projected shortcut of c2 channels
// (besides being valid for the convolution itself)
bool igemm_param_takes_projection(int dtype, int param, int layout, int n, int c, int h, int w, int r, int s,
                                  int stride, int pad, int k, int c2);
// workspace bytes (c2 > 0: with a projected shortcut of c2 channels)
size_t igemm_ws_bytes(int dtype, int param, const TDesc& xd, const TDesc& yd, int r, int s, int c2 = 0);
// 3x3 stride-1 or stride-2 convolution with the input patch in LDS (an
// implicit-GEMM parameter family; see conv_patch.hip)
struct PatchCfg {
  int fmt, bn, pwt, wm, wn, tg, st, prows;  // one PATCH_CONFIGS tuple
  int sd = 1;                               // convolution stride
  int occ = 1;                              // workgroups per CU the tile is sized for
  int ra = 0;                               // 1: row-aligned row blocks (stride 1)
};
// Instantiated patch tiles (FMT, BN, PWT, WM, WN, TG, ST, PROWS): FMT row
// blocks of 16 output pixels, BN output channels, patch row pitch PWT, 8
// waves as TG tap groups of WM x WN, ST LDS stages, PROWS patch rows per
// stage.  Each is one implicit-GEMM routine parameter.
#define PATCH_CONFIGS(X)         \
  X(25, 64, 64, 4, 2, 1, 2, 576) \
  X(13, 64, 32, 4, 2, 1, 2, 288) \
  X(13, 64, 32, 2, 2, 2, 2, 288) \
  X(13, 32, 16, 4, 1, 2, 3, 256) \
  X(13, 32, 16, 4, 2, 1, 3, 256) \
  X(7, 32, 16, 4, 1, 2, 3, 288)  \
  X(7, 32, 64, 4, 1, 2, 2, 256)  \
  X(25, 64, 64, 4, 1, 2, 2, 576) \
  X(13, 64, 32, 4, 1, 2, 2, 288) \
  X(7, 64, 16, 4, 1, 2, 2, 288)
// Stride-2 patch tiles (same fields): ResNet-50's first 3x3 of stages 2-4
// at 56->28, 28->14 and 14->7 (patch width 2Q + 1 within PWT)
#define PATCH2_CONFIGS(X)        \
  X(7, 64, 64, 4, 1, 2, 2, 576)  \
  X(7, 64, 32, 4, 1, 2, 2, 480)  \
  X(7, 64, 16, 4, 1, 2, 2, 480)  \
  X(4, 64, 16, 4, 1, 2, 2, 240)  \
  X(7, 32, 16, 4, 1, 2, 3, 480)
// Stride-1 patch tiles for two workgroups per CU (at most 80 KB of LDS and
// 128 registers each), so that one workgroup's prologue and stores overlap
// the other's steps (7 x 7 and 14 x 14 at 32 output channels per tile)
#define PATCH_OCC2_CONFIGS(X)    \
  X(7, 32, 16, 4, 1, 2, 2, 288)
// Row-aligned stride-1 patch tiles (same fields): a row block is 16
// consecutive patch columns of one output row (PWT / 16 blocks per row, the
// columns past Q computed and dropped), so every operand read covers 16
// consecutive LDS rows; at 56, 28 and 14 columns the blocks computed are as
// many as the unaligned tiles' waves cover anyway
// (the last field: workgroups per CU the tile is sized for)
#define PATCH_RA_CONFIGS(X)         \
  X(28, 64, 64, 4, 2, 1, 2, 576, 1) \
  X(14, 64, 32, 4, 2, 1, 2, 288, 1) \
  X(8, 64, 16, 4, 1, 2, 2, 288, 1)  \
  X(8, 32, 16, 4, 1, 2, 2, 160, 2)
bool patch_applicable(int layout, int c, int h, int w, int r, int s, int stride, int pad, int n,
                      int fmt, int pwt, int prows, int sd, int ra = 0);
void conv_patch(int dtype, const PatchCfg& cfg, const ConvArgs& a, hipStream_t st);
// Stride-1 or -2 convolution of an NHWC input with C <= 4 (a CNN stem; see
// conv_smallc.hip); gmax: filter chunks the kernel holds (28 for 7 x 7, 8 for 3 x 3)
bool smallc_applicable(int layout, int c, int h, int w, int r, int s, int stride, int pad, int n,
                       int k, int fmt, int ppx, int gmax);
// wm: wave rows (of 4 waves); occ: workgroups per CU the persistent grid and
// the register budget are sized for
void conv_smallc(int dtype, int fmt, int gmax, const ConvArgs& a, hipStream_t st, int wm = 2, int occ = 3);
// 1x1 convolution (stride 1 or 2, no padding) of an NHWC input with cc =
// 64, 128, 256 or 512 channels by persistent workgroups streaming pixel tiles
// (see conv1x1_stream.hip).  Instantiated tiles (CC, BM, BN, WM, PD): BM
// pixels x BN channels per tile, WM wave rows, loads PD tiles ahead; each is
// one implicit-GEMM routine parameter.
#define STREAM_CONFIGS(X) \
  X(64, 64, 256, 2, 1)    \
  X(64, 128, 128, 4, 1)   \
  X(64, 128, 64, 4, 1)    \
  X(128, 64, 128, 2, 1)   \
  X(128, 32, 256, 1, 1)   \
  X(256, 64, 64, 4, 1)    \
  X(256, 32, 128, 2, 1)   \
  X(64, 64, 256, 2, 2)    \
  X(64, 128, 128, 4, 2)   \
  X(128, 64, 128, 2, 2)   \
  X(128, 32, 256, 1, 3)   \
  X(256, 64, 64, 4, 2)    \
  X(256, 32, 128, 2, 2)   \
  X(256, 32, 128, 2, 3)
// 512-channel inputs, and 384 = 128 + 256 (a 128-channel 1x1 convolution
// with a 256-channel projected shortcut) with the sums staged in the pixel
// buffer; routine parameters after the others
#define STREAM512_CONFIGS(X) \
  X(512, 32, 64, 2, 1)       \
  X(384, 32, 128, 2, 1)
// Streaming tiles sized for two workgroups per CU (at most 80 KB of LDS and
// 128 registers each), so that one workgroup's loads and epilogue overlap
// the other's MFMAs
#define STREAM_OCC2_CONFIGS(X) \
  X(256, 32, 64, 2, 1)         \
  X(128, 32, 64, 2, 2)         \
  X(64, 64, 64, 4, 2)          \
  X(64, 64, 128, 4, 2)         \
  X(128, 32, 128, 2, 1)
bool stream1x1_applicable(int layout, int c, int cs, int n, int h, int w, int r, int s, int stride, int pad,
                          int k, int cc);
// the streaming kernel with a projected shortcut of c2 channels (slabs of
// the main input, then of the shortcut: c + c2 = cc, both multiples of 64)
bool stream1x1_takes_projection(int layout, int c, int cs, int n, int h, int w, int r, int s, int stride, int pad,
                                int k, int c2, int cc);
// occ: workgroups per CU the persistent grid and the LDS are sized for
void conv1x1_stream(int dtype, int cc, int bm, int bn, int pd, const ConvArgs& a, hipStream_t st, int occ = 1);
// Winograd F(m x m, 3x3), m = tile 2 or 4, as three sub-layers (a
// childnet): sub 0 = input transform, 1 = the (m+2)^2 batched GEMMs with
// GEMM tile `cfg` (one of winograd_gemm_num_configs), 2 = output transform;
// V and M in the workspace (winograd_ws_bytes)
size_t winograd_ws_bytes(int dtype, const TDesc& xd, int k, int tile = 2);
int winograd_gemm_num_configs(int dtype);
void winograd_sub(int dtype, int tile, int sub, int cfg, const ConvArgs& a, hipStream_t st);
void conv_winograd(int dtype, int tile, const ConvArgs& a, int gemm_cfg, hipStream_t st);
// routine parameter of the F(4x4,3x3) routine (after the fused F(2x2,3x3) ones)
int winograd_f4_param();
// param 0: the strip kernel (16-bit NHWC with C % 8 == 0 or NC8HW8, 3x3,
// stride 1 or 2) with its strip length chosen by the thread count, else the
// general kernel; param p >= 1: the strip kernel with strips of
// dw_strip_len(p) output rows (valid for p <= dw_num_strip_params(...)).
void dwconv(int dtype, const ConvArgs& a, int param, hipStream_t st);
int dw_num_strip_params(int dtype, int layout, int c, int r, int s, int stride);
int dw_strip_len(int param);

void maxpool(int dtype, const void* x, const TDesc& xd, void* y, const TDesc& yd, int k,
             int stride, int pad, hipStream_t st);
void gap(int dtype, const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t st);
void add_act(int dtype, const void* a, const void* b, void* y, int64_t n, int act, hipStream_t st);
// FC: x [N][cin_s] (stored), w [Kp][C8], y [N][kout_s] = act(W x + b); small
// 16-bit batches run on MFMA, the rest as VALU dot products
void fc_direct(int dtype, const void* x, int n, int cin, int cin_s, const void* w, int c8,
               const float* bias, void* y, int kout, int kout_s, int act, hipStream_t st);
void convert(int dtype, const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t st);
// 16-byte vector layout converters for 16-bit tensors (convert.hip); false
// when the shape needs the element-wise converter
bool convert_vec16(const void* x, const TDesc& xd, void* y, const TDesc& yd, hipStream_t st);
// schema conversion: layout and element type (sdt -> ddt) at once; equal
// dtypes fall back to convert (see convert.hip)
void convert_cast(int sdt, const void* x, const TDesc& xd, int ddt, void* y, const TDesc& yd, hipStream_t st);
void fill_random(int dtype, void* p, int64_t n, uint64_t seed, hipStream_t st);

}  // namespace k
}  // namespace sn
