// Fully connected layer for a small batch (y = act(W x + b) with W [K][C], the
// FC layer type of Sec. III-B) on MFMA, 16-bit types.
//
// With a batch of at most 64 the layer is a skinny GEMM whose cost is
// reading W once (2048 x 1000 bf16 = 4 MB for a ResNet classifier).  A
// workgroup owns 16 output features and 16 rows of the batch; its 8 waves split
// the input features (wave w takes the 32-wide reduction steps w, w + 8, ...)
// so every workgroup keeps many 16-byte loads in flight, and the 8 partial
// sums meet in LDS.  Operands come straight from global memory: W rows are
// read once, x rows (shared by all workgroups) come from L2.
#include "gemm_common.hpp"
#include "kcommon.hpp"
#include "launch.hpp"

namespace sn {
namespace k {

constexpr int kFcWaves = 8;

// NB: 16-row batch blocks (batch <= 16 NB); U: reduction steps per wave issued together
template <typename T, int NB, int U>
__global__ __launch_bounds__(64 * kFcWaves) void fc_mfma_kernel(const T* __restrict__ x, int N, int cin,
                                                                int cin_s, const T* __restrict__ w,
                                                                int c8, int kp,
                                                                const float* __restrict__ bias,
                                                                T* __restrict__ y, int kout_s, int act) {
  typedef typename Mfma<T>::frag frag;
  __shared__ f32x4 red[kFcWaves][NB][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int k0 = blockIdx.x * 16;
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(w, (long long)kp * c8 * 2);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (long long)N * cin_s * 2);
  // lane l: W row k0 + (l & 15) and batch row (l & 15) of each block, 8
  // input features at (l >> 4) * 8 within the 32-wide step
  const int sub = (lane >> 4) * 8;
  const unsigned wrow = (unsigned)(k0 + (lane & 15)) * (unsigned)c8;
  unsigned xrow[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int n = (blockIdx.y * NB + j) * 16 + (lane & 15);
    xrow[j] = n < N ? (unsigned)n * (unsigned)cin_s : kOOB;
  }
  f32x4 acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int steps = (cin + 31) / 32;
  for (int s0 = wave; s0 < steps; s0 += kFcWaves * U) {
    frag fw[U], fx[U][NB];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = (s0 + u * kFcWaves) * 32 + sub;
      const bool in = c < cin;  // cin % 8 == 0: a chunk is wholly in or out
      fw[u] = __builtin_bit_cast(frag, __builtin_amdgcn_raw_buffer_load_b128(
                                          rw, in ? (int)((wrow + c) * 2u) : (int)kOOB, 0, 0));
#pragma unroll
      for (int j = 0; j < NB; ++j)
        fx[u][j] = __builtin_bit_cast(
            frag, __builtin_amdgcn_raw_buffer_load_b128(
                      rx, in && xrow[j] != kOOB ? (int)((xrow[j] + c) * 2u) : (int)kOOB, 0, 0));
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[j] = Mfma<T>::run(fw[u], fx[u][j], acc[j]);
  }
#pragma unroll
  for (int j = 0; j < NB; ++j) red[wave][j][lane] = acc[j];
  __syncthreads();
  // thread t < 64 NB sums block j = t / 64 over the waves; its lane holds
  // batch row j * 16 + (t & 15) and features k0 + ((t & 63) >> 4) * 4 + v
  const int t = threadIdx.x;
  if (t >= 64 * NB) return;
  const int j = t >> 6, l = t & 63;
  f32x4 s = red[0][j][l];
#pragma unroll
  for (int v = 1; v < kFcWaves; ++v) s += red[v][j][l];
  const int n = (blockIdx.y * NB + j) * 16 + (l & 15);
  const int kb = k0 + (l >> 4) * 4;
  if (n >= N) return;
  T o[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) o[v] = from_f<T>(act_f(s[v] + (kb + v < kout_s ? bias[kb + v] : 0.f), act));
  T* yp = y + (long long)n * kout_s + kb;
  if (kout_s % 4 == 0 && kb + 4 <= kout_s) {
    u32x2 pk;
    __builtin_memcpy(&pk, o, 8);
    *reinterpret_cast<u32x2*>(yp) = pk;
  } else {
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (kb + v < kout_s) yp[v] = o[v];
  }
}

bool fc_mfma_applicable(int dtype, int n, int cin, int cin_s) {
  return dtype != 0 && n >= 1 && n <= 64 && cin % 8 == 0 && cin_s % 8 == 0 &&
         (long long)n * cin_s * 2 < (long long)kOOB;
}

template <typename T>
static void fc_mfma_t(const void* x, int n, int cin, int cin_s, const void* w, int c8, const float* bias,
                      void* y, int kout, int kout_s, int act, hipStream_t st) {
  const int kp = (kout + 7) / 8 * 8;
  check((long long)kp * c8 * 2 < (long long)kOOB, "FC weights too large for 32-bit offsets");
  check(kout_s <= kp && c8 >= cin, "FC shapes");
  // one 16-row batch block per workgroup (grid.y): more workgroups to read
  // W, whose rows the batch blocks then share through L2
  const dim3 grid((kout_s + 15) / 16, (n + 15) / 16), block(64 * kFcWaves);
  const T* xp = static_cast<const T*>(x);
  const T* wp = static_cast<const T*>(w);
  T* yp = static_cast<T*>(y);
  SN_LAUNCH((fc_mfma_kernel<T, 1, 4>), grid, block, 0, st, xp, n, cin, cin_s, wp, c8, kp, bias, yp, kout_s, act);
}

void fc_mfma(int dtype, const void* x, int n, int cin, int cin_s, const void* w, int c8, const float* bias,
             void* y, int kout, int kout_s, int act, hipStream_t st) {
  check(fc_mfma_applicable(dtype, n, cin, cin_s), "FC on MFMA: 16-bit types, batch <= 64, C % 8 == 0");
  if (dtype == 1) fc_mfma_t<f16>(x, n, cin, cin_s, w, c8, bias, y, kout, kout_s, act, st);
  else fc_mfma_t<bf16>(x, n, cin, cin_s, w, c8, bias, y, kout, kout_s, act, st);
}

}  // namespace k
}  // namespace sn
