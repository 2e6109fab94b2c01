// Fused Winograd F(2x2, 3x3) routines (wino_fused.hip): the input
// transform, the 16 tile GEMMs on MFMA and the output transform in one
// kernel, with nothing but the input, the transformed filters and the output
// in memory.
#pragma once

#include "launch.hpp"

namespace sn {
namespace k {

// Tile configurations (waves per workgroup NW: 16 output tiles each; FN
// blocks of 16 output channels per wave).  Routine parameter p of the fused
// Winograd routine runs configuration p.
#define WINO_CONFIGS(X) \
  X(4, 4)               \
  X(4, 2)               \
  X(2, 4)               \
  X(2, 2)
int wino_fused_num_configs();
// 16-bit, 3x3 stride 1 pad 1, channels in steps of 32 (NHWC with C % 32 == 0,
// or NC8HW8 with C rounded to 8 a multiple of 32)
bool wino_fused_applicable(int dtype, int layout, int c);
// a.w: transformed filters U [16][Kp][C8] in the dtype
void conv_wino_fused(int dtype, int cfg, const ConvArgs& a, hipStream_t st);

}  // namespace k
}  // namespace sn
