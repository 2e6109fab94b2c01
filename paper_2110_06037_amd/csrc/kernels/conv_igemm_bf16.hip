// The bf16 instantiations of the implicit-GEMM convolution routines (the
// kernels and their dispatch live in igemm.hpp).
#include "igemm.hpp"

namespace sn {
namespace k {

void conv_igemm_bf16(int param, const ConvArgs& c, hipStream_t st) { igemm_dispatch<bf16>(2, param, c, st); }

}  // namespace k
}  // namespace sn
