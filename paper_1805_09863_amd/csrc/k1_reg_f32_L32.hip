// Instantiations of the register-staged projection kernel: f32 operands, layout L32.
#include "k1_fused.hpp"

namespace kb {
hipError_t launch_k1_reg_f32_L32(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_reg<false, LayL32>(kc, grid, a, st);
}
}  // namespace kb
