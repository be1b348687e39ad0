// Instantiations of the register-staged projection kernel: f32 operands,
// 32-row layouts with 256- and 128-word tiles.
#include "k1_fused.hpp"

namespace kb {
hipError_t launch_k1_reg_f32_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_reg<false, LayL32M>(kc, grid, a, st);
}
hipError_t launch_k1_reg_f32_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_reg<false, LayL32S>(kc, grid, a, st);
}
}  // namespace kb
