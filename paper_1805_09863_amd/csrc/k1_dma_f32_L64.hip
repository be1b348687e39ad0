// Instantiations of the DMA-pipelined float32 projection kernel, layout L64.
#include "k1_dma.hpp"

namespace kb {
hipError_t launch_k1_dma_f32_L64(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_dma_layout<LayL64, true>(kc, grid, a, st);
}
}  // namespace kb
