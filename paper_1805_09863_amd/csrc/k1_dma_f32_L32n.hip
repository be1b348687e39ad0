// Instantiations of the DMA-pipelined float32 projection kernel, 32-row
// layouts with 256- and 128-word tiles.
#include "k1_dma.hpp"

namespace kb {
hipError_t launch_k1_dma_f32_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_dma_layout<LayL32M, true>(kc, grid, a, st);
}
hipError_t launch_k1_dma_f32_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_dma_layout<LayL32S, true>(kc, grid, a, st);
}
}  // namespace kb
