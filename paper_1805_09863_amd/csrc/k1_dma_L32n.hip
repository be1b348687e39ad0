// Instantiations of the DMA-pipelined bf16 projection kernel, 32-row layouts
// with 256- and 128-word tiles.
#include "k1_dma.hpp"

namespace kb {
hipError_t launch_k1_dma_L32M(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_dma_layout<LayL32M>(kc, grid, a, st);
}
hipError_t launch_k1_dma_L32S(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_dma_layout<LayL32S>(kc, grid, a, st);
}
}  // namespace kb
