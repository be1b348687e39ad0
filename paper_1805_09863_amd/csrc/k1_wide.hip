// Instantiations of the wide (256 x 256 tile) bf16 projection kernel.
#include "k1_wide.hpp"

namespace kb {
hipError_t launch_k1_wide(int kc, dim3 grid, const K1Args& a, hipStream_t st) {
  if (a.no_stats) return kc == 4 ? launch_k1_wide_kc<4, kWideArgmax>(grid, a, st) : hipErrorInvalidValue;
  switch (kc) {
    case 4: return launch_k1_wide_kc<4>(grid, a, st);
    case 8: return launch_k1_wide_kc<8>(grid, a, st);
    case 12: return launch_k1_wide_kc<12>(grid, a, st);
    case 16: return launch_k1_wide_kc<16>(grid, a, st);
    default: return hipErrorInvalidValue;
  }
}


// The plain projection of the unfused baseline: p = W h stored to a.logits.
hipError_t launch_k1_wide_store(dim3 grid, const K1Args& a, hipStream_t st) {
  return launch_k1_wide_kc<4, kWideStore>(grid, a, st);
}
}  // namespace kb
