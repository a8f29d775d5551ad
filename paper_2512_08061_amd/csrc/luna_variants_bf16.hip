// luna_variants_bf16.hip -- the feature-map variant kernels of bf16 inputs, a
// translation unit of their own so that the two input types compile in parallel.
#include "luna_variants.hpp"

namespace luna {

hipError_t variant_map_bf16(int d, const VariantArgs& a, int64_t items, int* grid, hipStream_t s) {
  return variant_dispatch_d<__bf16>(d, a, items, grid, s);
}

}  // namespace luna
