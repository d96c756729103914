// Linear-prior FEM read (chunked scan) -- placeholder until the scan kernels land.
#include "fem_internal.h"

namespace fem {
hipError_t launch_linear_bf16(const void*, const void*, const void*, const float*, float*, int,
                              int, int, int, int, int, hipStream_t) {
  return hipErrorNotSupported;
}
}  // namespace fem
