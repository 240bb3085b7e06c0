// The empty kernel: the launch-cost yardstick (no arguments, no work).
#include <hip/hip_runtime.h>

namespace tri {

__global__ void k_empty() {}

const void *empty_kernel() { return reinterpret_cast<const void *>(&k_empty); }

}  // namespace tri
