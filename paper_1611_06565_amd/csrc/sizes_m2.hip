// Kernel instances of F(2^N, 3^N) in 2-D and 3-D (m = 2: k_input, k_gemm_acc, k_part_reduce).
#include "launch.hpp"

namespace wino {

WINO_DEFINE_OPS(2, 2, 3)
WINO_DEFINE_OPS(3, 2, 3)

}  // namespace wino
