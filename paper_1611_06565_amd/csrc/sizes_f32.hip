// Kernel instances of F(3,2) of Table 1 in 2-D and 3-D (k_input, k_gemm_inv).
#include "launch.hpp"

namespace wino {

WINO_DEFINE_OPS(2, 3, 2)
WINO_DEFINE_OPS(3, 3, 2)

}  // namespace wino
