// Kernel instances of the 2-D size F(3,6) of Table 1 (k_input, k_gemm_inv).
#include "launch.hpp"

namespace wino {

WINO_DEFINE_OPS(2, 3, 6)

}  // namespace wino
