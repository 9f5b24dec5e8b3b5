// Kernel instances of F(4^3, 3^3) (k_input_split, k_gemm_inv).
#include "launch.hpp"

namespace wino {

WINO_DEFINE_OPS(3, 4, 3)

}  // namespace wino
