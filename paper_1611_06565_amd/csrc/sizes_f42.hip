// Kernel instances of F(4^2, 3^2) (k_input, k_gemm_acc4, k_part_reduce).
#include "launch.hpp"

namespace wino {

WINO_DEFINE_OPS(2, 4, 3)

}  // namespace wino
