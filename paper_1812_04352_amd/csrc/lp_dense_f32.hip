// Dense VALU kernels instantiated for float (widths 8, 16, 32, 64).
#include "lp_dense_impl.h"

LP_DENSE_DEFINE(float, f32, true)
