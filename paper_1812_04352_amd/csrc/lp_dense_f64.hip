// Dense VALU kernels instantiated for double (widths 8, 16, 32).
#include "lp_dense_impl.h"

LP_DENSE_DEFINE(double, f64, false)
