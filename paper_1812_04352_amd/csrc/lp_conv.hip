// 3x3 convolution layers (placeholder until the conv kernels land).
#include "lp_internal.h"

namespace lp {
bool conv_supported(const Shape&) { return false; }
int conv_grad_chunks(int, int) { return 1; }
int conv_tile(const Shape&) { return 1; }
hipError_t conv_sweep(const Shape&, int, const SweepArgs&, hipStream_t, int*) { return hipErrorNotSupported; }
hipError_t conv_serial(const Shape&, int, const SerialArgs&, hipStream_t) { return hipErrorNotSupported; }
hipError_t conv_resid(const Shape&, int, const ResidArgs&, hipStream_t, int*) { return hipErrorNotSupported; }
hipError_t conv_grad(const Shape&, const GradArgs&, hipStream_t) { return hipErrorNotSupported; }
}  // namespace lp
