// Backward kernels (placeholder until the backward sweep lands).
#include "flex_common.hpp"
#include "flex_kernels.hpp"

namespace flex {

size_t bwd_state_floats(const KernelShape& ks) { return fwd_state_floats(ks); }
size_t bwd_dw_floats(const KernelShape& ks) { return (size_t)(ks.nonstationary ? 2 : 1) * ks.m * ks.d; }
hipError_t launch_bwd(const BwdArgs&, const KernelShape&, hipStream_t) { return hipErrorNotSupported; }

}  // namespace flex
