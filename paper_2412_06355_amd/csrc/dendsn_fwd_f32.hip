// Forward-kernel instantiations and dispatch for f32 storage.
#include "dendsn_kernels.h"

namespace dendsn {

hipError_t launch_fwd_f32(const Plan& pl, const FwdArgs& fa, int psi, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G)), block(kThreads);
#define DENDSN_CASE(BL_, L_)                                                        \
  if (pl.BL == BL_ && pl.L == L_) {                                                 \
    if (psi)                                                                        \
      dendsn_fwd_kernel<float, BL_, L_, 1><<<grid, block, 0, stream>>>(fa);          \
    else                                                                            \
      dendsn_fwd_kernel<float, BL_, L_, 0><<<grid, block, 0, stream>>>(fa);          \
    return hipGetLastError();                                                       \
  }
  DENDSN_FAST_F32(DENDSN_CASE)
  DENDSN_GENERIC(DENDSN_CASE)
#undef DENDSN_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
