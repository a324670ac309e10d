// Backward-kernel instantiations and dispatch for f32 storage.
#include "dendsn_kernels.h"

namespace dendsn {

template <int BL, int L, int KS>
static hipError_t launch_bwd_ks(const dim3& grid, const BwdArgs& ba, int psi, hipStream_t stream) {
  if (psi)
    dendsn_bwd_kernel<float, BL, L, 1, KS><<<grid, dim3(kThreads), 0, stream>>>(ba);
  else
    dendsn_bwd_kernel<float, BL, L, 0, KS><<<grid, dim3(kThreads), 0, stream>>>(ba);
  return hipGetLastError();
}

hipError_t launch_bwd_f32(const Plan& pl, const BwdArgs& ba, int psi, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
#define DENDSN_FAST_CASE(BL_, L_)                                                   \
  if (pl.BL == BL_ && pl.L == L_ && pl.fast) {                                      \
    if (pl.KS == 4) return launch_bwd_ks<BL_, L_, 4>(grid, ba, psi, stream);        \
    if constexpr (BL_ <= 4)                                                         \
      if (pl.KS == 8) return launch_bwd_ks<BL_, L_, 8>(grid, ba, psi, stream);      \
    return hipErrorInvalidValue;                                                    \
  }
#define DENDSN_GENERIC_CASE(BL_, L_)                                                \
  if (pl.BL == BL_ && pl.L == L_ && !pl.fast && pl.KS == DENDSN_GENERIC_KS)         \
    return launch_bwd_ks<BL_, L_, DENDSN_GENERIC_KS>(grid, ba, psi, stream);
  DENDSN_FAST_F32(DENDSN_FAST_CASE)
  DENDSN_BWD_HALF(DENDSN_FAST_CASE)
  DENDSN_GENERIC(DENDSN_GENERIC_CASE)
#undef DENDSN_FAST_CASE
#undef DENDSN_GENERIC_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
