// Forward-kernel instantiations and dispatch for bf16 storage in the
// channel-major layout (X / grad_x [T, batch, C, P, S]).
// V: bit 0 = Mexican-hat activation, bit 1 = residual dendrite, bits 2-3 =
// log2(KC), bit 4 = channel-major.
#include "dendsn_kernels.h"

namespace dendsn {

template <int BL, int L, int KC>
static hipError_t launch_fwd_cm_v(const dim3& grid, const FwdArgs& fa, int v, size_t lds, hipStream_t stream) {
  constexpr int VK = 16 | ((KC == 1 ? 0 : (KC == 2 ? 1 : 2)) << 2);
  switch (v & 3) {
    case 0: dendsn_fwd_kernel<bf16_t, BL, L, VK | 0><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    case 1: dendsn_fwd_kernel<bf16_t, BL, L, VK | 1><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    case 2: dendsn_fwd_kernel<bf16_t, BL, L, VK | 2><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
    case 3: dendsn_fwd_kernel<bf16_t, BL, L, VK | 3><<<grid, dim3(kThreads), lds, stream>>>(fa); break;
  }
  return hipGetLastError();
}

hipError_t launch_fwd_bf16_cm(const Plan& pl, const FwdArgs& fa, int v, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>(pl.ntiles * pl.G));
  if (!pl.cm) return hipErrorInvalidValue;
#define DENDSN_CASE(BL_, L_, KC_) \
  if (pl.BL == BL_ && pl.L == L_ && pl.KC == KC_) return launch_fwd_cm_v<BL_, L_, KC_>(grid, fa, v, size_t(pl.lds), stream);
  DENDSN_CM_FWD(DENDSN_CASE)
#undef DENDSN_CASE
  return hipErrorInvalidValue;
}

}  // namespace dendsn
