// Register Sinkhorn kernel with 2 waves per multi-wave problem and 8 waves
// per workgroup (its own translation unit, so the register kernels compile in
// parallel).
#include "sk_register.h"

namespace taot {

taot_status launch_reg_w2g8(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                            hipStream_t stream) {
  return launch_reg_kernel<2, 8>(p, multi, single, counts, stream);
}

}  // namespace taot
