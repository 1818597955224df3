// Register Sinkhorn kernel with 4 waves per multi-wave problem and 4 waves
// per workgroup (its own translation unit, so the register kernels compile in
// parallel).
#include "sk_register.h"

namespace taot {

taot_status launch_reg_w4g4(const SkParams& p, const int32_t* multi, const int32_t* single, const int32_t* counts,
                            hipStream_t stream) {
  return launch_reg_kernel<4, 4>(p, multi, single, counts, stream);
}

}  // namespace taot
