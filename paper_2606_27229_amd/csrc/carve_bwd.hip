// carve_bwd.hip -- chunked CARVE backward on gfx950 (placeholder until the
// reverse chain lands).
#include "carve_kernels.h"

namespace carve {

int launch_bwd(const BwdArgs& a, int dtype, int D, int LW, hipStream_t s) {
  (void)a; (void)dtype; (void)D; (void)LW; (void)s;
  return CARVE_ERR_UNSUPPORTED;
}

size_t bwd_lds_bytes(int dtype, int D, int LW, int RP) {
  (void)dtype; (void)D; (void)LW; (void)RP;
  return 0;
}

int launch_param_reduce(const float* part, int nparts, int R, int D, float* dUb, float* dUw,
                        float* dVb, float* dVw, hipStream_t s) {
  (void)part; (void)nparts; (void)R; (void)D; (void)dUb; (void)dUw; (void)dVb; (void)dVw; (void)s;
  return CARVE_ERR_UNSUPPORTED;
}

}  // namespace carve
