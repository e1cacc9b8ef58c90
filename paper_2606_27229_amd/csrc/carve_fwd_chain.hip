// carve_fwd_chain.hip -- variant dispatch and LDS sizing of the chain forward
// (the kernels are in carve_fwd_chain.h, instantiated per variant in
// carve_variant.hip).
#include "carve_kernels.h"

namespace carve {

int launch_chain_fwd(const FwdArgs& a, int dtype, int D, int WB, int var, hipStream_t s) {
  switch (var) {
    case 0: return launch_chain_fwd_var<0>(a, dtype, D, WB, s);
    case kVarGated: return launch_chain_fwd_var<kVarGated>(a, dtype, D, WB, s);
    case kVarScalarW: return launch_chain_fwd_var<kVarScalarW>(a, dtype, D, WB, s);
    case kVarGated | kVarScalarW: return launch_chain_fwd_var<kVarGated | kVarScalarW>(a, dtype, D, WB, s);
    case kVarAct: return launch_chain_fwd_var<kVarAct>(a, dtype, D, WB, s);
    default: return CARVE_ERR_UNSUPPORTED;
  }
}

template <typename T, int D, int RP>
static size_t chain_lds_w(int WB) {
  if (WB == 16) return chain_lds<T, D, 16, RP, 0>().total;
  if (WB == 32) return chain_lds<T, D, 32, RP, 0>().total;
  if (WB == 64) return chain_lds<T, D, 64, RP, 0>().total;
  return (size_t)-1;
}

template <typename T>
static size_t chain_lds_d(int D, int WB, int RP) {
  if (RP == 32) {
    if (D == 32) return chain_lds_w<T, 32, 32>(WB);
    if (D == 64) return chain_lds_w<T, 64, 32>(WB);
    if (D == 128) return chain_lds_w<T, 128, 32>(WB);
  } else if (RP == 64) {
    if (D == 32) return chain_lds_w<T, 32, 64>(WB);
    if (D == 64) return chain_lds_w<T, 64, 64>(WB);
    if (D == 128) return chain_lds_w<T, 128, 64>(WB);
  }
  return (size_t)-1;
}

size_t chain_lds_bytes(int dtype, int D, int WB, int RP) {
  return dtype == CARVE_BF16 ? chain_lds_d<bf16_t>(D, WB, RP) : chain_lds_d<float>(D, WB, RP);
}

}  // namespace carve
