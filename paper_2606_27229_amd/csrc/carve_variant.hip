// carve_variant.hip -- the kernels of one layer variant (CARVE_VARIANT, a bit
// set of kVarGated, kVarScalarW, kVarAct): the chain forward and the fused chunk
// recompute + adjoint, for every supported dtype, head size, rank and block
// length.  The build compiles this file once per variant, so the variants
// compile in parallel.
#include "carve_bwd.h"
#include "carve_fwd_chain.h"

#ifndef CARVE_VARIANT
#error "compile with -DCARVE_VARIANT=<0..4> (one object per layer variant)"
#endif

namespace carve {
static_assert(var_built(CARVE_VARIANT), "layer variant not built");
template int launch_chain_fwd_var<CARVE_VARIANT>(const FwdArgs&, int, int, int, hipStream_t);
template int launch_bwd_fused_var<CARVE_VARIANT>(const FwdArgs&, const BwdArgs&, int*, int, int, int, int,
                                                 hipStream_t);
}  // namespace carve
