// Instantiates the backward kernels for f32 operands, variant VAR_DECAY.
#include "gdn_bwd.hpp"
namespace gdn {
template hipError_t launch_bwd_var<DT_F32, VAR_DECAY>(const BwdArgs&);
}
