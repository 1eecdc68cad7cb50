// Instantiates the forward kernels for float operands, variant VAR_DECAY.
#include "gdn_fwd.hpp"
namespace gdn {
template hipError_t launch_fwd_var<DT_F32, VAR_DECAY>(const FwdArgs&);
}
