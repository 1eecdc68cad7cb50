// Instantiates the forward kernels for bf16 operands, variant VAR_DELTA.
#include "gdn_fwd.hpp"
namespace gdn {
template hipError_t launch_fwd_var<DT_BF16, VAR_DELTA>(const FwdArgs&);
}
