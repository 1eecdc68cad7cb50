// Instantiates the backward kernels for bf16 operands, variant VAR_GATED.
#include "gdn_bwd.hpp"
namespace gdn {
template hipError_t launch_bwd_var<DT_BF16, VAR_GATED>(const BwdArgs&);
}
