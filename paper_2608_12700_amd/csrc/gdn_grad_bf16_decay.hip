// Instantiates the bf16 chunk-gradient kernel, variant VAR_DECAY.  Its tile loop
// needs the loop-safe thread index (GDN_TILE_LOOP), so it has a translation
// unit of its own.
#define GDN_TILE_LOOP
#include "gdn_bwd.hpp"
namespace gdn {
template hipError_t launch_grad_bf<64, 64, VAR_DECAY>(const BwdArgs&);
template hipError_t launch_grad_bf<64, 128, VAR_DECAY>(const BwdArgs&);
template hipError_t launch_grad_bf<64, 256, VAR_DECAY>(const BwdArgs&);
template hipError_t launch_grad_bf<128, 64, VAR_DECAY>(const BwdArgs&);
template hipError_t launch_grad_bf<128, 128, VAR_DECAY>(const BwdArgs&);
template hipError_t launch_grad_bf<128, 256, VAR_DECAY>(const BwdArgs&);
}
