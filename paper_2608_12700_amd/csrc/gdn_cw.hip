// Instantiates the channel-wise kernels (fp32 operands) for every supported
// (d_k, d_v).
#include "gdn_cw.hpp"
namespace gdn {

hipError_t launch_cw_fwd(const CwFwdArgs& a) {
  const int dk = a.dk, dv = a.dv;
  if (dk == 64 && dv == 64) return launch_cw_fwd_t<64, 64>(a);
  if (dk == 64 && dv == 128) return launch_cw_fwd_t<64, 128>(a);
  if (dk == 64 && dv == 256) return launch_cw_fwd_t<64, 256>(a);
  if (dk == 128 && dv == 64) return launch_cw_fwd_t<128, 64>(a);
  if (dk == 128 && dv == 128) return launch_cw_fwd_t<128, 128>(a);
  if (dk == 128 && dv == 256) return launch_cw_fwd_t<128, 256>(a);
  return hipErrorInvalidValue;
}

hipError_t launch_cw_bwd(const CwBwdArgs& a) {
  const int dk = a.dk, dv = a.dv;
  if (dk == 64 && dv == 64) return launch_cw_bwd_t<64, 64>(a);
  if (dk == 64 && dv == 128) return launch_cw_bwd_t<64, 128>(a);
  if (dk == 64 && dv == 256) return launch_cw_bwd_t<64, 256>(a);
  if (dk == 128 && dv == 64) return launch_cw_bwd_t<128, 64>(a);
  if (dk == 128 && dv == 128) return launch_cw_bwd_t<128, 128>(a);
  if (dk == 128 && dv == 256) return launch_cw_bwd_t<128, 256>(a);
  return hipErrorInvalidValue;
}

}  // namespace gdn
