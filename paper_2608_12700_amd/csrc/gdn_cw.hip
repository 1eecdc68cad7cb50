// Instantiates the channel-wise kernels for every supported (d_k, d_v) and
// activation type.
#include "gdn_cw.hpp"
namespace gdn {

template <typename IO>
static hipError_t cw_fwd_io(const CwFwdArgs& a) {
  const int dk = a.dk, dv = a.dv;
  if (dk == 64 && dv == 64) return launch_cw_fwd_t<64, 64, IO>(a);
  if (dk == 64 && dv == 128) return launch_cw_fwd_t<64, 128, IO>(a);
  if (dk == 64 && dv == 256) return launch_cw_fwd_t<64, 256, IO>(a);
  if (dk == 128 && dv == 64) return launch_cw_fwd_t<128, 64, IO>(a);
  if (dk == 128 && dv == 128) return launch_cw_fwd_t<128, 128, IO>(a);
  if (dk == 128 && dv == 256) return launch_cw_fwd_t<128, 256, IO>(a);
  return hipErrorInvalidValue;
}

template <typename IO>
static hipError_t cw_bwd_io(const CwBwdArgs& a) {
  const int dk = a.dk, dv = a.dv;
  if (dk == 64 && dv == 64) return launch_cw_bwd_t<64, 64, IO>(a);
  if (dk == 64 && dv == 128) return launch_cw_bwd_t<64, 128, IO>(a);
  if (dk == 64 && dv == 256) return launch_cw_bwd_t<64, 256, IO>(a);
  if (dk == 128 && dv == 64) return launch_cw_bwd_t<128, 64, IO>(a);
  if (dk == 128 && dv == 128) return launch_cw_bwd_t<128, 128, IO>(a);
  if (dk == 128 && dv == 256) return launch_cw_bwd_t<128, 256, IO>(a);
  return hipErrorInvalidValue;
}

hipError_t launch_cw_fwd(const CwFwdArgs& a) { return a.io == DT_BF16 ? cw_fwd_io<bf16>(a) : cw_fwd_io<float>(a); }
hipError_t launch_cw_bwd(const CwBwdArgs& a) { return a.io == DT_BF16 ? cw_bwd_io<bf16>(a) : cw_bwd_io<float>(a); }

}  // namespace gdn
