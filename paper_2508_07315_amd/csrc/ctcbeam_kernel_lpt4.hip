// Instantiation unit: decode kernels for up to 2048 tokens (4 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt4(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<4, false>(p, s); }
}  // namespace ctcbeam
