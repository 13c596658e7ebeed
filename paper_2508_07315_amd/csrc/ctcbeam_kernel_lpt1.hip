// Instantiation unit: decode kernels for up to 512 tokens (1 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt1(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<1, false>(p, s); }
}  // namespace ctcbeam
