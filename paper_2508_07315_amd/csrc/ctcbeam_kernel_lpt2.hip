// Instantiation unit: decode kernels for up to 1024 tokens (2 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt2(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<2, false>(p, s); }
}  // namespace ctcbeam
