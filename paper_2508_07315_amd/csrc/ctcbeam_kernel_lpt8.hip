// Instantiation unit: decode kernels for up to 4096 tokens (8 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt8(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<8, false>(p, s); }
}  // namespace ctcbeam
