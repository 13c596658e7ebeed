// Instantiation unit: repeat-scoring decode kernels (CTCBEAM_FLAG_REPEAT_SCORE)
// for up to 2048 tokens (4 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt4_rep(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<4, true>(p, s); }
}  // namespace ctcbeam
