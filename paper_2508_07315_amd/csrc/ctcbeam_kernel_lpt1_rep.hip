// Instantiation unit: repeat-scoring decode kernels (CTCBEAM_FLAG_REPEAT_SCORE)
// for up to 512 tokens (1 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt1_rep(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<1, true>(p, s); }
}  // namespace ctcbeam
