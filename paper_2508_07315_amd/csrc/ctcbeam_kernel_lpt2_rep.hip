// Instantiation unit: repeat-scoring decode kernels (CTCBEAM_FLAG_REPEAT_SCORE)
// for up to 1024 tokens (2 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt2_rep(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<2, true>(p, s); }
}  // namespace ctcbeam
