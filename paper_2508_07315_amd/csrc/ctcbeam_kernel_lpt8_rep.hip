// Instantiation unit: repeat-scoring decode kernels (CTCBEAM_FLAG_REPEAT_SCORE)
// for up to 4096 tokens (8 label(s) per lane).
#include "ctcbeam_decode.inl"

namespace ctcbeam {
hipError_t launch_lpt8_rep(const KernelParams& p, hipStream_t s) { return detail::launch_lpt_impl<8, true>(p, s); }
}  // namespace ctcbeam
