// Instantiation unit: greedy decode kernels for up to 1024 tokens (16 label(s) per lane).
#include "ctcbeam_greedy.inl"

namespace ctcbeam {
hipError_t launch_greedy_nj16(const KernelParams& p, hipStream_t s) { return greedy::launch_greedy_impl<16>(p, s); }
}  // namespace ctcbeam
