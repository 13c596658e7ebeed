// Instantiation unit: greedy decode kernels for up to 256 tokens (4 label(s) per lane).
#include "ctcbeam_greedy.inl"

namespace ctcbeam {
hipError_t launch_greedy_nj4(const KernelParams& p, hipStream_t s) { return greedy::launch_greedy_impl<4>(p, s); }
}  // namespace ctcbeam
