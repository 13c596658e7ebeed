// Instantiation unit: greedy decode kernels for up to 4096 tokens (64 label(s) per lane).
#include "ctcbeam_greedy.inl"

namespace ctcbeam {
hipError_t launch_greedy_nj64(const KernelParams& p, hipStream_t s) { return greedy::launch_greedy_impl<64>(p, s); }
}  // namespace ctcbeam
