// Instantiation unit: greedy decode kernels for up to 4096 tokens (4 wave(s) of
// 16 labels per thread).
#include "ctcbeam_greedy.inl"

namespace ctcbeam {
hipError_t launch_greedy_v4096(const KernelParams& p, hipStream_t s) { return greedy::launch_greedy_impl<4, 16>(p, s); }
}  // namespace ctcbeam
