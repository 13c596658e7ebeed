// Instantiation unit: greedy decode kernels for up to 256 tokens (1 wave(s) of
// 4 labels per thread).
#include "ctcbeam_greedy.inl"

namespace ctcbeam {
hipError_t launch_greedy_v256(const KernelParams& p, hipStream_t s) { return greedy::launch_greedy_impl<1, 4>(p, s); }
}  // namespace ctcbeam
