// Instantiation unit: greedy decode kernels for up to 1024 tokens (one wave
// of 16 labels per thread: four waves with their per-frame exchange measured
// slower at this size).
#include "ctcbeam_greedy.inl"

namespace ctcbeam {
hipError_t launch_greedy_v1024(const KernelParams& p, hipStream_t s) { return greedy::launch_greedy_impl<1, 16>(p, s); }
}  // namespace ctcbeam
