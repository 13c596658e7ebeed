// ctcbeam_decode_noalloc: ctcbeam_decode_ex for callers that cannot allocate
// device memory (code under stream capture, tight serving loops, harnesses
// that forbid allocation).  The workspace of the decode kernels (the header,
// the status words and the back-pointers [B, T, K]) lives in a fixed device
// array instead of a caller buffer; the caller still passes inputs and
// outputs.
//
// Each device that runs the library holds its own copy of the array until
// the process ends.  Host code never uses the array's name as an address:
// the device address is looked up once per device with hipGetSymbolAddress
// (with that device current) and kept.  Every call on a device shares that
// device's array, so calls that overlap on one device race; the kernels
// write every word of the workspace they later read, so nothing needs
// clearing between calls.
#include <mutex>
#include <string>

#include "../../include/ctcbeam.h"
#include "ctcbeam_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t(16) << 20;  // CTCBEAM_NOALLOC_MAX_WORKSPACE
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of the array (looked up on the first
// call on the device, with the device current).
int scratch_for_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return ctcbeam::set_last_error(4, "no HIP device");
  if (dev >= kMaxDevices) return ctcbeam::set_last_error(2, "device index above the supported count");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return ctcbeam::set_last_error(4, (std::string("scratch address: ") + hipGetErrorString(e)).c_str());
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return 0;
}

}  // namespace

static_assert(kScratchBytes == CTCBEAM_NOALLOC_MAX_WORKSPACE, "scratch size");

extern "C" int ctcbeam_decode_noalloc(const float* logprobs, const int32_t* lengths, int B, int T, int V,
                                      int K, float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                                      const ctcbeam_boost* boost, int32_t* out_tokens, int32_t* out_lengths,
                                      float* out_scores, hipStream_t stream, const ctcbeam_opts* opts) {
  if (B < 0 || T < 0 || K < 1) return ctcbeam::set_last_error(1, "B and T must be >= 0, K >= 1");
  const size_t need = ctcbeam_workspace_bytes(B, T, K);
  if (need > kScratchBytes)
    return ctcbeam::set_last_error(
        2, ("workspace of " + std::to_string(need) + " bytes above the no-allocation limit of " +
            std::to_string(kScratchBytes))
               .c_str());
  void* ws = nullptr;
  if (const int rc = scratch_for_current_device(&ws)) return rc;
  return ctcbeam::decode_with_workspace(logprobs, lengths, B, T, V, K, alpha, beta, boost_w, lm, boost, ws,
                                        kScratchBytes, out_tokens, out_lengths, out_scores, stream, opts);
}
