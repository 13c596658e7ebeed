// Internal layouts shared by the host builders and the gfx950 kernel.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

struct ctcbeam_lm;
struct ctcbeam_boost;
struct ctcbeam_opts;

namespace ctcbeam {

constexpr int kThreads = 512;         // threads per workgroup (8 wave64)
constexpr int kWaves = kThreads / 64;
constexpr int kMaxK = 128;            // beam size limit
constexpr int kMaxKWideV = 64;        // beam size limit above 1024 tokens
constexpr int kLmStage = 4096;        // staged LM arcs per chunk (12-bit slot)
constexpr int kCap = 512;             // survivor pool entries
constexpr uint32_t kExists = 0x80000000u;
constexpr int kFlagLogSumExp = 1;      // recombination by log-sum-exp
constexpr int kFlagBoostRollback = 2;  // pending boosting taken back at the end
constexpr int kFlagNoRowCache = 4;     // LM key rows refilled for every beam every frame
constexpr int kFlagRepeatScore = 8;    // repeated tokens get their LM / boosting terms again
// Workspace: [header, kWsHeaderBytes][status word per utterance, padded to
// 256 B][back-pointers [B, T, K] int32].  The header records the batch size
// of the last decode that used the workspace, so that its status can be read
// back from the workspace alone: {kWsMagic, B, ~B}.
constexpr size_t kWsHeaderBytes = 256;
constexpr uint32_t kWsMagic = 0x42435443u;  // "CTCB"

// LM state record, one per chain level l (context of length l+1):
//   {arc_begin, arc_count | kExists, backoff bits}
// Per-phase clocks of the kernels in profiling builds (-DCTCBEAM_PHASE_CLOCKS):
// a kernel declares uint64_t ph_acc (lane k of each wave holds word k) and
// ph_t0; each CTCBEAM_PHASE_MARK(k) adds the s_memtime cycles since the
// previous mark to word k, CTCBEAM_PHASE_COUNT(k) adds one.  One register
// pair per wave keeps the profiling build's register use close to the
// product's.  Product builds compile none of it.
constexpr int kPhaseWords = 20;
#ifdef CTCBEAM_PHASE_CLOCKS
#define CTCBEAM_PHASE_MARK(k)                                          \
  do {                                                                 \
    const uint64_t now_ = __builtin_amdgcn_s_memtime();                \
    ph_acc += ((threadIdx.x & 63u) == (k)) ? now_ - ph_t0 : 0ull;      \
    ph_t0 = now_;                                                      \
  } while (0)
#define CTCBEAM_PHASE_COUNT(k)                                 \
  do {                                                         \
    ph_acc += ((threadIdx.x & 63u) == (k)) ? 1ull : 0ull;      \
  } while (0)
#else
#define CTCBEAM_PHASE_MARK(k) \
  do {                        \
  } while (0)
#define CTCBEAM_PHASE_COUNT(k) \
  do {                         \
  } while (0)
#endif

struct LmLevel {
  uint32_t begin;
  uint32_t count;   // low 31 bits: arcs; bit 31: the context is an entry
  float bo;
};
// LM arc: ln probability of (context, token), next state after emitting token
struct LmArc {
  float logp;
  uint32_t target;
  uint32_t token;
};
// Boosting tree state record.
struct BtNode {
  uint32_t list_begin;
  uint32_t list_count;
  uint32_t pot;        // low 8 bits: pot; bits 8..31: chain nodes (statistics)
  uint32_t chain_arcs; // statistics only
};
struct BtEntry {
  uint32_t token;
  uint32_t key;        // (prio << 26) | (pre << 20) | child
};
constexpr uint32_t kBtChildMask = (1u << 20) - 1;

struct KernelParams {
  const float* logprobs;
  const int32_t* lengths;
  int B, T, V, K;
  float alpha, beta, boost_w, theta;
  int flags;                 // kFlag* bits
  // LM (null when disabled)
  const LmLevel* lm_states;
  const LmArc* lm_arcs;
  const float* lm_unigram;   // [V+1], index V = </s>
  int lm_nlev;
  uint32_t lm_bos_state;
  int lm_states_below_2p23;  // every LM state id fits 23 bits
  int64_t lm_n_states;       // number of LM states
  // boosting (null when disabled)
  const BtNode* bt_nodes;
  const BtEntry* bt_list;
  const uint32_t* bt_root_key;  // [V]
  // workspace / outputs
  uint32_t* ws_header;       // workspace header (written by workgroup 0)
  uint32_t* status;          // [B]
  int32_t* bp;               // [B, T, K]
  int32_t* out_tokens;       // [B, T] or null (then no 1-best output)
  int32_t* out_lengths;      // [B] or null
  float* out_scores;         // [B] or null
  int64_t* stats;            // [B, 8] or null
  // N-best output (nbest_scores null: none; nbest_tokens may be null when
  // T = 0): every slot's final hypothesis ordered by
  // final score, lowest slot on ties; dead slots last, empty, -inf
  int32_t* nbest_tokens;     // [B, K, T]
  int32_t* nbest_lengths;    // [B, K]
  float* nbest_scores;       // [B, K]
};

// Record the batch size in the workspace header (one thread of one workgroup).
__device__ __forceinline__ void write_ws_header(uint32_t* hdr, int B) {
  hdr[0] = kWsMagic;
  hdr[1] = static_cast<uint32_t>(B);
  hdr[2] = ~static_cast<uint32_t>(B);
}

// Kernel variants by labels per lane (V <= 512 * LPT); each dispatches on the
// LM order and on boosting.  Return the launch's hipError_t.
hipError_t launch_lpt1(const KernelParams& p, hipStream_t stream);
hipError_t launch_lpt2(const KernelParams& p, hipStream_t stream);
hipError_t launch_lpt4(const KernelParams& p, hipStream_t stream);
hipError_t launch_lpt8(const KernelParams& p, hipStream_t stream);
// the same for the repeat-scoring variant (CTCBEAM_FLAG_REPEAT_SCORE with an
// LM or boosting)
hipError_t launch_lpt1_rep(const KernelParams& p, hipStream_t stream);
hipError_t launch_lpt2_rep(const KernelParams& p, hipStream_t stream);
hipError_t launch_lpt4_rep(const KernelParams& p, hipStream_t stream);
hipError_t launch_lpt8_rep(const KernelParams& p, hipStream_t stream);

// Greedy (one hypothesis) kernels by vocabulary: up to 256 tokens (one wave
// per utterance), 1024 and 4096 tokens (four waves).
hipError_t launch_greedy_v256(const KernelParams& p, hipStream_t stream);
hipError_t launch_greedy_v1024(const KernelParams& p, hipStream_t stream);
hipError_t launch_greedy_v4096(const KernelParams& p, hipStream_t stream);

// Writes the header of an empty batch (B = 0: no decode kernel runs).
hipError_t launch_ws_header(uint32_t* hdr, int B, hipStream_t stream);

inline hipError_t launch_greedy(const KernelParams& p, hipStream_t stream) {
  if (p.B == 0) return hipSuccess;
  if (p.V <= 256) return launch_greedy_v256(p, stream);
  if (p.V <= 1024) return launch_greedy_v1024(p, stream);
  return launch_greedy_v4096(p, stream);
}

// The 1-best decode of ctcbeam_decode_ex into a given workspace (host side,
// ctcbeam_host.cpp): validation, parameter block, launch; the C entry
// points' return codes.  set_last_error records the message that
// ctcbeam_last_error returns and passes the code through.
int decode_with_workspace(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K,
                          float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                          const ctcbeam_boost* boost, void* workspace, size_t workspace_bytes,
                          int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                          hipStream_t stream, const ctcbeam_opts* opts);
int set_last_error(int code, const char* msg);

// Small-beam decoder (ctcbeam_small.inl): beams of at most 8, at most 1024
// tokens, no LM and no boosting, max recombination.
bool small_beam_eligible(const KernelParams& p);
hipError_t launch_small(const KernelParams& p, hipStream_t stream);

inline hipError_t launch_decode(const KernelParams& p, hipStream_t stream) {
  if (p.B == 0) return hipSuccess;
  if (small_beam_eligible(p)) return launch_small(p, stream);
  // repeat scoring changes nothing without an LM or boosting
  if ((p.flags & kFlagRepeatScore) && (p.lm_states != nullptr || p.lm_arcs != nullptr || p.bt_nodes != nullptr)) {
    if (p.V <= 512) return launch_lpt1_rep(p, stream);
    if (p.V <= 1024) return launch_lpt2_rep(p, stream);
    if (p.V <= 2048) return launch_lpt4_rep(p, stream);
    return launch_lpt8_rep(p, stream);
  }
  if (p.V <= 512) return launch_lpt1(p, stream);
  if (p.V <= 1024) return launch_lpt2(p, stream);
  if (p.V <= 2048) return launch_lpt4(p, stream);
  return launch_lpt8(p, stream);
}

}  // namespace ctcbeam
