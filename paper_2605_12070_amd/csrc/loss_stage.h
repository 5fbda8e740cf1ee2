// Internal interface between the C-ABI layer and the loss-stage kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "dppo.h"

namespace dppo {

constexpr int kModeLogprob = 0;  // log-prob (and lse) only
constexpr int kModeLoss = 1;     // decoupled PPO loss, optional dlogits

// Row-kernel policy (dppo_set_path_policy): bit 0 forces the streaming kernel; the ABI layer
// also reads bit 1 (counters by prep_stats and atomics only).
constexpr int kForceAuto = 0;
constexpr int kForceStream = 1;  // use the two-pass streaming kernel even when resident fits

// Arguments of every per-row kernel (passed by value).
struct RowArgs {
  const void* logits;   // row t at logits + t * ld (RowArgsV: unless a version table is set)
  int64_t ld;
  void* dlogits;        // NULL: forward only
  int64_t ldd;
  const int64_t* ids;
  const float* lp_mu;
  const float* lp_ref;
  const float* adv;
  const uint8_t* mask;  // NULL: all valid
  const float* tscale;  // NULL: all 1
  float* lp_out;
  float* loss_tok;
  uint8_t* flags;       // NULL: not written
  int32_t* stats;
  float* lse_out;       // log-prob mode only, may be NULL
  int32_t T;            // rows (persistent kernels loop over them)
  int32_t V;
  int32_t mode;
  float band_lo, band_hi;
  float clip_lo, clip_hi;  // 1 - eps_lo, 1 + eps_hi
  float loss_scale;
  int32_t rd_mode;
  int32_t scale_mode;
  int32_t ref_mode;     // dppo_ref_mode; lp_ref is NULL unless GIVEN
  float alpha;          // behaviour-policy weight of an interpolated reference
  int32_t stagger;      // persistent bf16 kernels: start delay per XCD-local workgroup index,
                        // in s_sleep(6) units (set by the launcher from RowLaunch)
  int32_t count_mode;   // 1 (persistent fp32 resident loss calls that write flags): no
                        // prep_stats; each workgroup counts the valid tokens itself for the
                        // token-mean scale (workgroup 0 stores the count), no counter
                        // atomics; loss_sum derives the counters from the flags
};

// Arguments of the kernels without the backward sweep: the row arguments plus an optional
// per-token version table (versioned log-prob call). The gradient kernels take RowArgs
// alone, so their argument block is not widened by a table they never read.
struct RowArgsV : RowArgs {
  const int32_t* version;                  // per-token policy version, or NULL
  int32_t nver;                            // number of versions (1..DPPO_MAX_VERSIONS)
  const void* vlogits[DPPO_MAX_VERSIONS];  // version v's logits; row t at vlogits[v] + t * ld
};

template <bool BWD>
using RowArgsOf = typename std::conditional<BWD, RowArgs, RowArgsV>::type;

struct RowLaunch {
  const void* fn = nullptr;  // kernel taking RowArgsOf<bwd>
  bool bwd = false;
  int threads = 0;
  int chunks = 0;            // resident kernels: 16-byte chunks per thread
  bool resident = false;
  bool persistent = false;  // grid = resident workgroups on the device, rows looped over
  bool two_buffers = false; // resident backward kernel with two row buffers
  bool prefix = false;       // backward kernel with a resident prefix and a streamed tail
  bool phase = false;        // bf16 resident kernel for rows with a phase (rows_bf16_*phase*)
  bool counts = false;       // the kernel supports count mode (RowArgs::count_mode)
  int fill = 27;             // persistent grids: workgroups launched per 32 resident slots
  int stagger = 2;           // RowArgs::stagger for the kernels that stagger their starts
};

constexpr int kPrefixNC = 19;  // resident 16-byte chunks per thread of the prefix kernels
// tail chunks per thread the fp32 prefix kernel also keeps in LDS (16 KB per unit at 1024
// threads)
constexpr int kPrefixKeepF32 = 9;
// and the bf16 prefix kernel, beside its 76 KB shift table
constexpr int kPrefixKeepBf16 = 5;

// aligned: the rows (and dlogits rows) start on 16-byte boundaries. phase_ok: bf16 rows that
// start anywhere (2-byte aligned), with dlogits (if any) at the logits' phase on every row;
// rows that are not aligned or not a whole number of chunks then use the phase kernels.
RowLaunch select_row_kernel(int32_t dtype, int64_t V, bool aligned, bool bwd, int force,
                            bool phase_ok = false);
void launch_prep_stats(const uint8_t* mask, int64_t T, int32_t* stats, hipStream_t st);
// With flags (a count-mode row kernel ran before), also stores the five counters derived
// from the flags (rd_mode decides which tokens are active).
void launch_loss_sum(const float* loss_tok, const uint8_t* mask, const float* tscale,
                     int32_t* stats, int64_t T, float loss_scale, int32_t scale_mode,
                     float* loss_out, hipStream_t st, const uint8_t* flags = nullptr,
                     int32_t rd_mode = 0);
// Longest batch whose loss call may run in count mode (every workgroup reads the whole mask).
constexpr int64_t kCountModeMaxT = 65536;

}  // namespace dppo
