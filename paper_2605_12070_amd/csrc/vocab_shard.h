// Internal interface of the vocabulary-shard kernels (loss stage on a [T, Vs] column block
// of the logits, columns [vstart, vstart + Vs) of a V-column vocabulary).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "loss_stage.h"

namespace dppo {

struct ShardArgs {
  RowArgs a;            // a.logits / a.ld / a.V: the shard ([T, Vs], row stride ld);
                        // a.dlogits / a.ldd: the shard's gradient; per-token arrays as usual
  int64_t vstart;       // global column of the shard's first column
  int64_t vtot;         // V, the whole vocabulary (token-id range check)
  const float* lse_in;  // loss: global log-sum-exp per token
  const float* zy_in;   // loss: global z[t, y_t] per token
  float* lse_out;       // stats: the shard's log-sum-exp per token
  float* zy_out;        // stats: z[t, y_t] when the shard holds column y_t, else 0
};

hipError_t launch_shard_stats(const ShardArgs& s, bool bf16, bool vec, hipStream_t st);
hipError_t launch_shard_combine(const float* lse_s, int32_t P, int64_t T, float* lse,
                                hipStream_t st);
hipError_t launch_shard_loss(const ShardArgs& s, bool bf16, bool vec, hipStream_t st);

}  // namespace dppo
