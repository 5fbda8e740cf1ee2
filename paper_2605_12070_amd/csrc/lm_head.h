// Loss stage with the LM head folded in: logits z = hidden weight^T are formed tile by tile
// on the matrix cores and never written to memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "loss_stage.h"

namespace dppo {

// Tile of the GEMM kernels: LMH_WM x LMH_WN waves (one per SIMD), each with LMH_TM x LMH_TN
// matrix-core tiles of 32 x 32, so a workgroup of LMH_THREADS threads covers LMH_BM tokens x
// LMH_BN vocabulary rows; K advances LMH_BK hidden features per LDS stage.
constexpr int LMH_WM = 2, LMH_WN = 2;
constexpr int LMH_TM = 4, LMH_TN = 4;
constexpr int LMH_BM = 32 * LMH_WM * LMH_TM;
constexpr int LMH_BN = 32 * LMH_WN * LMH_TN;
constexpr int LMH_BK = 64;
constexpr int LMH_THREADS = 64 * LMH_WM * LMH_WN;
constexpr int LMH_STAGES = 2;

struct LmhArgs {
  const uint16_t* hidden;  // [T, d] bf16, rows contiguous
  const uint16_t* weight;  // [V, d] bf16 (LM head, [out, in] layout)
  int32_t T, d, V;
  int32_t n0, n1;          // vocabulary rows [n0, n1) covered by a launch
  float* part;             // forward: (max * log2 e, sum 2^(z log2 e - max)) per (tile, token)
  float* zy;               // z[t, y_t] (dot-product kernel)
  float* w;                // MIS weight per token (0 where the gradient is zero)
  float* lse2;             // log2 sum_v 2^(z log2 e) per token
  uint8_t* ev;             // 1 where the token was evaluated (valid row, good id)
  const int64_t* ids;
  uint16_t* g;             // backward: w (softmax - onehot) for rows [n0, n1), [T, ldg] bf16
  int64_t ldg;
};

__host__ __device__ inline int lmh_tiles(int n) { return (n + LMH_BN - 1) / LMH_BN; }

hipError_t launch_lmh_zy(const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_fwd_tiles(const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_finish(const RowArgs& a, const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_bwd_tiles(const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_zero(float* p, int64_t n, hipStream_t st);  // fill kernel (no memset)

}  // namespace dppo
