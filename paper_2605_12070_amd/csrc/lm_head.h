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

// Partial log-sum-exps are kept per token and 128-entry vocabulary group (one wave's share
// of a tile's columns).
constexpr int LMH_GROUP = 128;

struct LmhArgs {
  const uint16_t* hidden;  // [T, d] bf16, rows contiguous
  const uint16_t* weight;  // [V, d] bf16 (LM head, [out, in] layout)
  int32_t T, d, V;
  int32_t n0, n1;          // vocabulary rows [n0, n1) covered by a launch
  float* part;             // forward: (m2, sum 2^(z log2 e - m2)) per (token, group), with
                           // m2 = log2 e * the group's maximum; [T][groups] float pairs, so a
                           // token's partials are contiguous for the row pass
  float* zy;               // z[t, y_t] (dot-product kernel)
  float* w;                // MIS weight per token (0 where the gradient is zero)
  float* lse2;             // log2 sum_v 2^(z log2 e) per token
  float* dy;               // w (p_y - 1) per token: the sampled entry of G (one pass)
  uint8_t* ev;             // 1 where the token was evaluated (valid row, good id)
  const int64_t* ids;
  uint16_t* g;             // [T, ldg]: the forward tiles' fp16 exponentials 2^(z log2 e - m2)
                           // (store_p), turned in place into G = w (softmax - onehot) in
                           // bf16; or, chunk by chunk, G for rows [n0, n1) (backward tiles)
  int64_t ldg;
  int32_t store_p;         // forward tiles: also store the exponentials into g
};

__host__ __device__ inline int lmh_tiles(int n) { return (n + LMH_BN - 1) / LMH_BN; }
// Groups per token: every tile's two groups, the last one possibly past V (empty: -inf, 0).
__host__ __device__ inline int lmh_groups(int n) { return lmh_tiles(n) * (LMH_BN / LMH_GROUP); }

// C[m, n] (+)= sum_k A[m, k] B[n, k] for the gradient products (bf16 operands, fp32 C).
// An operand is K-major (element [i, k] at p[i ld + k]) or MN-major (element [i, k] at
// p[k ld + i]); ext is its M (or N) extent: the row count when K-major, the row length in
// use (a multiple of 8, entries past the matrix's own end zero) when MN-major.
struct GemmArgs {
  const uint16_t* a;
  int64_t lda;
  int32_t a_ext;
  const uint16_t* b;
  int64_t ldb;
  int32_t b_ext;
  int32_t M, N, K;
  float* c;                // [M, ldc] fp32
  int64_t ldc;
  int32_t accumulate;      // 1: C += A B^T; 0: C = A B^T
  int32_t tiles_m, tiles_n;  // set by the launcher
};
constexpr int LMH_GBM = 256, LMH_GBN = 256;  // C tile of one workgroup

hipError_t launch_lmh_zy(const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_fwd_tiles(const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_finish(const RowArgs& a, const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_bwd_tiles(const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_zero(float* p, int64_t n, hipStream_t st);  // fill kernel (no memset)
hipError_t launch_lmh_grad_rows(const RowArgs& a, const LmhArgs& m, hipStream_t st);
hipError_t launch_lmh_grad_gemm(const GemmArgs& g, bool a_mn, bool b_mn, hipStream_t st);

}  // namespace dppo
