// Loss stage with the LM head folded in (gfx950). The logits z = hidden weight^T exist only
// as 128 x 128 tiles in registers and LDS:
//   lmh_fwd_tiles  one tile per workgroup on the matrix cores, reduced to a per-token
//                  partial log-sum-exp of the tile's 128 vocabulary entries;
//   lmh_zy         z[t, y_t] as one dot product per token;
//   lmh_finish     merges the partials into lse_t and runs the token math of Eq. 1-4
//                  (ratios, band, PPO clip, loss, MIS weight w_t);
//   lmh_bwd_tiles  recomputes a tile and writes g = w_t (softmax - onehot) for one
//                  vocabulary chunk, the operand of the two gradient products.
#include "dppo.h"
#include "dppo_device.h"
#include "lm_head.h"
#include "token_math.h"

namespace dppo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int kLdk = LMH_BK + 8;                 // padded LDS row of an operand tile (bf16)
constexpr int kTileElems = LMH_BM * kLdk;        // one operand tile (LMH_BM == LMH_BN)
constexpr int kLdc = LMH_BN + 4;                 // padded fp32 row of the staged C tile
constexpr int kStageBytes = 2 * kTileElems * 2;  // A and B tiles of one stage
constexpr int kSmemBytes = (2 * kStageBytes > LMH_BM * kLdc * 4) ? 2 * kStageBytes : LMH_BM * kLdc * 4;
static_assert(LMH_BM == 128 && LMH_BN == 128 && LMH_BK == 64, "tile shape assumed below");

// C tile = hidden[m0 : m0+128] . weight[r0 : r0+128]^T with fp32 accumulation, staged in
// LDS as Cs[row][col] (row = token, col = vocabulary entry) on return. 256 threads: wave
// (wm, wn) owns the 64 x 64 quarter (wm, wn), four 32 x 32 x 16 bf16 MFMA tiles. Rows past
// T or V read as zeros (buffer range checks); K is consumed in steps of 64 through two LDS
// stages, the next stage's global loads in flight while the current one is multiplied.
__device__ __forceinline__ void lmh_tile(const LmhArgs& m, int m0, int r0, char* smem) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int d = m.d;
  const int rows_a = min(LMH_BM, m.T - m0);
  const int rows_b = min(LMH_BN, m.V - r0);
  const __amdgpu_buffer_rsrc_t ra = row_rsrc(m.hidden + (int64_t)m0 * d, rows_a * d * 2);
  const __amdgpu_buffer_rsrc_t rb = row_rsrc(m.weight + (int64_t)r0 * d, rows_b * d * 2);

  // Each thread moves four 16-byte chunks of each operand per stage: chunk c = tid + 256 i
  // is row c / 8, columns 8 (c % 8) .. +7 of the 128 x 64 tile.
  int goff[4], loff[4], kcol[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int row = c >> 3, kc = (c & 7) * 8;
    kcol[i] = kc;
    goff[i] = (row * d + kc) * 2;
    loff[i] = row * kLdk + kc;
  }
  u32x4 ga[4], gb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // a K tail past d reads zeros through an offset outside the resource
      const int off = (k0 + kcol[i] < d) ? goff[i] + k0 * 2 : 0x7fffff00;
      ga[i] = buf_load16(ra, off, 0);
      gb[i] = buf_load16(rb, off, 0);
    }
  };
  auto lstore = [&](int stage) {
    uint16_t* As = (uint16_t*)(smem + stage * kStageBytes);
    uint16_t* Bs = As + kTileElems;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *(u32x4*)(As + loff[i]) = ga[i];
      *(u32x4*)(Bs + loff[i]) = gb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;

  const int nk = (d + LMH_BK - 1) / LMH_BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kb = 0; kb < nk; ++kb) {
    const int cur = kb & 1;
    if (kb + 1 < nk) gload((kb + 1) * LMH_BK);
    const uint16_t* As = (const uint16_t*)(smem + cur * kStageBytes);
    const uint16_t* Bs = As + kTileElems;
#pragma unroll
    for (int ks = 0; ks < LMH_BK / 16; ++ks) {
      // 32x32x16 operands: lane l holds row (l % 32), k = 8 (l / 32) .. +7
      const int kk = ks * 16 + 8 * (lane >> 5);
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        af[mi] = __builtin_bit_cast(bf16x8, *(const u32x4*)(As + (wm * 64 + mi * 32 + (lane & 31)) * kLdk + kk));
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bfr[ni] = __builtin_bit_cast(bf16x8, *(const u32x4*)(Bs + (wn * 64 + ni * 32 + (lane & 31)) * kLdk + kk));
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kb + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // 32x32 accumulator layout: register r of lane l is row 8 (r / 4) + 4 (l / 32) + r % 4,
  // column l % 32.
  float* Cs = (float*)smem;
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * 64 + mi * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int col = wn * 64 + ni * 32 + (lane & 31);
        Cs[row * kLdc + col] = acc[mi][ni][r];
      }
  __syncthreads();
}

}  // namespace

// Forward: per-token partial log-sum-exp (log2 domain) of one 128-entry vocabulary tile.
// An entry of z that is NaN or +inf makes the partial sum NaN; a tile of only -inf logits
// contributes nothing.
__global__ __launch_bounds__(256) void lmh_fwd_tiles(LmhArgs m) {
  __shared__ __align__(16) char smem[kSmemBytes];
  const int m0 = blockIdx.x * LMH_BM;
  const int nt = blockIdx.y;
  const int r0 = m.n0 + nt * LMH_BN;
  lmh_tile(m, m0, r0, smem);
  const float* Cs = (const float*)smem;
  const int tid = threadIdx.x;
  const int row = tid >> 1, half = tid & 1;
  const int ncols = min(LMH_BN, m.n1 - r0);
  const float* cr = Cs + row * kLdc + half * 64;
  float mx = -INFINITY;
#pragma unroll 16
  for (int j = 0; j < 64; ++j)
    if (half * 64 + j < ncols) mx = fmaxf(mx, cr[j]);
  const float m2 = mx * kLog2e;
  float s = 0.0f;
  if (mx != -INFINITY) {
#pragma unroll 16
    for (int j = 0; j < 64; ++j)
      if (half * 64 + j < ncols) s += exp2_hw(__builtin_fmaf(cr[j], kLog2e, -m2));
  }
  float n = (mx == -INFINITY) ? -INFINITY : m2;
  merge_ns(n, s, __shfl_xor(n, 1, 64), __shfl_xor(s, 1, 64));
  const int t = m0 + row;
  if (half == 0 && t < m.T) {
    float* p = m.part + ((int64_t)nt * m.T + t) * 2;
    p[0] = n;
    p[1] = s;
  }
}

// z[t, y_t] = hidden[t] . weight[y_t]: one wave per token, fp32 accumulation.
__global__ __launch_bounds__(256) void lmh_zy(LmhArgs m) {
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= m.T) return;
  const int64_t y = m.ids[t];
  float acc = 0.0f;
  if (y >= 0 && y < m.V) {
    const uint16_t* h = m.hidden + (int64_t)t * m.d;
    const uint16_t* wr = m.weight + y * m.d;
    for (int k = lane * 8; k < m.d; k += 512) {
      const u32x4 hv = *(const u32x4*)(h + k);
      const u32x4 wv = *(const u32x4*)(wr + k);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc = __builtin_fmaf(bf16_lo(hv[i]), bf16_lo(wv[i]), acc);
        acc = __builtin_fmaf(bf16_hi(hv[i]), bf16_hi(wv[i]), acc);
      }
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0) m.zy[t] = acc;
}

// One thread per token: merge the tile partials into lse, then the token math. Writes the
// per-token outputs and the backward constants; counters are reduced per workgroup.
__global__ __launch_bounds__(256) void lmh_finish(RowArgs a, LmhArgs m) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  bool band = false, ppo = false, active = false, bad = false;
  if (t < m.T) {
    const bool valid = a.mask == nullptr || a.mask[t] != 0;
    const int64_t y = m.ids[t];
    const bool good = y >= 0 && y < m.V;
    float w = 0.0f, l2 = 0.0f;
    uint8_t ev = 0;
    if (!valid) {
      a.lp_out[t] = 0.0f;
      a.loss_tok[t] = 0.0f;
      if (a.flags) a.flags[t] = 0;
    } else if (!good) {
      a.lp_out[t] = __builtin_nanf("");
      a.loss_tok[t] = 0.0f;
      if (a.flags) a.flags[t] = (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID);
      bad = true;
    } else {
      float n = -INFINITY, s = 0.0f;
      const int ntiles = lmh_tiles(m.V);
      const float* p = m.part + (int64_t)t * 2;
      for (int i = 0; i < ntiles; ++i) merge_ns(n, s, p[(int64_t)i * m.T * 2], p[(int64_t)i * m.T * 2 + 1]);
      l2 = (n == -INFINITY) ? __builtin_nanf("") : n + log2f(s);
      const TokenOut o = token_math(a, token_inputs_lane(a, t), m.zy[t], l2);
      a.lp_out[t] = o.lp;
      a.loss_tok[t] = o.loss;
      if (a.flags) a.flags[t] = o.flags;
      w = o.w;
      ev = 1;
      band = o.flags & DPPO_FLAG_BAND;
      ppo = o.flags & DPPO_FLAG_PPO;
      const bool uses_mask = a.rd_mode == DPPO_RD_MASK || a.rd_mode == DPPO_RD_MASK_WEIGHT;
      active = ppo && (band || !uses_mask);
    }
    m.w[t] = w;
    m.lse2[t] = l2;
    m.ev[t] = ev;
  }
  const int nb = __syncthreads_count(band);
  const int np = __syncthreads_count(ppo);
  const int na = __syncthreads_count(active);
  const int nbad = __syncthreads_count(bad);
  if (threadIdx.x == 0) {
    if (nb) atomicAdd(&a.stats[DPPO_STAT_N_BAND], nb);
    if (np) atomicAdd(&a.stats[DPPO_STAT_N_PPO], np);
    if (na) atomicAdd(&a.stats[DPPO_STAT_N_ACTIVE], na);
    if (nbad) atomicAdd(&a.stats[DPPO_STAT_N_BAD], nbad);
  }
}

// Backward: g[t, v - n0] = w_t (softmax(z_t)[v] - 1{v = y_t}) in bf16 for the tile's rows
// of the chunk [n0, n1); tokens that were not evaluated get zeros.
__global__ __launch_bounds__(256) void lmh_bwd_tiles(LmhArgs m) {
  __shared__ __align__(16) char smem[kSmemBytes];
  const int m0 = blockIdx.x * LMH_BM;
  const int r0 = m.n0 + blockIdx.y * LMH_BN;
  lmh_tile(m, m0, r0, smem);
  const float* Cs = (const float*)smem;
  const int ncols = min(LMH_BN, m.n1 - r0);
#pragma unroll 2
  for (int i = 0; i < 8; ++i) {
    const int idx = threadIdx.x + 256 * i;
    const int row = idx >> 4, c0 = (idx & 15) * 8;
    const int t = m0 + row;
    if (t >= m.T || c0 >= ncols) continue;
    const bool ev = m.ev[t] != 0;
    const float wt = m.w[t], l2 = m.lse2[t];
    const int64_t y = m.ids[t];
    const float* cr = Cs + row * kLdc + c0;
    float o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float p = exp2_hw(__builtin_fmaf(cr[j], kLog2e, -l2));
      const float oh = (int64_t)(r0 + c0 + j) == y ? 1.0f : 0.0f;
      o[j] = ev ? wt * (p - oh) : 0.0f;
    }
    uint16_t* dst = m.g + (int64_t)t * m.ldg + (r0 - m.n0) + c0;
    if (c0 + 8 <= ncols) {
      u32x4 v;
      v.x = pack_bf16(o[0], o[1]);
      v.y = pack_bf16(o[2], o[3]);
      v.z = pack_bf16(o[4], o[5]);
      v.w = pack_bf16(o[6], o[7]);
      *(u32x4*)dst = v;
    } else {
      for (int j = 0; j < ncols - c0; ++j) dst[j] = to_bf16(o[j]);
    }
  }
}

hipError_t launch_lmh_zy(const LmhArgs& m, hipStream_t st) {
  lmh_zy<<<(m.T + 3) / 4, 256, 0, st>>>(m);
  return hipGetLastError();
}

hipError_t launch_lmh_fwd_tiles(const LmhArgs& m, hipStream_t st) {
  const dim3 grid((m.T + LMH_BM - 1) / LMH_BM, lmh_tiles(m.n1 - m.n0));
  lmh_fwd_tiles<<<grid, 256, 0, st>>>(m);
  return hipGetLastError();
}

hipError_t launch_lmh_finish(const RowArgs& a, const LmhArgs& m, hipStream_t st) {
  lmh_finish<<<(m.T + 255) / 256, 256, 0, st>>>(a, m);
  return hipGetLastError();
}

hipError_t launch_lmh_bwd_tiles(const LmhArgs& m, hipStream_t st) {
  const dim3 grid((m.T + LMH_BM - 1) / LMH_BM, lmh_tiles(m.n1 - m.n0));
  lmh_bwd_tiles<<<grid, 256, 0, st>>>(m);
  return hipGetLastError();
}

}  // namespace dppo

namespace dppo {

__global__ __launch_bounds__(256) void lmh_fill_zero(float* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0.0f;
}

hipError_t launch_lmh_zero(float* p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  lmh_fill_zero<<<(unsigned)blocks, 256, 0, st>>>(p, n);
  return hipGetLastError();
}

}  // namespace dppo
