// Loss stage with the LM head folded in (gfx950). The logits z = hidden weight^T exist only
// as LMH_BM x LMH_BN tiles in registers and LDS:
//   lmh_fwd_tiles  one tile per workgroup on the matrix cores, reduced to a per-token
//                  partial log-sum-exp of the tile's LMH_BN vocabulary entries;
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

// Tile engine. 256 threads = 4 waves in a 2 x 2 arrangement; wave (wm, wn) owns TM x TN
// MFMA tiles of 32 x 32, so the workgroup tile is (64 TM) tokens x (64 TN) vocabulary rows.
// K advances LMH_BK at a time through two LDS stages (rows padded by 8 bf16 so that the 16-byte
// fragment reads of 16 lanes hit distinct banks); the next stage's global loads are in
// flight while the current stage is multiplied.
template <int TM, int TN>
struct Cfg {
  static constexpr int BM = 64 * TM, BN = 64 * TN, BK = LMH_BK, LDK = BK + 8;
  static constexpr int KC = BK / 8;                     // 16-byte chunks per tile row
  static constexpr int A_EL = BM * LDK, B_EL = BN * LDK;
  static constexpr int STAGE = (A_EL + B_EL) * 2;       // bytes of one stage (A and B)
  static constexpr int CA = BM * BK / 8 / 256;          // 16-byte chunks per thread, A
  static constexpr int CB = BN * BK / 8 / 256;          // and B
  static constexpr int LDC = BN + 4;                    // staged C row (fp32)
  static constexpr int STG = 64 * LDC * 4;              // one pass: 64 token rows
  static constexpr int SMEM = 2 * STAGE > STG ? 2 * STAGE : STG;
};
using LC = Cfg<LMH_BM / 64, LMH_BN / 64>;
static_assert(LC::BM == LMH_BM && LC::BN == LMH_BN && LC::BK == LMH_BK, "tile constants");

// Computes the tile hidden[m0 : m0 + BM] . weight[r0 : r0 + BN]^T (rows past T or V read as
// zeros through the buffer range checks; a K tail past d reads zeros through an offset
// outside the resource), then hands it to epi(Cs, mi) in TM passes: pass mi stages, for
// both wave rows wm, the 32 token rows wm * 32 TM + mi * 32 + [0, 32) as Cs[s][col] with
// s = wm * 32 + row % 32 and col in [0, BN).
template <int TM, int TN, typename Epi>
__device__ __forceinline__ void lmh_engine(const LmhArgs& m, int m0, int r0, char* smem, Epi&& epi) {
  using C = Cfg<TM, TN>;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int d = m.d;
  const int rows_a = min(C::BM, m.T - m0);
  const int rows_b = min(C::BN, m.V - r0);
  const __amdgpu_buffer_rsrc_t ra = row_rsrc(m.hidden + (int64_t)m0 * d, rows_a * d * 2);
  const __amdgpu_buffer_rsrc_t rb = row_rsrc(m.weight + (int64_t)r0 * d, rows_b * d * 2);

  // chunk c = tid + 256 i of a tile is row c / KC, columns 8 (c % KC) .. +7
  int ga_off[C::CA], la_off[C::CA], gb_off[C::CB], lb_off[C::CB];
  int kcol_a[C::CA], kcol_b[C::CB];
#pragma unroll
  for (int i = 0; i < C::CA; ++i) {
    const int c = tid + 256 * i, row = c / C::KC, kc = (c % C::KC) * 8;
    kcol_a[i] = kc;
    ga_off[i] = (row * d + kc) * 2;
    la_off[i] = row * C::LDK + kc;
  }
#pragma unroll
  for (int i = 0; i < C::CB; ++i) {
    const int c = tid + 256 * i, row = c / C::KC, kc = (c % C::KC) * 8;
    kcol_b[i] = kc;
    gb_off[i] = (row * d + kc) * 2;
    lb_off[i] = C::A_EL + row * C::LDK + kc;
  }
  u32x4 ga[C::CA], gb[C::CB];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::CA; ++i)
      ga[i] = buf_load16(ra, (k0 + kcol_a[i] < d) ? ga_off[i] + k0 * 2 : 0x7fffff00, 0);
#pragma unroll
    for (int i = 0; i < C::CB; ++i)
      gb[i] = buf_load16(rb, (k0 + kcol_b[i] < d) ? gb_off[i] + k0 * 2 : 0x7fffff00, 0);
  };
  auto lstore = [&](int stage) {
    uint16_t* S = (uint16_t*)(smem + stage * C::STAGE);
#pragma unroll
    for (int i = 0; i < C::CA; ++i) *(u32x4*)(S + la_off[i]) = ga[i];
#pragma unroll
    for (int i = 0; i < C::CB; ++i) *(u32x4*)(S + lb_off[i]) = gb[i];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;

  const int nk = (d + C::BK - 1) / C::BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kb = 0; kb < nk; ++kb) {
    const int cur = kb & 1;
    if (kb + 1 < nk) gload((kb + 1) * C::BK);
    const uint16_t* As = (const uint16_t*)(smem + cur * C::STAGE);
    const uint16_t* Bs = As + C::A_EL;
#pragma unroll
    for (int ks = 0; ks < C::BK / 16; ++ks) {
      // 32x32x16 operands: lane l holds row (l % 32), k = 8 (l / 32) .. +7
      const int kk = ks * 16 + 8 * (lane >> 5);
      bf16x8 af[TM], bfr[TN];
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
        af[mi] = __builtin_bit_cast(bf16x8, *(const u32x4*)(As + (wm * 32 * TM + mi * 32 + (lane & 31)) * C::LDK + kk));
#pragma unroll
      for (int ni = 0; ni < TN; ++ni)
        bfr[ni] = __builtin_bit_cast(bf16x8, *(const u32x4*)(Bs + (wn * 32 * TN + ni * 32 + (lane & 31)) * C::LDK + kk));
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kb + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // 32x32 accumulator layout: register r of lane l is row 8 (r / 4) + 4 (l / 32) + r % 4,
  // column l % 32.
  float* Cs = (float*)smem;
#pragma unroll
  for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int s = wm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int col = wn * 32 * TN + ni * 32 + (lane & 31);
        Cs[s * C::LDC + col] = acc[mi][ni][r];
      }
    __syncthreads();
    epi((const float*)Cs, mi);
    __syncthreads();
  }
}

// Token row of staged row s in pass mi.
__device__ __forceinline__ int lmh_token(int m0, int s, int mi) {
  return m0 + (s >> 5) * 32 * (LMH_BM / 64) + mi * 32 + (s & 31);
}

}  // namespace

// Forward: per-token partial log-sum-exp (log2 domain) of one LMH_BN-entry vocabulary tile.
// An entry of z that is NaN or +inf makes the partial sum NaN; a tile of only -inf logits
// contributes nothing.
__global__ __launch_bounds__(256) void lmh_fwd_tiles(LmhArgs m) {
  __shared__ __align__(16) char smem[LC::SMEM];
  const int m0 = blockIdx.x * LMH_BM;
  const int nt = blockIdx.y;
  const int r0 = m.n0 + nt * LMH_BN;
  const int ncols = min(LMH_BN, m.n1 - r0);
  const int tid = threadIdx.x;
  const int s = tid >> 2, q = tid & 3;          // 4 threads per staged row
  constexpr int QC = LMH_BN / 4;                // columns per thread
  lmh_engine<LMH_BM / 64, LMH_BN / 64>(m, m0, r0, smem, [&](const float* Cs, int mi) {
    const float* cr = Cs + s * LC::LDC + q * QC;
    const int lim = ncols - q * QC;              // valid columns of this quarter
    float mx = -INFINITY;
#pragma unroll 16
    for (int j = 0; j < QC; ++j)
      if (j < lim) mx = fmaxf(mx, cr[j]);
    const float m2 = mx * kLog2e;
    float sum = 0.0f;
    if (mx != -INFINITY) {
#pragma unroll 16
      for (int j = 0; j < QC; ++j)
        if (j < lim) sum += exp2_hw(__builtin_fmaf(cr[j], kLog2e, -m2));
    }
    float n = (mx == -INFINITY) ? -INFINITY : m2;
    merge_ns(n, sum, __shfl_xor(n, 1, 64), __shfl_xor(sum, 1, 64));
    merge_ns(n, sum, __shfl_xor(n, 2, 64), __shfl_xor(sum, 2, 64));
    const int t = lmh_token(m0, s, mi);
    if (q == 0 && t < m.T) {
      float* p = m.part + ((int64_t)nt * m.T + t) * 2;
      p[0] = n;
      p[1] = sum;
    }
  });
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
  __shared__ __align__(16) char smem[LC::SMEM];
  const int m0 = blockIdx.x * LMH_BM;
  const int r0 = m.n0 + blockIdx.y * LMH_BN;
  const int ncols = min(LMH_BN, m.n1 - r0);
  constexpr int SEGS = LMH_BN / 8;              // 8-column segments of a staged row
  lmh_engine<LMH_BM / 64, LMH_BN / 64>(m, m0, r0, smem, [&](const float* Cs, int mi) {
#pragma unroll 2
    for (int i = 0; i < 64 * SEGS / 256; ++i) {
      const int idx = threadIdx.x + 256 * i;
      const int s = idx / SEGS, c0 = (idx % SEGS) * 8;
      const int t = lmh_token(m0, s, mi);
      if (t >= m.T || c0 >= ncols) continue;
      const bool ev = m.ev[t] != 0;
      const float wt = m.w[t], l2 = m.lse2[t];
      const int64_t y = m.ids[t];
      const float* cr = Cs + s * LC::LDC + c0;
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
  });
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
