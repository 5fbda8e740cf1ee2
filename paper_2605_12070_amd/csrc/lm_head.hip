// Loss stage with the LM head folded in (gfx950). The logits z = hidden weight^T exist only
// as LMH_BM x LMH_BN tiles in registers and LDS:
//   lmh_fwd_tiles  one tile per workgroup on the matrix cores, reduced to per-token partial
//                  log-sum-exps of each 128-entry vocabulary group; optionally also stores
//                  the group-normalised exponentials 2^(z log2 e - m2) as fp16;
//   lmh_zy         z[t, y_t] as one dot product per token;
//   lmh_row_stats  per token row: merges the partials into lse_t and runs the token math
//                  of Eq. 1-4 (ratios, band, PPO clip, loss, MIS weight w_t);
//   lmh_grad_scale turns the stored exponentials into G = w_t (softmax - onehot) in bf16,
//                  the operand of the two gradient products (lm_head_grad.hip);
//   lmh_finish     the same merge and token math without G (forward only, or the
//                  vocabulary-chunk mode);
//   lmh_bwd_tiles  vocabulary-chunk mode: recomputes a tile and writes G for one chunk.
#include <type_traits>
#include <utility>

#include "dppo.h"
#include "dppo_device.h"
#include "lm_head.h"
#include "token_math.h"

namespace dppo {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

// Tile engine: hidden[m0 : m0 + BM] . weight[r0 : r0 + BN]^T on the matrix cores, fed by
// buffer-to-LDS loads (gfx950 writes lane l's 16 bytes at the wave's LDS base + 16 l, and
// zeros for a lane whose offset lies outside the resource, which bounds every access to
// the tile's rows and turns a K tail past d into zeros). There is no register staging:
// LMH_STAGES LDS stages form a ring. A stage holds the A and B tiles as rows of LMH_BK bf16
// of K (128 bytes); the 16-byte chunk c of row r sits at position c ^ sw(r), sw(r) = (r / 2)
// % 8, so the fragment reads of 16 lanes (16 consecutive rows, one chunk) cover all 64 banks.
// Each stage is its own LDS object, which lets the compiler track the loads into each
// separately.
// Wave (wm, wn) owns TM x TN tiles of 32 x 32 (v_mfma_f32_32x32x16_bf16, fp32 accumulation;
// operand lane l holds row l % 32, K 8 (l / 32) .. +7). With 4 waves, one per SIMD, a wave
// holds 128 x 128 accumulators in its 256 accumulation registers, which halves the LDS
// fragment reads per matrix-core instruction against a 128 x 64 wave tile. The vocabulary
// tile is the A operand, so an accumulator holds vocabulary rows in its registers and
// tokens across its lanes: a lane reduces over the vocabulary of its own tokens without
// crossing lanes (LmhLane below).
// With a single wave per SIMD no other wave covers a stall, so the instruction order is
// fixed by hand (scheduling fences between steps):
//  * a K step of 16 is TM TN MFMAs; the fragments of the next K step are read during it,
//    one read after each of the first TM + TN MFMAs (two fragment register sets, by the
//    parity of the step);
//  * the stage barrier sits before the last K step of a stage: by then every wave has read
//    all of that stage's fragments, so its slot is refilled (with stage kb + LMH_STAGES)
//    by loads spread one per MFMA over that last step, whose MFMAs also overlap the reads of
//    the next stage's first fragments;
//  * K is padded to whole turns of the ring; stages past d load zeros (the out-of-range
//    offset) and add nothing, which keeps the loop free of branches.
// After the K loop, epi(acc, scratch) runs on the accumulators, with the ring as scratch.
constexpr int kWaves = LMH_WM * LMH_WN;
constexpr int kChunks = LMH_BK / 8;             // 16-byte chunks per staged row
constexpr int kRL = 64 / kChunks;               // rows covered by one wave-wide load
constexpr int kIA = LMH_BM / kRL / kWaves;      // loads per wave and stage, A
constexpr int kIB = LMH_BN / kRL / kWaves;      // and B
constexpr int kAEl = LMH_BM * LMH_BK;           // bf16 elements of the A tile (B follows)
constexpr int kStageEl = (LMH_BM + LMH_BN) * LMH_BK;
static_assert(LMH_BK == 64 && LMH_BM % (kRL * kWaves) == 0 && LMH_BN % (kRL * kWaves) == 0,
              "tile shape");
static_assert(LMH_STAGES >= 2 && (LMH_STAGES - 2) * (kIA + kIB) <= 63, "ring depth");
static_assert((LMH_BK / 16) % 2 == 0, "an even number of K steps per stage");

// Swizzled position of 16-byte chunk c in staged row r.
__device__ __forceinline__ int lmh_sw(int r) { return (r >> 1) & 7; }

template <int N> using IC = std::integral_constant<int, N>;

template <typename Epi>
__device__ __forceinline__ void lmh_engine(const LmhArgs& m, int m0, int r0,
                                           uint16_t* (&st)[LMH_STAGES], Epi&& epi) {
  constexpr int TM = LMH_TM, TN = LMH_TN, BK = LMH_BK, KS = BK / 16, S = LMH_STAGES;
  constexpr int L = kIA + kIB;                  // loads per wave and stage
  constexpr int NF = TM + TN;                   // fragment reads per K step
  constexpr int NM = TM * TN;                   // MFMAs per K step
  constexpr int LPM = (L + NM - 1) / NM;        // refill loads per MFMA
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / LMH_WN, wn = wave % LMH_WN;
  const int d = m.d;
  const int rows_a = min(LMH_BM, m.T - m0);
  const int rows_b = min(LMH_BN, m.V - r0);
  const __amdgpu_buffer_rsrc_t ra = row_rsrc(m.hidden + (int64_t)m0 * d, rows_a * d * 2);
  const __amdgpu_buffer_rsrc_t rb = row_rsrc(m.weight + (int64_t)r0 * d, rows_b * d * 2);

  // Load i of wave w covers tile rows kRL (w I + i) .. +kRL-1: lane l takes row
  // kRL (w I + i) + l / kChunks at position l % kChunks, i.e. K chunk (l % kChunks) ^ sw(row).
  int goa[kIA], gob[kIB];
#pragma unroll
  for (int i = 0; i < kIA; ++i) {
    const int row = kRL * (wave * kIA + i) + lane / kChunks;
    goa[i] = (row * d + ((lane % kChunks) ^ lmh_sw(row)) * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < kIB; ++i) {
    const int row = kRL * (wave * kIB + i) + lane / kChunks;
    gob[i] = (row * d + ((lane % kChunks) ^ lmh_sw(row)) * 8) * 2;
  }
  // refill load i of stage kb into slot s: i < kIA of the A tile, else of the B tile
  auto load_one = [&](uint16_t* s, int kb, auto I) {
    constexpr int i = decltype(I)::value;
    const int k0 = kb * BK;
    if constexpr (i < kIA) {
      const int row = kRL * (wave * kIA + i) + lane / kChunks;
      const int kc = (lane % kChunks) ^ lmh_sw(row);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ra, (__attribute__((address_space(3))) void*)(s + (wave * kIA + i) * 512), 16,
          (k0 + kc * 8 < d) ? goa[i] + k0 * 2 : 0x7fffff00, 0, 0, 0);
    } else {
      constexpr int ib = i - kIA;
      const int row = kRL * (wave * kIB + ib) + lane / kChunks;
      const int kc = (lane % kChunks) ^ lmh_sw(row);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rb, (__attribute__((address_space(3))) void*)(s + kAEl + (wave * kIB + ib) * 512), 16,
          (k0 + kc * 8 < d) ? gob[ib] + k0 * 2 : 0x7fffff00, 0, 0, 0);
    }
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;

  // Fragment sets by K-step parity. A fragment row's swizzle depends only on lane % 32 (the
  // rows of a wave's tiles step by 32), so every read is a per-lane base plus a constant.
  bf16x8 fa[2][TM], fb[2][TN];
  const int swz = lmh_sw(lane & 31);
  const int rowa = (wm * 32 * TM + (lane & 31)) * BK;
  const int rowb = kAEl + (wn * 32 * TN + (lane & 31)) * BK;
  // fragment read i of K step ks of slot s into set f: i < TM the A fragment mi = i, else
  // the B fragment ni = i - TM
  auto read_one = [&](const uint16_t* s, int ks, auto F, auto I) {
    constexpr int f = decltype(F)::value, i = decltype(I)::value;
    const int col = ((2 * ks + (lane >> 5)) ^ swz) * 8;
    if constexpr (i < TM)
      fa[f][i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(s + rowa + col + i * 32 * BK));
    else
      fb[f][i - TM] = __builtin_bit_cast(bf16x8, *(const u32x4*)(s + rowb + col + (i - TM) * 32 * BK));
  };
  // MFMA i of a K step on set f: mi = i / TN, ni = i % TN
  auto mfma_one = [&](auto F, auto I) {
    constexpr int f = decltype(F)::value, i = decltype(I)::value;
    acc[i / TN][i % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
        fb[f][i % TN], fa[f][i / TN], acc[i / TN][i % TN], 0, 0, 0);
  };
  // One K step on set f, reading K step rks of slot rs into set f ^ 1; with LOADS, the
  // refill of slot dst with stage kb as well. Order per MFMA: read, loads, MFMA.
  auto kstep = [&](auto F, const uint16_t* rs, int rks, auto LOADS, uint16_t* dst, int kb) {
    constexpr int f = decltype(F)::value;
    constexpr bool loads = decltype(LOADS)::value;
    auto one = [&](auto I) {
      constexpr int i = decltype(I)::value;
      if constexpr (i < NF) read_one(rs, rks, IC<f ^ 1>{}, IC<i>{});
      if constexpr (loads) {
        [&]<int... vs>(std::integer_sequence<int, vs...>) {
          ((i * LPM + vs < L ? load_one(dst, kb, IC<(i * LPM + vs < L ? i * LPM + vs : 0)>{})
                             : void()), ...);
        }(std::make_integer_sequence<int, LPM>{});
      }
      mfma_one(IC<f>{}, IC<i>{});
      __builtin_amdgcn_sched_barrier(0);
    };
    [&]<int... is>(std::integer_sequence<int, is...>) {
      (one(IC<is>{}), ...);
    }(std::make_integer_sequence<int, NM>{});
  };
  // Barrier without a memory fence (a fence would wait for the loads still in flight); the
  // empty asm statements keep the compiler from moving memory accesses across it.
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  const int nk = (d + BK - 1) / BK;
#pragma unroll
  for (int s = 0; s < S; ++s)
    [&]<int... vs>(std::integer_sequence<int, vs...>) {
      (load_one(st[s], s, IC<vs>{}), ...);
    }(std::make_integer_sequence<int, L>{});
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"((S - 1) * L) : "memory");
  barrier();
  [&]<int... is>(std::integer_sequence<int, is...>) {
    (read_one(st[0], 0, IC<0>{}, IC<is>{}), ...);
  }(std::make_integer_sequence<int, NF>{});
  // stage kb in slot J
  auto stage = [&](auto J, int kb) {
    constexpr int j = decltype(J)::value;
    [&]<int... ks>(std::integer_sequence<int, ks...>) {
      (kstep(IC<ks & 1>{}, st[j], ks + 1, std::false_type{}, st[j], kb), ...);
    }(std::make_integer_sequence<int, KS - 1>{});
    // This wave's reads of slot j are done, and its loads of stage kb + 1 are once at most
    // the loads of the S - 2 later stages are outstanding; after the barrier, every wave's.
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"((S - 2) * L) : "memory");
    barrier();
    __builtin_amdgcn_sched_barrier(0);
    kstep(IC<(KS - 1) & 1>{}, st[(j + 1) % S], 0, std::true_type{}, st[j], kb + S);
  };
  for (int kb0 = 0; kb0 < nk; kb0 += S) {
    [&]<int... js>(std::integer_sequence<int, js...>) {
      (stage(IC<js>{}, kb0 + js), ...);
    }(std::make_integer_sequence<int, S>{});
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  barrier();

  // The ring is free from here on; the epilogue works on the accumulators in registers and
  // may use the ring as scratch.
  epi(acc, (float*)st[0]);
}

// Accumulator layout (v_mfma_f32_32x32x16_bf16 with the vocabulary tile as the A operand):
// acc[mi][ni] register r of lane l holds z for token
//   m0 + wm 32 TM + mi 32 + l % 32
// and vocabulary row
//   r0 + wn 32 TN + ni 32 + 8 (r / 4) + 4 (l / 32) + r % 4,
// so a lane sees one token per mi and, for each (ni, r / 4), four consecutive vocabulary rows.
struct LmhLane {
  int wm, wn, lane;
  __device__ LmhLane() : wm((threadIdx.x >> 6) / LMH_WN), wn((threadIdx.x >> 6) % LMH_WN), lane(threadIdx.x & 63) {}
  __device__ int token(int m0, int mi) const { return m0 + wm * 32 * LMH_TM + mi * 32 + (lane & 31); }
  // tile-relative vocabulary row of register r of tile ni
  __device__ int vrow(int ni, int r) const {
    return wn * 32 * LMH_TN + ni * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
  }
};

}  // namespace

#define LMH_RUN_ENGINE(m, m0, r0, epi)                                                    \
  do {                                                                                    \
    __shared__ __align__(16) uint16_t lmh_st[LMH_STAGES][kStageEl];                       \
    uint16_t* ring[LMH_STAGES];                                                           \
    _Pragma("unroll") for (int i = 0; i < LMH_STAGES; ++i) ring[i] = lmh_st[i];            \
    lmh_engine(m, m0, r0, ring, epi);                                                     \
  } while (0)

// Forward: per-token partial log-sum-exp (log2 domain) of each 128-entry vocabulary group of
// the tile (one wave's columns): m2 = log2 e * the group's maximum, sum 2^(z log2 e - m2).
// With store_p the exponentials 2^(z log2 e - m2) in (0, 1] are also stored as fp16 into
// g [T, ldg], four consecutive vocabulary entries (8 bytes) per store: the row pass later
// scales them by w 2^(m2 - lse2) into the gradient, so the backward needs no second product.
// ldg is then a multiple of the tile width, so every tile's columns lie inside the row
// (entries past V are overwritten by the row pass); a buffer resource over the tile's token
// rows drops the stores of rows past T.
// An entry of z that is NaN or +inf makes the partial sum NaN; a group of only -inf logits
// contributes nothing.
__global__ __launch_bounds__(LMH_THREADS) void lmh_fwd_tiles(LmhArgs m) {
  const int m0 = blockIdx.x * LMH_BM;
  const int nt = blockIdx.y;
  const int r0 = m.n0 + nt * LMH_BN;
  const int ncols = min(LMH_BN, m.n1 - r0);
  auto epi = [&](f32x16 (&acc)[LMH_TM][LMH_TN], float*) {
    const LmhLane L;
    const bool ragged = ncols < LMH_BN;       // only the last vocabulary tile
    const int grp = (r0 / LMH_GROUP) + L.wn;  // this wave's 128 columns
    const int prows = m.store_p ? min(LMH_BM, m.T - m0) : 0;
    const __amdgpu_buffer_rsrc_t rp = row_rsrc(m.g + (int64_t)m0 * m.ldg, (int)(prows * m.ldg * 2));
    static_assert(LMH_TN * 32 == LMH_GROUP, "a wave's columns form one group");
#pragma unroll
    for (int mi = 0; mi < LMH_TM; ++mi) {
      float mx = -INFINITY;
#pragma unroll
      for (int ni = 0; ni < LMH_TN; ++ni)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float x = acc[mi][ni][r];
          mx = fmaxf(mx, (ragged && L.vrow(ni, r) >= ncols) ? -INFINITY : x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));  // the two lanes that hold the token's group
      const float m2 = mx * kLog2e;
      const float sh = (mx == -INFINITY) ? 0.0f : m2;
      const int t = L.token(m0, mi);
      const int poff = (int)(((int64_t)(t - m0) * m.ldg + r0) * 2);
      float sum = 0.0f;
#pragma unroll
      for (int ni = 0; ni < LMH_TN; ++ni)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int v0 = L.vrow(ni, 4 * q);
          float e[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            e[j] = exp2_hw(__builtin_fmaf(acc[mi][ni][4 * q + j], kLog2e, -sh));
            sum += (ragged && v0 + j >= ncols) ? 0.0f : e[j];
          }
          if (m.store_p) {
            u32x2 v;
            v.x = pack_f16(e[0], e[1]);
            v.y = pack_f16(e[2], e[3]);
            __builtin_amdgcn_raw_buffer_store_b64(v, rp, poff + v0 * 2, 0, 0);
          }
        }
      sum += __shfl_xor(sum, 32, 64);
      if (L.lane < 32 && t < m.T) {
        float* p = m.part + ((int64_t)t * lmh_groups(m.V) + grp) * 2;
        p[0] = (mx == -INFINITY) ? -INFINITY : m2;
        p[1] = sum;
      }
    }
  };
  LMH_RUN_ENGINE(m, m0, r0, epi);
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
      const int ngroups = lmh_groups(m.V);
      const float* p = m.part + (int64_t)t * ngroups * 2;
      for (int i = 0; i < ngroups; ++i) merge_ns(n, s, p[2 * i], p[2 * i + 1]);
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

// Full-vocabulary backward without a second product, in two passes.
// lmh_row_stats, one 256-thread workgroup per token row (looping over rows): merges the
// row's group partials into lse2, runs the token math (per-token outputs, counters kept per
// workgroup) and leaves the backward constants w, lse2, dy = w (p_y - 1) (as token_math
// computes it from z[y]) and ev for the scale pass.
// lmh_grad_scale turns the stored exponentials into G = w (softmax - onehot) in place, one
// 16-byte chunk (8 entries) per thread: entry v of group q becomes w 2^(m2_q - lse2) e_v in
// bf16, the sampled entry dy, and the entries from V up to ldg zeros; a row that is not
// evaluated (masked, or a bad id) becomes zeros without being read. One chunk per thread
// and a grid of (chunks per row / 256) x T workgroups is the shape in which a read-write
// stream moves the most bytes per second on MI355X (as a per-row loop over four chunks per
// thread it took 1.0 ms at T = 8192, V = 151936).
constexpr int kGR = 256;

__global__ __launch_bounds__(kGR) void lmh_row_stats(RowArgs a, LmhArgs m) {
  __shared__ float red[2 * (kGR / 64) + 2];
  StatCount sc;
  const int tid = threadIdx.x;
  const int ngroups = lmh_groups(m.V);
  for (int64_t row = blockIdx.x; row < m.T; row += gridDim.x) {
    const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
    const int64_t y = uload(m.ids + row);
    const bool ev = valid && y >= 0 && y < m.V;           // uniform over the workgroup
    if (ev) {
      float n = -INFINITY, s = 0.0f;
      for (int q = tid; q < ngroups; q += kGR) {
        const float* p = m.part + (row * ngroups + q) * 2;
        merge_ns(n, s, p[0], p[1]);
      }
      block_merge_ns<kGR>(n, s, red);  // once per row: its second barrier orders the reuse
      const float l2 = (n == -INFINITY) ? __builtin_nanf("") : n + log2f(s);
      if (tid == 0) {
        const TokenOut o = token_math(a, token_inputs(a, row), uload(m.zy + row), l2);
        a.lp_out[row] = o.lp;
        a.loss_tok[row] = o.loss;
        if (a.flags) a.flags[row] = o.flags;
        count_stats(a, o.flags, sc);
        m.w[row] = o.w;
        m.lse2[row] = l2;
        m.dy[row] = o.dy;
        m.ev[row] = 1;
      }
    } else if (tid == 0) {
      a.lp_out[row] = valid ? __builtin_nanf("") : 0.0f;
      a.loss_tok[row] = 0.0f;
      if (a.flags) a.flags[row] = valid ? (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID) : (uint8_t)0;
      if (valid) sc.bad += 1;
      m.w[row] = 0.0f;
      m.lse2[row] = 0.0f;
      m.dy[row] = 0.0f;
      m.ev[row] = 0;
    }
  }
  if (tid == 0) flush_stats(a, sc);
}

__global__ __launch_bounds__(256) void lmh_grad_scale(LmhArgs m, int per_row) {
  // per_row workgroups cover a row's chunks; consecutive workgroups walk along a row
  const int64_t row = blockIdx.x / per_row;
  const int c = (int)(blockIdx.x % per_row) * 256 + threadIdx.x;
  if (c >= (int)(m.ldg / 8)) return;
  const int v0 = 8 * c;
  uint16_t* grow = m.g + row * m.ldg;
  const bool ev = uload_u8(m.ev + row) != 0;              // uniform over the workgroup
  u32x4 out = {0u, 0u, 0u, 0u};
  if (ev && v0 < m.V) {
    const u32x4 e = __builtin_nontemporal_load((const u32x4*)(grow + v0));
    const float w = uload(m.w + row), l2 = uload(m.lse2 + row), dy = uload(m.dy + row);
    const int64_t y = uload(m.ids + row);
    const float m2 = m.part[(row * lmh_groups(m.V) + v0 / LMH_GROUP) * 2];
    const float f = w * exp2_hw(m2 - l2);
    float x[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[2 * j] = f16_lo_mul(e[j], f);
      x[2 * j + 1] = f16_hi_mul(e[j], f);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if ((int64_t)(v0 + j) == y) x[j] = dy;
      if (v0 + j >= m.V) x[j] = 0.0f;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) out[j] = pack_bf16(x[2 * j], x[2 * j + 1]);
  }
  __builtin_nontemporal_store(out, (u32x4*)(grow + v0));
}

// Backward (vocabulary chunks): g[t, v - n0] = w_t (softmax(z_t)[v] - 1{v = y_t}) in bf16
// for the tile's rows of the chunk [n0, n1); tokens that were not evaluated get zeros. The
// last tile also zeroes the entries past the chunk up to the next multiple of 8, which the
// gradient products read as whole 16-byte chunks.
__global__ __launch_bounds__(LMH_THREADS) void lmh_bwd_tiles(LmhArgs m) {
  const int m0 = blockIdx.x * LMH_BM;
  const int r0 = m.n0 + blockIdx.y * LMH_BN;
  const int ncols = min(LMH_BN, m.n1 - r0);
  auto epi = [&](f32x16 (&acc)[LMH_TM][LMH_TN], float*) {
    const LmhLane L;
#pragma unroll
    for (int mi = 0; mi < LMH_TM; ++mi) {
      const int t = L.token(m0, mi);
      if (t >= m.T) continue;
      const bool ev = m.ev[t] != 0;
      const float wt = ev ? m.w[t] : 0.0f;
      const float l2 = m.lse2[t];
      const int64_t yr = m.ids[t] - r0;        // the token's id relative to the tile
      uint16_t* grow = m.g + (int64_t)t * m.ldg + (r0 - m.n0);
#pragma unroll
      for (int ni = 0; ni < LMH_TN; ++ni)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // four consecutive vocabulary rows v0 .. v0 + 3 of this token
          const int v0 = L.vrow(ni, 4 * q);
          float o[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float p = exp2_hw(__builtin_fmaf(acc[mi][ni][4 * q + j], kLog2e, -l2));
            o[j] = ev ? wt * (p - ((int64_t)(v0 + j) == yr ? 1.0f : 0.0f)) : 0.0f;
          }
          if (v0 + 4 <= ncols) {
            u32x2 v;
            v.x = pack_bf16(o[0], o[1]);
            v.y = pack_bf16(o[2], o[3]);
            *(u32x2*)(grow + v0) = v;
          } else {
            const int end8 = (ncols + 7) & ~7;
            for (int j = 0; j < 4 && v0 + j < end8; ++j)
              grow[v0 + j] = v0 + j < ncols ? to_bf16(o[j]) : (uint16_t)0;
          }
        }
    }
  };
  LMH_RUN_ENGINE(m, m0, r0, epi);
}

hipError_t launch_lmh_zy(const LmhArgs& m, hipStream_t st) {
  lmh_zy<<<(m.T + 3) / 4, 256, 0, st>>>(m);
  return hipGetLastError();
}

hipError_t launch_lmh_fwd_tiles(const LmhArgs& m, hipStream_t st) {
  const dim3 grid((m.T + LMH_BM - 1) / LMH_BM, lmh_tiles(m.n1 - m.n0));
  lmh_fwd_tiles<<<grid, LMH_THREADS, 0, st>>>(m);
  return hipGetLastError();
}

hipError_t launch_lmh_finish(const RowArgs& a, const LmhArgs& m, hipStream_t st) {
  lmh_finish<<<(m.T + 255) / 256, 256, 0, st>>>(a, m);
  return hipGetLastError();
}

hipError_t launch_lmh_grad_rows(const RowArgs& a, const LmhArgs& m, hipStream_t st) {
  if (m.ldg % 8 != 0 || m.ldg / 8 > 0x7fffffff) return hipErrorInvalidValue;
  if (m.T <= 0) return hipSuccess;
  const int grid = m.T < 2048 ? m.T : 2048;
  lmh_row_stats<<<grid, kGR, 0, st>>>(a, m);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t per_row = (m.ldg / 8 + 255) / 256;
  if (per_row * m.T > 0x7fffffff) return hipErrorInvalidValue;
  lmh_grad_scale<<<(unsigned)(per_row * m.T), 256, 0, st>>>(m, (int)per_row);
  return hipGetLastError();
}

hipError_t launch_lmh_bwd_tiles(const LmhArgs& m, hipStream_t st) {
  const dim3 grid((m.T + LMH_BM - 1) / LMH_BM, lmh_tiles(m.n1 - m.n0));
  lmh_bwd_tiles<<<grid, LMH_THREADS, 0, st>>>(m);
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
