// Loss stage on one vocabulary shard (gfx950): the kernels a GPU runs when the LM head's
// output dimension is split over GPUs (vocabulary / tensor parallelism), at the shard's
// real shape [T, Vs]. Between the two calls the shards exchange their row statistics (an
// all-gather of the shard log-sum-exps and an all-reduce sum of z[y]); shard_combine is
// the local step after that exchange.
//   shard_stats  per row: log-sum-exp over the shard's columns, and z[y] when the shard
//                holds column y (0 otherwise);
//   shard_combine  lse = log sum_s exp(lse_s) over the gathered shard statistics;
//   shard_loss   per row: the token math of Eq. 1-4 from the global lse and z[y] (every
//                shard computes the same per-token values), then this shard's columns of
//                dlogits = w (softmax - onehot).
// One workgroup of 256 threads per row; 16-byte vector accesses on aligned rows.
#include "dppo.h"
#include "dppo_device.h"
#include "loss_stage.h"
#include "token_math.h"
#include "vocab_shard.h"

namespace dppo {

namespace {

constexpr int kNT = 256;
constexpr int kGroup = 8;  // 16-byte chunks whose loads a thread issues together

// Elements of a 16-byte chunk as floats.
template <bool BF16>
__device__ __forceinline__ void unpack(const u32x4& v, float (&x)[BF16 ? 8 : 4]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (BF16) {
      x[2 * k] = bf16_lo(v[k]);
      x[2 * k + 1] = bf16_hi(v[k]);
    } else {
      x[k] = __uint_as_float(v[k]);
    }
  }
}

template <bool BF16>
__device__ __forceinline__ float elem(const char* row, int64_t i) {
  return BF16 ? bf16_to_f32(((const uint16_t*)row)[i]) : ((const float*)row)[i];
}

// This thread's log2-domain partial (n, s) of the row's Vs elements: chunks of one 16-byte
// vector get an integer shift n_c = ceil(L max), as in the row kernels, so that partials
// merge exactly (merge_ns_int).
template <bool BF16, bool VEC>
__device__ __forceinline__ void row_partial(const char* row, int Vs, float& N, float& S) {
  constexpr int E = BF16 ? 8 : 4;
  const int tid = threadIdx.x;
  int64_t tail0 = 0;
  if (VEC) {
    const int nfull = Vs / E;
    const __amdgpu_buffer_rsrc_t rz = row_rsrc(row, nfull * 16);
    for (int c0 = 0; c0 < nfull; c0 += kNT * kGroup) {
      u32x4 v[kGroup];
#pragma unroll
      for (int g = 0; g < kGroup; ++g) v[g] = buf_load16<kAuxLast>(rz, (c0 + g * kNT + tid) * 16, 0);
#pragma unroll
      for (int g = 0; g < kGroup; ++g) {
        if (c0 + g * kNT + tid >= nfull) continue;
        float x[E];
        unpack<BF16>(v[g], x);
        float cm = x[0];
#pragma unroll
        for (int j = 1; j < E; ++j) cm = fmaxf(cm, x[j]);
        const float nc = __builtin_ceilf(cm * kLog2e);
        const float sh = (nc == -INFINITY) ? 0.0f : nc;
        float sc = 0.0f;
#pragma unroll
        for (int j = 0; j < E; ++j) sc += exp2_hw(__builtin_fmaf(x[j], kLog2e, -sh));
        merge_ns_int(N, S, nc, sc);
      }
    }
    tail0 = (int64_t)nfull * E;
  }
  for (int64_t i = tail0 + tid; i < Vs; i += kNT) {
    const float z = elem<BF16>(row, i);
    const float nc = __builtin_ceilf(z * kLog2e);
    const float sh = (nc == -INFINITY) ? 0.0f : nc;
    merge_ns_int(N, S, nc, exp2_hw(__builtin_fmaf(z, kLog2e, -sh)));
  }
}

}  // namespace

// One workgroup per row. (A persistent grid looping over rows measured 12-80 % slower for
// this read-only kernel: every row's load, merge and barrier then run back to back.)
template <bool BF16, bool VEC>
__global__ __launch_bounds__(kNT) void shard_stats(ShardArgs s) {
  __shared__ float red[2 * (kNT / 64)];
  const RowArgs& a = s.a;
  const int64_t row = blockIdx.x;
  constexpr int ES = BF16 ? 2 : 4;
  const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
  if (!valid) {                        // not read: its statistics never reach a loss
    if (threadIdx.x == 0) {
      s.lse_out[row] = -INFINITY;
      s.zy_out[row] = 0.0f;
    }
    return;
  }
  const char* rp = (const char*)a.logits + row * a.ld * ES;
  float N = -INFINITY, S = 0.0f;
  row_partial<BF16, VEC>(rp, a.V, N, S);
  block_merge_ns_int<kNT>(N, S, red);
  if (threadIdx.x == 0) {
    // an empty or all -inf shard contributes exp(-inf) = 0 to the global sum
    s.lse_out[row] = (N == -INFINITY) ? -INFINITY : (N + log2f(S)) * kLn2;
    const int64_t yl = uload(a.ids + row) - s.vstart;
    s.zy_out[row] = (yl >= 0 && yl < a.V) ? elem<BF16>(rp, yl) : 0.0f;
  }
}

// lse_t = log sum_s exp(lse_s,t), shards in index order around their maximum. No finite
// shard (every column of the row -inf, or the row masked) gives NaN, as the unsharded
// log-sum-exp does for a row of -inf.
__global__ __launch_bounds__(256) void shard_combine(const float* lse_s, int32_t P, int64_t T,
                                                     float* lse) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  float m = -INFINITY;
  for (int p = 0; p < P; ++p) m = fmaxf(m, lse_s[(int64_t)p * T + t]);
  float sum = 0.0f;
  for (int p = 0; p < P; ++p) sum += expf(lse_s[(int64_t)p * T + t] - m);
  lse[t] = (m == -INFINITY) ? __builtin_nanf("") : m + logf(sum);
}

// Persistent: workgroup g takes rows g, g + grid, ... Each row's first chunks are loaded
// before thread 0 runs the row's token math, so the two overlap; the counters are summed in
// the workgroup and added to stats once at the end. (Loading the next row's chunks before
// this row's stores, in a second register set, measured no faster: the occupancy it costs
// cancels the overlap.)
template <bool BF16, bool VEC>
__global__ __launch_bounds__(kNT) void shard_loss(ShardArgs s) {
  struct Row {
    float w, lse2, dy;
    int ev;
  };
  __shared__ Row rb[2];                  // alternated by row parity: one barrier per row
  const RowArgs& a = s.a;
  constexpr int ES = BF16 ? 2 : 4;
  constexpr int E = 16 / ES;
  const int tid = threadIdx.x;
  const int Vs = a.V;
  const int nfull = VEC ? Vs / E : 0;
  const int64_t tail0 = (int64_t)nfull * E;
  const bool want_d = a.dlogits != nullptr;
  const bool uses_mask = a.rd_mode == DPPO_RD_MASK || a.rd_mode == DPPO_RD_MASK_WEIGHT;
  int n_band = 0, n_ppo = 0, n_active = 0, n_bad = 0;   // thread 0's counts
  int parity = 0;
  for (int64_t row = blockIdx.x; row < a.T; row += gridDim.x, parity ^= 1) {
    // uniform: every thread reads the row's mask and id through the scalar unit
    const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
    const int64_t y = uload(a.ids + row);
    const bool ev = valid && y >= 0 && y < s.vtot;
    const int64_t yl = y - s.vstart;
    const char* zp = (const char*)a.logits + row * a.ld * ES;
    char* dp = (char*)a.dlogits + row * a.ldd * ES;
    // a zero-size resource turns the loads of a row that is not evaluated into zeros
    const __amdgpu_buffer_rsrc_t rz = row_rsrc(zp, (ev && want_d) ? nfull * 16 : 0);
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(dp, want_d ? nfull * 16 : 0);
    u32x4 v[kGroup];
    if (VEC && want_d) {
#pragma unroll
      for (int g = 0; g < kGroup; ++g) v[g] = buf_load16(rz, (g * kNT + tid) * 16, 0);
    }
    if (tid == 0) {
      Row r = {0.0f, 0.0f, 0.0f, 0};
      if (!valid) {
        a.lp_out[row] = 0.0f;
        a.loss_tok[row] = 0.0f;
        if (a.flags) a.flags[row] = 0;
      } else if (!ev) {
        a.lp_out[row] = __builtin_nanf("");
        a.loss_tok[row] = 0.0f;
        if (a.flags) a.flags[row] = (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID);
        ++n_bad;
      } else {
        const float lse2 = uload(s.lse_in + row) * kLog2e;
        const TokenOut o = token_math(a, token_inputs(a, row), uload(s.zy_in + row), lse2);
        a.lp_out[row] = o.lp;
        a.loss_tok[row] = o.loss;
        if (a.flags) a.flags[row] = o.flags;
        const bool band = o.flags & DPPO_FLAG_BAND, ppo = o.flags & DPPO_FLAG_PPO;
        n_band += band;
        n_ppo += ppo;
        n_active += ppo && (band || !uses_mask);
        r = {o.w, lse2, o.dy, 1};
      }
      rb[parity] = r;
    }
    if (!want_d) continue;               // uniform
    __syncthreads();
    const Row r = rb[parity];
    auto grad = [&](float z) -> float {
      return r.ev ? r.w * exp2_hw(__builtin_fmaf(z, kLog2e, -r.lse2)) : 0.0f;
    };
    auto chunk_out = [&](const u32x4& cv, int ci) {
      float x[E];
      unpack<BF16>(cv, x);
      u32x4 o;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (BF16) o[k] = pack_bf16(grad(x[2 * k]), grad(x[2 * k + 1]));
        else o[k] = __float_as_uint(grad(x[k]));
      }
      buf_store16_nt(o, rd, ci * 16, 0);                       // past the row: dropped
    };
    if (VEC) {
#pragma unroll
      for (int g = 0; g < kGroup; ++g) chunk_out(v[g], g * kNT + tid);
      // rows wider than one group (Vs > kGroup kNT E): the rest, four chunks per thread at
      // a time
      for (int c0 = kNT * kGroup; c0 < nfull; c0 += kNT * 4) {
        u32x4 w[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) w[g] = buf_load16(rz, (c0 + g * kNT + tid) * 16, 0);
#pragma unroll
        for (int g = 0; g < 4; ++g) chunk_out(w[g], c0 + g * kNT + tid);
      }
    }
    for (int64_t i = tail0 + tid; i < Vs; i += kNT) {
      const float g = grad(r.ev ? elem<BF16>(zp, i) : 0.0f);
      if (BF16) ((uint16_t*)dp)[i] = to_bf16(g);
      else ((float*)dp)[i] = g;
    }
    // the sampled column, when this shard holds it: w (p_y - 1), written by the thread that
    // wrote its chunk, after that chunk and through the same kind of store
    if (r.ev && yl >= 0 && yl < Vs) {
      const bool in_vec = VEC && yl < tail0;
      const int64_t owner = in_vec ? (yl / E) % kNT : (yl - tail0) % kNT;
      if (tid == owner) {
        if (in_vec) {
          if (BF16) __builtin_amdgcn_raw_buffer_store_b16(to_bf16(r.dy), rd, (int)(yl * 2), 0, kAuxNT);
          else __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(r.dy), rd, (int)(yl * 4), 0, kAuxNT);
        } else if (BF16) {
          ((uint16_t*)dp)[yl] = to_bf16(r.dy);
        } else {
          ((float*)dp)[yl] = r.dy;
        }
      }
    }
  }
  if (tid == 0) {
    if (n_band) atomicAdd(&a.stats[DPPO_STAT_N_BAND], n_band);
    if (n_ppo) atomicAdd(&a.stats[DPPO_STAT_N_PPO], n_ppo);
    if (n_active) atomicAdd(&a.stats[DPPO_STAT_N_ACTIVE], n_active);
    if (n_bad) atomicAdd(&a.stats[DPPO_STAT_N_BAD], n_bad);
  }
}

hipError_t launch_shard_stats(const ShardArgs& s, bool bf16, bool vec, hipStream_t st) {
  const dim3 g((unsigned)s.a.T), b(kNT);
  if (bf16) {
    if (vec) shard_stats<true, true><<<g, b, 0, st>>>(s);
    else shard_stats<true, false><<<g, b, 0, st>>>(s);
  } else {
    if (vec) shard_stats<false, true><<<g, b, 0, st>>>(s);
    else shard_stats<false, false><<<g, b, 0, st>>>(s);
  }
  return hipGetLastError();
}

hipError_t launch_shard_combine(const float* lse_s, int32_t P, int64_t T, float* lse, hipStream_t st) {
  const int64_t blocks = (T + 255) / 256;
  shard_combine<<<(unsigned)blocks, 256, 0, st>>>(lse_s, P, T, lse);
  return hipGetLastError();
}

constexpr int kShardLossFill = 27;  // CUs used per 32

hipError_t launch_shard_loss(const ShardArgs& s, bool bf16, bool vec, hipStream_t st) {
  const void* fn = bf16 ? (vec ? (const void*)shard_loss<true, true> : (const void*)shard_loss<true, false>)
                        : (vec ? (const void*)shard_loss<false, true> : (const void*)shard_loss<false, false>);
  // Persistent grid: two workgroups on 27 of every 32 CUs, each looping over rows. At
  // T = 16384, Vs = 18992 on MI355X this beat every other grid measured: all resident slots
  // (five per CU) 9 % slower, two per CU on all CUs 4 %, three per CU 11 %, one per CU 29 %.
  int dev = 0, cus = 0, per_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kNT, 0);
  if (e != hipSuccess) return e;
  const int64_t used_cus = cus * kShardLossFill / 32 > 0 ? cus * kShardLossFill / 32 : 1;
  const int64_t slots = used_cus * (per_cu >= 2 ? 2 : (per_cu > 0 ? per_cu : 1));
  const unsigned grid = (unsigned)(s.a.T < slots ? s.a.T : slots);
  void* args[] = {const_cast<ShardArgs*>(&s)};
  e = hipLaunchKernel(fn, dim3(grid), dim3(kNT), args, 0, st);
  return e != hipSuccess ? e : hipGetLastError();
}

}  // namespace dppo
