// Loss stage on one vocabulary shard (gfx950): the kernels a GPU runs when the LM head's
// output dimension is split over GPUs (vocabulary / tensor parallelism), at the shard's
// real shape [T, Vs]. Between the two calls the shards exchange their row statistics (an
// all-gather of the shard log-sum-exps and an all-reduce sum of z[y]); shard_combine is
// the local step after that exchange.
//   shard_stats  per row: log-sum-exp over the shard's columns, and z[y] when the shard
//                holds column y (0 otherwise);
//   shard_combine  lse = log sum_s exp(lse_s) over the gathered shard statistics;
//   shard_token, shard_grad (aligned rows with dlogits) or shard_loss (otherwise): the
//                token math of Eq. 1-4 from the global lse and z[y] (every shard computes
//                the same per-token values), then this shard's columns of
//                dlogits = w (softmax - onehot).
// 16-byte vector accesses on aligned rows.
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

// The shard loss on aligned rows as two kernels instead of shard_loss:
//   shard_token  one thread per token: the token math from the global lse and z[y], the
//                per-token outputs, and the counters (one add per workgroup);
//   shard_grad   one 16-byte chunk of dlogits per thread, (chunks per row / kGradNT) workgroups
//                per row: thread 0 repeats the row's token math for w, lse2 and dy (the same
//                operations on the same inputs, so the same values), the workgroup shares
//                them through LDS, and every thread writes w 2^(z log2 e - lse2) for its
//                chunk; the thread whose chunk holds the sampled column then writes dy there.
//                A row that is not evaluated is written as zeros without being read.
// One chunk per thread over many small workgroups is the shape in which a read-write stream
// moves the most bytes per second on MI355X.
__global__ __launch_bounds__(256) void shard_token(ShardArgs s) {
  const RowArgs& a = s.a;
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool uses_mask = a.rd_mode == DPPO_RD_MASK || a.rd_mode == DPPO_RD_MASK_WEIGHT;
  bool band = false, ppo = false, active = false, bad = false;
  if (row < a.T) {
    const bool valid = a.mask == nullptr || a.mask[row] != 0;
    const int64_t y = a.ids[row];
    const bool ev = valid && y >= 0 && y < s.vtot;
    if (!valid) {
      a.lp_out[row] = 0.0f;
      a.loss_tok[row] = 0.0f;
      if (a.flags) a.flags[row] = 0;
    } else if (!ev) {
      a.lp_out[row] = __builtin_nanf("");
      a.loss_tok[row] = 0.0f;
      if (a.flags) a.flags[row] = (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID);
      bad = true;
    } else {
      const float lse2 = s.lse_in[row] * kLog2e;
      const TokenOut o = token_math(a, token_inputs_lane(a, row), s.zy_in[row], lse2);
      a.lp_out[row] = o.lp;
      a.loss_tok[row] = o.loss;
      if (a.flags) a.flags[row] = o.flags;
      band = o.flags & DPPO_FLAG_BAND;
      ppo = o.flags & DPPO_FLAG_PPO;
      active = ppo && (band || !uses_mask);
    }
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

constexpr int kGradNT = 512;  // threads of a shard_grad workgroup (128-1024 measured)

template <bool BF16>
__global__ __launch_bounds__(kGradNT) void shard_grad(ShardArgs s, int per_row) {
  __shared__ float rb[4];
  const RowArgs& a = s.a;
  constexpr int ES = BF16 ? 2 : 4;
  constexpr int E = 16 / ES;
  const int64_t row = blockIdx.x / per_row;
  const int c = (int)(blockIdx.x % per_row) * kGradNT + threadIdx.x;
  const int Vs = a.V;
  const int nfull = Vs / E;
  const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
  const int64_t y = uload(a.ids + row);
  const bool ev = valid && y >= 0 && y < s.vtot;          // uniform over the workgroup
  const char* zp = (const char*)a.logits + row * a.ld * ES;
  char* dp = (char*)a.dlogits + row * a.ldd * ES;
  const __amdgpu_buffer_rsrc_t rz = row_rsrc(zp, ev ? nfull * 16 : 0);
  const __amdgpu_buffer_rsrc_t rd = row_rsrc(dp, nfull * 16);
  const u32x4 v = buf_load16<kAuxLast>(rz, c * 16, 0);     // past the row or not read: zeros
  if (ev && threadIdx.x == 0) {
    const float lse2 = uload(s.lse_in + row) * kLog2e;
    const TokenOut o = token_math(a, token_inputs(a, row), uload(s.zy_in + row), lse2);
    rb[0] = o.w;
    rb[1] = lse2;
    rb[2] = o.dy;
  }
  __syncthreads();
  const float w = ev ? rb[0] : 0.0f, lse2 = ev ? rb[1] : 0.0f;
  float x[E];
  unpack<BF16>(v, x);
  u32x4 o;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (BF16) {
      o[k] = pack_bf16(ev ? w * exp2_hw(__builtin_fmaf(x[2 * k], kLog2e, -lse2)) : 0.0f,
                       ev ? w * exp2_hw(__builtin_fmaf(x[2 * k + 1], kLog2e, -lse2)) : 0.0f);
    } else {
      o[k] = __float_as_uint(ev ? w * exp2_hw(__builtin_fmaf(x[k], kLog2e, -lse2)) : 0.0f);
    }
  }
  buf_store16_nt(o, rd, c * 16, 0);                        // past the row: dropped
  // the V % E last entries of the row, by the thread after the last whole chunk
  if (c == nfull) {
    for (int i = nfull * E; i < Vs; ++i) {
      const float g = ev ? w * exp2_hw(__builtin_fmaf(elem<BF16>(zp, i), kLog2e, -lse2)) : 0.0f;
      if (BF16) ((uint16_t*)dp)[i] = to_bf16(g);
      else ((float*)dp)[i] = g;
    }
  }
  // the sampled column, when this shard holds it, by the thread that wrote its entry
  const int64_t yl = y - s.vstart;
  if (ev && yl >= 0 && yl < Vs && c == (yl < (int64_t)nfull * E ? (int)(yl / E) : nfull)) {
    const float dy = rb[2];
    if (yl < (int64_t)nfull * E) {
      if (BF16) __builtin_amdgcn_raw_buffer_store_b16(to_bf16(dy), rd, (int)(yl * 2), 0, kAuxNT);
      else __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(dy), rd, (int)(yl * 4), 0, kAuxNT);
    } else if (BF16) {
      ((uint16_t*)dp)[yl] = to_bf16(dy);
    } else {
      ((float*)dp)[yl] = dy;
    }
  }
}


hipError_t launch_shard_loss(const ShardArgs& s, bool bf16, bool vec, hipStream_t st) {
  if (vec && s.a.dlogits != nullptr) {                    // shard_token + shard_grad
    if (s.a.T <= 0) return hipSuccess;
    shard_token<<<(unsigned)((s.a.T + 255) / 256), 256, 0, st>>>(s);
    const hipError_t e0 = hipGetLastError();
    if (e0 != hipSuccess) return e0;
    const int E = bf16 ? 8 : 4;
    const int64_t per_row = (s.a.V / E + kGradNT) / kGradNT;  // whole chunks, the tail thread
    if (per_row * s.a.T > 0x7fffffff) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)(per_row * s.a.T);
    if (bf16) shard_grad<true><<<grid, kGradNT, 0, st>>>(s, (int)per_row);
    else shard_grad<false><<<grid, kGradNT, 0, st>>>(s, (int)per_row);
    return hipGetLastError();
  }
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
