// Device-side helpers for the gfx950 loss-stage kernels.
//
// Numerics of the vocabulary-wide log-sum-exp. Every thread keeps its share of a row's
// logits and works in log2 units: with n = L * m (L = log2 e, m = the thread's maximum,
// rounded once to float), each element contributes e = 2^(z L - n), evaluated as one FMA
// (z L is exact inside the FMA, one rounding) and one v_exp_f32. Thread partials (n, s)
// merge as N = max n, S = sum s * 2^(n - N), where n - N is a difference of floats (exact
// when the shifts are close), so lse2 = N + log2 S carries about one ulp of error however
// large the logits are. lse = lse2 * ln 2 and softmax(z)[v] = 2^(z L - lse2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dppo {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;
constexpr uint32_t kBf16NegInfPair = 0xFF80FF80u;  // two bf16 -inf
constexpr uint32_t kF32NegInf = 0xFF800000u;

// 2^x on the transcendental unit (v_exp_f32); about 1 ulp for normal results.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// max(a, b, c) in one v_max3_f32. A quiet-NaN operand is ignored, as by fmaxf; NaN logits
// still reach the sum of exponentials, which turns NaN.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// bf16 halves of a 32-bit word as exact floats.
__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// Two floats -> two bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}
__device__ __forceinline__ uint16_t to_bf16(float x) {
  return (uint16_t)(pack_bf16(x, 0.0f) & 0xFFFFu);
}

// Two floats -> two fp16, round to nearest even (v_cvt_pk_f16_f32).
__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, f16x2));
}

// fp16 half of a word times a float scale, fused (v_fma_mix_f32).
__device__ __forceinline__ float f16_lo_mul(uint32_t u, float f) {
  f16x2 h = __builtin_bit_cast(f16x2, u);
  return __builtin_fmaf((float)h[0], f, 0.0f);
}
__device__ __forceinline__ float f16_hi_mul(uint32_t u, float f) {
  f16x2 h = __builtin_bit_cast(f16x2, u);
  return __builtin_fmaf((float)h[1], f, 0.0f);
}

// Merge two log2-domain partials (n, s) into (n, s). A partial with n = -inf is empty.
// Symmetric: merge(a, b) and merge(b, a) give the same bits, so every lane of a butterfly
// ends with the same result.
__device__ __forceinline__ void merge_ns(float& n, float& s, float n2, float s2) {
  const float N = fmaxf(n, n2);
  const float fa = (n == N) ? 1.0f : exp2f(n - N);
  const float fb = (n2 == N) ? 1.0f : exp2f(n2 - N);
  s = s * fa + s2 * fb;
  n = N;
}

// The same merge for integer-valued shifts, where 2^(n - N) is exact on v_exp_f32.
__device__ __forceinline__ void merge_ns_int(float& n, float& s, float n2, float s2) {
  const float N = fmaxf(n, n2);
  const float fa = (n == N) ? 1.0f : exp2_hw(n - N);
  const float fb = (n2 == N) ? 1.0f : exp2_hw(n2 - N);
  s = s * fa + s2 * fb;
  n = N;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}

// Wave-wide merge of integer-shift partials; every lane returns the wave's result.
// Quad xor 1 and xor 2, half-row and row mirrors (DPP) reduce each 16-lane row; the
// permlane swaps combine rows 0-1, 2-3 and then the two halves.
__device__ __forceinline__ void wave_merge_ns_int(float& n, float& s) {
  merge_ns_int(n, s, dpp_f<0xB1>(n), dpp_f<0xB1>(s));    // quad_perm [1,0,3,2]
  merge_ns_int(n, s, dpp_f<0x4E>(n), dpp_f<0x4E>(s));    // quad_perm [2,3,0,1]
  merge_ns_int(n, s, dpp_f<0x141>(n), dpp_f<0x141>(s));  // row_half_mirror
  merge_ns_int(n, s, dpp_f<0x140>(n), dpp_f<0x140>(s));  // row_mirror
  {
    const auto pn = __builtin_amdgcn_permlane16_swap(__float_as_uint(n), __float_as_uint(n), false, false);
    const auto ps = __builtin_amdgcn_permlane16_swap(__float_as_uint(s), __float_as_uint(s), false, false);
    n = __uint_as_float(pn[0]);
    s = __uint_as_float(ps[0]);
    merge_ns_int(n, s, __uint_as_float(pn[1]), __uint_as_float(ps[1]));
  }
  {
    const auto pn = __builtin_amdgcn_permlane32_swap(__float_as_uint(n), __float_as_uint(n), false, false);
    const auto ps = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
    n = __uint_as_float(pn[0]);
    s = __uint_as_float(ps[0]);
    merge_ns_int(n, s, __uint_as_float(pn[1]), __uint_as_float(ps[1]));
  }
}

// Workgroup-wide merge of integer-shift partials with a single barrier. `lds` holds
// 2 * (NT / 64) floats and must not be written again before the workgroup's next barrier:
// callers alternate two buffers from one merge to the next (not by row: a row that runs no
// merge must not flip the buffer, or two merges in a row would share one with no barrier
// between them). Every thread returns the same bits: each wave merges the NT / 64 wave
// results in the same fixed tree.
template <int NT>
__device__ __forceinline__ void block_merge_ns_int(float& n, float& s, float* lds) {
  constexpr int NW = NT / 64;
  static_assert(NW <= 16, "one 16-lane row merges the wave results");
  wave_merge_ns_int(n, s);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    lds[wave] = n;
    lds[NW + wave] = s;
  }
  __syncthreads();
  const int l = threadIdx.x & 15;
  n = l < NW ? lds[l] : -INFINITY;
  s = l < NW ? lds[NW + l] : 0.0f;
  merge_ns_int(n, s, dpp_f<0xB1>(n), dpp_f<0xB1>(s));
  merge_ns_int(n, s, dpp_f<0x4E>(n), dpp_f<0x4E>(s));
  merge_ns_int(n, s, dpp_f<0x141>(n), dpp_f<0x141>(s));
  merge_ns_int(n, s, dpp_f<0x140>(n), dpp_f<0x140>(s));
}

// Raw buffer resources (gfx9-family descriptor: stride 0, 32-bit data format). Loads past
// num_records return zeros and stores past it are dropped, so a row's resource bounds
// every access to that row.
constexpr int kRsrcFlags = 0x00020000;
constexpr int kAuxNT = 2;  // non-temporal cache policy bit for buffer accesses on gfx950

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, kRsrcFlags);
}
// Cache policy of a row load. Data read for the last time is loaded non-temporal
// (kAuxLast), so that its lines do not displace data that is read again. Same-process A/B
// on MI355X: the flagship row kernel 0.5 % faster, the forward-only kernel 3-5 %, the
// shard statistics 11 %, the fp32 resident and prefix kernels 2 %. The first read of a
// tail that is streamed twice keeps the default policy (kAuxKeep): non-temporal there made
// the prefix kernels 8-17 % slower, as it made the shard loss kernel 6 % slower.
constexpr int kAuxKeep = 0;
constexpr int kAuxLast = kAuxNT;
template <int AUX = kAuxKeep>
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX);
}
template <int AUX = kAuxKeep>
__device__ __forceinline__ void load16(uint32_t (&d)[4], __amdgpu_buffer_rsrc_t r, int voff, int soff) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX);
  d[0] = v.x;
  d[1] = v.y;
  d[2] = v.z;
  d[3] = v.w;
}
// A 16-byte store, then two wait states. On gfx950 a VALU write of a 16-byte buffer store's
// data VGPRs issued right behind the store (seen: a v_mov_b64 into the first two) changed
// the data being stored, and the compiler inserts no wait after a buffer store whose
// offset is an SGPR. The scheduling barriers keep the wait directly behind the store.
__device__ __forceinline__ void buf_store16_nt(u32x4 v, __amdgpu_buffer_rsrc_t r, int voff, int soff) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, kAuxNT);
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 1");
  __builtin_amdgcn_sched_barrier(0);
}

// Load of a value at a workgroup-uniform address through the scalar unit (constant
// address space): waited on with lgkmcnt, so it never waits behind the row's vector loads.
template <typename T>
__device__ __forceinline__ T uload(const T* p) {
  return *(const __attribute__((address_space(4))) T*)p;
}

// A uniform byte through the scalar unit, which has no byte loads: the aligned 32-bit word
// holding the byte is loaded and shifted. A plain byte load would become a vector load. The
// word can reach up to 3 bytes past the last mask byte; the ABI therefore asks for a mask
// allocation readable up to the next 4-byte boundary (every device allocation is).
__device__ __forceinline__ uint32_t uload_u8(const uint8_t* p) {
  const uintptr_t a = (uintptr_t)p;
  const uint32_t w = uload((const uint32_t*)(a & ~(uintptr_t)3));
  return (w >> ((uint32_t)(a & 3u) * 8u)) & 0xffu;
}

// Workgroup-wide merge of general (n, s) partials (two barriers, shuffles). Fixed
// reduction order: the result is reproducible.
template <int NT>
__device__ __forceinline__ void block_merge_ns(float& n, float& s, float* lds) {
  constexpr int NW = NT / 64;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float n2 = __shfl_xor(n, off, 64);
    const float s2 = __shfl_xor(s, off, 64);
    merge_ns(n, s, n2, s2);
  }
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  if (NW > 1) {
    if (lane == 0) {
      lds[wave] = n;
      lds[NW + wave] = s;
    }
    __syncthreads();
    if (wave == 0) {
      n = lane < NW ? lds[lane] : -INFINITY;
      s = lane < NW ? lds[NW + lane] : 0.0f;
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) {
        const float n2 = __shfl_xor(n, off, 64);
        const float s2 = __shfl_xor(s, off, 64);
        merge_ns(n, s, n2, s2);
      }
      if (lane == 0) {
        lds[2 * NW] = n;
        lds[2 * NW + 1] = s;
      }
    }
    __syncthreads();
    n = lds[2 * NW];
    s = lds[2 * NW + 1];
  }
}

// numpy-style minimum: NaN if either operand is NaN.
__device__ __forceinline__ float nan_min(float a, float b) {
  return (a != a || b != b) ? __builtin_nanf("") : fminf(a, b);
}

}  // namespace dppo
