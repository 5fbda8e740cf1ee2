// Gradient products of the loss stage with the LM head folded in (gfx950 matrix cores):
//   dL/dhidden = G W          [T, d] = [T, V] x [V, d]
//   dL/dW      = G^T hidden   [V, d] = [V, T] x [T, d]
// where G = w (softmax - onehot) is the bf16 dlogits matrix (Sec. 3.1, the MIS gradient,
// chained through z = hidden W^T), and the row pass that forms G in place from the
// exponentials the forward tiles stored.
//
// Both products are C[m, n] = sum_k A[m, k] B[n, k] with fp32 accumulation and an fp32 C.
// An operand lies in memory either K-major (A[m, k] at p[m ld + k]: a row holds K) or
// MN-major (A[m, k] at p[k ld + m]: a row holds M). G is K-major for dhidden (K = V) and
// MN-major for dW (K = T); W and hidden are MN-major in both (their rows hold d = N).
//
// Tile engine: 4 waves (2 x 2, one per SIMD), each with 4 x 4 tiles of
// v_mfma_f32_32x32x16_bf16, so a workgroup covers 256 x 256 of C and a wave 128 x 128 (256
// accumulation registers). K advances GBK = 32 per LDS stage; four stages of 32 KB form a
// ring (each slot its own LDS object), filled by 16-byte buffer-to-LDS loads (lane l's 16
// bytes land at the wave's LDS base + 16 l; a lane whose offset lies outside the buffer
// resource receives zeros, which bounds every access to the matrix and turns every tail into
// zeros). A slot is refilled three stages ahead of its use: on MI355X four 32-deep stages
// ran 3 % faster than two 64-deep ones, and five (the whole 160 KB of LDS) no faster.
//  * A K-major operand tile is 256 staged rows of GBK K (GBK / 8 16-byte chunks); chunk c of
//    row r sits at position c ^ sw_k(r), so the 16 consecutive rows of one fragment read
//    pass cover all 64 banks. A fragment (one lane: 8 consecutive K of one row) is one
//    16-byte LDS read.
//  * An MN-major operand tile is GBK staged rows of K, each 256 M (or N) entries (512
//    bytes); chunk c of row r sits at position c ^ (4 (r % 4)). A fragment is read with two
//    transposing LDS reads (ds_read_b64_tr_b16): within each 16-lane block, lane s reads 4
//    consecutive entries of row k0 + s / 4 at column c0 + 4 (s % 4), and lane i receives
//    column c0 + i of rows k0 .. k0 + 3 (the layout was checked on MI355X with an in-bounds
//    probe). The swizzle puts the 32 lanes of one read pass on 64 distinct banks.
// The instruction order is fixed by hand, as in the logit-tile engine: during each K step
// of 16 (16 MFMAs) the next step's fragments are read, one read after each MFMA; the stage
// barrier sits before a stage's last K step, whose MFMAs also carry the refill loads of the
// slot just consumed, one per MFMA. K is padded to whole turns of the ring (stages past K
// load zeros), which keeps the loop free of branches.
//
// Tile order. Workgroups are dealt to the 8 XCDs in turn, and each XCD has its own L2. The
// 1-D grid index i is first mapped to L(i) so that one XCD's workgroups take consecutive
// L; L then walks the tile grid in groups of kGroupM = 4 tile rows, M fastest within a
// group, so the 32 workgroups an XCD runs at once cover a 4 x 8 block of tiles: 12 operand
// panels per K stage instead of the 2 + 16 of a row-major walk (N fastest). On MI355X this
// cut the L2 misses of dhidden from 22.4 to 16.4 GB and of dW from 33.1 to 17.3 GB per
// launch (T = 8192, d = 4096, V = 151936) at the same speed: the products are not bound by
// L2 misses.
#include <type_traits>
#include <utility>

#include "dppo.h"
#include "dppo_device.h"
#include "lm_head.h"
#include "token_math.h"

namespace dppo {

typedef __bf16 bf16x8g __attribute__((ext_vector_type(8)));
typedef float f32x16g __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int GW_M = 2, GW_N = 2;                // waves
constexpr int GTM = 4, GTN = 4;                  // 32 x 32 tiles per wave
constexpr int GBM = 32 * GW_M * GTM;             // 256
constexpr int GBN = 32 * GW_N * GTN;             // 256
#ifndef LMG_BK
#define LMG_BK 32
#endif
#ifndef LMG_STAGES
#define LMG_STAGES 4
#endif
constexpr int GBK = LMG_BK;                      // K per LDS stage
constexpr int GTHREADS = 64 * GW_M * GW_N;
constexpr int GS = LMG_STAGES;                   // LDS stages
constexpr int kOpEl = 256 * GBK;                 // bf16 elements of one operand tile
constexpr int kLoads = kOpEl * 2 / 1024 / (GW_M * GW_N);  // wave loads per operand, stage
constexpr int kC = GBK / 8;                      // 16-byte chunks per K-major staged row
constexpr int kRL = 64 / kC;                     // K-major rows per wave load
static_assert(GBM == LMH_GBM && GBN == LMH_GBN && (GBK == 64 || GBK == 32), "tile shape");

template <int N> using IC = std::integral_constant<int, N>;

// K-major rows: 16 consecutive rows (one 16-lane read pass) land on 16 distinct bank groups
__device__ __forceinline__ int sw_k(int r) { return (r / (16 / kC)) % kC; }
__device__ __forceinline__ int sw_mn(int r) { return (r & 3) << 2; }  // MN-major rows

constexpr int kOob = 0x7fffff00;  // an offset past every resource: the load returns zeros

// One operand of a product as the engine loads it.
template <bool MN>
struct Operand {
  const uint16_t* p;   // bf16
  int64_t ld;          // row stride, elements
  int32_t ext;         // K-major: rows of the matrix (its M or N extent);
                       // MN-major: row length in use (the M or N extent), a multiple of 8
  int32_t K;
  int32_t o0;          // first M (or N) index of the workgroup's tile
  int off[kLoads];     // per-load lane offsets in bytes (the stage-independent part)
  __amdgpu_buffer_rsrc_t rs;  // K-major: the tile's rows, for the whole K loop

  __device__ __forceinline__ void init(const uint16_t* p_, int64_t ld_, int ext_, int K_, int o0_) {
    p = p_;
    ld = ld_;
    ext = ext_;
    K = K_;
    o0 = o0_;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if constexpr (!MN) {
      // load i: tile rows kRL (wave kLoads + i) .. +kRL-1; lane -> row l / kC, position l % kC
      const int rows = min(256, ext - o0);
      rs = row_rsrc(p + (int64_t)o0 * ld, rows > 0 ? (int)(rows * ld * 2) : 0);
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        const int row = kRL * (wave * kLoads + i) + lane / kC;
        off[i] = (int)(row * ld * 2) + (((lane % kC) ^ sw_k(row)) * 16);
      }
    } else {
      // load i: staged rows (K) 2 (wave kLoads + i), +1; lane -> row l / 32, position l % 32
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        const int row = 2 * (wave * kLoads + i) + (lane >> 5);
        const int c = (lane & 31) ^ sw_mn(row);
        off[i] = (o0 + 8 * c < ext) ? (int)(row * ld * 2) + c * 16 : kOob;
      }
    }
  }

  // Resource of stage kb. MN-major: rows k0 .. k0 + 63 from column o0, up to the end of the
  // columns in use of the last row (so every lane past K or past the columns lies outside);
  // empty past K.
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t stage_rsrc(int kb) const {
    if constexpr (!MN) {
      return rs;
    } else {
      const int k0 = kb * GBK;
      const int nrows = min(GBK, K - k0);
      if (nrows <= 0) return row_rsrc(p, 0);
      const int64_t bytes = (int64_t)(nrows - 1) * ld * 2 + (int64_t)(ext - o0) * 2;
      return row_rsrc(p + (int64_t)k0 * ld + o0, (int)bytes);
    }
  }

  // Refill load I of stage kb into the operand tile at dst.
  template <int I>
  __device__ __forceinline__ void load(uint16_t* dst, int kb, __amdgpu_buffer_rsrc_t r) const {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    int o;
    if constexpr (!MN) {
      const int k0 = kb * GBK;
      const int row = kRL * (wave * kLoads + I) + lane / kC;
      const int kc = (lane % kC) ^ sw_k(row);
      o = (k0 + kc * 8 < K) ? off[I] + k0 * 2 : kOob;
    } else {
      o = off[I];
    }
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        r, (__attribute__((address_space(3))) void*)(dst + (wave * kLoads + I) * 512), 16, o, 0, 0, 0);
  }
};

// Fragment reads of one operand for the wave's four 32-row tiles at tile offset wo (0 or
// 128). K-major: one 16-byte read per fragment. MN-major: two transposing 8-byte reads,
// K 0..3 and 4..7 of the lane's eight.
template <bool MN>
struct Frags {
  int base[4];  // per-fragment lane byte offsets into an operand tile

  __device__ __forceinline__ void init(int wo) {
    const int lane = threadIdx.x & 63;
    if constexpr (!MN) {
      const int row = wo + (lane & 31);
#pragma unroll
      for (int f = 0; f < 4; ++f) base[f] = (row + 32 * f) * GBK * 2;
    } else {
      const int b = lane >> 4, s = lane & 15, q = s >> 2, e = s & 3;
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        const int pos = 4 * ((wo >> 5) + (f ^ q)) + 2 * (b & 1) + (e >> 1);
        base[f] = (8 * (b >> 1) + q) * 512 + pos * 16 + (e & 1) * 8;
      }
    }
  }

  // Part H (MN-major: 0 or 1; K-major: 0 only) of fragment F of K step ks from tile t.
  template <int F, int H>
  __device__ __forceinline__ void read(const uint16_t* t, int ks, u32x4& out) const {
    const char* tb = (const char*)t;
    if constexpr (!MN) {
      const int lane = threadIdx.x & 63;
      const int col = ((2 * ks + (lane >> 5)) ^ sw_k(lane & 31)) * 16;
      out = *(const u32x4*)(tb + base[F] + col);
    } else {
      auto* pp = (__attribute__((address_space(3))) s16x4*)(tb + base[F] + ks * 8192 + H * 2048);
      const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(pp));
      if constexpr (H == 0) {
        out.x = v.x;
        out.y = v.y;
      } else {
        out.z = v.x;
        out.w = v.y;
      }
    }
  }
};

// The LDS ring: each stage's A and B tiles are LDS objects of their own, so that the
// compiler can tell the loads into one slot from the fragment reads of the other and does
// not make the reads wait for the loads in flight.
struct Ring {
  uint16_t* a[GS];
  uint16_t* b[GS];
};

template <bool AMN, bool BMN, typename Epi>
__device__ __forceinline__ void grad_engine(const GemmArgs& g, int m0, int n0, const Ring& ring,
                                            Epi&& epi) {
  constexpr int RA = AMN ? 2 : 1, RB = BMN ? 2 : 1;   // reads per fragment
  constexpr int NR = GTM * RA + GTN * RB;              // fragment reads per K step
  constexpr int NM = GTM * GTN;                         // MFMAs per K step
  constexpr int L = 2 * kLoads;                         // refill loads per stage and wave
  constexpr int KS = GBK / 16;                          // K steps per stage
  static_assert(NR <= NM && L <= NM && KS % 2 == 0, "schedule");
  const int wave = threadIdx.x >> 6;
  const int wm = wave / GW_N, wn = wave % GW_N;
  Operand<AMN> A;
  Operand<BMN> B;
  A.init(g.a, g.lda, g.a_ext, g.K, m0);
  B.init(g.b, g.ldb, g.b_ext, g.K, n0);
  Frags<AMN> FA;
  Frags<BMN> FB;
  FA.init(wm * 128);
  FB.init(wn * 128);

  f32x16g acc[GTM][GTN];
#pragma unroll
  for (int mi = 0; mi < GTM; ++mi)
#pragma unroll
    for (int ni = 0; ni < GTN; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;
  u32x4 fa[2][GTM], fb[2][GTN];

  // read op I of K step ks of slot s into set S_, in the order the next step's MFMAs first
  // use the fragments (MFMA i takes A fragment i / GTN and B fragment i % GTN): A 0, then
  // B 0 .. GTN - 1, then A 1 .. GTM - 1. Read I is issued after MFMA I of this step, so
  // every fragment has at least 8 MFMAs to arrive.
  auto read_one = [&](auto J, int ks, auto S_, auto I) {
    constexpr int j0 = decltype(J)::value, f = decltype(S_)::value, i = decltype(I)::value;
    if constexpr (i < RA) {
      FA.template read<0, i>(ring.a[j0], ks, fa[f][0]);
    } else if constexpr (i < RA + GTN * RB) {
      constexpr int j = i - RA;
      FB.template read<j / RB, j % RB>(ring.b[j0], ks, fb[f][j / RB]);
    } else {
      constexpr int j = i - RA - GTN * RB;
      FA.template read<1 + j / RA, j % RA>(ring.a[j0], ks, fa[f][1 + j / RA]);
    }
  };
  auto load_one = [&](auto J, int kb, __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb,
                      auto I) {
    constexpr int j0 = decltype(J)::value, i = decltype(I)::value;
    if constexpr (i < kLoads) A.template load<i>(ring.a[j0], kb, ra);
    else B.template load<i - kLoads>(ring.b[j0], kb, rb);
  };
  auto mfma_one = [&](auto S_, auto I) {
    constexpr int f = decltype(S_)::value, i = decltype(I)::value;
    acc[i / GTN][i % GTN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
        __builtin_bit_cast(bf16x8g, fa[f][i / GTN]), __builtin_bit_cast(bf16x8g, fb[f][i % GTN]),
        acc[i / GTN][i % GTN], 0, 0, 0);
  };
  // One K step on set S_, reading K step rks of slot RS into the other set; with LOADS, the
  // refill of slot DST with stage kb as well. Order per MFMA: read, load, MFMA.
  auto kstep = [&](auto S_, auto RS, int rks, auto LOADS, auto DST, int kb,
                   __amdgpu_buffer_rsrc_t ra, __amdgpu_buffer_rsrc_t rb) {
    constexpr int f = decltype(S_)::value;
    constexpr bool loads = decltype(LOADS)::value;
    auto one = [&](auto I) {
      constexpr int i = decltype(I)::value;
      if constexpr (i < NR) read_one(RS, rks, IC<f ^ 1>{}, IC<i>{});
      if constexpr (loads && i < L) load_one(DST, kb, ra, rb, IC<i>{});
      mfma_one(IC<f>{}, IC<i>{});
      __builtin_amdgcn_sched_barrier(0);
    };
    [&]<int... is>(std::integer_sequence<int, is...>) {
      (one(IC<is>{}), ...);
    }(std::make_integer_sequence<int, NM>{});
  };
  // barrier without a memory fence (a fence would wait for the loads in flight)
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  const int nk = (g.K + GBK - 1) / GBK;
  [&]<int... ss>(std::integer_sequence<int, ss...>) {
    auto prologue = [&](auto S_) {
      constexpr int s0 = decltype(S_)::value;
      const __amdgpu_buffer_rsrc_t ra = A.stage_rsrc(s0), rb = B.stage_rsrc(s0);
      [&]<int... vs>(std::integer_sequence<int, vs...>) {
        (load_one(IC<s0>{}, s0, ra, rb, IC<vs>{}), ...);
      }(std::make_integer_sequence<int, L>{});
    };
    (prologue(IC<ss>{}), ...);
  }(std::make_integer_sequence<int, GS>{});
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"((GS - 1) * L) : "memory");
  barrier();
  [&]<int... is>(std::integer_sequence<int, is...>) {
    (read_one(IC<0>{}, 0, IC<0>{}, IC<is>{}), ...);
  }(std::make_integer_sequence<int, NR>{});
  // stage kb in slot J
  auto stage = [&](auto J, int kb) {
    constexpr int j = decltype(J)::value;
    const __amdgpu_buffer_rsrc_t ra = A.stage_rsrc(kb + GS), rb = B.stage_rsrc(kb + GS);
    [&]<int... ks>(std::integer_sequence<int, ks...>) {
      (kstep(IC<ks & 1>{}, IC<j>{}, ks + 1, std::false_type{}, IC<j>{}, kb, ra, rb), ...);
    }(std::make_integer_sequence<int, KS - 1>{});
    // This wave's reads of slot j are done, and its loads of stage kb + 1 are once at most
    // the loads of the GS - 2 later stages are outstanding; after the barrier, every wave's.
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"((GS - 2) * L) : "memory");
    barrier();
    __builtin_amdgcn_sched_barrier(0);
    kstep(IC<(KS - 1) & 1>{}, IC<(j + 1) % GS>{}, 0, std::true_type{}, IC<j>{}, kb + GS, ra, rb);
  };
  for (int kb0 = 0; kb0 < nk; kb0 += GS) {
    [&]<int... js>(std::integer_sequence<int, js...>) {
      (stage(IC<js>{}, kb0 + js), ...);
    }(std::make_integer_sequence<int, GS>{});
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  barrier();
  epi(acc, wm, wn);
}

// Index i of the 1-D grid -> the tile order's L: with nt tiles, the first 8 floor(nt / 8)
// workgroups are dealt to XCD i % 8, which takes the consecutive L (i % 8) floor(nt / 8) +
// i / 8; the rest keep their own index.
__device__ __forceinline__ int xcd_tile(int i, int nt) {
  const int per = nt >> 3;
  return i < 8 * per ? (i & 7) * per + (i >> 3) : i;
}

constexpr int kGroupM = 4;  // tile rows per group of the tile order

// L -> tile (tm, tn): groups of kGroupM tile rows (fewer in the last group), M fastest.
__device__ __forceinline__ void grouped_tile(int L, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int per_group = kGroupM * tiles_n;
  const int grp = L / per_group, r = L - grp * per_group;
  const int rows = min(kGroupM, tiles_m - grp * kGroupM);
  tm = grp * kGroupM + r % rows;
  tn = r / rows;
}

}  // namespace

// C (+)= A B^T over the tile of workgroup blockIdx.x; fp32 C stored non-temporally.
template <bool AMN, bool BMN>
__global__ __launch_bounds__(GTHREADS) void lmh_grad_gemm(GemmArgs g) {
  // one LDS object per slot and operand (a 2-D array is one object: the transposing reads of
  // one slot would then wait for the loads into another); unused ones are not allocated
  static_assert(GS >= 2 && GS <= 5, "LDS slots");
  __shared__ __align__(16) uint16_t la0[kOpEl], la1[kOpEl], la2[kOpEl], la3[kOpEl], la4[kOpEl];
  __shared__ __align__(16) uint16_t lb0[kOpEl], lb1[kOpEl], lb2[kOpEl], lb3[kOpEl], lb4[kOpEl];
  uint16_t* const as[5] = {la0, la1, la2, la3, la4};
  uint16_t* const bs[5] = {lb0, lb1, lb2, lb3, lb4};
  Ring ring;
#pragma unroll
  for (int i = 0; i < GS; ++i) {
    ring.a[i] = as[i];
    ring.b[i] = bs[i];
  }
  int tm, tn;
  grouped_tile(xcd_tile(blockIdx.x, g.tiles_m * g.tiles_n), g.tiles_m, g.tiles_n, tm, tn);
  const int m0 = tm * GBM;
  const int n0 = tn * GBN;
  auto epi = [&](f32x16g (&acc)[GTM][GTN], int wm, int wn) {
    const int lane = threadIdx.x & 63;
    const int n_l = n0 + wn * 128 + (lane & 31);
    const int m_l = m0 + wm * 128 + 4 * (lane >> 5);
#pragma unroll
    for (int mi = 0; mi < GTM; ++mi)
#pragma unroll
      for (int ni = 0; ni < GTN; ++ni) {
        const int n = n_l + ni * 32;
        if (n >= g.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m_l + mi * 32 + 8 * (r >> 2) + (r & 3);
          if (m >= g.M) continue;
          float* p = g.c + (int64_t)m * g.ldc + n;
          float v = acc[mi][ni][r];
          if (g.accumulate) v += *p;
          __builtin_nontemporal_store(v, p);
        }
      }
  };
  grad_engine<AMN, BMN>(g, m0, n0, ring, epi);
}

template __global__ void lmh_grad_gemm<false, true>(GemmArgs);
template __global__ void lmh_grad_gemm<true, true>(GemmArgs);

hipError_t launch_lmh_grad_gemm(const GemmArgs& g0, bool a_mn, bool b_mn, hipStream_t st) {
  GemmArgs g = g0;
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  g.tiles_m = (g.M + GBM - 1) / GBM;
  g.tiles_n = (g.N + GBN - 1) / GBN;
  const int64_t nt = (int64_t)g.tiles_m * g.tiles_n;
  if (nt > 0x7fffffff) return hipErrorInvalidValue;
  if (!b_mn) return hipErrorInvalidValue;
  if (a_mn) lmh_grad_gemm<true, true><<<(unsigned)nt, GTHREADS, 0, st>>>(g);
  else lmh_grad_gemm<false, true><<<(unsigned)nt, GTHREADS, 0, st>>>(g);
  return hipGetLastError();
}

}  // namespace dppo
