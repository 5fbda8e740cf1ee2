// Per-row kernels of the loss stage (gfx950): vocabulary-wide log-sum-exp, the decoupled
// MIS token math (Eq. 1-4 of arXiv 2605.12070) and the fused dlogits sweep, plus the two
// small kernels around them (valid-token count, deterministic loss sum).
//
// Launch shape: each token row is handled by one workgroup (persistent workgroups loop over
// rows). A row of V = 151936 bf16 logits (297 KiB) is loaded once with 16-byte loads and
// kept in registers (1024 threads x 19 x 16 B); the thread's exponentials replace the
// logits in the same registers as fp16 pairs, so the backward sweep reads nothing from
// memory and writes dlogits once with 16-byte non-temporal stores. bf16 rows that start
// anywhere or end in a partial chunk run in the same kernels with the neighbouring entries
// masked (the phase kernels). Rows longer than the register budget keep a resident prefix
// and read only the rest twice (the prefix kernels); what is left (fp32 rows off a 16-byte
// boundary, forward calls on rows past the budget) uses a streaming kernel that reads the
// row twice.
#include "dppo.h"
#include "dppo_device.h"
#include "loss_stage.h"
#include "token_math.h"

namespace dppo {

// Logits matrix holding token row `row`: with a version table (RowArgsV), the matrix of the
// token's policy version. An out-of-range version reads version 0's matrix (always mapped)
// and version_ok rejects the token. The pointer is picked with a chain of uniform selects:
// indexing the by-value argument array with a run-time index would make the compiler copy
// the arguments to scratch.
template <class A>
__device__ __forceinline__ const void* logits_of(const A& a, int64_t row) {
  const void* base = a.logits;
  if constexpr (std::is_same<A, RowArgsV>::value) {
    if (a.version) {
      const int v = (int)uload((const uint32_t*)(a.version + row));
#pragma unroll
      for (int i = 1; i < DPPO_MAX_VERSIONS; ++i)
        if (v == i && i < a.nver) base = a.vlogits[i];
    }
  }
  return base;
}
template <class T, class A>
__device__ __forceinline__ const T* row_ptr(const A& a, int64_t row) {
  return (const T*)logits_of(a, row) + row * a.ld;
}
template <class A>
__device__ __forceinline__ bool version_ok(const A& a, int64_t row) {
  if constexpr (std::is_same<A, RowArgsV>::value) {
    if (!a.version) return true;
    const int v = (int)uload((const uint32_t*)(a.version + row));
    return v >= 0 && v < a.nver;
  }
  return true;
}

// The call's loss scale (Eq. 2: the token-mean normaliser, or the constant), once per
// workgroup; every thread calls it. Normally prep_stats has stored the valid-token count; in
// count mode the workgroup counts the mask itself (workgroup 0 also stores the count, for
// loss_sum), which saves that launch for a short batch. The fp32 resident kernel (before
// its first row) and the bf16 kernels with two row buffers (behind their first row's loads)
// take this path; in the single-buffer bf16 kernels the extra prologue cost 0.7 % of the
// flagship's time even with count mode off. Counting behind the first row's loads in the
// fp32 kernel too was measured slower (the tiny batch's step 27.5 us against 25.6 us).
template <int NT>
__device__ float call_scale(const RowArgs& a) {
  if (a.mode == kModeLogprob) return 1.0f;
  if (!a.count_mode) return row_scale(a);
  if (a.scale_mode != DPPO_SCALE_TOKEN_MEAN) return a.loss_scale;
  __shared__ int part[NT / 64];
  int cnt = 0;
  if (a.mask != nullptr) {
    // 16-byte chunks from the 16-byte boundary at or below the mask, four per thread in
    // flight (T <= kCountModeMaxT); a byte counts when it lies in [mask, mask + T)
    const uintptr_t m0 = (uintptr_t)a.mask;
    const int ph = (int)(m0 & 15u);
    const int nb = ph + a.T;
    // The range check drops a 4-byte word that reaches past the resource's end, so the
    // resource runs to the next 4-byte boundary (readable, see the mask's requirement in the
    // ABI); bytes past the mask are not counted.
    const __amdgpu_buffer_rsrc_t r =
        row_rsrc((const void*)(m0 - (uintptr_t)ph), (nb + 3) & ~3);
    const int nch = (nb + 15) >> 4;
    for (int c0 = threadIdx.x; c0 < nch; c0 += 4 * NT) {
      u32x4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + u * NT;
        v[u] = buf_load16(r, c < nch ? c * 16 : 0x7fffff00, 0);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int base = (c0 + u * NT) * 16;
#pragma unroll
        for (int b = 0; b < 16; ++b) {
          const int pos = base + b;
          const uint32_t byte = (v[u][b >> 2] >> (8 * (b & 3))) & 0xffu;
          cnt += (byte != 0u) & (pos >= ph) & (pos < nb);
        }
      }
    }
  } else if (threadIdx.x == 0) {
    cnt = a.T;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) cnt += __shfl_xor(cnt, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = cnt;
  __syncthreads();
  int n = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) n += part[i];
  if (blockIdx.x == 0 && threadIdx.x == 0) a.stats[DPPO_STAT_N_VALID] = n;
  return a.loss_scale / (float)(n > 1 ? n : 1);
}

// Rows that are not evaluated (loss mask 0, or a bad token id on a valid row).
template <typename Tin, int NT>
__device__ void skip_row(const RowArgs& a, int64_t row, bool valid, StatCount& sc) {
  if (a.dlogits) {
    Tin* d = (Tin*)a.dlogits + row * a.ldd;
    for (int v = threadIdx.x; v < a.V; v += NT) d[v] = (Tin)0;
  }
  if (threadIdx.x == 0) {
    a.lp_out[row] = valid ? __builtin_nanf("") : 0.0f;
    a.loss_tok[row] = 0.0f;
    if (a.flags) a.flags[row] = valid ? (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID) : (uint8_t)0;
    if (valid) sc.bad += 1;
  }
}

// Zero dlogits row for the register-resident paths: NC 16-byte buffer stores per thread
// (stores past the row are dropped by the buffer range check) plus a ragged tail.
template <int NT, int NC, int ES>
__device__ void skip_row_resident(const RowArgs& a, int64_t row, bool valid, StatCount& sc) {
  if (a.dlogits) {
    constexpr int E = 16 / ES;
    char* d = (char*)a.dlogits + row * a.ldd * ES;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(d, a.V * ES);
    const int nfull = a.V / E;
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int c = 0; c < NC; ++c)
      if (c * NT + (int)threadIdx.x < nfull) buf_store16_nt(z, rd, threadIdx.x * 16, c * NT * 16);
    for (int e = nfull * E + threadIdx.x; e < a.V; e += NT) {
      if (ES == 2) ((uint16_t*)d)[e] = 0;
      else ((float*)d)[e] = 0.0f;
    }
  }
  if (threadIdx.x == 0) {
    a.lp_out[row] = valid ? __builtin_nanf("") : 0.0f;
    a.loss_tok[row] = 0.0f;
    if (a.flags) a.flags[row] = valid ? (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID) : (uint8_t)0;
    if (valid) sc.bad += 1;
  }
}

// Per-thread factor turning stored exponentials 2^(zL - n_mine) into w * softmax.
__device__ __forceinline__ float row_factor(float w, float n_mine, float lse2) {
  if (lse2 != lse2) return __builtin_nanf("");
  return (n_mine == -INFINITY) ? 0.0f : w * exp2f(n_mine - lse2);
}

// Thread 0 finishes a row: writes per-token outputs, counts stats, and publishes the
// backward constants (w, lse2, dy) in LDS. Returns through `bc`.
struct Bcast {
  float w, lse2, dy;
  float zy;  // z[y], published by the thread that holds it
};

__device__ __forceinline__ void finish_row(const RowArgs& a, int64_t row, float zy,
                                           float lse2, bool good, Bcast* bc, const TokenIn& tin,
                                           StatCount& sc) {
  if (a.mode == kModeLogprob) {
    if (threadIdx.x == 0) {
      a.lp_out[row] = good ? zy - lse2 * kLn2 : __builtin_nanf("");
      if (a.lse_out) a.lse_out[row] = lse2 * kLn2;
    }
    return;
  }
  if (threadIdx.x == 0) {
    const TokenOut o = token_math(a, tin, zy, lse2);
    a.lp_out[row] = o.lp;
    a.loss_tok[row] = o.loss;
    if (a.flags) a.flags[row] = o.flags;
    count_stats(a, o.flags, sc);
    bc->w = o.w;
    bc->lse2 = lse2;
    bc->dy = o.dy;
  }
}

// ---------------------------------------------------------------------------------------
// Register-resident row kernel, bf16 logits: persistent, one workgroup per CU slot.
//
// NT threads x NC 16-byte chunks hold a whole row; thread tid owns chunks c * NT + tid.
// All row traffic uses raw buffer accesses (one VGPR offset per thread, the chunk offset
// c * NT * 16 in an SGPR, range-checked against the row). Per row:
//   pass A  chunks are consumed in arrival order; chunk c gets an integer log2 shift
//           n_c = ceil(L * max(chunk)), its elements become 2^(zL - n_c) in (0, 1], are
//           summed and stored back in place as fp16 pairs; (n_c, sum) merges into (N, S);
//   merge   workgroup merge of (N, S) -> lse2; thread 0 does the token math;
//   pass B  dlogits chunk c = w * 2^(n_c - lse2) * e (v_fma_mix), bf16-packed and stored
//           non-temporally; once every store of the row is issued, the registers receive
//           the workgroup's next row (all loads issued back to back), so those loads are in
//           flight while this row's stores drain. Stores go first because the vector
//           memory counter retires in order: a load queued behind a store would make the
//           next row's first wait also wait for that store.
// With DB (two row buffers, for shapes whose registers allow it) the next row's loads go
// out as soon as this row has arrived, into the other buffer, before this row's stores;
// the next row's wait then leaves this row's NC stores outstanding (vmcnt(NC)), so a
// workgroup's next row streams in while its current row is reduced and stored (5-10 %
// faster for the shapes 512 x 4 .. 1024 x 8 on MI355X).
// ---------------------------------------------------------------------------------------
// With PH (rows that do not start on a 16-byte boundary, or whose length is not a whole number
// of chunks) a row is read as the aligned chunks that cover it, from the 16-byte boundary at
// or below its start: the first ph = (start / 2) % 8 entries of the first chunk belong to the
// row before, and the last chunk may run past the row's end (at most 7 entries, inside the
// 16-byte boundary after it). Those entries are read but count as -inf in the sums, and are
// never written: the first and last chunks of the gradient are stored entry by entry, so the
// neighbouring rows (other workgroups' dlogits, or their logits in place) are left alone.
// dlogits must then have the logits' phase on every row (the launcher checks it).
template <int NT, int NC, bool BWD, bool DB, bool PH>
__device__ __forceinline__ void resident_rows(const RowArgsOf<BWD>& a) {
  __shared__ float red[2][2 * (NT / 64)];   // alternated merge by merge: one barrier per merge
  __shared__ Bcast bc;
  // Per-chunk shifts n_c live in LDS (NC x NT floats, conflict-free [c][tid] layout): the
  // registers are reserved for the row itself.
  __shared__ float nch[BWD ? NC : 1][NT];
  const bool loss_mode = a.mode != kModeLogprob;
  const bool want_d = BWD && a.dlogits != nullptr;

  // A row is read unless it is a masked or bad-id row of the loss.
  auto reads = [&](int64_t rr) -> bool {
    if (!loss_mode) return true;
    if (a.mask != nullptr && uload_u8(a.mask + rr) == 0) return false;
    const int64_t yy = uload(a.ids + rr);
    return yy >= 0 && yy < a.V;
  };
  // The same decision in two halves (single-buffer kernels): the scalar loads it needs,
  // issued at the top of a row for the next one (rr clamped into the batch), then the
  // decision at the end of the row, when they have long arrived. A branch on a loaded value
  // makes the wave wait for every scalar load in flight, so nothing branches on these
  // before the end.
  struct RowMeta {
    uint32_t mword;   // the 32-bit word holding the mask byte (all ones without a mask)
    int64_t y;
  };
  auto meta_load = [&](int64_t rr) -> RowMeta {
    const int64_t q = rr < a.T ? rr : a.T - 1;
    RowMeta m;
    m.mword = (loss_mode && a.mask != nullptr)
                  ? uload((const uint32_t*)(((uintptr_t)a.mask + (uintptr_t)q) & ~(uintptr_t)3))
                  : 0xffffffffu;
    m.y = uload(a.ids + q);
    return m;
  };
  auto meta_reads = [&](int64_t rr, const RowMeta& m) -> bool {
    if (!loss_mode) return true;
    const uint32_t sh = 8u * (uint32_t)(((uintptr_t)a.mask + (uintptr_t)rr) & 3u);
    return ((m.mword >> sh) & 0xffu) != 0 && m.y >= 0 && m.y < a.V;
  };
  // Every load and store of the row goes through a buffer resource; a resource with
  // num_records = 0 turns an access into a no-op (loads read zeros, stores are dropped),
  // which keeps the chunk loops free of branches.
  // The resource over row rr's chunks (size 0 when rd is false); with PH it starts at the
  // 16-byte boundary at or below the row and covers the chunks the row touches.
  auto load_rsrc = [&](int64_t rr, bool rd) -> __amdgpu_buffer_rsrc_t {
    const uint16_t* p = row_ptr<uint16_t>(a, rd ? rr : 0);
    if constexpr (PH) {
      const int ph = (int)(((uintptr_t)p >> 1) & 7);
      return row_rsrc(p - ph, rd ? ((ph + a.V + 7) >> 3) * 16 : 0);
    } else {
      return row_rsrc(p, rd ? a.V * 2 : 0);
    }
  };
  uint32_t r1[NC][4];
  uint32_t r2[DB ? NC : 1][4];             // the second row buffer (DB)
  StatCount sc;                            // thread 0's counters over this workgroup's rows
  int64_t row = blockIdx.x;
  // the call's scale (token-mean: from the valid-token count, fixed while the kernel runs);
  // DB kernels take it after the first row's loads are issued (see below)
  const float scale_top = (!DB && loss_mode) ? row_scale(a) : 1.0f;
  // Stagger the start of the workgroups that share an XCD: workgroups are dealt to the
  // eight XCDs in turn, so blockIdx / 8 numbers them within their XCD. Started together,
  // they would load, compute and store in lockstep and leave the XCD's memory path idle
  // while they all compute; offsets of up to a third of a row's time keep it busy (1-4 %
  // faster on MI355X, the offset chosen per shape by the launcher).
  if (a.T >= 4 * (int64_t)gridDim.x) {
    const int steps = (int)((blockIdx.x >> 3) & 31) * a.stagger;
    for (int i = 0; i < steps; ++i) __builtin_amdgcn_s_sleep(6);
  }
  bool rd_cur = row < a.T && reads(row);
  {
    const __amdgpu_buffer_rsrc_t rz = load_rsrc(row, rd_cur);
#pragma unroll
    for (int c = 0; c < NC; ++c) load16<kAuxLast>(r1[c], rz, threadIdx.x * 16, c * NT * 16);
  }
  // In count mode the workgroup counts the mask here, its loads in flight together with the
  // first row's: one memory round trip for both, where a counting kernel before this one
  // costs a launch.
  const float scale = DB ? call_scale<NT>(a) : scale_top;
  // Without DB the token id of a row comes with the metadata loaded a row ahead of it.
  // It is waited for here: a load still in flight on entry would make the loop wait for every
  // scalar load at the top of every row.
  int64_t y_cur = 0;
  if constexpr (!DB) {
    y_cur = row < a.T ? uload(a.ids + row) : 0;
    asm volatile("" :: "s"(y_cur));
  }
  int parity = 0;
  // One row: its chunks are in r (cur); nx receives the next row's chunks (nx is r itself
  // without DB). `first`: nothing but this row's loads is outstanding.
  auto step = [&](uint32_t (&r)[NC][4], uint32_t (&nx)[NC][4], bool first) {
    // Start a row only once all of it has arrived, rather than consuming chunks as they
    // land: measured faster on MI355X, by 1-2 %, with the staggered starts and the reduced
    // grid described above. Without DB this also waits for the previous row's stores; with
    // DB at least NC stores of the previous row were issued after this row's loads.
    if (DB && want_d && !first) {
      asm volatile("s_waitcnt vmcnt(%0)" :: "n"(NC) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    const int tid = threadIdx.x;
    const int V = a.V;
    const int voff = tid * 16;
    const int nfull = V >> 3;               // 16-byte chunks of a row (V % 8 == 0 here)
    // Slots c < cb are inside the row for every thread, slot cb only for threads with
    // lane_in, slots above cb for none. Chunks outside the row read as zeros (buffer
    // range check) and are dropped from the sums and from the stores.
    const int cb = nfull / NT;
    const bool lane_in = tid < nfull - cb * NT;
    // PH: the row's phase; entry k of this thread's chunk in slot c lies inside the row iff
    // ph_lo(c) <= k < ph_hi(c).
    const int ph = PH ? (int)(((uintptr_t)row_ptr<uint16_t>(a, row) >> 1) & 7) : 0;
    auto ph_lo = [&](int c) { return ph - 8 * (c * NT + tid); };
    auto ph_hi = [&](int c) { return ph + V - 8 * (c * NT + tid); };

    const int64_t next = row + gridDim.x;
    // Without DB, the scalar loads are all issued here and waited for only where they are
    // used, after the merge: the mask word and id of the next row (whose loads follow pass
    // B), this row's token inputs and the word holding z[y] (its id came with the previous
    // row's metadata); waiting for them at the top of the row took several scalar round
    // trips per row (0.3 % of the large_vocab and long_agentic steps). DB issues the next
    // row's loads here and decides first whether it is read (the look-ahead measured 2 %
    // slower there).
    const RowMeta mt = DB ? RowMeta{0u, 0} : meta_load(next);
    bool rd_next = false;
    int64_t y = y_cur;
    if constexpr (DB) {
      rd_next = next < a.T && reads(next);
      const __amdgpu_buffer_rsrc_t rn = load_rsrc(rd_next ? next : row, rd_next);
#pragma unroll
      for (int c = 0; c < NC; ++c) load16<kAuxLast>(nx[c], rn, voff, c * NT * 16);
      y = uload(a.ids + row);
    }
    const TokenIn tin = token_inputs(a, row, scale);
    const bool good = (y >= 0) && (y < V) && version_ok(a, row);
    float w = 0.0f, dy = 0.0f, l2 = 0.0f;

    if (rd_cur) {
      // z[y] through the scalar unit (the aligned 32-bit word holding it; a bad id reads the
      // row's first word, unused), unpacked after the merge. The row's bytes are written,
      // in place, only by this workgroup and only after this read.
      const uintptr_t at = (uintptr_t)logits_of(a, row) + (uintptr_t)(row * a.ld + (good ? y : 0)) * 2u;
      const uint32_t zword = uload((const uint32_t*)(at & ~(uintptr_t)3));
      // Pass A.
      float N = -INFINITY, S = 0.0f;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        float x[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          x[2 * k] = bf16_lo(r[c][k]);
          x[2 * k + 1] = bf16_hi(r[c][k]);
        }
        if constexpr (PH) {                 // entries of the neighbouring rows
          const int lo = ph_lo(c), hi = ph_hi(c);
#pragma unroll
          for (int k = 0; k < 8; ++k) x[k] = (k >= lo && k < hi) ? x[k] : -INFINITY;
        }
        const float cm = max3(max3(x[0], x[1], x[2]), max3(x[3], x[4], x[5]), max3(x[6], x[7], x[7]));
        float nc = __builtin_ceilf(cm * kLog2e);
        const float sh = (nc == -INFINITY) ? 0.0f : nc;
        float e[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) e[j] = exp2_hw(__builtin_fmaf(x[j], kLog2e, -sh));
        float sc = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
        // a chunk outside the row contributes nothing
        const bool dead = PH ? ph_hi(c) <= 0 : ((c > cb) || (c == cb && !lane_in));
        nc = dead ? -INFINITY : nc;
        sc = dead ? 0.0f : sc;
        if (BWD) {
          // Pack here: left to itself the compiler sinks the packing to pass B and keeps
          // the fp32 exponentials of every chunk alive across the merge.
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            r[c][k] = pack_f16(e[2 * k], e[2 * k + 1]);
            asm volatile("" : "+v"(r[c][k]));
          }
          nch[c][tid] = nc;
        }
        merge_ns_int(N, S, nc, sc);
        // Keep chunk order: the loads were issued in the previous iteration, so the
        // scheduler would otherwise unpack every chunk at once.
        __builtin_amdgcn_sched_barrier(0);
      }
      float n = N;
      float s = S;
      block_merge_ns_int<NT>(n, s, red[parity]);
      parity ^= 1;                          // the buffers alternate between merges
      // An all -inf row has no finite shift: lse is NaN, as in IEEE max-shifted evaluation.
      const float lse2 = (n == -INFINITY) ? __builtin_nanf("") : n + log2f(s);
      const float zy = good ? ((at & 2u) ? bf16_hi(zword) : bf16_lo(zword)) : 0.0f;
      finish_row(a, row, zy, lse2, good, &bc, tin, sc);
      if (want_d) {
        __syncthreads();
        w = bc.w;
        dy = bc.dy;
        l2 = bc.lse2;
      }
    } else {                                // masked row, or a bad id on a valid row
      // Redefine the registers on this path too, so that both paths leave a fresh value
      // (otherwise the allocator keeps the row and its exponentials apart).
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int k = 0; k < 4; ++k) r[c][k] = 0u;
    }
    if (!rd_cur && tid == 0) {
      const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
      a.lp_out[row] = valid ? __builtin_nanf("") : 0.0f;
      a.loss_tok[row] = 0.0f;
      if (a.flags) a.flags[row] = valid ? (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID) : (uint8_t)0;
      if (valid) sc.bad += 1;
    }

    // Pass B: dlogits of this row, then the only place the registers are refilled: the
    // next row's chunks. For a row that was not read the dlogits stores are dropped and
    // zeros are written below.
    uint16_t* drow = want_d ? (uint16_t*)a.dlogits + row * a.ldd : nullptr;
    // PH: a resource from the 16-byte boundary at or below the row, over the chunks it
    // touches (dlogits has the logits' phase)
    uint16_t* dbase = PH ? drow - ph : drow;
    const int dbytes = PH ? ((ph + V + 7) >> 3) * 16 : V * 2;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(dbase, (want_d && rd_cur) ? dbytes : 0);
    const float wf = rd_cur ? w : 0.0f;
    // PH: chunk c is stored whole when it lies inside the row, else entry by entry
    auto store_chunk = [&](const u32x4& v, const __amdgpu_buffer_rsrc_t& res, int c) {
      if constexpr (PH) {
        const int lo = ph_lo(c), hi = ph_hi(c);
        if (lo <= 0 && hi >= 8) {
          buf_store16_nt(v, res, voff, c * NT * 16);
        } else {
#pragma unroll
          for (int k = 0; k < 8; ++k)
            if (k >= lo && k < hi)
              __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(v[k >> 1] >> (16 * (k & 1))), res,
                                                    voff + 2 * k, c * NT * 16, kAuxNT);
        }
      } else {
        buf_store16_nt(v, res, voff, c * NT * 16);
      }
    };
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (BWD) {
        // softmax(z)[v] = e_v * 2^(n_c - lse2); a chunk of -inf holds zeros; a NaN lse
        // (non-finite row) makes every element NaN, as 0 * NaN does.
        const float ncv = nch[c][tid];
        const float f = (l2 != l2) ? l2 : ((ncv == -INFINITY) ? 0.0f : wf * exp2_hw(ncv - l2));
        float o[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          o[2 * k] = f16_lo_mul(r[c][k], f);
          o[2 * k + 1] = f16_hi_mul(r[c][k], f);
        }
        // stores past the row fall outside the buffer range and are dropped
        u32x4 v;
        v.x = pack_bf16(o[0], o[1]);
        v.y = pack_bf16(o[2], o[3]);
        v.z = pack_bf16(o[4], o[5]);
        v.w = pack_bf16(o[6], o[7]);
        store_chunk(v, rd, c);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    // All of this row's stores are issued before any load of the next row: the vector
    // memory counter retires in order, and loads queued behind interleaved stores would
    // make every wait in the next row's pass A also wait for store acknowledgements.
    if constexpr (!DB) {
      rd_next = next < a.T && meta_reads(next, mt);
      const __amdgpu_buffer_rsrc_t rn = load_rsrc(rd_next ? next : row, rd_next);
#pragma unroll
      for (int c = 0; c < NC; ++c) load16<kAuxLast>(nx[c], rn, voff, c * NT * 16);
      y_cur = mt.y;
    }
    if (want_d && !rd_cur) {                // zeros for a row that was not read
      const __amdgpu_buffer_rsrc_t rz = row_rsrc(dbase, dbytes);
      const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int c = 0; c < NC; ++c) store_chunk(zero, rz, c);
    }
    // dlogits at v = y is w (p_y - 1) = w expm1(lp), computed once by thread 0. The thread
    // whose chunk holds y writes it over its own vector store above: two stores of one
    // thread to one address, through the same buffer path, land in program order.
    if (want_d && rd_cur && good && tid == (int)(((y + ph) >> 3) % NT))
      __builtin_amdgcn_raw_buffer_store_b16(to_bf16(dy), rd, (int)((y + ph) * 2), 0, kAuxNT);
    rd_cur = rd_next;
  };
  if constexpr (DB) {
    // unrolled twice, so that the buffers swap roles without register copies
    bool first = true;
    while (row < a.T) {
      step(r1, r2, first);
      first = false;
      row += gridDim.x;
      if (row >= a.T) break;
      step(r2, r1, false);
      row += gridDim.x;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the loads past the last row
  } else {
    for (; row < a.T; row += gridDim.x) step(r1, r1, false);
  }
  // count mode: loss_sum derives the counters from the flags
  if (threadIdx.x == 0 && !(DB && a.count_mode)) flush_stats(a, sc);
}

template <int NT, int NC, bool BWD>
__global__ __launch_bounds__(NT) void rows_bf16_resident(RowArgsOf<BWD> a) {
  resident_rows<NT, NC, BWD, false, false>(a);
}
// Rows with a phase (see resident_rows).
template <int NT, int NC, bool BWD>
__global__ __launch_bounds__(NT) void rows_bf16_phase(RowArgsOf<BWD> a) {
  resident_rows<NT, NC, BWD, false, true>(a);
}
// The two-buffer form, with dlogits (the backward kernel).
template <int NT, int NC>
__global__ __launch_bounds__(NT) void rows_bf16_resident_db(RowArgs a) {
  resident_rows<NT, NC, true, true, false>(a);
}
template <int NT, int NC>
__global__ __launch_bounds__(NT) void rows_bf16_phase_db(RowArgs a) {
  resident_rows<NT, NC, true, true, true>(a);
}

// ---------------------------------------------------------------------------------------
// Forward-only row kernel, bf16 logits (log-prob calls, versioned or not, and the loss
// without dlogits): persistent like rows_bf16_resident, NT threads x NC 16-byte chunks per
// row. With no backward sweep a chunk's registers are free as soon as the chunk has been
// unpacked, so the next row's chunk is loaded into them at once: the next row streams in
// while this row is summed, merged and finished, and the loop waits for memory only at its
// top. Rows that are not read (masked or bad-id loss rows) still run the chunk loop on
// zeros, so that every row issues its successor's loads from the same place.
// ---------------------------------------------------------------------------------------
// PH: rows with a phase, read as in resident_rows.
template <int NT, int NC, bool PH>
__device__ __forceinline__ void fwd_rows(const RowArgsV& a) {
  __shared__ float red[2][2 * (NT / 64)];
  __shared__ Bcast bc;
  const bool loss_mode = a.mode != kModeLogprob;
  auto load_rsrc = [&](int64_t rr, bool rd) -> __amdgpu_buffer_rsrc_t {
    const uint16_t* p = row_ptr<uint16_t>(a, rd ? rr : 0);
    if constexpr (PH) {
      const int ph = (int)(((uintptr_t)p >> 1) & 7);
      return row_rsrc(p - ph, rd ? ((ph + a.V + 7) >> 3) * 16 : 0);
    } else {
      return row_rsrc(p, rd ? a.V * 2 : 0);
    }
  };
  auto reads = [&](int64_t rr) -> bool {
    if (!loss_mode) return true;
    if (a.mask != nullptr && uload_u8(a.mask + rr) == 0) return false;
    const int64_t yy = uload(a.ids + rr);
    return yy >= 0 && yy < a.V;
  };
  uint32_t r[NC][4];
  StatCount sc;
  int64_t row = blockIdx.x;
  if (a.T >= 4 * (int64_t)gridDim.x) {      // staggered starts, as in rows_bf16_resident
    const int steps = (int)((blockIdx.x >> 3) & 31) * a.stagger;
    for (int i = 0; i < steps; ++i) __builtin_amdgcn_s_sleep(6);
  }
  // the call's scale (token-mean: from the valid-token count, fixed while the kernel runs)
  const float scale = loss_mode ? row_scale(a) : 1.0f;
  bool rd_cur = row < a.T && reads(row);
  {
    const __amdgpu_buffer_rsrc_t rz = load_rsrc(row, rd_cur);
#pragma unroll
    for (int c = 0; c < NC; ++c) load16<kAuxLast>(r[c], rz, threadIdx.x * 16, c * NT * 16);
  }
  int parity = 0;                          // flips after each merge that ran
  for (; row < a.T; row += gridDim.x) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const int tid = threadIdx.x;
    const int V = a.V;
    const int voff = tid * 16;
    const int nfull = V >> 3;
    const int cb = nfull / NT;
    const bool lane_in = tid < nfull - cb * NT;
    const int ph = PH ? (int)(((uintptr_t)row_ptr<uint16_t>(a, row) >> 1) & 7) : 0;
    const int64_t next = row + gridDim.x;
    const bool rd_next = next < a.T && reads(next);
    const __amdgpu_buffer_rsrc_t rn = load_rsrc(rd_next ? next : row, rd_next);
    const int64_t y = uload(a.ids + row);
    const bool good = (y >= 0) && (y < V) && version_ok(a, row);
    const TokenIn tin = token_inputs(a, row, scale);
    float zy = 0.0f;
    if (rd_cur && good) {
      const uintptr_t at = (uintptr_t)logits_of(a, row) + (uintptr_t)(row * a.ld + y) * 2u;
      const uint32_t wv = uload((const uint32_t*)(at & ~(uintptr_t)3));
      zy = (at & 2u) ? bf16_hi(wv) : bf16_lo(wv);
    }
    float N = -INFINITY, S = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float x[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        x[2 * k] = bf16_lo(r[c][k]);
        x[2 * k + 1] = bf16_hi(r[c][k]);
      }
      load16<kAuxLast>(r[c], rn, voff, c * NT * 16);
      const int lo = ph - 8 * (c * NT + tid), hi = ph + V - 8 * (c * NT + tid);
      if constexpr (PH) {                   // entries of the neighbouring rows
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = (k >= lo && k < hi) ? x[k] : -INFINITY;
      }
      const float cm = max3(max3(x[0], x[1], x[2]), max3(x[3], x[4], x[5]), max3(x[6], x[7], x[7]));
      float nc = __builtin_ceilf(cm * kLog2e);
      const float sh = (nc == -INFINITY) ? 0.0f : nc;
      // the same operations in the same order as rows_bf16_resident's pass A, so that the
      // forward-only and the gradient calls return bit-identical log-probs and losses
      float e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = exp2_hw(__builtin_fmaf(x[j], kLog2e, -sh));
      const float sc = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
      const bool dead = PH ? hi <= 0 : ((c > cb) || (c == cb && !lane_in));
      merge_ns_int(N, S, dead ? -INFINITY : nc, dead ? 0.0f : sc);
      // Pin the chunk's work here: otherwise the exponentials are sunk past the later
      // chunks and every chunk's unpacked values stay live at once.
      asm volatile("" : "+v"(N), "+v"(S));
      __builtin_amdgcn_sched_barrier(0);
    }
    if (rd_cur) {
      block_merge_ns_int<NT>(N, S, red[parity]);
      parity ^= 1;
      const float lse2 = (N == -INFINITY) ? __builtin_nanf("") : N + log2f(S);
      finish_row(a, row, zy, lse2, good, &bc, tin, sc);
    } else if (tid == 0) {                  // masked row, or a bad id on a valid loss row
      const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
      a.lp_out[row] = valid ? __builtin_nanf("") : 0.0f;
      a.loss_tok[row] = 0.0f;
      if (a.flags) a.flags[row] = valid ? (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID) : (uint8_t)0;
      if (valid) sc.bad += 1;
    }
    rd_cur = rd_next;
  }
  if (threadIdx.x == 0) flush_stats(a, sc);
}

template <int NT, int NC>
__global__ __launch_bounds__(NT) void rows_bf16_fwd(RowArgsV a) {
  fwd_rows<NT, NC, false>(a);
}
template <int NT, int NC>
__global__ __launch_bounds__(NT) void rows_bf16_fwd_phase(RowArgsV a) {
  fwd_rows<NT, NC, true>(a);
}

// ---------------------------------------------------------------------------------------
// Register-resident row kernel, fp32 logits (4 per 16-byte chunk; exps stored as fp32).
// ---------------------------------------------------------------------------------------
template <int NT, int NC, bool BWD>
__global__ __launch_bounds__(NT) void rows_f32_resident(RowArgsOf<BWD> a) {
  __shared__ float red[2 * (NT / 64) + 2];
  __shared__ Bcast bc;
  StatCount sc;
  const bool loss_mode = a.mode != kModeLogprob;
  // the call's scale (token-mean: from the valid-token count, fixed while the kernel runs)
  const float scale = call_scale<NT>(a);
  // one row; the merge's second barrier orders the LDS reuse between consecutive rows
  auto one = [&](const int64_t row) {
    const int tid = threadIdx.x;
    const int V = a.V;
    const int nfull = V >> 2;
    // Every scalar load of the row is issued before the first branch on any of them (a
    // branch on a loaded value waits for all scalar loads in flight), so they share one
    // round trip; the token inputs are used after the merge. With one row per workgroup
    // (a short batch) the chain of round trips was most of the kernel's time.
    const uint32_t mword =
        (loss_mode && a.mask != nullptr)
            ? uload((const uint32_t*)(((uintptr_t)a.mask + (uintptr_t)row) & ~(uintptr_t)3))
            : 0xffffffffu;
    const int64_t y = uload(a.ids + row);
    const TokenIn tin = token_inputs(a, row, scale);
    const bool valid = ((mword >> (8u * (uint32_t)(((uintptr_t)a.mask + (uintptr_t)row) & 3u))) & 0xffu) != 0;
    const bool good = (y >= 0) && (y < V) && version_ok(a, row);
    if (loss_mode && !(valid && good)) {
      skip_row_resident<NT, NC, 4>(a, row, valid, sc);
      return;
    }
    const float* zrow = row_ptr<float>(a, row);
    float zy = 0.0f;
    if (tid == 0 && good) zy = zrow[y];

    const __amdgpu_buffer_rsrc_t rz = row_rsrc(zrow, V * 4);
    const int voff = tid * 16;
    float r[NC][4];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const u32x4 v = buf_load16<kAuxLast>(rz, voff, c * NT * 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) r[c][j] = __uint_as_float(v[j]);
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if ((c + 1) * NT > nfull && c * NT + tid >= nfull) {
        r[c][0] = r[c][1] = r[c][2] = r[c][3] = -INFINITY;
      }
    }
    const int tail_slot = nfull / NT;
    const bool tail_owner = (V & 3) != 0 && tid == nfull % NT;
    if (tail_owner) {
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        if (c == tail_slot) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int e = nfull * 4 + j;
            if (e < V) r[c][j] = zrow[e];
          }
        }
      }
    }

    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      m = max3(m, r[c][0], r[c][1]);
      m = max3(m, r[c][2], r[c][3]);
    }
    const float n_shift = (m == -INFINITY) ? 0.0f : m * kLog2e;
    const float nb = -n_shift;
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float e[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) e[j] = exp2_hw(__builtin_fmaf(r[c][j], kLog2e, nb));
      s0 += e[0]; s1 += e[1]; s2 += e[2]; s3 += e[3];
      if (BWD) {
#pragma unroll
        for (int j = 0; j < 4; ++j) r[c][j] = e[j];
      }
    }
    float n = (m == -INFINITY) ? -INFINITY : n_shift;
    float s = (s0 + s1) + (s2 + s3);
    const float n_mine = n;
    block_merge_ns<NT>(n, s, red);
    const float lse2 = (n == -INFINITY) ? __builtin_nanf("") : n + log2f(s);

    finish_row(a, row, zy, lse2, good, &bc, tin, sc);
    if (!BWD || !a.dlogits) return;
    __syncthreads();
    const float w = bc.w;
    const float dy = bc.dy;
    const float f = row_factor(w, n_mine, bc.lse2);
    float* drow = (float*)a.dlogits + row * a.ldd;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, V * 4);
    const int cy = (int)(y >> 2);
    const int my_slot = (cy % NT == tid) ? cy / NT : -1;
    const int jy = (int)(y & 3);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int idx = c * NT + tid;
      float o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = r[c][j] * f;
      if (c == my_slot) {
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = (j == jy) ? dy : o[j];
      }
      if ((c + 1) * NT <= nfull || idx < nfull) {
        const u32x4 v = {__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                         __float_as_uint(o[3])};
        buf_store16_nt(v, rd, voff, c * NT * 16);
      } else if (tail_owner && c == tail_slot) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int e = nfull * 4 + j;
          if (e < V) drow[e] = o[j];
        }
      }
    }
  };
  for (int64_t row = blockIdx.x; row < a.T; row += gridDim.x) one(row);
  // in count mode the counters come from the flags (loss_sum)
  if (threadIdx.x == 0 && !a.count_mode) flush_stats(a, sc);
}

// ---------------------------------------------------------------------------------------
// Streaming row kernel: any V, any alignment. Pass A reads the row once for (n, s); pass
// B reads it again to write dlogits. Element e of the row is read and written by the same
// thread, so dlogits may alias the logits.
// ---------------------------------------------------------------------------------------
template <typename Tin>
__device__ __forceinline__ float load_elem(const Tin* p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_to_f32(p[i]);
}
template <typename Tin>
__device__ __forceinline__ void store_elem(Tin* p, int64_t i, float x);
template <>
__device__ __forceinline__ void store_elem<float>(float* p, int64_t i, float x) { p[i] = x; }
template <>
__device__ __forceinline__ void store_elem<uint16_t>(uint16_t* p, int64_t i, float x) {
  p[i] = to_bf16(x);
}

// E elements per chunk: 16-byte vectors when VEC, single elements otherwise.
template <typename Tin, bool VEC>
struct Chunk {
  static constexpr int E = VEC ? (int)(16 / sizeof(Tin)) : 1;
  __device__ static void load(const Tin* row, int idx, int V, float (&x)[E]) {
    if constexpr (VEC) {
      if ((idx + 1) * E <= V) {
        const u32x4 v = ((const u32x4*)row)[idx];
        if constexpr (sizeof(Tin) == 2) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            x[2 * k] = bf16_lo(v[k]);
            x[2 * k + 1] = bf16_hi(v[k]);
          }
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k) x[k] = __uint_as_float(v[k]);
        }
        return;
      }
    }
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int e = idx * E + j;
      x[j] = e < V ? load_elem<Tin>(row, e) : -INFINITY;
    }
  }
  __device__ static void store(Tin* row, int idx, int V, const float (&o)[E]) {
    if constexpr (VEC) {
      if ((idx + 1) * E <= V) {
        u32x4 v;
        if constexpr (sizeof(Tin) == 2) {
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = pack_bf16(o[2 * k], o[2 * k + 1]);
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k) v[k] = __float_as_uint(o[k]);
        }
        __builtin_nontemporal_store(v, ((u32x4*)row) + idx);
        return;
      }
    }
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int e = idx * E + j;
      if (e < V) store_elem<Tin>(row, e, o[j]);
    }
  }
};

template <typename Tin, int NT, bool BWD, bool VEC>
__global__ __launch_bounds__(NT) void rows_stream(RowArgsOf<BWD> a) {
  using C = Chunk<Tin, VEC>;
  constexpr int E = C::E;
  __shared__ float red[2 * (NT / 64) + 2];
  __shared__ Bcast bc;
  StatCount sc;
  const bool loss_mode = a.mode != kModeLogprob;
  // the call's scale (token-mean: from the valid-token count, fixed while the kernel runs)
  const float scale = loss_mode ? row_scale(a) : 1.0f;
  // one row; the merge's second barrier orders the LDS reuse between consecutive rows
  auto one = [&](const int64_t row) {
    const int tid = threadIdx.x;
    const int V = a.V;
    const int nchunk = (V + E - 1) / E;
    // the row's scalar loads, issued before the first branch on any of them (the token
    // inputs are used after the merge)
    const uint32_t mword =
        (loss_mode && a.mask != nullptr)
            ? uload((const uint32_t*)(((uintptr_t)a.mask + (uintptr_t)row) & ~(uintptr_t)3))
            : 0xffffffffu;
    const int64_t y = uload(a.ids + row);
    const TokenIn tin = token_inputs(a, row, scale);
    const bool valid = ((mword >> (8u * (uint32_t)(((uintptr_t)a.mask + (uintptr_t)row) & 3u))) & 0xffu) != 0;
    const bool good = (y >= 0) && (y < V) && version_ok(a, row);
    if (loss_mode && !(valid && good)) {
      skip_row<Tin, NT>(a, row, valid, sc);
      return;
    }
    const Tin* zrow = row_ptr<Tin>(a, row);
    float zy = 0.0f;
    if (tid == 0 && good) zy = load_elem<Tin>(zrow, y);

    float n = -INFINITY, s = 0.0f;
    for (int idx = tid; idx < nchunk; idx += NT) {
      float x[E];
      C::load(zrow, idx, V, x);
      float m = -INFINITY;
#pragma unroll
      for (int j = 0; j < E; ++j) m = fmaxf(m, x[j]);
      const float ns = (m == -INFINITY) ? 0.0f : m * kLog2e;
      float cs = 0.0f;
#pragma unroll
      for (int j = 0; j < E; ++j) cs += exp2_hw(__builtin_fmaf(x[j], kLog2e, -ns));
      merge_ns(n, s, (m == -INFINITY) ? -INFINITY : ns, cs);
    }
    block_merge_ns<NT>(n, s, red);
    const float lse2 = (n == -INFINITY) ? __builtin_nanf("") : n + log2f(s);

    finish_row(a, row, zy, lse2, good, &bc, tin, sc);
    if (!BWD || !a.dlogits) return;
    __syncthreads();
    const float w = bc.w;
    const float dy = bc.dy;
    const float nl = -bc.lse2;
    Tin* drow = (Tin*)a.dlogits + row * a.ldd;
    for (int idx = tid; idx < nchunk; idx += NT) {
      float x[E];
      C::load(zrow, idx, V, x);
      float o[E];
#pragma unroll
      for (int j = 0; j < E; ++j) {
        o[j] = w * exp2_hw(__builtin_fmaf(x[j], kLog2e, nl));
        if ((int64_t)idx * E + j == y) o[j] = dy;
      }
      C::store(drow, idx, V, o);
    }
  };
  for (int64_t row = blockIdx.x; row < a.T; row += gridDim.x) one(row);
  if (threadIdx.x == 0) flush_stats(a, sc);
}

// ---------------------------------------------------------------------------------------
// fp32 rows with dlogits that are longer than the register-resident kernels hold
// (V > 4 NT NC): the first NT x NC 16-byte chunks of a row stay in registers between the
// two passes, exponentials written back in place as in rows_f32_resident, the next 9 NT
// chunks of the row wait in LDS, and only the rest of the row (the tail past those) is read a
// second time. Per row: V elements read, V - 4 (NT NC + 9 NT) read again, V written, against
// 2 V read and V written by the streaming kernel. Persistent, one workgroup per row at a
// time.
// Pass A streams the tail eight chunks per thread at a time (chunks NT NC + tid, + NT, ...;
// the last may be partial), keeps the first ones in LDS, and merges each as a general (max,
// sum) partial, then loads the resident chunks and gives them one shift per thread, as the
// resident kernel does. Pass B scales the resident exponentials into dlogits, then takes the
// tail from LDS or reads it again. Element e of the row is read and written by the same
// thread, so dlogits may alias the logits.
// ---------------------------------------------------------------------------------------
template <typename Tin, int NT>
__device__ void skip_row_long(const RowArgs& a, int64_t row, bool valid, StatCount& sc) {
  using C = Chunk<Tin, true>;
  if (a.dlogits) {
    Tin* d = (Tin*)a.dlogits + row * a.ldd;
    const int nchunk = (a.V + C::E - 1) / C::E;
    float z[C::E];
#pragma unroll
    for (int j = 0; j < C::E; ++j) z[j] = 0.0f;
    for (int idx = threadIdx.x; idx < nchunk; idx += NT) C::store(d, idx, a.V, z);
  }
  if (threadIdx.x == 0) {
    a.lp_out[row] = valid ? __builtin_nanf("") : 0.0f;
    a.loss_tok[row] = 0.0f;
    if (a.flags) a.flags[row] = valid ? (uint8_t)(DPPO_FLAG_VALID | DPPO_FLAG_BAD_ID) : (uint8_t)0;
    if (valid) sc.bad += 1;
  }
}

template <int NT, int NC>
__global__ __launch_bounds__(NT) void rows_f32_prefix(RowArgs a) {
  constexpr int P = NT * NC;              // resident chunks of a row
  // Tail chunks per thread in flight: 8 was 1.5 % faster than 4 at T = 8192, V = 151936 (the
  // resident chunks are not live yet in pass A, and no longer in pass B); the bf16 prefix
  // kernel was 1 % slower with 8 and keeps 4.
  constexpr int U = 8;
  // The first KS of each thread's tail chunks are also kept in LDS between the passes (each
  // thread reads back only what it wrote), so that only the rest of the tail is read twice:
  // 2.2 % faster with 9 (144 KB) than with none at T = 8192, V = 151936. The second read
  // mostly hits the Infinity Cache, which is why the gain is far below the 10 % of traffic
  // it saves.
  constexpr int KS = kPrefixKeepF32;
  __shared__ float red[2 * (NT / 64) + 2];
  __shared__ Bcast bc;
  __shared__ u32x4 keep[KS * NT];
  StatCount sc;
  // the call's scale (token-mean: from the valid-token count, fixed while the kernel runs)
  const float scale = row_scale(a);
  for (int64_t row = blockIdx.x; row < a.T; row += gridDim.x) {
    const int tid = threadIdx.x;
    const int V = a.V;
    const int nfull = V >> 2;             // whole 16-byte chunks, > P by the selection
    const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
    const int64_t y = uload(a.ids + row);
    // issued with the row's other scalar loads, before the first branch on them; used after
    // the merge
    const TokenIn tin = token_inputs(a, row, scale);
    const bool good = (y >= 0) && (y < V);
    if (!(valid && good)) {               // uniform
      skip_row_long<float, NT>(a, row, valid, sc);
      continue;
    }
    const float* zrow = (const float*)a.logits + row * a.ld;
    float zy = 0.0f;
    if (tid == 0) zy = zrow[y];
    // Whole chunks through a resource over the row: a chunk past the end (offset kOff)
    // loads zeros, replaced by -inf below. The V % 4 last elements belong to one thread.
    const __amdgpu_buffer_rsrc_t rz = row_rsrc(zrow, nfull * 16);
    constexpr int kOff = 0x7fffff00;
    const bool rag_owner = (V & 3) != 0 && tid == nfull % NT;
    // pass A, tail first, so that its registers and the resident chunks are never live
    // together
    float nt = -INFINITY, st = 0.0f;
    for (int i0 = P + tid, s0 = 0; i0 < nfull; i0 += U * NT, s0 += U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = i0 + u * NT;
        // a chunk kept in LDS is read here for the last time (uniform condition)
        if (s0 + u < KS) v[u] = buf_load16<kAuxLast>(rz, idx < nfull ? idx * 16 : kOff, 0);
        else v[u] = buf_load16(rz, idx < nfull ? idx * 16 : kOff, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (s0 + u < KS) keep[(s0 + u) * NT + tid] = v[u];   // uniform condition
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = i0 + u * NT < nfull;
        float x[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = in ? __uint_as_float(v[u][j]) : -INFINITY;
        const float m = fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]));
        const float ns = (m == -INFINITY) ? 0.0f : m * kLog2e;
        float cs = 0.0f;
#pragma unroll
        for (int j = 0; j < 4; ++j) cs += exp2_hw(__builtin_fmaf(x[j], kLog2e, -ns));
        merge_ns(nt, st, (m == -INFINITY) ? -INFINITY : ns, cs);
      }
    }
    if (rag_owner) {
      for (int e = nfull * 4; e < V; ++e) {
        const float x = zrow[e];
        const float ns = (x == -INFINITY) ? 0.0f : x * kLog2e;
        merge_ns(nt, st, (x == -INFINITY) ? -INFINITY : ns, exp2_hw(__builtin_fmaf(x, kLog2e, -ns)));
      }
    }
    // pass A, resident chunks: one shift per thread, exponentials in place
    float r[NC][4];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const u32x4 v = buf_load16<kAuxLast>(rz, tid * 16, c * NT * 16);
#pragma unroll
      for (int j = 0; j < 4; ++j) r[c][j] = __uint_as_float(v[j]);
    }
    float m = -INFINITY;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      m = max3(m, r[c][0], r[c][1]);
      m = max3(m, r[c][2], r[c][3]);
    }
    const float n_shift = (m == -INFINITY) ? 0.0f : m * kLog2e;
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int j = 0; j < 4; ++j) r[c][j] = exp2_hw(__builtin_fmaf(r[c][j], kLog2e, -n_shift));
      s0 += r[c][0]; s1 += r[c][1]; s2 += r[c][2]; s3 += r[c][3];
    }
    const float n_mine = (m == -INFINITY) ? -INFINITY : n_shift;
    float n = n_mine;
    float s = (s0 + s1) + (s2 + s3);
    merge_ns(n, s, nt, st);
    block_merge_ns<NT>(n, s, red);
    const float lse2 = (n == -INFINITY) ? __builtin_nanf("") : n + log2f(s);
    finish_row(a, row, zy, lse2, good, &bc, tin, sc);
    if (!a.dlogits) continue;             // uniform
    __syncthreads();
    const float w = bc.w;
    const float dy = bc.dy;
    const float l2 = bc.lse2;
    const float f = row_factor(w, n_mine, l2);
    float* drow = (float*)a.dlogits + row * a.ldd;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, nfull * 16);
    // pass B, resident chunks (the sampled entry: the thread that holds it)
    const int cy = (int)(y >> 2);
    const int jy = (int)(y & 3);
    const int my_slot = (cy < P && cy % NT == tid) ? cy / NT : -1;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = (c == my_slot && j == jy) ? dy : r[c][j] * f;
      const u32x4 v = {__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                       __float_as_uint(o[3])};
      buf_store16_nt(v, rd, tid * 16, c * NT * 16);
    }
    // pass B, tail: from LDS or read again, scale, store (stores past the row are dropped)
    for (int i0 = P + tid, s0 = 0; i0 < nfull; i0 += U * NT, s0 += U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = i0 + u * NT;
        if (s0 + u < KS) v[u] = keep[(s0 + u) * NT + tid];     // uniform condition
        else v[u] = buf_load16<kAuxLast>(rz, idx < nfull ? idx * 16 : kOff, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = i0 + u * NT;
        float o[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          o[j] = w * exp2_hw(__builtin_fmaf(__uint_as_float(v[u][j]), kLog2e, -l2));
          o[j] = (idx == cy && j == jy) ? dy : o[j];
        }
        const u32x4 ov = {__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]),
                          __float_as_uint(o[3])};
        buf_store16_nt(ov, rd, idx < nfull ? idx * 16 : kOff, 0);
      }
    }
    if (rag_owner) {
      for (int e = nfull * 4; e < V; ++e)
        drow[e] = (e == y) ? dy : w * exp2_hw(__builtin_fmaf(zrow[e], kLog2e, -l2));
    }
  }
  if (threadIdx.x == 0) flush_stats(a, sc);
}

// ---------------------------------------------------------------------------------------
// bf16 rows with dlogits that are longer than the register-resident kernels hold
// (V > 8 NT NC): the first NT x NC 16-byte chunks of a row stay in registers between the two
// passes with the numerics of rows_bf16_resident (an integer log2 shift per chunk, kept in
// LDS, and the exponentials stored in place as fp16 pairs); the rest of the row (the tail)
// is read a second time and its gradient formed in fp32 from the logits. Per row: V elements
// read, V - 8 NT NC read again, V written, against 2 V read and V written by the streaming
// kernel. Persistent, one workgroup per row at a time; pass A streams the tail first, so
// that its registers and the resident chunks are never live together. Element e of the row
// is read and written by the same thread, so dlogits may alias the logits.
// ---------------------------------------------------------------------------------------
template <int NT, int NC>
__global__ __launch_bounds__(NT) void rows_bf16_prefix(RowArgs a) {
  constexpr int P = NT * NC;              // resident chunks of a row
  constexpr int U = 4;                    // tail chunks per thread in flight
  // the first KS of each thread's tail chunks also wait in LDS between the passes (each
  // thread reads back only what it wrote), beside the shift table
  constexpr int KS = kPrefixKeepBf16;
  __shared__ float red[2 * (NT / 64) + 2];
  __shared__ Bcast bc;
  __shared__ float nch[NC][NT];           // per-chunk shifts, [c][tid]: conflict-free
  __shared__ u32x4 keep[KS * NT];
  StatCount sc;
  // the call's scale (token-mean: from the valid-token count, fixed while the kernel runs)
  const float scale = row_scale(a);
  for (int64_t row = blockIdx.x; row < a.T; row += gridDim.x) {
    const int tid = threadIdx.x;
    const int V = a.V;
    const int nfull = V >> 3;             // whole 16-byte chunks, >= P by the selection
    const bool valid = a.mask == nullptr || uload_u8(a.mask + row) != 0;
    const int64_t y = uload(a.ids + row);
    // issued with the row's other scalar loads, before the first branch on them; used after
    // the merge
    const TokenIn tin = token_inputs(a, row, scale);
    const bool good = (y >= 0) && (y < V);
    if (!(valid && good)) {               // uniform
      skip_row_long<uint16_t, NT>(a, row, valid, sc);
      continue;
    }
    const uint16_t* zrow = (const uint16_t*)a.logits + row * a.ld;
    float zy = 0.0f;
    if (tid == 0) zy = bf16_to_f32(zrow[y]);
    // Whole chunks through a resource over the row: a chunk past the end (offset kOff)
    // loads zeros, replaced by -inf below. The V % 8 last elements belong to one thread.
    const __amdgpu_buffer_rsrc_t rz = row_rsrc(zrow, nfull * 16);
    constexpr int kOff = 0x7fffff00;
    const bool rag_owner = (V & 7) != 0 && tid == nfull % NT;
    // pass A, tail: general (max, sum) partials per chunk
    float nt = -INFINITY, st = 0.0f;
    for (int i0 = P + tid, s0 = 0; i0 < nfull; i0 += U * NT, s0 += U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = i0 + u * NT;
        // a chunk kept in LDS is read here for the last time (uniform condition)
        if (s0 + u < KS) v[u] = buf_load16<kAuxLast>(rz, idx < nfull ? idx * 16 : kOff, 0);
        else v[u] = buf_load16(rz, idx < nfull ? idx * 16 : kOff, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (s0 + u < KS) keep[(s0 + u) * NT + tid] = v[u];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = i0 + u * NT < nfull;
        float x[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          x[2 * k] = in ? bf16_lo(v[u][k]) : -INFINITY;
          x[2 * k + 1] = in ? bf16_hi(v[u][k]) : -INFINITY;
        }
        const float m = max3(max3(x[0], x[1], x[2]), max3(x[3], x[4], x[5]), max3(x[6], x[7], x[7]));
        const float ns = (m == -INFINITY) ? 0.0f : m * kLog2e;
        float cs = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) cs += exp2_hw(__builtin_fmaf(x[j], kLog2e, -ns));
        merge_ns(nt, st, (m == -INFINITY) ? -INFINITY : ns, cs);
      }
    }
    if (rag_owner) {
      for (int e = nfull * 8; e < V; ++e) {
        const float x = bf16_to_f32(zrow[e]);
        const float ns = (x == -INFINITY) ? 0.0f : x * kLog2e;
        merge_ns(nt, st, (x == -INFINITY) ? -INFINITY : ns, exp2_hw(__builtin_fmaf(x, kLog2e, -ns)));
      }
    }
    // pass A, resident chunks: shift n_c = ceil(L max(chunk)), fp16 exponentials in place
    uint32_t r[NC][4];
#pragma unroll
    for (int c = 0; c < NC; ++c) load16<kAuxLast>(r[c], rz, tid * 16, c * NT * 16);
    float N = -INFINITY, S = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      float x[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        x[2 * k] = bf16_lo(r[c][k]);
        x[2 * k + 1] = bf16_hi(r[c][k]);
      }
      const float cm = max3(max3(x[0], x[1], x[2]), max3(x[3], x[4], x[5]), max3(x[6], x[7], x[7]));
      const float nc = __builtin_ceilf(cm * kLog2e);
      const float sh = (nc == -INFINITY) ? 0.0f : nc;
      float e[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = exp2_hw(__builtin_fmaf(x[j], kLog2e, -sh));
      const float cs = ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        r[c][k] = pack_f16(e[2 * k], e[2 * k + 1]);
        asm volatile("" : "+v"(r[c][k]));
      }
      nch[c][tid] = nc;
      merge_ns_int(N, S, nc, cs);
      __builtin_amdgcn_sched_barrier(0);
    }
    merge_ns(N, S, nt, st);
    block_merge_ns<NT>(N, S, red);
    const float lse2 = (N == -INFINITY) ? __builtin_nanf("") : N + log2f(S);
    finish_row(a, row, zy, lse2, good, &bc, tin, sc);
    if (!a.dlogits) continue;             // uniform
    __syncthreads();
    const float w = bc.w;
    const float dy = bc.dy;
    const float l2 = bc.lse2;
    uint16_t* drow = (uint16_t*)a.dlogits + row * a.ldd;
    const __amdgpu_buffer_rsrc_t rd = row_rsrc(drow, nfull * 16);
    // pass B, resident chunks: w 2^(n_c - lse2) e (the sampled entry: the thread that holds
    // it); a NaN lse (non-finite row) makes every element NaN
    const int cy = (int)(y >> 3);
    const int jy = (int)(y & 7);
    const int my_slot = (cy < P && cy % NT == tid) ? cy / NT : -1;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float ncv = nch[c][tid];
      const float f = (l2 != l2) ? l2 : ((ncv == -INFINITY) ? 0.0f : w * exp2_hw(ncv - l2));
      float o[8];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        o[2 * k] = f16_lo_mul(r[c][k], f);
        o[2 * k + 1] = f16_hi_mul(r[c][k], f);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (c == my_slot && j == jy) ? dy : o[j];
      u32x4 v;
      v.x = pack_bf16(o[0], o[1]);
      v.y = pack_bf16(o[2], o[3]);
      v.z = pack_bf16(o[4], o[5]);
      v.w = pack_bf16(o[6], o[7]);
      buf_store16_nt(v, rd, tid * 16, c * NT * 16);
    }
    // pass B, tail: re-read, w 2^(z L - lse2), store (stores past the row are dropped)
    for (int i0 = P + tid, s0 = 0; i0 < nfull; i0 += U * NT, s0 += U) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = i0 + u * NT;
        if (s0 + u < KS) v[u] = keep[(s0 + u) * NT + tid];
        else v[u] = buf_load16<kAuxLast>(rz, idx < nfull ? idx * 16 : kOff, 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int idx = i0 + u * NT;
        float o[8];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          o[2 * k] = w * exp2_hw(__builtin_fmaf(bf16_lo(v[u][k]), kLog2e, -l2));
          o[2 * k + 1] = w * exp2_hw(__builtin_fmaf(bf16_hi(v[u][k]), kLog2e, -l2));
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = (idx == cy && j == jy) ? dy : o[j];
        u32x4 ov;
        ov.x = pack_bf16(o[0], o[1]);
        ov.y = pack_bf16(o[2], o[3]);
        ov.z = pack_bf16(o[4], o[5]);
        ov.w = pack_bf16(o[6], o[7]);
        buf_store16_nt(ov, rd, idx < nfull ? idx * 16 : kOff, 0);
      }
    }
    if (rag_owner) {
      for (int e = nfull * 8; e < V; ++e)
        drow[e] = to_bf16((e == y) ? dy : w * exp2_hw(__builtin_fmaf(bf16_to_f32(zrow[e]), kLog2e, -l2)));
    }
  }
  if (threadIdx.x == 0) flush_stats(a, sc);
}

// ---------------------------------------------------------------------------------------
// Valid-token count (prepares stats for the token-mean scale) and the loss sum.
// ---------------------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void prep_stats(const uint8_t* mask, int64_t T, int32_t* stats) {
  __shared__ int part[16];
  int cnt = 0;
  if (mask) {
    for (int64_t i = threadIdx.x; i < T; i += 1024) cnt += mask[i] != 0;
  } else if (threadIdx.x == 0) {
    cnt = (int)T;
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) cnt += __shfl_xor(cnt, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int tot = 0;
    for (int i = 0; i < 16; ++i) tot += part[i];
    stats[DPPO_STAT_N_VALID] = tot;
    stats[DPPO_STAT_N_BAND] = 0;
    stats[DPPO_STAT_N_PPO] = 0;
    stats[DPPO_STAT_N_ACTIVE] = 0;
    stats[DPPO_STAT_N_BAD] = 0;
  }
}

// L = sum_t m_t s_t l_t in float64, each thread over a fixed stride, then a fixed tree:
// the same inputs give the same bits on every run.
template <bool HAS_MASK, bool HAS_TSCALE>
// With flags (count mode), the counters are derived from them as well: n_valid, n_band,
// n_ppo, n_active (PPO-active, and in the band when rd_mode masks by it) and n_bad.
__global__ __launch_bounds__(1024) void loss_sum(const float* loss_tok, const uint8_t* mask,
                                                 const float* tscale, int32_t* stats,
                                                 int64_t T, float loss_scale, int32_t scale_mode,
                                                 float* loss_out, const uint8_t* flags,
                                                 int32_t rd_mode) {
  __shared__ double part[16];
  __shared__ int cpart[16][5];
  float scale = loss_scale;
  if (scale_mode == DPPO_SCALE_TOKEN_MEAN) {
    const int n = stats[DPPO_STAT_N_VALID];
    scale = loss_scale / (float)(n > 1 ? n : 1);
  }
  const bool uses_band = rd_mode == DPPO_RD_MASK || rd_mode == DPPO_RD_MASK_WEIGHT;
  // Thread k adds tokens k, k + 1024, k + 2048, ... in that order; the loads of 16 of them
  // are issued together so that their latencies overlap.
  constexpr int U = 16;
  double acc = 0.0;
  int c[5] = {0, 0, 0, 0, 0};
  for (int64_t base = threadIdx.x; base < T; base += 1024 * U) {
    float lt[U], ts[U];
    bool on[U];
    uint32_t fl[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + (int64_t)u * 1024;
      const int64_t j = i < T ? i : T - 1;   // in bounds (T >= 1 here): loads without branches
      lt[u] = loss_tok[j];
      ts[u] = HAS_TSCALE ? tscale[j] : 1.0f;
      on[u] = (i < T) & ((HAS_MASK ? mask[j] : (uint8_t)1) != 0);
      fl[u] = (flags != nullptr && i < T) ? flags[j] : 0u;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (on[u]) acc += (double)(scale * ts[u]) * (double)lt[u];
      const bool band = fl[u] & DPPO_FLAG_BAND, ppo = fl[u] & DPPO_FLAG_PPO;
      c[DPPO_STAT_N_VALID] += (fl[u] & DPPO_FLAG_VALID) != 0;
      c[DPPO_STAT_N_BAND] += band;
      c[DPPO_STAT_N_PPO] += ppo;
      c[DPPO_STAT_N_ACTIVE] += ppo && (band || !uses_band);
      c[DPPO_STAT_N_BAD] += (fl[u] & DPPO_FLAG_BAD_ID) != 0;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
#pragma unroll
  for (int k = 0; k < 5; ++k)
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) c[k] += __shfl_xor(c[k], off, 64);
  if ((threadIdx.x & 63) == 0) {
    part[threadIdx.x >> 6] = acc;
#pragma unroll
    for (int k = 0; k < 5; ++k) cpart[threadIdx.x >> 6][k] = c[k];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double tot = 0.0;
    for (int i = 0; i < 16; ++i) tot += part[i];
    loss_out[0] = (float)tot;
    if (flags != nullptr) {
      for (int k = 0; k < 5; ++k) {
        int n = 0;
        for (int i = 0; i < 16; ++i) n += cpart[i][k];
        stats[k] = n;
      }
    }
  }
}

// ---------------------------------------------------------------------------------------
// Kernel selection.
// ---------------------------------------------------------------------------------------
namespace {
struct ResCfg {
  int nt, nc;
};
// Resident shapes, by capacity in 16-byte chunks (NT * NC).
constexpr ResCfg kResident[] = {{256, 1},  {256, 2},   {256, 4},   {512, 4},   {512, 6},
                                {512, 8},  {1024, 6}, {1024, 8}, {1024, 12}, {1024, 19}};
constexpr int kNumResident = sizeof(kResident) / sizeof(kResident[0]);
// Per-shape launch choices, each from same-box A/B timings at T = 16384 (MI355X):
//  * bf16 backward with two row buffers: 5-10 % faster for 512 x 4 .. 1024 x 8; within
//    +-4 % (either way) for the 256-thread shapes and 1024 x 12; 1024 x 19 has no registers
//    for a second row;
//  * fp32 persistent (a loop over rows, counters flushed once per workgroup) rather than one
//    workgroup per row: 2-6x faster up to 512 x 8 and 6 % at 1024 x 19, 0-7 % slower for
//    1024 x 6 .. 1024 x 12.
constexpr bool kResidentDB[kNumResident] = {false, false, false, true, true,
                                            true,  true,  true,  false, false};
constexpr bool kF32Persistent[kNumResident] = {true,  true,  true,  true,  true,
                                               true,  false, false, false, true};
// Persistent grids launch kFill* of every 32 resident workgroup slots. A gradient kernel
// moves fewer bytes per second with every CU streaming than with a few CUs of each XCD
// idle; the read-only forward kernels mostly want every slot. Same-box A/B at T = 16384 over
// fills of 24 to 32, per kernel and shape (the shapes not listed as measured take a measured
// neighbour's value): the flagship (bf16 backward 1024 x 19) is fastest at 27 (29-32: 2-3 %
// slower, 25: 3 %); the forward kernel at 32 for 512 x 4 .. 1024 x 8 (7-13 % faster than
// 27) and 30 for 1024 x 12 and 19 (6 %, 3 %); the long-row prefix kernels at 31 (bf16, 6 %)
// and 32 (fp32, 2 %). The bf16 backward 512 x 8 shape is set for the small_vocab batch
// (T = 4096, count mode): 31 gives a 1.4-1.7 % shorter step than 29 (27: 1.6 % longer, 30:
// 0.6 % shorter, 32: 0.3 % shorter; same-process runs), the same time at
// T = 16384, 0.3-0.5 % less at T = 8192 and 1-2 % more at T = 2048.
// Shapes:                                   256x1 256x2 256x4 512x4 512x6 512x8 1Kx6 1Kx8 1Kx12 1Kx19
constexpr int kFillBf16Bwd[kNumResident] = {27,   27,   27,   32,   29,   31,   27,  27,  29,   27};
constexpr int kFillBf16Fwd[kNumResident] = {30,   30,   30,   32,   32,   32,   32,  32,  30,   30};
constexpr int kFillF32Bwd[kNumResident] = {27,    27,   27,   30,   30,   30,   27,  27,  27,   25};
constexpr int kFillF32Fwd[kNumResident] = {27,    27,   27,   32,   32,   32,   27,  27,  27,   32};
// Measured: bf16 backward from 256 x 4 up; bf16 forward all but 256 x 2; fp32 backward
// 512 x 4, 512 x 8 and 1024 x 19; fp32 forward 512 x 4 and 1024 x 19. fp32 backward
// 1024 x 6 .. 12 run one workgroup per row (kF32Persistent), so their fill is unused.
constexpr int kFillF32Prefix = 32;
constexpr int kFillBf16Prefix = 31;
// Start stagger of the persistent bf16 kernels (RowArgs::stagger: s_sleep(6) units per
// XCD-local workgroup index, up to 31 indices): longer rows want longer offsets. Same-box
// sweeps of 0 to 6: the flagship is fastest at 4 (0.5 % faster than 2), 512 x 4 backward and
// 512 x 8 forward at 0 (4 %), the small_vocab shape (512 x 8 backward, T = 4096) at 1 (1 %);
// 1024 x 8 and 1024 x 12 backward are flat from 1 to 4.
// Shapes:                                   256x1 256x2 256x4 512x4 512x6 512x8 1Kx6 1Kx8 1Kx12 1Kx19
constexpr int kStagBf16Bwd[kNumResident] = {0,    0,    0,    0,    1,    1,    2,   2,   2,    4};
constexpr int kStagBf16Fwd[kNumResident] = {0,    0,    0,    0,    0,    0,    1,   1,   2,    2};

const void* pick_bf16_fwd(int i) {
  switch (i) {
    case 0: return (const void*)rows_bf16_fwd<256, 1>;
    case 1: return (const void*)rows_bf16_fwd<256, 2>;
    case 2: return (const void*)rows_bf16_fwd<256, 4>;
    case 3: return (const void*)rows_bf16_fwd<512, 4>;
    case 4: return (const void*)rows_bf16_fwd<512, 6>;
    case 5: return (const void*)rows_bf16_fwd<512, 8>;
    case 6: return (const void*)rows_bf16_fwd<1024, 6>;
    case 7: return (const void*)rows_bf16_fwd<1024, 8>;
    case 8: return (const void*)rows_bf16_fwd<1024, 12>;
    default: return (const void*)rows_bf16_fwd<1024, 19>;
  }
}
const void* pick_bf16_fwd_phase(int i) {
  switch (i) {
    case 0: return (const void*)rows_bf16_fwd_phase<256, 1>;
    case 1: return (const void*)rows_bf16_fwd_phase<256, 2>;
    case 2: return (const void*)rows_bf16_fwd_phase<256, 4>;
    case 3: return (const void*)rows_bf16_fwd_phase<512, 4>;
    case 4: return (const void*)rows_bf16_fwd_phase<512, 6>;
    case 5: return (const void*)rows_bf16_fwd_phase<512, 8>;
    case 6: return (const void*)rows_bf16_fwd_phase<1024, 6>;
    case 7: return (const void*)rows_bf16_fwd_phase<1024, 8>;
    case 8: return (const void*)rows_bf16_fwd_phase<1024, 12>;
    default: return (const void*)rows_bf16_fwd_phase<1024, 19>;
  }
}
const void* pick_bf16_phase_db(int i) {
  switch (i) {
    case 3: return (const void*)rows_bf16_phase_db<512, 4>;
    case 4: return (const void*)rows_bf16_phase_db<512, 6>;
    case 5: return (const void*)rows_bf16_phase_db<512, 8>;
    case 6: return (const void*)rows_bf16_phase_db<1024, 6>;
    case 7: return (const void*)rows_bf16_phase_db<1024, 8>;
    default: return nullptr;
  }
}
template <bool BWD>
const void* pick_bf16_phase(int i) {
  switch (i) {
    case 0: return (const void*)rows_bf16_phase<256, 1, BWD>;
    case 1: return (const void*)rows_bf16_phase<256, 2, BWD>;
    case 2: return (const void*)rows_bf16_phase<256, 4, BWD>;
    case 3: return (const void*)rows_bf16_phase<512, 4, BWD>;
    case 4: return (const void*)rows_bf16_phase<512, 6, BWD>;
    case 5: return (const void*)rows_bf16_phase<512, 8, BWD>;
    case 6: return (const void*)rows_bf16_phase<1024, 6, BWD>;
    case 7: return (const void*)rows_bf16_phase<1024, 8, BWD>;
    case 8: return (const void*)rows_bf16_phase<1024, 12, BWD>;
    default: return (const void*)rows_bf16_phase<1024, 19, BWD>;
  }
}
// Two-buffer backward kernels, for the shapes kResidentDB selects.
const void* pick_bf16_db(int i) {
  switch (i) {
    case 3: return (const void*)rows_bf16_resident_db<512, 4>;
    case 4: return (const void*)rows_bf16_resident_db<512, 6>;
    case 5: return (const void*)rows_bf16_resident_db<512, 8>;
    case 6: return (const void*)rows_bf16_resident_db<1024, 6>;
    case 7: return (const void*)rows_bf16_resident_db<1024, 8>;
    default: return nullptr;
  }
}
template <bool BWD>
const void* pick_bf16(int i) {
  switch (i) {
    case 0: return (const void*)rows_bf16_resident<256, 1, BWD>;
    case 1: return (const void*)rows_bf16_resident<256, 2, BWD>;
    case 2: return (const void*)rows_bf16_resident<256, 4, BWD>;
    case 3: return (const void*)rows_bf16_resident<512, 4, BWD>;
    case 4: return (const void*)rows_bf16_resident<512, 6, BWD>;
    case 5: return (const void*)rows_bf16_resident<512, 8, BWD>;
    case 6: return (const void*)rows_bf16_resident<1024, 6, BWD>;
    case 7: return (const void*)rows_bf16_resident<1024, 8, BWD>;
    case 8: return (const void*)rows_bf16_resident<1024, 12, BWD>;
    default: return (const void*)rows_bf16_resident<1024, 19, BWD>;
  }
}
template <bool BWD>
const void* pick_f32(int i) {
  switch (i) {
    case 0: return (const void*)rows_f32_resident<256, 1, BWD>;
    case 1: return (const void*)rows_f32_resident<256, 2, BWD>;
    case 2: return (const void*)rows_f32_resident<256, 4, BWD>;
    case 3: return (const void*)rows_f32_resident<512, 4, BWD>;
    case 4: return (const void*)rows_f32_resident<512, 6, BWD>;
    case 5: return (const void*)rows_f32_resident<512, 8, BWD>;
    case 6: return (const void*)rows_f32_resident<1024, 6, BWD>;
    case 7: return (const void*)rows_f32_resident<1024, 8, BWD>;
    case 8: return (const void*)rows_f32_resident<1024, 12, BWD>;
    default: return (const void*)rows_f32_resident<1024, 19, BWD>;
  }
}
}  // namespace

RowLaunch select_row_kernel(int32_t dtype, int64_t V, bool aligned, bool bwd, int force,
                            bool phase_ok) {
  RowLaunch L;
  L.bwd = bwd;
  const int esize = dtype == DPPO_BF16 ? 2 : 4;
  int64_t chunks = (V * esize + 15) / 16;
  int pick = -1;
  const bool whole_chunks = (V * esize) % 16 == 0;
  // a row with a phase touches at most ceil((V + 7) / 8) chunks (ceil(V / 8) when every row
  // starts on a 16-byte boundary)
  const bool ph = !(aligned && whole_chunks) && dtype == DPPO_BF16 && phase_ok;
  if (ph && !aligned) chunks = (V + 14) / 8;
  // fp32 rows on an aligned stride may end in a partial chunk: rows_f32_resident loads and
  // stores its last V % 4 entries one by one
  const bool f32_ragged = dtype == DPPO_F32 && aligned && !whole_chunks;
  if (((aligned && whole_chunks) || ph || f32_ragged) && !(force & kForceStream)) {
    for (int i = 0; i < kNumResident; ++i) {
      if ((int64_t)kResident[i].nt * kResident[i].nc >= chunks) {
        pick = i;
        break;
      }
    }
  }
  if (pick >= 0) {
    L.threads = kResident[pick].nt;
    L.chunks = kResident[pick].nc;
    L.phase = ph;
    if (dtype == DPPO_BF16 && ph)
      L.fn = bwd ? (kResidentDB[pick] ? pick_bf16_phase_db(pick) : pick_bf16_phase<true>(pick))
                 : pick_bf16_fwd_phase(pick);
    else
      L.fn = dtype == DPPO_BF16
                 ? (bwd ? (kResidentDB[pick] ? pick_bf16_db(pick) : pick_bf16<true>(pick))
                        : pick_bf16_fwd(pick))
                 : (bwd ? pick_f32<true>(pick) : pick_f32<false>(pick));
    L.two_buffers = dtype == DPPO_BF16 && bwd && kResidentDB[pick];
    // the fp32 resident kernel and the bf16 two-buffer kernels can count the valid tokens
    // themselves (count mode)
    L.counts = dtype == DPPO_F32 || L.two_buffers;
    L.resident = true;
    // fp32 forward rows loop persistently at every shape: 0-2.5 % faster than one workgroup
    // per row for 1024 x 6 .. 12 (the gradient kernel there is 0-6 % slower persistent)
    L.persistent = dtype == DPPO_BF16 || kF32Persistent[pick] || !bwd;
    L.fill = dtype == DPPO_BF16 ? (bwd ? kFillBf16Bwd[pick] : kFillBf16Fwd[pick])
                                : (bwd ? kFillF32Bwd[pick] : kFillF32Fwd[pick]);
    L.stagger = dtype == DPPO_BF16 ? (bwd ? kStagBf16Bwd[pick] : kStagBf16Fwd[pick]) : 0;
    return L;
  }
  L.threads = 1024;
  L.resident = false;
  if (bwd && aligned && !(force & kForceStream) && (V * esize) / 16 >= (int64_t)1024 * kPrefixNC) {
    // longer rows: a resident prefix of 1024 x kPrefixNC whole chunks, the rest (and a
    // ragged end) streamed twice
    L.fn = dtype == DPPO_F32 ? (const void*)rows_f32_prefix<1024, kPrefixNC>
                             : (const void*)rows_bf16_prefix<1024, kPrefixNC>;
    L.chunks = kPrefixNC;
    L.prefix = true;
    L.persistent = true;
    L.fill = dtype == DPPO_F32 ? kFillF32Prefix : kFillBf16Prefix;
    return L;
  }
  if (dtype == DPPO_BF16) {
    L.fn = aligned ? (bwd ? (const void*)rows_stream<uint16_t, 1024, true, true>
                          : (const void*)rows_stream<uint16_t, 1024, false, true>)
                   : (bwd ? (const void*)rows_stream<uint16_t, 1024, true, false>
                          : (const void*)rows_stream<uint16_t, 1024, false, false>);
  } else {
    L.fn = aligned ? (bwd ? (const void*)rows_stream<float, 1024, true, true>
                          : (const void*)rows_stream<float, 1024, false, true>)
                   : (bwd ? (const void*)rows_stream<float, 1024, true, false>
                          : (const void*)rows_stream<float, 1024, false, false>);
  }
  return L;
}

void launch_prep_stats(const uint8_t* mask, int64_t T, int32_t* stats, hipStream_t st) {
  prep_stats<<<1, 1024, 0, st>>>(mask, T, stats);
}

void launch_loss_sum(const float* loss_tok, const uint8_t* mask, const float* tscale,
                     int32_t* stats, int64_t T, float loss_scale, int32_t scale_mode,
                     float* loss_out, hipStream_t st, const uint8_t* flags, int32_t rd_mode) {
  auto k = mask ? (tscale ? loss_sum<true, true> : loss_sum<true, false>)
                : (tscale ? loss_sum<false, true> : loss_sum<false, false>);
  k<<<1, 1024, 0, st>>>(loss_tok, mask, tscale, stats, T, loss_scale, scale_mode, loss_out,
                        flags, rd_mode);
}

}  // namespace dppo
