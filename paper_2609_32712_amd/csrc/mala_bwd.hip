// MALA backward (Algorithm 2) for gfx950, as two kernels that use the same tile
// decisions.
//
// mala_bwd_dq_kernel (query-major, like the forward) runs first and takes every
// tile decision: one workgroup = 8 wavefronts = 256 query rows; K and V stream
// through double-buffered LDS one 128-key block at a time (four decision tiles per
// wavefront between barriers, which evens out the work of wavefronts that retain
// different numbers of tiles).  It computes the transposed products (S^T = K Q^T,
// dP^T = V dO^T, dQ^T += K^T dS^T), so that a lane holds one query row and dS feeds
// the dQ MFMA straight from registers.  It records its decisions, one byte per
// (query tile, query head, 128-key block), for the key-major kernel.  dQ needs no
// atomics and is bitwise reproducible.
//   S^T = K_w Q_i^T       8 MFMAs per 32 x 32 tile
//   offline test          retain iff some valid entry has
//                         s - lse_q >= log2(tau) - log2(L_q) (base-2 units); ballot
//   retained path         P = exp2(S - lse); dP^T = V dO^T; dS = P (dP - D_q);
//                         dQ^T += K^T dS^T
// mala_bwd_dkdv_kernel (key-major, Algorithm 2's traversal): one workgroup owns 128
// keys of one (batch, KV head) and keeps their dK and dV in registers (no atomics,
// bitwise reproducible); it sweeps the query tiles of every query head of the GQA
// group from the end down to the diagonal, stepping only through the query tiles
// that the dQ kernel retained for some of its four key tiles.  Sixteen wavefronts,
// four roles per 32 keys on one SIMD, pipelined over those tiles: role 0 forms P
// (fp32, handed on through LDS) and, when counters are requested, re-runs the
// offline test as a check; role 1 accumulates dV one tile later and moves the query
// tiles into LDS; role 2 forms dP and dS; role 3 accumulates dK two tiles later (dS
// handed on as bf16 operands).
// On small grids the sweeps run in parts whose sums mala_bwd_dkdv_reduce_kernel
// adds.  An MFMA with its operands exchanged gives the transposed scores bit for
// bit, so both kernels see the same scores.
// P and dS enter the post-score MFMAs as two bf16 terms (hi + lo) unless an error
// budget allows the hi term alone; the transposed A operands come through
// ds_read_b64_tr_b16.  A skipped tile costs its QK MFMAs and the test in the dQ
// kernel and nothing in the key-major kernel unless a neighbouring key tile of the
// same query tile is retained.
#include <algorithm>

#include "mala_device.h"
#include "mala_kernels.h"

namespace mala {

__global__ __launch_bounds__(256) void mala_fill_zero_kernel(float4* p, size_t n16) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}
__global__ void mala_fill_zero_tail_kernel(unsigned char* p, size_t n) {
  for (size_t i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t st) {
  // Clears with kernels (not hipMemsetAsync) so that a captured graph replays it safely.
  if (bytes == 0) return hipSuccess;
  const size_t n16 = bytes / 16;
  if (n16) {
    const size_t blocks = (n16 + 255) / 256;
    const unsigned grid = (unsigned)(blocks < 8192 ? blocks : 8192);
    hipLaunchKernelGGL(mala_fill_zero_kernel, dim3(grid), dim3(256), 0, st, (float4*)ptr, n16);
  }
  if (bytes % 16)
    hipLaunchKernelGGL(mala_fill_zero_tail_kernel, dim3(1), dim3(64), 0, st,
                       (unsigned char*)ptr + n16 * 16, bytes % 16);
  return hipGetLastError();
}

// D_q = sum_d O[q][d] * dO[q][d]; 16 lanes per row; O in fp32 or bf16 (OT).
template <int D, typename OT>
__global__ __launch_bounds__(256) void mala_bwd_preprocess_kernel(const OT* o, const bf16* dout,
                                                                  float* dvec, long rows) {
  constexpr int PER = D / 16;
  const long row = (long)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int part = threadIdx.x & 15;
  float s = 0.f;
  if (row < rows) {
    const OT* op = o + row * D + part * PER;
    const bf16* dp = dout + row * D + part * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) s += (float)op[e] * (float)dp[e];
  }
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1) s += __shfl_xor(s, w, 16);
  if (row < rows && part == 0) dvec[row] = s;
}

template <typename OT>
static void launch_preprocess_t(const OT* o, const bf16* dout, float* dvec, long rows, int D,
                                hipStream_t st) {
  const unsigned grid = (unsigned)((rows + 15) / 16);
  if (D == 128)
    hipLaunchKernelGGL((mala_bwd_preprocess_kernel<128, OT>), dim3(grid), dim3(256), 0, st, o,
                       dout, dvec, rows);
  else
    hipLaunchKernelGGL((mala_bwd_preprocess_kernel<64, OT>), dim3(grid), dim3(256), 0, st, o,
                       dout, dvec, rows);
}

hipError_t launch_bwd_preprocess(const void* o, bool o_bf16, const bf16* dout, float* dvec,
                                 long rows, int D, hipStream_t st) {
  if (o_bf16)
    launch_preprocess_t(static_cast<const bf16*>(o), dout, dvec, rows, D, st);
  else
    launch_preprocess_t(static_cast<const float*>(o), dout, dvec, rows, D, st);
  return hipGetLastError();
}


// S = Q K^T for one 32 x 32 tile: A = Q rows (lane row q, 8 of d), B = K rows
// (lane column key, 8 of d); the k-steps accumulate in order in one chain.  Both
// backward kernels use exactly this sequence, so their scores are identical.
template <int KS>
__device__ __forceinline__ f32x16 qk_tile(const bf16x8 (&a)[KS], const bf16x8 (&b)[KS]) {
  f32x16 s;
#pragma unroll
  for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) s = mfma32(a[kk], b[kk], s);
  return s;
}

// Offline test of one tile in the C layout of qk_tile (lane = key column, rows
// 8 g + 4 h + e of the query tile).  Copies the raw scores into sv (-inf where
// masked) and returns whether some legal entry of this lane reaches its row's
// threshold (lse2 + log2(tau / L), base 2): max(s * scale2 - thr) >= 0 with one
// rounding (fma).  For finite values this is exactly the comparison of the
// rounded base-2 score with thr; padded rows have thr = +inf, tau = 0 gives
// thr = -inf.  klo / qlim bound the legal rows: 8 g + e in [klo, qlim); the bounds
// are only consulted on tiles that cross the diagonal or the end of the sequence
// (need_mask, uniform over the wavefront).  The probability of an entry is then
// exp2(fma(s, scale2, -lse2)).
template <bool MASK>
__device__ __forceinline__ bool offline_test(const f32x16& s, float scale2, int klo, int qlim,
                                             const float* thrs, int h, float (&sv)[16]) {
  // both backward kernels must round identically: explicit fma, no contraction
#pragma clang fp contract(off)
  float dm = kNegInf;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const f32x4 th = *reinterpret_cast<const f32x4*>(thrs + 8 * g + 4 * h);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float x = s[4 * g + e];
      if (MASK) {
        const bool legal = (8 * g + e >= klo) && (8 * g + e < qlim);
        sv[4 * g + e] = legal ? x : kNegInf;
        dm = fmaxf(dm, legal ? __builtin_fmaf(x, scale2, -th[e]) : kNegInf);
      } else {
        sv[4 * g + e] = x;
        dm = fmaxf(dm, __builtin_fmaf(x, scale2, -th[e]));
      }
    }
  }
  return dm >= 0.f;
}
__device__ __forceinline__ bool offline_entries(const f32x16& s, float scale2, bool need_mask,
                                                int klo, int qlim, const float* thrs, int h,
                                                float (&sv)[16]) {
  return need_mask ? offline_test<true>(s, scale2, klo, qlim, thrs, h, sv)
                   : offline_test<false>(s, scale2, klo, qlim, thrs, h, sv);
}

// P = exp2(s * scale2 - lse2) in place, for the C layout of qk_tile.
__device__ __forceinline__ void probabilities(float (&sv)[16], float scale2, const float* lse2,
                                              int h) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse2 + 8 * g + 4 * h);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      sv[4 * g + e] = fast_exp2(__builtin_fmaf(sv[4 * g + e], scale2, -l4[e]));
  }
}

// Per-row vectors of a query tile: base-2 lse, test threshold, D_q.
__device__ __forceinline__ void row_vectors(const BwdParams& p, long qbase, int Nq, long qq,
                                            long off, float* lse2, float* thr, float* dv) {
#pragma clang fp contract(off)
  if (qq < Nq) {
    const float l2 = p.lse[qbase + qq] * kLog2e;
    *lse2 = l2;
    *thr = l2 + p.log2tau - log2f((float)(qq + 1 + off));
    *dv = p.dvec[qbase + qq];
  } else {
    *lse2 = 0.f;
    *thr = __builtin_huge_valf();   // padded rows never retain
    *dv = 0.f;
  }
}

template <int D>
__global__ __launch_bounds__(1024) void mala_bwd_dkdv_kernel(BwdParams p) {
  constexpr int KS = D / 16;       // k-steps over head_dim
  constexpr int DB = D / 32;       // 32-wide column blocks
  constexpr int TILE = tile_elems<D>(kBq);          // one Q or dO tile in LDS
  constexpr int RC = D / 8 + 1;                     // 16-byte chunk positions per LDS row
  constexpr int NI = (kBq * RC + 63) / 64;          // 64-chunk LDS-DMA loads per tile
  constexpr int TS = NI * 64 * 8;                   // tile slot stride (elements)
  static_assert(TS >= TILE, "slot holds the tile");
  static_assert(kDkdvChunk % 256 == 0, "whole sweep iterations per compacting thread");
  // rings of query tiles: Q_k is read at steps k and k + 1, dO_k and the row vectors
  // at step k + 1 (k counts the processed tiles)
  __shared__ __attribute__((aligned(16))) bf16 Qs[4 * TS];
  __shared__ __attribute__((aligned(16))) bf16 dOs[3 * TS];
  // per-row vectors of the ring's tiles: lse2, test threshold (written only when
  // counters are requested), -D_q
  __shared__ __attribute__((aligned(16))) float rowv[3][3][kBq];
  // hand-offs per key group: P in fp32 as [buf][group][C registers 4g .. 4g+3][lane];
  // dS as the B operands [buf][group][hi0, hi1, lo0, lo1][lane]
  __shared__ __attribute__((aligned(16))) f32x4 Pf[2][4][4][64];
  __shared__ __attribute__((aligned(16))) bf16x8 dSop[2][4][4][64];
  __shared__ int Pflag[3][4];    // 0 skipped, 1 retained, 3 retained with P's lo term
  __shared__ int dSlo[2][4];     // dS of the tile needs its lo term
  // the processed tiles of the current chunk of the sweep: (iteration - chunk start)
  // << 4 | the tile's decisions for the four key groups
  __shared__ uint16_t plist[kDkdvChunk];
  __shared__ int wsum[5];      // per-wavefront counts of the compaction, then the total
  __shared__ unsigned long long bcnt[kNumCounters];   // the workgroup's counter sums

  // Sixteen wavefronts, four per 32 keys [32 g, +32) of the block (g = w % 4, so a
  // key group's four wavefronts share one SIMD), in a pipeline over the query tiles
  // that some key group retains (processed tile k):
  //   role 0, step k:   S_k = Q_k K^T, P_k (fp32) -> LDS
  //   role 1, step k+1: dV^T += dO_k^T P_k (16 MFMAs)
  //   role 2, step k+1: dP_k = dO_k V^T, dS_k = P_k (dP_k - D) -> LDS
  //   role 3, step k+2: dK^T += Q_k^T dS_k (16 MFMAs)
  // Each role runs its own loop (one barrier per step, the same count in all roles),
  // so that the register allocation of one role carries no values of another: no
  // wavefront needs more than 128 registers and four share a SIMD.
  //
  // The tile decisions are the dQ pass's (it runs first and records, per query tile,
  // head and 128-key block, which of the four 32-key tiles it retained): a query tile
  // that no key group retains costs no score MFMAs, no Q / dO load and no pipeline
  // step here.  When counters are requested, role 0 also evaluates the offline test on
  // the tiles it processes and counts those it confirms (a statistic: equal to the
  // retained count when the two passes agree).
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int role = wave >> 2, grp_k = wave & 3;
  const int h = lane >> 5, c = lane & 31, G = lane >> 4, t16 = lane & 15;
  // lane bases of the LDS tile reads: operand rows (row c) and transposed rows
  const int rdo = rd_base<D>(c, h), tro = tr_base<D>(4 * h + (t16 >> 2), G & 1, t16);
  const int BHk = p.B * p.Hkv;
  const int part = blockIdx.x / (p.nkblk * BHk);   // part of the sweep (split sweeps)
  const int bhk = blockIdx.x % BHk;
  const int kblk = (blockIdx.x / BHk) % p.nkblk;   // ascending: the longest key blocks first
  const int b = bhk / p.Hkv, hkv = bhk % p.Hkv, grp = p.Hq / p.Hkv;
  const Seg sg = seq_slice(p, b);
  const int Nq = sg.Nq, Nk = sg.Nk;
  const long off = (long)Nk - Nq;
  const int kb0 = kblk * kBwdKeys;
  if (kb0 >= Nk || Nq == 0) return;        // past the end of (or a skipped) packed sequence
  const long kbase = sg.kb + (long)hkv * p.Nk;   // key 0 of this (sequence, KV head)
  const int kw = kb0 + grp_k * kBk;        // first key of this wavefront's decision tile
  const int key = kw + c;                  // this lane's key (C-layout column)

  const int nqt = (Nq + kBq - 1) / kBq;
  // >= grp: key kb0 < Nk is visible to row Nq - 1
  const int total = dkdv_iterations(Nq, Nk, kb0, grp);
  // this workgroup's part of the sweep; the parts of a split sweep share the lo-term
  // budgets of the key (each part keeps 1 / parts of them), so the error bound of
  // the whole sweep holds
  const int it0 = part * p.psize, it1 = min(total, it0 + p.psize);
  if (it0 >= total) return;
  const float budget_share = 1.f / (float)((total + p.psize - 1) / p.psize);
  if (p.counters) blk_init(bcnt);

  // Query tiles are swept from the last one down to the block's diagonal, the
  // heads of the group innermost (iteration it: tile nqt - 1 - it / grp, head
  // it % grp): all co-resident workgroups of the same KV head then step through the
  // same Q / dO tiles in near lockstep, so that one fetch from HBM serves the XCD
  // through its L2.  The dV wavefronts (role 1, which wait longest at the barrier)
  // move the tiles with buffer loads straight into LDS: the 64 lanes of one load fill
  // 64 consecutive 16-byte positions of the tile's slot, each lane fetching the chunk
  // that the LDS layout keeps there (row padding positions and the slack at the
  // slot's end receive harmless data); the range check reads rows past the end of the
  // sequence as zeros.  Loads for tile k + 1 are issued at the start of step k in the
  // compiler-tracked form, so the dV wavefront waits for them at its first read of the
  // dO tile (after reading and splitting P): that also holds its MFMAs back until the
  // S wavefronts' dependent chains are under way, which measured faster than the
  // untracked form with the wait at the barrier.
  auto tile_q0 = [&](int it) { return (nqt - 1 - it / grp) * kBq; };
  const int mrow0 = mask_row0(p, b, sg);
  // decisions of iteration it (query tile nqt - 1 - it / grp, head it % grp): bit g for
  // key group g
  auto decisions = [&](int it) {
    return (int)p.mask[mask_index(p, mrow0 + nqt - 1 - it / grp, hkv * grp + it % grp, kblk)];
  };
  const bool mover = role == 1;
  const int mt = tid & 255;                  // thread index within the moving role
  const int mw = grp_k;                      // moving wavefront 0..3: loads mw, mw + 4, ...
  constexpr int NJ = (NI + 3) / 4;           // loads per moving wavefront and tile
  float plse = 0.f, pdv = 0.f;
  int pq0 = 0;                               // first row of the staged tile
  // Q / dO tiles of iteration it into ring slot k
  auto fetch = [&](int it, int k) {
    const int q0 = tile_q0(it);
    pq0 = q0;
    const long r0 = sg.qb + (long)(hkv * grp + it % grp) * p.Nq + q0;
    if (mt < kBq) {
      const uint32_t nr = (uint32_t)(Nq - q0) * 4u;
      plse = buf_load1(make_rsrc(p.lse + r0, nr), mt * 4u);
      pdv = buf_load1(make_rsrc(p.dvec + r0, nr), mt * 4u);
    }
    const uint32_t nb = (uint32_t)(Nq - q0) * (uint32_t)D * 2u;
    const auto rq = make_rsrc(p.q + r0 * D, nb), ro = make_rsrc(p.dout + r0 * D, nb);
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
      const int j = mw + 4 * u;
      if (j < NI) {
        // the chunk this lane fetches so that LDS position 64 j + lane holds it
        const int pos = 64 * j + lane;
        const int row = pos / RC, pc = pos % RC;
        const int L = pc < D / 8 ? pc / (D / 32) + 4 * (pc % (D / 32)) : 0;   // logical chunk
        const uint32_t off_b = (uint32_t)(row * D + 8 * L) * 2u;
        buf_load_lds16_tracked(rq, off_b, Qs + (k & 3) * TS + 512 * j);
        buf_load_lds16_tracked(ro, off_b, dOs + (k % 3) * TS + 512 * j);
      }
    }
  };
  auto stash = [&](int k) {
    if (mt < kBq) {
      // the same arithmetic as row_vectors (the query-major kernel must agree bitwise)
#pragma clang fp contract(off)
      const bool prow = pq0 + mt < Nq;
      const float l2 = plse * kLog2e;
      rowv[k % 3][0][mt] = prow ? l2 : 0.f;
      if (p.counters) {   // the threshold feeds only the statistics' re-run of the test
        const float plg = log2f((float)((long)pq0 + mt + 1 + off));
        rowv[k % 3][1][mt] = prow ? l2 + p.log2tau - plg : __builtin_huge_valf();
      }
      rowv[k % 3][2][mt] = prow ? -pdv : 0.f;   // -D: the dP accumulator starts there
    }
    wait_vm();
  };
  // Compacts iterations [c0, c0 + kDkdvChunk) of the sweep into plist and returns how
  // many there are (every thread calls it; the dP / dS wavefronts, which hold the
  // least state, do the work: sixteen iterations per thread and a prefix sum of the
  // processed counts over the four wavefronts).  The pipeline over the chunk then
  // starts at step -1, in which the first tile is staged.
  auto begin_chunk = [&](int c0) {
    if (role == 2) {
      const int t2 = tid & 255, w2 = wave & 3;
      constexpr int PER = kDkdvChunk / 256;
      int dec[PER], cnt = 0;
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int it = c0 + PER * t2 + u;
        dec[u] = it < it1 ? decisions(it) : 0;
        cnt += dec[u] != 0;
      }
      int x = cnt;   // inclusive scan over the wavefront
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(x, d);
        if (lane >= d) x += y;
      }
      if (lane == 63) wsum[w2] = x;
      __syncthreads();
      int before = 0, np = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const int s_ = wsum[w];
        before += w < w2 ? s_ : 0;
        np += s_;
      }
      int pos = before + x - cnt;
#pragma unroll
      for (int u = 0; u < PER; ++u)
        if (dec[u]) plist[pos++] = (uint16_t)(((PER * t2 + u) << 4) | dec[u]);
      if (tid == 512) wsum[4] = np;
    } else {
      __syncthreads();
    }
    __syncthreads();
    return __builtin_amdgcn_readfirstlane(wsum[4]);
  };

  if (role == 0 || role == 2) {
    // K rows (role 0, B operand of S = Q K^T) or V rows (role 2, of dP = dO V^T)
    bf16x8 kv[KS];
    {
      const bf16* src = (role == 0 ? p.k : p.v) + kbase * D;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        kv[kk] = key < Nk ? load8(src + (long)key * D + 16 * kk + 8 * h) : zero8();
    }
    if (role == 0) {
      float fdv = 0.f;   // P mass of this lane's key in tiles run without the lo term
      unsigned n_ret_kv = 0;          // statistics: processed tiles whose test this pass confirms
      unsigned long long hsum = 0;    // and their fingerprints
      for (int c0 = it0; c0 < it1; c0 += kDkdvChunk) {
        const int np = begin_chunk(c0);
        if (!np) continue;
        // the list entry of the next step, read during this one (the step's closing
        // barrier waits for it, so the next step finds it in place)
        int e_next = plist[0];
        for (int k = -1; k < np + 2; ++k) {
          if (k >= 0 && k < np) {
            const int e = __builtin_amdgcn_readfirstlane(e_next);
            if (k + 1 < np) e_next = plist[k + 1];
            const int it = c0 + (e >> 4);
            const bool ret = (e >> grp_k) & 1;
            bool with_lo = false;
            if (ret) {
              // tile k: score discovery, offline test (statistics), P
              const int q0 = tile_q0(it);
              const float* rv = &rowv[k % 3][0][0];
              bf16x8 qa[KS];
              const bf16* qr = lds_pin(Qs + (k & 3) * TS + rdo);
#pragma unroll
              for (int kk = 0; kk < KS; ++kk) qa[kk] = load8(qr + rd_step<D>(kk));
              const f32x16 sc = qk_tile<KS>(qa, kv);
              // tiles that cross the diagonal or the end of the sequence (or whose keys
              // all lie beyond this tile's rows) take the masked test
              const bool need_mask =
                  ((long)kw + kBk - 1 > (long)q0 + off) || (q0 + kBq > Nq) || (kw + kBk > Nk);
              const int klo = key < Nk ? (int)((long)key - off - q0) - 4 * h : 1000000;
              float sv[16];
              if (p.counters) {
                // the offline test again, as a statistic: it confirms the dQ pass's decision
                const bool dem =
                    offline_entries(sc, p.scale2, need_mask, klo, Nq - q0 - 4 * h, rv + kBq, h, sv);
                if (wave_any(dem)) {
                  ++n_ret_kv;
                  hsum += tile_hash(b, hkv * grp + it % grp, q0 / kBq, kw / kBk);
                }
              } else if (need_mask) {
                const int qlim = Nq - q0 - 4 * h;
#pragma unroll
                for (int g = 0; g < 4; ++g)
#pragma unroll
                  for (int e = 0; e < 4; ++e)
                    sv[4 * g + e] = (8 * g + e >= klo) && (8 * g + e < qlim) ? sc[4 * g + e] : kNegInf;
              } else {
#pragma unroll
                for (int r = 0; r < 16; ++r) sv[r] = sc[r];
              }
              probabilities(sv, p.scale2, rv, h);
#pragma unroll
              for (int g = 0; g < 4; ++g)
                Pf[k & 1][grp_k][g][lane] =
                    f32x4{sv[4 * g], sv[4 * g + 1], sv[4 * g + 2], sv[4 * g + 3]};
              // dV runs this tile without P's lo term while the key's P mass in such
              // tiles stays within kLoMassDv (for every key of the tile)
              float ps = 0.f;
#pragma unroll
              for (int r = 0; r < 16; ++r) ps += sv[r];
              const float fv_new = fdv + halves_sum(ps);
              with_lo = wave_any(fv_new > kLoMassDv * budget_share);
              if (!with_lo) fdv = fv_new;
            }
            if (lane == 0) Pflag[k % 3][grp_k] = ret ? (with_lo ? 3 : 1) : 0;
          }
          __syncthreads();
        }
      }
      if (p.counters && lane == 0) {
        blk_add(bcnt, kCntRetainedKV, n_ret_kv);
        blk_add(bcnt, kCntSetHashKV, hsum);
      }
    } else {
      float fdk = 0.f;   // sum of |dS| of this lane's key in tiles run without the lo term
      for (int c0 = it0; c0 < it1; c0 += kDkdvChunk) {
        const int np = begin_chunk(c0);
        if (!np) continue;
        for (int k = -1; k < np + 2; ++k) {
          const int t = k - 1;
          if (t >= 0 && t < np && Pflag[t % 3][grp_k]) {
            // tile t: dP = dO V^T; dS = P (dP - D) -> LDS as hi / lo B operands
            const float* rv = &rowv[t % 3][0][0];
            bf16x8 oa[KS];
            const bf16* orr = lds_pin(dOs + (t % 3) * TS + rdo);
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) oa[kk] = load8(orr + rd_step<D>(kk));
            // dP - D: the accumulator starts at -D of each row (C layout: register 4 g + e
            // holds row 8 g + 4 h + e)
            f32x16 dpd;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const f32x4 d4 = *reinterpret_cast<const f32x4*>(rv + 2 * kBq + 8 * g + 4 * h);
#pragma unroll
              for (int e = 0; e < 4; ++e) dpd[4 * g + e] = d4[e];
            }
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) dpd = mfma32(oa[kk], kv[kk], dpd);
            float ds[16];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const f32x4 p4 = Pf[t & 1][grp_k][g][lane];
#pragma unroll
              for (int e = 0; e < 4; ++e) ds[4 * g + e] = p4[e] * dpd[4 * g + e];
            }
            // dK runs this tile without dS's lo term while the key's sum of |dS| in
            // such tiles stays within kLoMassDk (for every key of the tile); a tile
            // holding more than kLoTileDk of some key's |dS| always takes the lo term
            float as = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) as += fabsf(ds[r]);
            const float as_key = halves_sum(as);
            const float fk_new = fdk + as_key;
            const bool with_lo = wave_any(fk_new > kLoMassDk * budget_share || as_key > kLoTileDk);
            if (!with_lo) fdk = fk_new;
            bf16x8 xh[2], xl[2];
            if (with_lo) {
              split_bf16x8(ds, xh[0], xl[0]);
              split_bf16x8(ds + 8, xh[1], xl[1]);
              dSop[t & 1][grp_k][2][lane] = xl[0];
              dSop[t & 1][grp_k][3][lane] = xl[1];
            } else {
              xh[0] = hi_bf16x8(ds);
              xh[1] = hi_bf16x8(ds + 8);
            }
            dSop[t & 1][grp_k][0][lane] = xh[0];
            dSop[t & 1][grp_k][1][lane] = xh[1];
            if (lane == 0) dSlo[t & 1][grp_k] = with_lo ? 1 : 0;
          }
          __syncthreads();
        }
      }
    }
  } else {
    // roles 1 (dV^T += dO^T P, one tile behind) and 3 (dK^T += Q^T dS, two behind),
    // each in its own loop
    f32x16 acc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;
    auto accumulate = [&](const bf16* atb, bf16x8 b0, bf16x8 b1) {
      const bf16* ab = lds_pin(atb);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const bf16* at = ab + 16 * ks * (D + 8) + tr_step<D>(db);
          acc[db] = mfma32(cat(lds_read_tr(at), lds_read_tr(at + 8 * (D + 8))), ks ? b1 : b0, acc[db]);
        }
    };
    if (role == 1) {
      unsigned n_do = 0;   // statistics: dO tiles staged (some key group retained the tile)
      for (int c0 = it0; c0 < it1; c0 += kDkdvChunk) {
        const int np = begin_chunk(c0);
        if (!np) continue;
        n_do += np;
        int e_next = plist[0];   // the entry to fetch next, read a step ahead
        for (int k = -1; k < np + 2; ++k) {
          if (k + 1 < np) {
            fetch(c0 + (__builtin_amdgcn_readfirstlane(e_next) >> 4), k + 1);
            if (k + 2 < np) e_next = plist[k + 2];
          }
          const int t = k - 1;
          const int pf = (t >= 0 && t < np) ? Pflag[t % 3][grp_k] : 0;
          if (pf) {
            float pv[16];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const f32x4 p4 = Pf[t & 1][grp_k][g][lane];
#pragma unroll
              for (int e = 0; e < 4; ++e) pv[4 * g + e] = p4[e];
            }
            const bf16* atb = dOs + (t % 3) * TS + tro;
            accumulate(atb, hi_bf16x8(pv), hi_bf16x8(pv + 8));
            if (pf & 2) {
              bf16x8 hh[2], bl[2];
              split_bf16x8(pv, hh[0], bl[0]);
              split_bf16x8(pv + 8, hh[1], bl[1]);
              accumulate(atb, bl[0], bl[1]);
            }
          }
          if (k + 1 < np) stash(k + 1);
          __syncthreads();
        }
      }
      if (p.counters && grp_k == 0 && lane == 0) {
        blk_add(bcnt, kCntVTiles, n_do);
        blk_add(bcnt, kCntVNeeded, n_do);
      }
    } else {
      // the decision of tile k - 2 is known since the end of step k - 2: it is read one
      // step early, off the critical path
      int fl3 = 0;
      // the Q^T operands of the next step's tile for its first k-step, read at the end
      // of this step (the second k-step's are read in the step itself: holding both
      // across the barrier would exceed the registers of four wavefronts per SIMD)
      bf16x8 a0[DB], a1[DB];
      auto load_a = [&](int tt, int ks, bf16x8 (&a)[DB]) {
        const bf16* ab = lds_pin(Qs + (tt & 3) * TS + tro);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16* at = ab + 16 * ks * (D + 8) + tr_step<D>(db);
          a[db] = cat(lds_read_tr(at), lds_read_tr(at + 8 * (D + 8)));
        }
      };
      auto acc_a = [&](bf16x8 b0, bf16x8 b1) {
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] = mfma32(a0[db], b0, acc[db]);
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] = mfma32(a1[db], b1, acc[db]);
      };
      for (int c0 = it0; c0 < it1; c0 += kDkdvChunk) {
        const int np = begin_chunk(c0);
        if (!np) continue;
        fl3 = 0;
        for (int k = -1; k < np + 2; ++k) {
          const int t = k - 2;
          if (fl3) {
            // the dS operands first: the first k-step's MFMAs wait only for them
            const bf16x8 b0 = dSop[t & 1][grp_k][0][lane], b1 = dSop[t & 1][grp_k][1][lane];
            load_a(t, 1, a1);
            acc_a(b0, b1);
            if (dSlo[t & 1][grp_k]) acc_a(dSop[t & 1][grp_k][2][lane], dSop[t & 1][grp_k][3][lane]);
          }
          const int tn = k - 1;   // the tile of the next step
          fl3 = (tn >= 0 && tn < np) ? Pflag[tn % 3][grp_k] : 0;
          if (fl3) load_a(tn, 0, a0);
          __syncthreads();
        }
      }
    }
    // dV = sum P^T dO (role 1), dK = scale * sum dS^T Q (role 3); lane (h, c)
    // holds key kw + c
    // (split sweeps: this part's fp32 sums to its slots of the partial buffer)
    if (key < Nk) {
      const float f = role == 1 ? 1.f : p.scale;
      const bool split = p.nparts > 1;
      void* dst = split ? (void*)(p.part + (size_t)(2 * part + (role == 1 ? 0 : 1)) *
                                               ((size_t)p.B * p.Hkv * p.Nk) * D)
                        : (role == 1 ? p.dv : p.dk);
      const long krow = (kbase + key) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 v4 = {acc[db][4 * g] * f, acc[db][4 * g + 1] * f, acc[db][4 * g + 2] * f,
                      acc[db][4 * g + 3] * f};
          store_out4(dst, krow + 32 * db + 8 * g + 4 * h, v4, split ? 0 : p.grad_bf16);
        }
    }
  }
  // every role ends here, after the same number of barriers
  if (p.counters) blk_flush(bcnt, p.counters);
}

// Offline test of one tile in the transposed C layout of the dQ pass: the lane
// holds one query row (threshold thr) and its 16 keys kb + 8 (r / 4) + 4 h + r % 4.
// The per-entry test of offline_test, fma(s, scale2, -thr) >= 0 with one rounding,
// is monotonic in s (scale2 > 0), so with one threshold per lane it is taken once,
// on the lane's largest legal score: the same decision with one fma instead of
// sixteen.  Keys with 8 (r / 4) + r % 4 > kmax lie beyond the row's causal limit,
// those with 8 (r / 4) + r % 4 >= klim beyond the sequence; both are only consulted
// on tiles that cross the diagonal or an end (need_mask, uniform over the
// wavefront).  Rows past the end have thr = +inf and never retain.
template <bool MASK>
__device__ __forceinline__ bool offline_test_t(const f32x16& s, float scale2, int kmax, int klim,
                                               float thr, float (&sv)[16]) {
#pragma clang fp contract(off)
  float mx = kNegInf;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int kr = 8 * (r >> 2) + (r & 3);
    const float x = (!MASK || (kr <= kmax && kr < klim)) ? s[r] : kNegInf;
    sv[r] = x;
    mx = fmaxf(mx, x);
  }
  return __builtin_fmaf(mx, scale2, -thr) >= 0.f;
}

// dQ pass (query-major).  Each wavefront owns 32 query rows and computes the
// transposed products, so that every lane holds one query row: S^T = K Q^T and
// dP^T = V dO^T (A = K / V rows from the LDS stage, B = the wavefront's Q / dO rows
// in registers), then dQ^T += K^T dS^T with dS^T fed straight back from the C
// registers as the B operand (the contraction index permuted as in the forward's
// P.V) and K^T through transposed LDS reads.  An MFMA with its two operands
// exchanged gives the transposed result bit for bit (checked by a probe on gfx950),
// so the scores, and with them the retention decisions, equal those of the
// key-major kernel (same operand values, k-step order and threshold arithmetic).
template <int D>
__global__ __launch_bounds__(kDqWaves * 64) void mala_bwd_dq_kernel(BwdParams p) {
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int kDqStage = kBwdKeys;             // keys per K / V stage: one 128-key block
  constexpr int TPS = kDqStage / kBk;            // decision tiles per stage
  constexpr int STAGE = tile_elems<D>(kDqStage);
  static_assert(TPS == 4, "a stage is one decision byte's block");
  __shared__ __attribute__((aligned(16))) bf16 Ks[2 * STAGE];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2 * STAGE];
  __shared__ unsigned long long bcnt[kNumCounters];   // the workgroup's counter sums

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, c = lane & 31, G = lane >> 4, t16 = lane & 15;
  // lane bases of the LDS tile reads: operand rows (row c) and transposed rows
  const int rdo = rd_base<D>(c, h), tro = tr_base<D>(4 * h + (t16 >> 2), G & 1, t16);
  const int BH = p.B * p.Hq;
  const int bh = blockIdx.x % BH;
  const int qblk = p.nqblk - 1 - (int)(blockIdx.x / BH);   // longest rows first
  const int b = bh / p.Hq, hq = bh % p.Hq, hkv = hq / (p.Hq / p.Hkv);
  const Seg sg = seq_slice(p, b);
  const int Nq = sg.Nq, Nk = sg.Nk;
  if (qblk * kDqRows >= Nq) return;   // past the end of a packed sequence
  const long off = (long)Nk - Nq;
  const int q0w = qblk * kDqRows + wave * kBq;
  const int offi = Nk - Nq;   // off as an int (|off| < 2^31)
  const int qrow = q0w + c;
  const bool row_valid = qrow < Nq;
  const long qbase = sg.qb + (long)hq * p.Nq;    // row 0 of this (sequence, head)
  const long kbase = sg.kb + (long)hkv * p.Nk;
  const bf16* Kp = p.k + kbase * D;
  const bf16* Vp = p.v + kbase * D;
  if (p.counters) blk_init(bcnt);

  // Q and dO rows of this wavefront as B operands (lane column qrow)
  bf16x8 qb[KS], ob[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    const long off_e = (qbase + qrow) * D + 16 * kk + 8 * h;
    qb[kk] = row_valid ? load8(p.q + off_e) : zero8();
    ob[kk] = row_valid ? load8(p.dout + off_e) : zero8();
  }
  // this lane's row vectors: base-2 lse, test threshold, D_q
  float lse2, thr, dvq;
  row_vectors(p, qbase, Nq, (long)qrow, off, &lse2, &thr, &dvq);
  f32x16 negd;
#pragma unroll
  for (int r = 0; r < 16; ++r) negd[r] = -dvq;

  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  const int qlast_w = min(q0w + kBq - 1, Nq - 1);
  const int jdiag = (q0w < Nq) ? (int)((qlast_w + off) / kBk) : -1;
  const int nvalid = max(0, min(kBq, Nq - q0w));
  const int qlast_g = min(qblk * kDqRows + kDqRows - 1, Nq - 1);
  const int ttop = (int)((qlast_g + off) / kDqStage);
  unsigned n_legal = 0, n_ret = 0;
  unsigned long long hsum = 0;   // fingerprints of the retained tiles
  int cnt_row = 0;   // retained diagonal tiles in which row qrow has a legal key
  unsigned n_ret_m = 0;  // retained diagonal tiles
  // The decisions for the key-major pass: one byte per 128-key block of this
  // wavefront's query tile and head, bit j % 4 for key tile j, the blocks contiguous
  // (mask_index).  Stage t is block t (key tiles 4t .. 4t + 3); the block's byte is
  // complete after the stage and goes into lane t % 64 of pack; after block 64 m the
  // group of 64 blocks goes out in one coalesced store (the first group only up to
  // the workgroup's top block).  Every
  // block up to the diagonal is written (blocks above this wavefront's diagonal get
  // zero), so the buffer needs no clearing.
  uint8_t* mrow = p.mask + mask_index(p, mask_row0(p, b, sg) + q0w / kBq, hq, 0);
  const bool mwave = q0w < Nq;               // this wavefront has query rows
  int nib = 0, stored = 0;
  uint32_t pack = 0;
  float fdq = 0.f;   // this row's sum of |dS| in tiles run without the lo term
  // K / V stages move with buffer loads straight into LDS (keys past the end read
  // as zeros): wavefront w issues the 64-position loads w, w + 8, ... of each slot.
  // The loads of stage t - 1 overlap the compute of stage t (untracked form) and
  // are waited for just before the stage's closing barrier.
  constexpr int NIS = STAGE / 512;           // 64-position loads per stage slot
  static_assert(NIS * 512 == STAGE, "whole loads per slot");
  constexpr int NJS = (NIS + kDqWaves - 1) / kDqWaves;
  uint32_t dma_off[NJS];
#pragma unroll
  for (int u = 0; u < NJS; ++u) dma_off[u] = dma_lane_offset<D>(64 * (wave + kDqWaves * u) + lane);
  auto fetch = [&](int t, int buf) {
    const long k0 = (long)t * kDqStage;
    const uint32_t nb = (uint32_t)(Nk - k0) * (uint32_t)D * 2u;
    const i32x4 rk = rsrc_words(Kp + k0 * D, nb), rvv = rsrc_words(Vp + k0 * D, nb);
#pragma unroll
    for (int u = 0; u < NJS; ++u) {
      const int j = wave + kDqWaves * u;
      if (j < NIS) {
        buf_load_lds16(rk, dma_off[u], Ks + buf * STAGE + 512 * j);
        buf_load_lds16(rvv, dma_off[u], Vs + buf * STAGE + 512 * j);
      }
    }
  };

  fetch(ttop, 0);
  wait_vm();   // (also the loads above, so that no wait for them lands in the loop)
  __syncthreads();

  for (int t = ttop; t >= 0; --t) {
    const int buf = (ttop - t) & 1;
    if (t > 0) fetch(t - 1, buf ^ 1);
    const bf16* Kb = Ks + buf * STAGE;
    const bf16* Vb = Vs + buf * STAGE;
    const bf16* kr = lds_pin(Kb + rdo);
    const bf16* vr = lds_pin(Vb + rdo);
    const bf16* ktb = lds_pin(Kb + tro);
    // the two wavefronts of a SIMD keep pace: the one with more of the stage left
    // issues first (priority 2 for the first two tiles, then 1, 0 at the barrier)
#pragma unroll 1
    for (int sub = TPS - 1; sub >= 0; --sub) {
      if (sub > 1) __builtin_amdgcn_s_setprio(2); else __builtin_amdgcn_s_setprio(1);
      const int j = TPS * t + sub;
      if (j > jdiag) continue;
      const int kb = j * kBk;
      ++n_legal;
      bf16x8 kop[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) kop[kk] = load8(kr + sub * kBk * (D + 8) + rd_step<D>(kk));
      const f32x16 s = qk_tile<KS>(kop, qb);
      const bool need_mask = (kb + kBk - 1 > q0w + offi) || (q0w + kBq > Nq) || (kb + kBk > Nk);
      const int kmax = qrow + offi - kb - 4 * h;
      const int klim = min(Nk - kb, kBk) - 4 * h;
      float sv[16];
      const bool dem = need_mask ? offline_test_t<true>(s, p.scale2, kmax, klim, thr, sv)
                                 : offline_test_t<false>(s, p.scale2, kmax, klim, thr, sv);
      const bool ret = wave_any(dem);
      nib |= (ret ? 1 : 0) << (j & 3);
      if (!ret) continue;
      ++n_ret;
      if (p.counters) hsum += tile_hash(b, hq, q0w / kBq, j);
      // off the diagonal and the sequence end every row has a legal key: those tiles
      // are counted per wavefront
      if (need_mask) {
        ++n_ret_m;
        cnt_row += (row_valid && kb <= qrow + offi) ? 1 : 0;
      }
      // P^T = exp2(s * scale2 - lse2), the key-major kernel's arithmetic
#pragma unroll
      for (int r = 0; r < 16; ++r) sv[r] = fast_exp2(__builtin_fmaf(sv[r], p.scale2, -lse2));
      bf16x8 vop[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) vop[kk] = load8(vr + sub * kBk * (D + 8) + rd_step<D>(kk));
      // dP^T - D: the accumulator starts at -D_q (one row per lane)
      f32x16 dpd = negd;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) dpd = mfma32(vop[kk], ob[kk], dpd);
      float dsv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) dsv[r] = sv[r] * dpd[r];
      // dQ runs this tile without dS's lo term while this row's sum of |dS| over
      // such tiles stays within kLoMassDq (for every row of the wavefront); a tile
      // holding more than kLoTileDq of some row's |dS| always takes the lo term, so
      // that the budget goes to the many small tiles
      float as = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) as += fabsf(dsv[r]);
      const float as_row = halves_sum(as);
      const float fq_new = fdq + as_row;
      const bool with_lo = wave_any(fq_new > kLoMassDq || as_row > kLoTileDq);
      if (!with_lo) fdq = fq_new;
      // dQ^T[d][q] += K^T[d][key] dS^T[key][q]: k-step ks takes C registers
      // 8 ks .. 8 ks + 7 as the B operand, K^T through transposed reads of the same
      // key rows.  The hi MFMAs run with no branch among them; the lo ones, when
      // needed, in a second pass that reads the K operands again.
      auto k_operand = [&](int ks, int db) {
        const bf16* kt = ktb + (sub * kBk + 16 * ks) * (D + 8) + tr_step<D>(db);
        return cat(lds_read_tr(kt), lds_read_tr(kt + 8 * (D + 8)));
      };
      const bf16x8 dh[2] = {hi_bf16x8(dsv), hi_bf16x8(dsv + 8)};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] = mfma32(k_operand(ks, db), dh[ks], acc[db]);
      if (with_lo) {
        bf16x8 dl[2], hh[2];
        split_bf16x8(dsv, hh[0], dl[0]);
        split_bf16x8(dsv + 8, hh[1], dl[1]);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int db = 0; db < DB; ++db) acc[db] = mfma32(k_operand(ks, db), dl[ks], acc[db]);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    if (mwave) {
      // block t is complete
      const int blk = t;
      if (lane == (blk & 63)) pack = (uint32_t)nib;
      nib = 0;
      if (!(blk & 63)) {
        // the group's blocks blk .. blk + 63, up to the workgroup's top block ttop
        if (lane <= ttop - blk) mrow[blk + lane] = (uint8_t)pack;
        stored = 1;
      }
    }
    // the next stage's loads have landed; a decision store issued in this stage
    // (issued after those loads: vector memory operations complete in order) may
    // still be in flight
    if (stored)
      wait_vm_keep<1>();
    else
      wait_vm();
    stored = 0;
    __syncthreads();
  }

  // dQ = scale * sum dS K; lane (h, c) holds row qrow, columns 32 db + 8 g + 4 h + e
  if (row_valid) {
    const long qr = (qbase + qrow) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 v4 = {acc[db][4 * g] * p.scale, acc[db][4 * g + 1] * p.scale,
                          acc[db][4 * g + 2] * p.scale, acc[db][4 * g + 3] * p.scale};
        store_out4(p.dq, qr + 32 * db + 8 * g + 4 * h, v4, p.grad_bf16);
      }
    if (p.row_tiles && h == 0) p.row_tiles[qbase + qrow] = cnt_row + (int)(n_ret - n_ret_m);
  }
  if (p.counters) {
    if (lane == 0) {
      blk_add(bcnt, kCntLegal, n_legal);
      blk_add(bcnt, kCntRetained, n_ret);
      blk_add(bcnt, kCntSlots, (unsigned long long)n_ret * kBk * nvalid);
      blk_add(bcnt, kCntSetHash, hsum);
    }
    blk_flush(bcnt, p.counters);
  }
}

// Sum of the parts of split dK/dV sweeps in part order (fixed-length batches): one
// thread per four columns of a K-shaped row; a row's key block has
// ceil(iterations / psize) parts.
template <int D>
__global__ __launch_bounds__(256) void mala_bwd_dkdv_reduce_kernel(BwdParams p) {
  const long rows = (long)p.B * p.Hkv * p.Nk;
  const long n4 = rows * (D / 4);
  const size_t slot = (size_t)rows * D;
  const int grp = p.Hq / p.Hkv;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < n4;
       i += (long)gridDim.x * blockDim.x) {
    const long row = i / (D / 4);
    const long e = row * D + (i % (D / 4)) * 4;
    const int kb0 = (int)(row % p.Nk) / kBwdKeys * kBwdKeys;
    const int np = (dkdv_iterations(p.Nq, p.Nk, kb0, grp) + p.psize - 1) / p.psize;
    f32x4 sv = {0.f, 0.f, 0.f, 0.f}, sk = {0.f, 0.f, 0.f, 0.f};
    for (int q = 0; q < np; ++q) {
      sv += *reinterpret_cast<const f32x4*>(p.part + (size_t)(2 * q) * slot + e);
      sk += *reinterpret_cast<const f32x4*>(p.part + (size_t)(2 * q + 1) * slot + e);
    }
    store_out4(p.dv, e, sv, p.grad_bf16);
    store_out4(p.dk, e, sk, p.grad_bf16);
  }
}

hipError_t launch_bwd(const BwdParams& p, int D, hipStream_t st) {
  dim3 grid_kv((unsigned)p.nkblk * p.B * p.Hkv * p.nparts), block_kv(1024);
  dim3 grid_q((unsigned)p.nqblk * p.B * p.Hq), block_q(kDqWaves * 64);
  const long n4 = (long)p.B * p.Hkv * p.Nk * (D / 4);
  dim3 grid_r((unsigned)std::min<long>((n4 + 255) / 256, 8192));
  // the dQ pass first: it records the tile decisions that the key-major pass follows
  if (D == 128) {
    hipLaunchKernelGGL(mala_bwd_dq_kernel<128>, grid_q, block_q, 0, st, p);
    hipLaunchKernelGGL(mala_bwd_dkdv_kernel<128>, grid_kv, block_kv, 0, st, p);
    if (p.nparts > 1) hipLaunchKernelGGL(mala_bwd_dkdv_reduce_kernel<128>, grid_r, dim3(256), 0, st, p);
  } else {
    hipLaunchKernelGGL(mala_bwd_dq_kernel<64>, grid_q, block_q, 0, st, p);
    hipLaunchKernelGGL(mala_bwd_dkdv_kernel<64>, grid_kv, block_kv, 0, st, p);
    if (p.nparts > 1) hipLaunchKernelGGL(mala_bwd_dkdv_reduce_kernel<64>, grid_r, dim3(256), 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace mala
