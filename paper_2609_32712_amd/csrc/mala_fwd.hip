// MALA forward (Algorithm 1) for gfx950.
//
// One workgroup = 8 wavefronts = 256 consecutive query rows of one (batch, query
// head); each wavefront owns 32 rows, which is the decision tile's B_q.  K and V
// are staged through double-buffered LDS 64 keys at a time, from the workgroup's
// highest legal key down to key 0 (the diagonal-first traversal of the Online
// Sparse Softmax paragraph); the next stage moves straight into LDS (buffer loads
// with the LDS flag) while the current one is processed.  Inside a stage each
// wavefront visits its two 32-key decision tiles high half first, so every
// wavefront sees its tiles in strictly descending order.
//
// Per decision tile (32 keys x the wavefront's 32 rows):
//   S^T = K_j Q_i^T       8 (D = 128) bf16 MFMAs 32x32x16, fp32 accumulate; each
//                         lane holds one query row and 16 of the 32 keys, so the
//                         row max is 15 in-lane max + one permlane32 swap;
//   online test           skip iff every row with a legal key has
//                         rowmax - m - log2(l) < log2(tau) - log2(L_q) (base-2 units,
//                         equivalent to the natural-log test), rows with l == 0
//                         always retain; one ballot makes the branch wave-uniform;
//   retained path         lazy rescale of O and l (only when some row's max grew by
//                         more than 2^8), P = exp2(S - m) as a bf16 hi term, plus a
//                         lo term when the tile holds more than kFwdLoShare of some
//                         row's normalizer, O^T += V^T P^T (8 MFMAs per term, V^T
//                         operand through ds_read_b64_tr_b16).
// A skipped tile costs its QK MFMAs, one max reduction and one compare.
#include "mala_device.h"
#include "mala_kernels.h"

namespace mala {

template <int D>
__global__ __launch_bounds__(kFwdWaves * 64) void mala_fwd_kernel(FwdParams p) {
  constexpr int NT = kFwdWaves * 64;     // threads per workgroup
  constexpr int KS = D / 16;             // k-steps of the QK product
  constexpr int DB = D / 32;             // 32-wide output column blocks
  constexpr int STAGE = tile_elems<D>(kFwdStage);
  // double-buffered K and V stages: the next stage is fetched while the current one
  // is processed
  __shared__ __attribute__((aligned(16))) bf16 Ks[2 * STAGE];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2 * STAGE];
  // statistics: per stage buffer and decision tile, t + 1 once some wavefront
  // retained the tile of stage t (stage-tagged: no clearing between stages); the
  // workgroup's counter sums
  __shared__ int vneed[2][kFwdStage / kBk];
  __shared__ unsigned long long bcnt[kNumCounters];

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
  if (qblk * kFwdRows >= Nq) return;   // past the end of a packed sequence
  const long off = (long)Nk - Nq;
  const int offi = Nk - Nq;   // off as an int (|off| < 2^31)
  const int q0w = qblk * kFwdRows + wave * kBq;
  const int qrow = q0w + c;
  const bool row_valid = qrow < Nq;

  const long qbase = sg.qb + (long)hq * p.Nq;    // row 0 of this (sequence, head)
  const long kbase = sg.kb + (long)hkv * p.Nk;
  const bf16* Qp = p.q + qbase * D;
  const bf16* Kp = p.k + kbase * D;
  const bf16* Vp = p.v + kbase * D;

  // Q^T as the B operand: lane (h, c) holds Q[qrow][16kk + 8h .. +7]
  bf16x8 qreg[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk)
    qreg[kk] = row_valid ? load8(Qp + (long)qrow * D + 16 * kk + 8 * h) : zero8();

  float m = kNegInf, l = 0.f;
  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;
  int cnt = 0;          // retained diagonal tiles in which this row has a legal key
  unsigned n_ret_m = 0;  // retained diagonal tiles
  const float thr = p.log2tau - log2f((float)(qrow + 1 + off));   // log2(tau / L_q)

  const int qlast_w = min(q0w + kBq - 1, Nq - 1);
  const int jdiag = (q0w < Nq) ? (int)((qlast_w + off) / kBk) : -1;
  const int nvalid = max(0, min(kBq, Nq - q0w));
  const int qlast_g = min(qblk * kFwdRows + kFwdRows - 1, Nq - 1);
  const int ttop = (int)((qlast_g + off) / kFwdStage);
  unsigned n_legal = 0, n_ret = 0, n_vneed = 0;
  unsigned long long hsum = 0;   // fingerprints of the retained tiles
  const bool stats = p.counters != nullptr;
  if (stats) {
    if (tid < 2 * (kFwdStage / kBk)) vneed[tid / (kFwdStage / kBk)][tid % (kFwdStage / kBk)] = 0;
    blk_init(bcnt);
  }

  // K / V stages move with buffer loads straight into LDS (keys past the end read
  // as zeros): wavefront w issues the 64-position loads w, w + 8, ... of each slot.
  // The loads of stage t - 1 overlap the compute of stage t and are waited for just
  // before the stage's closing barrier.
  constexpr int NIS = STAGE / 512;           // 64-position loads per stage slot
  static_assert(NIS * 512 == STAGE, "whole loads per slot");
  constexpr int NJS = (NIS + kFwdWaves - 1) / kFwdWaves;
  uint32_t dma_off[NJS];
#pragma unroll
  for (int u = 0; u < NJS; ++u) dma_off[u] = dma_lane_offset<D>(64 * (wave + kFwdWaves * u) + lane);
  auto fetch = [&](int t, int buf) {
    const long k0 = (long)t * kFwdStage;
    const uint32_t nb = (uint32_t)(Nk - k0) * (uint32_t)D * 2u;
    const i32x4 rk = rsrc_words(Kp + k0 * D, nb), rvv = rsrc_words(Vp + k0 * D, nb);
#pragma unroll
    for (int u = 0; u < NJS; ++u) {
      const int j = wave + kFwdWaves * u;
      if (j < NIS) {
        buf_load_lds16(rk, dma_off[u], Ks + buf * STAGE + 512 * j);
        buf_load_lds16(rvv, dma_off[u], Vs + buf * STAGE + 512 * j);
      }
    }
  };

  fetch(ttop, 0);
  wait_vm();   // (also the Q loads above, so that no wait for them lands in the loop)
  __syncthreads();

  for (int t = ttop; t >= 0; --t) {
    const int buf = (ttop - t) & 1;
    if (t > 0) fetch(t - 1, buf ^ 1);
    const bf16* kr = lds_pin(Ks + buf * STAGE + rdo);
    const bf16* vtb = lds_pin(Vs + buf * STAGE + tro);

    // statistics: the tag each retained tile of this stage found in vneed (t + 1:
    // another wavefront marked it first); compared after the stage, so that the
    // exchange's result is not waited for in the middle of the tile's work
    int vtag[2] = {t + 1, t + 1};
    if (2 * t <= jdiag) {
      // the two tiles in descending key order: the high half first
#pragma unroll
      for (int sub = 1; sub >= 0; --sub) {
        const int j = 2 * t + sub;
        if (j > jdiag) continue;            // above this wavefront's diagonal
        const int kb = j * kBk;
        ++n_legal;
        // score discovery (all K operands are read from LDS first)
        f32x16 s;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.f;
        {
          bf16x8 ka[KS];
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) ka[kk] = load8(kr + sub * kBk * (D + 8) + rd_step<D>(kk));
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) s = mfma32(ka[kk], qreg[kk], s);
        }

        const bool need_mask = (kb + kBk - 1 > q0w + offi) || (q0w + kBq > Nq);
        float sv[16];
        float mt = kNegInf;
        if (need_mask) {
          // keys of this lane: kb + 8 (r / 4) + 4 h + r % 4; legal iff key <= qrow + off
          const int lim = row_valid ? qrow + offi - kb - 4 * h : -1000000;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float x = (8 * (r >> 2) + (r & 3) <= lim) ? s[r] : kNegInf;
            sv[r] = x;
            mt = fmaxf(mt, x);
          }
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            sv[r] = s[r];
            mt = fmaxf(mt, sv[r]);
          }
        }
        // the row max of the raw scores, then scaled (scale2 > 0 and rounding is
        // monotonic, so this is the max of the scaled scores)
        mt = halves_max(mt) * p.scale2;

        // the online test (rows with no legal key in the tile do not vote); m + log2(l)
        // is log2 of the retained normalizer whichever reference m the row uses
        const bool voter = row_valid & (kb <= qrow + offi);
        const bool demand = voter & ((l == 0.f) | (mt - m - fast_log2(l) >= thr));
        if (!wave_any(demand)) continue;    // skipped: m, l and O unchanged
        ++n_ret;
        // off the diagonal every valid row votes: those tiles are counted per wavefront
        if (need_mask) {
          ++n_ret_m;
          cnt += voter ? 1 : 0;
        }
        // O^T[d][q] += V^T[d][key] P^T[key][q]; V^T rows through transposed LDS reads,
        // issued before the softmax work so that their latency hides under it
        bf16x8 va[DB][2];
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const bf16* vt = vtb + (sub * kBk + 16 * ks) * (D + 8) + tr_step<D>(db);
            va[db][ks] = cat(lds_read_tr(vt), lds_read_tr(vt + 8 * (D + 8)));
          }
        if (stats) {
          hsum += tile_hash(b, hq, q0w / kBq, j);
          // the first wavefront to retain this tile of the stage counts its V tile
          if (lane == 0) vtag[sub] = atomicExch(&vneed[buf][sub], t + 1);
        }

        // Lazy rescaling: a row's reference m moves only when some row of the
        // wavefront would otherwise see P = exp2(s - m) above 2^8; O and l are then
        // rescaled.  The result is the same softmax; P stays in [0, 2^8].
        if (wave_any(mt > m + 8.f)) {
          const float m_new = fmaxf(m, mt);
          const float alpha = (m_new == kNegInf) ? 1.f : fast_exp2(m - m_new);
          l *= alpha;
          m = m_new;
#pragma unroll
          for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[db][r] *= alpha;
        }
        // a row with no legal key so far keeps m = -inf: shift by 0 so exp2(-inf) = 0
        const float shift = (m == kNegInf) ? 0.f : m;
        // P = exp2(s scale2 - shift) with one rounding; the row sum as a tree
#pragma unroll
        for (int r = 0; r < 16; ++r) sv[r] = fast_exp2(__builtin_fmaf(sv[r], p.scale2, -shift));
        float ps4[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) ps4[g] = (sv[4 * g] + sv[4 * g + 1]) + (sv[4 * g + 2] + sv[4 * g + 3]);
        const float ps = halves_sum((ps4[0] + ps4[1]) + (ps4[2] + ps4[3]));
        l += ps;
        // P as two bf16 terms where it matters: the backward's D = rowsum(O * dO)
        // cancels against dP for dominant keys, so their probabilities must be
        // accurate well beyond one bf16 rounding.  A tile whose mass is a small
        // share of every row's retained normalizer (this tile included) runs the
        // high term only.
        const bool need_lo = wave_any(ps > kFwdLoShare * l);
        const bf16x8 ph[2] = {hi_bf16x8(sv), hi_bf16x8(sv + 8)};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int db = 0; db < DB; ++db) acc[db] = mfma32(va[db][ks], ph[ks], acc[db]);
        if (need_lo) {
          const bf16x8 pl[2] = {lo_bf16x8(sv, ph[0]), lo_bf16x8(sv + 8, ph[1])};
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int db = 0; db < DB; ++db) acc[db] = mfma32(va[db][ks], pl[ks], acc[db]);
        }
      }
    }
    wait_vm();
    __syncthreads();
    n_vneed += (vtag[0] != t + 1) + (vtag[1] != t + 1);
  }

  // epilogue: O <- O / l, LSE = (m + log2 l) * ln 2
  if (row_valid) {
    const float inv = 1.f / l;
    const long orow = (qbase + qrow) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 v4 = {acc[db][4 * g] * inv, acc[db][4 * g + 1] * inv, acc[db][4 * g + 2] * inv,
                    acc[db][4 * g + 3] * inv};
        store_out4(p.o, orow + 32 * db + 8 * g + 4 * h, v4, p.o_bf16);
      }
    if (h == 0) {
      p.lse[qbase + qrow] = (m + fast_log2(l)) * kLn2;
      if (p.row_tiles) p.row_tiles[qbase + qrow] = cnt + (int)(n_ret - n_ret_m);
    }
  }
  if (stats) {
    if (lane == 0) {
      blk_add(bcnt, kCntLegal, n_legal);
      blk_add(bcnt, kCntRetained, n_ret);
      blk_add(bcnt, kCntSlots, (unsigned long long)n_ret * kBk * nvalid);
      blk_add(bcnt, kCntSetHash, hsum);
      blk_add(bcnt, kCntVNeeded, n_vneed);
    }
    if (tid == 0) blk_add(bcnt, kCntVTiles, (unsigned long long)(ttop + 1) * (kFwdStage / kBk));
    blk_flush(bcnt, p.counters);
  }
}

hipError_t launch_fwd(const FwdParams& p, int D, hipStream_t st) {
  dim3 grid((unsigned)p.nqblk * p.B * p.Hq), block(kFwdWaves * 64);
  if (D == 128)
    hipLaunchKernelGGL(mala_fwd_kernel<128>, grid, block, 0, st, p);
  else
    hipLaunchKernelGGL(mala_fwd_kernel<64>, grid, block, 0, st, p);
  return hipGetLastError();
}

}  // namespace mala
