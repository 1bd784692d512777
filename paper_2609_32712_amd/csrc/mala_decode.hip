// MALA split-KV decode for gfx950 (Fused Execution section and its appendix:
// each split tests its tiles against its own partial normalizer, with L = Nk).
//
// One wavefront (= one workgroup) owns one split of one (batch, KV head) and
// serves up to 16 query heads of the GQA group at once (larger groups take
// ceil(group / 16) wavefronts), so the K and V bytes of a tile are read once per
// 16 heads.  Decode is HBM-bound: K is always read (score
// discovery), V only when at least one head of the group retains the tile.
//
// With per-sequence cache lengths n_b, sequence b sees keys [0, n_b) (L = n_b) and
// its ceil(n_b / 32) tiles are cut into the splits as for a cache of n_b tokens.
//
// Per 32-key tile, in descending order inside the split:
//   S^T = K_t Q^T     2 x 4 (D = 128) MFMAs 16x16x32; K arrives in registers in
//                     whole contiguous rows (1 KB per load instruction), passes
//                     through LDS and is read back as the A operands; lane
//                     (g, col) holds query head col and 8 of the 32 keys; K is
//                     prefetched two tiles ahead
//   test              per head against that head's running (m, l) of the split
//   retained (any)    V tile (fetched one tile ahead when a look-ahead test says
//                     it may be needed) -> LDS; per head P = exp2(S - m_new) (0 for
//                     heads that skip); O^T += V^T P^T with V^T through
//                     ds_read_b64_tr_b16.
// Every K and V load is a streaming buffer load (each byte is read once per call)
// that is always issued: rows past the cache length, tiles outside the split and V
// tiles the look-ahead test rules out have a resource of 0 bytes, read as zeros and
// move no data.  With no load under a
// branch, the compiler's waits count exactly the loads a step needs, so the next
// K tile and the next V tile stay in flight while a tile is processed.
// Partials (O / l, lse, count) go to the workspace; a second kernel merges the
// splits with the normalizer-aware (log-sum-exp weighted) reduction.
#include "mala_device.h"
#include "mala_kernels.h"

namespace mala {

template <int D>
__global__ __launch_bounds__(64) void mala_decode_split_kernel(DecParams p) {
  constexpr int KS = D / 32;   // k-steps of 32 over head_dim
  constexpr int NDB = D / 16;  // 16-row blocks of O^T
  constexpr int LD = D + 8;
  constexpr int VCH = kDecBk * D / 8 / 64;   // 16-byte V chunks per lane per tile
  __shared__ __attribute__((aligned(16))) bf16 Ks[kDecBk * LD];
  __shared__ __attribute__((aligned(16))) bf16 Vs[kDecBk * LD];

  const int lane = threadIdx.x, g = lane >> 4, col = lane & 15;
  const int s = blockIdx.x % p.S;
  const int chunk = (blockIdx.x / p.S) % p.nchunk;     // heads 16 chunk .. 16 chunk + 15
  const int bhk = blockIdx.x / p.S / p.nchunk;
  const int b = bhk / p.Hkv, hkv = bhk % p.Hkv, grp = p.Hq / p.Hkv;
  const int nh = min(16, grp - 16 * chunk);             // query heads of this wavefront
  // this sequence's cache length n (clamped into [0, Nk]), its tiles and split range
  int n = p.Nk, T = p.T, tps = p.tps;
  float thr2 = p.thr2;
  if (p.lens) {
    n = min(max(p.lens[b], 0), p.Nk);
    T = (n + kDecBk - 1) / kDecBk;
    tps = (T + p.S - 1) / p.S;
    thr2 = p.log2tau - log2f((float)n);   // L = n (n = 0 leaves no tile to test)
  }
  const int t_lo = s * tps, t_hi = min(T, t_lo + tps);
  const bool head_valid = col < nh;
  const int hq = hkv * grp + 16 * chunk + col;

  bf16x8 qreg[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk)
    qreg[kk] = head_valid ? load8(p.q + ((long)b * p.Hq + hq) * D + 32 * kk + 8 * g) : zero8();
  wait_vm();   // no wait for these loads is left for the tile loop

  const bf16* Kp = p.k + (long)bhk * p.Nk * D;
  const bf16* Vp = p.v + (long)bhk * p.Nk * D;

  float m = kNegInf, l = 0.f;
  f32x4 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  int cnt = 0;
  unsigned vloads = 0, vfetch = 0;   // V tiles consumed / fetched (statistics)
  unsigned long long hsum = 0;       // fingerprints of this head's retained tiles

  // A K or V tile in registers as whole rows: lane chunk e holds the 16 bytes at
  // byte 16 (lane + 64 e) of the tile, row (lane + 64 e) / (D / 8).  The resource
  // covers the tile's rows below n when the tile is wanted and nothing otherwise.
  auto tile_rsrc = [&](const bf16* base, int t, bool want) {
    const long k0 = (long)max(t, 0) * kDecBk;
    const long rows = want && t >= 0 ? min((long)kDecBk, (long)n - k0) : 0;
    return make_rsrc(base + k0 * D, (uint32_t)(rows > 0 ? rows * D * 2 : 0));
  };
  bf16x8 kr[VCH], vr[VCH];
  auto load_k = [&](int t) {
    const auto r = tile_rsrc(Kp, t, t >= t_lo);
#pragma unroll
    for (int e = 0; e < VCH; ++e) kr[e] = buf_load8_stream(r, 16u * (lane + 64 * e));
  };
  auto load_v = [&](int t, bool want) {
    const auto r = tile_rsrc(Vp, t, want && t >= t_lo);
#pragma unroll
    for (int e = 0; e < VCH; ++e) vr[e] = buf_load8_stream(r, 16u * (lane + 64 * e));
  };
  // tile rows to LDS (row stride LD keeps the operand reads below conflict-free)
  auto to_lds = [&](bf16* dst, const bf16x8 (&x)[VCH]) {
#pragma unroll
    for (int e = 0; e < VCH; ++e) {
      const int ch = lane + 64 * e;
      store8(dst + (ch / (D / 8)) * LD + (ch % (D / 8)) * 8, x[e]);
    }
  };
  // Base-2 scores of the tile whose K is in kr, for this lane's head (8 keys), and
  // their max over the tile; the next K tile (t - 1) starts loading as soon as kr
  // is in LDS.  One wavefront per workgroup: its LDS accesses complete in issue
  // order, so the reads below see the stores and the next stores follow the reads.
  auto scores = [&](int t, float (&sv)[8]) {
    to_lds(Ks, kr);
    load_k(t - 1);
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      s0 = mfma16(load8(Ks + col * LD + 32 * kk + 8 * g), qreg[kk], s0);
      s1 = mfma16(load8(Ks + (16 + col) * LD + 32 * kk + 8 * g), qreg[kk], s1);
    }
    const long kb = (long)t * kDecBk;
    float mt = kNegInf;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float x0 = s0[r] * p.scale2, x1 = s1[r] * p.scale2;
      if (kb + 4 * g + r >= n) x0 = kNegInf;
      if (kb + 16 + 4 * g + r >= n) x1 = kNegInf;
      sv[r] = x0;
      sv[4 + r] = x1;
      mt = fmaxf(mt, fmaxf(x0, x1));
    }
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    return fmaxf(mt, __shfl_xor(mt, 32));
  };

  // Pipeline: while tile t is decided and processed, K of tile t - 1 is already in
  // registers (its scores are computed first) and K of t - 2 is loading.  Whether
  // tile t - 1 can still be retained is checked against the state BEFORE tile t's
  // update; since the retained normalizer only grows, a tile that fails this check
  // fails the real test too, so V of t - 1 is fetched early exactly when it may be
  // needed (with a small margin against fp32 rounding of the normalizer).
  constexpr float kHintMargin = 1e-2f;
  float sv[8], sn[8];
  float mt = kNegInf, mtn = kNegInf;
  if (t_hi > t_lo) {
    load_k(t_hi - 1);
    mt = scores(t_hi - 1, sv);   // also starts K of t_hi - 2
    load_v(t_hi - 1, true);      // the first tile of a split is always retained (l = 0)
    ++vfetch;
  }
  for (int t = t_hi - 1; t >= t_lo; --t) {
    const bool has_next = t - 1 >= t_lo;
    mtn = scores(t - 1, sn);     // zeros past the split's first tile, not used then
    const float lse_run = m + fast_log2(l);
    const bool demand = head_valid && (l == 0.f || (mt - lse_run >= thr2));
    const bool hint =
        has_next && wave_any(head_valid && (l == 0.f || (mtn - lse_run >= thr2 - kHintMargin)));
    // V of tile t goes to LDS, and V of t - 1 (if the look-ahead test wants it) starts
    // loading into the freed registers before tile t's update runs
    const bool any_demand = wave_any(demand);
    if (any_demand) to_lds(Vs, vr);
    load_v(t - 1, hint);
    vfetch += hint ? 1u : 0u;
    if (any_demand) {
      ++vloads;
      float alpha = 1.f, m_new = m;
      if (demand) {
        m_new = fmaxf(m, mt);
        alpha = fast_exp2(m - m_new);
      }
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const float e = demand ? fast_exp2(sv[r] - m_new) : 0.f;
        sv[r] = e;
        ps += e;
      }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      if (demand) {
        l = alpha * l + ps;
        m = m_new;
        ++cnt;
        if (p.counters) hsum += tile_hash(b, hq, 0, t);
      }
      bf16x8 ph, pl;
      split_bf16x8(sv, ph, pl);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16* vrow = Vs + (4 * g + (col >> 2)) * LD + 16 * db + 4 * (col & 3);
        const bf16x8 a = cat(lds_read_tr(vrow), lds_read_tr(vrow + 16 * LD));
        acc[db] = mfma16(a, ph, acc[db] * alpha);
        acc[db] = mfma16(a, pl, acc[db]);
      }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) sv[r] = sn[r];
    mt = mtn;
  }

  // partial of this split: O / l, lse (natural log) and the retained-tile count.  A
  // split without tiles has l = 0 (o = 0, lse = -inf: the merge skips it); a NaN or
  // Inf input leaves l NaN, which must reach the merge as NaN, not as an empty split.
  float* pp = p.part + (((long)b * p.Hq + hq) * p.S + s) * (D + kDecStride);
  if (head_valid) {
    const float inv = l != 0.f ? 1.f / l : 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      *reinterpret_cast<f32x4*>(pp + 16 * db + 4 * g) = acc[db] * inv;
    if (g == 0) {
      pp[D] = l != 0.f ? (m + fast_log2(l)) * kLn2 : kNegInf;
      pp[D + 1] = __int_as_float(cnt);
    }
  }
  if (p.counters) {
    if (head_valid && g == 0 && cnt) {
      atomicAdd(&p.counters[kCntRetained], (unsigned long long)cnt);
      atomicAdd(&p.counters[kCntSlots], (unsigned long long)cnt * kDecBk);
      atomicAdd(&p.counters[kCntSetHash], hsum);
    }
    if (lane == 0) {
      atomicAdd(&p.counters[kCntLegal], (unsigned long long)(t_hi > t_lo ? t_hi - t_lo : 0) * nh);
      if (vfetch) atomicAdd(&p.counters[kCntVTiles], (unsigned long long)vfetch);
      if (vloads) atomicAdd(&p.counters[kCntVNeeded], (unsigned long long)vloads);
    }
  }
}

// Normalizer-aware merge of the split partials: lse = logsumexp_s lse_s,
// o = sum_s exp(lse_s - lse) o_s.  One workgroup per (batch, query head).
template <int D>
__global__ __launch_bounds__(64) void mala_decode_combine_kernel(const float* part, void* o,
                                                                 bool o_bf16, float* lse,
                                                                 int32_t* head_tiles, int S) {
  const long bh = blockIdx.x;
  const float* pp = part + bh * S * (D + kDecStride);
  float mx = kNegInf;
  for (int s = 0; s < S; ++s) mx = fmaxf(mx, pp[(long)s * (D + kDecStride) + D]);
  float z = 0.f;
  int cnt = 0;
  for (int s = 0; s < S; ++s) {
    const float ls = pp[(long)s * (D + kDecStride) + D];
    if (ls != kNegInf) z += expf(ls - mx);
    cnt += __float_as_int(pp[(long)s * (D + kDecStride) + D + 1]);
  }
  const float L = mx + logf(z);
  for (int d = threadIdx.x; d < D; d += 64) {
    float acc = 0.f;
    for (int s = 0; s < S; ++s) {
      const float ls = pp[(long)s * (D + kDecStride) + D];
      if (ls != kNegInf) acc += expf(ls - L) * pp[(long)s * (D + kDecStride) + d];
    }
    if (o_bf16)
      static_cast<bf16*>(o)[bh * D + d] = (bf16)acc;   // nearest even
    else
      static_cast<float*>(o)[bh * D + d] = acc;
  }
  if (threadIdx.x == 0) {
    lse[bh] = L;
    if (head_tiles) head_tiles[bh] = cnt;
  }
}

hipError_t launch_decode(const DecParams& p, int D, hipStream_t st) {
  dim3 grid((unsigned)p.B * p.Hkv * p.nchunk * p.S), block(64);
  if (D == 128)
    hipLaunchKernelGGL(mala_decode_split_kernel<128>, grid, block, 0, st, p);
  else
    hipLaunchKernelGGL(mala_decode_split_kernel<64>, grid, block, 0, st, p);
  return hipGetLastError();
}

hipError_t launch_decode_combine(const float* part, void* o, bool o_bf16, float* lse,
                                 int32_t* head_tiles, int BH, int S, int D, hipStream_t st) {
  dim3 grid((unsigned)BH), block(64);
  if (D == 128)
    hipLaunchKernelGGL(mala_decode_combine_kernel<128>, grid, block, 0, st, part, o, o_bf16,
                       lse, head_tiles, S);
  else
    hipLaunchKernelGGL(mala_decode_combine_kernel<64>, grid, block, 0, st, part, o, o_bf16,
                       lse, head_tiles, S);
  return hipGetLastError();
}

}  // namespace mala
