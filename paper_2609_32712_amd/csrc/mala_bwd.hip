// MALA backward (Algorithm 2) for gfx950.
//
// Key-major: one workgroup owns 128 keys of one (batch, KV head) and keeps their
// dK and dV in registers for the whole kernel (no atomics on dK/dV); it loops
// over every query head of the GQA group and over the query tiles from the
// diagonal to the end.  Wavefront w owns keys [32w, 32w + 32) of the block, so a
// wavefront's work on one query tile is exactly one 32 x 32 decision tile.
//
// Per query tile (32 rows), staged once per workgroup in double-buffered LDS (Q,
// dO, and the per-row base-2 LSE, test threshold and D_q = rowsum(O * dO)); the
// next tile is fetched into registers while the current one is processed:
//   S = Q_i K_w^T         8 MFMAs (lane = one key column, 16 query rows)
//   offline test          retain iff some valid entry has
//                         s - lse_q >= log2(tau) - log2(L_q) (base-2 units); ballot
//   retained path         P = exp2(S - lse); dP = dO_i V_w^T; dS = P (dP - D_q);
//                         P and dS are split into two bf16 terms (hi + lo), then
//                         dV^T += dO_i^T P; dK^T += Q_i^T dS (A operands through
//                         ds_read_b64_tr_b16); both dS planes are written to LDS
//   dQ                    after a barrier each wavefront forms one 32-column slice of
//                         dQ_i = dS K_j over the retained decision tiles of the block
//                         and adds it to dq with fp32 atomics.
// A skipped tile costs its QK MFMAs and the test only.
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

// D_q = sum_d O[q][d] * dO[q][d]; 16 lanes per row.
template <int D>
__global__ __launch_bounds__(256) void mala_bwd_preprocess_kernel(const float* o, const bf16* dout,
                                                                  float* dvec, long rows) {
  constexpr int PER = D / 16;
  const long row = (long)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int part = threadIdx.x & 15;
  float s = 0.f;
  if (row < rows) {
    const float* op = o + row * D + part * PER;
    const bf16* dp = dout + row * D + part * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) s += op[e] * (float)dp[e];
  }
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1) s += __shfl_xor(s, w, 16);
  if (row < rows && part == 0) dvec[row] = s;
}

hipError_t launch_bwd_preprocess(const float* o, const bf16* dout, float* dvec, long rows, int D,
                                 hipStream_t st) {
  const unsigned grid = (unsigned)((rows + 15) / 16);
  if (D == 128)
    hipLaunchKernelGGL(mala_bwd_preprocess_kernel<128>, dim3(grid), dim3(256), 0, st, o, dout,
                       dvec, rows);
  else
    hipLaunchKernelGGL(mala_bwd_preprocess_kernel<64>, dim3(grid), dim3(256), 0, st, o, dout,
                       dvec, rows);
  return hipGetLastError();
}

template <int D>
__global__ __launch_bounds__(256) void mala_bwd_kernel(BwdParams p) {
  constexpr int KS = D / 16;       // k-steps over head_dim
  constexpr int DB = D / 32;       // 32-wide column blocks
  constexpr int DSS = kBq + 16;    // dS row stride [key][q]: 24 dwords, conflict-free tr reads
  constexpr int WPB = 4 / DB;      // wavefronts per dQ column block
  constexpr int QK = kBwdKeys / WPB;   // keys one wavefront sums for its dQ slice
  constexpr int TILE = tile_elems<D>(kBq);   // one Q or dO tile in LDS
  constexpr int CPT = kBq * D / 8 / 256;   // 16-byte chunks per thread per tile
  // K_j (row-major) is only needed until the dQ operands are in registers; its LDS
  // is then reused for the two bf16 planes (hi, lo) of dS stored as [key][q].
  constexpr int KT_ELEMS = tile_elems<D>(kBwdKeys);
  constexpr int DS_ELEMS = 2 * kBwdKeys * DSS;
  __shared__ __attribute__((aligned(16))) bf16 shared_kt_ds[KT_ELEMS > DS_ELEMS ? KT_ELEMS : DS_ELEMS];
  // double-buffered query tiles: the next tile is fetched into registers while the
  // current one is processed, then written to the other buffer
  __shared__ __attribute__((aligned(16))) bf16 Qs[2 * TILE];
  __shared__ __attribute__((aligned(16))) bf16 dOs[2 * TILE];
  __shared__ __attribute__((aligned(16))) float rowv[2][3][kBq];   // base-2 lse, threshold, D_q
  __shared__ int flags[4];
  bf16* const Kt = shared_kt_ds;
  bf16* const dSh = shared_kt_ds;
  bf16* const dSl = shared_kt_ds + kBwdKeys * DSS;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, c = lane & 31, G = lane >> 4, t16 = lane & 15;
  const int BHk = p.B * p.Hkv;
  const int bhk = blockIdx.x % BHk;
  const int kblk = blockIdx.x / BHk;       // ascending: the longest key blocks first
  const int b = bhk / p.Hkv, hkv = bhk % p.Hkv, grp = p.Hq / p.Hkv;
  const long off = (long)p.Nk - p.Nq;
  const int kb0 = kblk * kBwdKeys;
  const int kw = kb0 + wave * kBk;         // first key of this wavefront's decision tile
  const int key = kw + c;                  // this lane's key (C-layout column)

  const bf16* Kp = p.k + (long)bhk * p.Nk * D;
  const bf16* Vp = p.v + (long)bhk * p.Nk * D;

  // K_j -> LDS (row-major) for the dQ product
  for (int ch = tid; ch < kBwdKeys * D / 8; ch += 256) {
    const int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
    const long kk = (long)kb0 + row;
    store8(Kt + tile_off<D>(row, col), kk < p.Nk ? load8(Kp + kk * D + col) : zero8());
  }
  // K_w, V_w rows as B operands of S = Q K^T and dP = dO V^T
  bf16x8 kreg[KS], vreg[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    kreg[kk] = key < p.Nk ? load8(Kp + (long)key * D + 16 * kk + 8 * h) : zero8();
    vreg[kk] = key < p.Nk ? load8(Vp + (long)key * D + 16 * kk + 8 * h) : zero8();
  }
  __syncthreads();
  // K rows [kq0, kq0 + QK) x columns [32 dqb, 32 dqb + 32) as B operands of dQ = dS K
  const int dqb = wave % DB;
  const int kq0 = (wave / DB) * QK;
  bf16x8 ktreg[QK / 16];
#pragma unroll
  for (int ks = 0; ks < QK / 16; ++ks) {
    const int krow = kq0 + 16 * ks + 4 * h + (t16 >> 2);
    const int kcol = 32 * dqb + 16 * (G & 1) + 4 * (t16 & 3);
    ktreg[ks] = cat(lds_read_tr(Kt + tile_off<D>(krow, kcol)), lds_read_tr(Kt + tile_off<D>(krow + 8, kcol)));
  }

  f32x16 dvacc[DB], dkacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dvacc[db][r] = dkacc[db][r] = 0.f;

  unsigned n_legal = 0, n_ret = 0;
  unsigned long long slots = 0;
  const long first_q = (long)kb0 - off;
  const int qi_start = first_q <= 0 ? 0 : (int)(first_q / kBq);
  const int nqt = (p.Nq + kBq - 1) / kBq;
  const int per_head = nqt - qi_start;     // >= 1: key kb0 < Nk is visible to row Nq - 1
  const int total = grp * per_head;

  // prefetch registers of the next query tile
  bf16x8 pq[CPT], pdo[CPT];
  float plse = 0.f, pdv = 0.f;
  auto fetch = [&](int it) {
    const long bhq = (long)b * p.Hq + hkv * grp + it / per_head;
    const int q0 = (qi_start + it % per_head) * kBq;
#pragma unroll
    for (int e = 0; e < CPT; ++e) {
      const int ch = tid + 256 * e;
      const int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
      const long qq = (long)q0 + row;
      const bool ok = qq < p.Nq;
      pq[e] = ok ? load8(p.q + (bhq * p.Nq + qq) * D + col) : zero8();
      pdo[e] = ok ? load8(p.dout + (bhq * p.Nq + qq) * D + col) : zero8();
    }
    if (tid < kBq) {
      const long qq = (long)q0 + tid;
      if (qq < p.Nq) {
        plse = p.lse[bhq * p.Nq + qq];
        pdv = p.dvec[bhq * p.Nq + qq];
      }
    }
  };
  auto stash = [&](int it, int buf) {
    const int q0 = (qi_start + it % per_head) * kBq;
#pragma unroll
    for (int e = 0; e < CPT; ++e) {
      const int ch = tid + 256 * e;
      const int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
      store8(Qs + buf * TILE + tile_off<D>(row, col), pq[e]);
      store8(dOs + buf * TILE + tile_off<D>(row, col), pdo[e]);
    }
    if (tid < kBq) {
      const long qq = (long)q0 + tid;
      if (qq < p.Nq) {
        const float l2 = plse * kLog2e;
        rowv[buf][0][tid] = l2;
        rowv[buf][1][tid] = l2 + p.log2tau - log2f((float)(qq + 1 + off));
        rowv[buf][2][tid] = pdv;
      } else {
        rowv[buf][0][tid] = 0.f;
        rowv[buf][1][tid] = __builtin_huge_valf();   // padded rows never retain
        rowv[buf][2][tid] = 0.f;
      }
    }
  };

  fetch(0);
  __syncthreads();   // every wavefront holds its dQ operands: K_j's LDS becomes the dS planes
  stash(0, 0);
  __syncthreads();

  for (int it = 0; it < total; ++it) {
    const int buf = it & 1;
    const long bhq = (long)b * p.Hq + hkv * grp + it / per_head;
    const int q0 = (qi_start + it % per_head) * kBq;
    if (it + 1 < total) fetch(it + 1);
    const bf16* Qb = Qs + buf * TILE;
    const bf16* dOb = dOs + buf * TILE;
    const float* lse2s = rowv[buf][0];
    const float* thrs = rowv[buf][1];
    const float* Dsv = rowv[buf][2];

    const int qlast = min(q0 + kBq - 1, p.Nq - 1);
    const bool legal_tile = (kw < p.Nk) && ((long)kw <= (long)qlast + off);
    bool ret = false;
    if (legal_tile) {
      ++n_legal;
      // S = Q_i K_w^T as two independent chains (even / odd k-steps), operands read first
      f32x16 s, s_odd;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = s_odd[r] = 0.f;
      {
        bf16x8 qa[KS];
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) qa[kk] = load8(Qb + tile_off<D>(c, 16 * kk + 8 * h));
#pragma unroll
        for (int kk = 0; kk < KS; kk += 2) {
          s = mfma32(qa[kk], kreg[kk], s);
          s_odd = mfma32(qa[kk + 1], kreg[kk + 1], s_odd);
        }
      }
      s += s_odd;
      const bool need_mask =
          ((long)kw + kBk - 1 > (long)q0 + off) || (q0 + kBq > p.Nq) || (kw + kBk > p.Nk);
      float sv[16];
      bool dem = false;
      // rows of this lane: q0 + 8 g + 4 h + e; entry legal iff row < Nq, key < Nk and
      // key <= row + off, i.e. 8 g + e in [klo, qlim)
      const int klo = key < p.Nk ? (int)((long)key - off - q0) - 4 * h : 1000000;
      const int qlim = p.Nq - q0 - 4 * h;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 th = *reinterpret_cast<const f32x4*>(thrs + 8 * g + 4 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * g + e;
          float x = s[r] * p.scale2;
          if (need_mask && (8 * g + e < klo || 8 * g + e >= qlim)) x = kNegInf;
          sv[r] = x;
          dem |= (x != kNegInf) && (x >= th[e]);
        }
      }
      ret = wave_any(dem);
      if (ret) {
        ++n_ret;
        slots += (unsigned long long)kBk * (unsigned)(qlast - q0 + 1);
        // P = exp2(S - lse)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse2s + 8 * g + 4 * h);
#pragma unroll
          for (int e = 0; e < 4; ++e) sv[4 * g + e] = fast_exp2(sv[4 * g + e] - l4[e]);
        }
        // dP = dO_i V_w^T
        f32x16 dp, dp_odd;
#pragma unroll
        for (int r = 0; r < 16; ++r) dp[r] = dp_odd[r] = 0.f;
        {
          bf16x8 oa[KS];
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) oa[kk] = load8(dOb + tile_off<D>(c, 16 * kk + 8 * h));
#pragma unroll
          for (int kk = 0; kk < KS; kk += 2) {
            dp = mfma32(oa[kk], vreg[kk], dp);
            dp_odd = mfma32(oa[kk + 1], vreg[kk + 1], dp_odd);
          }
        }
        dp += dp_odd;
        float dsv[16];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(Dsv + 8 * g + 4 * h);
#pragma unroll
          for (int e = 0; e < 4; ++e) dsv[4 * g + e] = sv[4 * g + e] * (dp[4 * g + e] - d4[e]);
        }
        bf16x8 ph[2], pl[2], dh[2], dl[2];
        split_bf16x8(sv, ph[0], pl[0]);
        split_bf16x8(sv + 8, ph[1], pl[1]);
        split_bf16x8(dsv, dh[0], dl[0]);
        split_bf16x8(dsv + 8, dh[1], dl[1]);
        // dV^T[d][key] += dO^T[d][q] P[q][key];  dK^T[d][key] += Q^T[d][q] dS[q][key]
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const int trow = 16 * ks + 4 * h + (t16 >> 2);
            const int tcol = 32 * db + 16 * (G & 1) + 4 * (t16 & 3);
            const int ro = tile_off<D>(trow, tcol), ro8 = tile_off<D>(trow + 8, tcol);
            const bf16x8 ao = cat(lds_read_tr(dOb + ro), lds_read_tr(dOb + ro8));
            dvacc[db] = mfma32(ao, ph[ks], dvacc[db]);
            dvacc[db] = mfma32(ao, pl[ks], dvacc[db]);
            const bf16x8 aq = cat(lds_read_tr(Qb + ro), lds_read_tr(Qb + ro8));
            dkacc[db] = mfma32(aq, dh[ks], dkacc[db]);
            dkacc[db] = mfma32(aq, dl[ks], dkacc[db]);
          }
        }
        // dS (hi and lo planes) -> LDS as [key][q] for the dQ product
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const bf16x8& hs = dh[g >> 1];
          const bf16x8& ls = dl[g >> 1];
          const int o4 = 4 * (g & 1);
          bf16x4 wh = {hs[o4], hs[o4 + 1], hs[o4 + 2], hs[o4 + 3]};
          bf16x4 wl = {ls[o4], ls[o4 + 1], ls[o4 + 2], ls[o4 + 3]};
          *reinterpret_cast<bf16x4*>(dSh + (wave * kBk + c) * DSS + 8 * g + 4 * h) = wh;
          *reinterpret_cast<bf16x4*>(dSl + (wave * kBk + c) * DSS + 8 * g + 4 * h) = wl;
        }
      }
    }
    if (lane == 0) flags[wave] = ret ? 1 : 0;
    __syncthreads();

    // per-row statistics: retained tiles of this workgroup in which the row has a key
    if (p.row_tiles && wave == 0 && lane < kBq) {
      const long qq = (long)q0 + lane;
      if (qq < p.Nq) {
        int n = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const long kww = (long)kb0 + w * kBk;
          n += (flags[w] && kww < p.Nk && kww <= qq + off) ? 1 : 0;
        }
        if (n) atomicAdd(p.row_tiles + bhq * p.Nq + qq, n);
      }
    }

    // dQ_i[:, 32 dqb .. +32] = sum over retained tiles of dS K  (fp32 atomics)
    // hi and lo planes accumulate in separate chains
    f32x16 dqacc, dqlo;
#pragma unroll
    for (int r = 0; r < 16; ++r) dqacc[r] = dqlo[r] = 0.f;
    bool any = false;
#pragma unroll
    for (int ks = 0; ks < QK / 16; ++ks) {
      if (!flags[(kq0 + 16 * ks) / kBk]) continue;
      any = true;
      const int ao = (kq0 + 16 * ks + 4 * h + (t16 >> 2)) * DSS + 16 * (G & 1) + 4 * (t16 & 3);
      const bf16x8 ah = cat(lds_read_tr(dSh + ao), lds_read_tr(dSh + ao + 8 * DSS));
      const bf16x8 al = cat(lds_read_tr(dSl + ao), lds_read_tr(dSl + ao + 8 * DSS));
      dqacc = mfma32(ah, ktreg[ks], dqacc);
      dqlo = mfma32(al, ktreg[ks], dqlo);
    }
    dqacc += dqlo;
    if (any) {
      float* dqp = p.dq + (bhq * p.Nq) * D + 32 * dqb + c;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const long qq = (long)q0 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (qq < p.Nq) atomicAdd(dqp + qq * D, dqacc[r] * p.scale);
      }
    }
    if (it + 1 < total) stash(it + 1, buf ^ 1);
    __syncthreads();
  }

  // dK = scale * sum dS^T Q, dV = sum P^T dO; lane (h, c) holds key kw + c
  if (key < p.Nk) {
    float* dkp = p.dk + ((long)bhk * p.Nk + key) * D;
    float* dvp = p.dv + ((long)bhk * p.Nk + key) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int d = 32 * db + 8 * g + 4 * h;
        f32x4 k4 = {dkacc[db][4 * g] * p.scale, dkacc[db][4 * g + 1] * p.scale,
                    dkacc[db][4 * g + 2] * p.scale, dkacc[db][4 * g + 3] * p.scale};
        f32x4 v4 = {dvacc[db][4 * g], dvacc[db][4 * g + 1], dvacc[db][4 * g + 2], dvacc[db][4 * g + 3]};
        *reinterpret_cast<f32x4*>(dkp + d) = k4;
        *reinterpret_cast<f32x4*>(dvp + d) = v4;
      }
  }
  if (p.counters) {
    if (lane == 0 && n_legal) {
      atomicAdd(&p.counters[0], (unsigned long long)n_legal);
      atomicAdd(&p.counters[1], (unsigned long long)n_ret);
      atomicAdd(&p.counters[3], slots);
    }
    if (tid == 0) atomicAdd(&p.counters[2], (unsigned long long)total);
  }
}

hipError_t launch_bwd(const BwdParams& p, int D, hipStream_t st) {
  dim3 grid((unsigned)p.nkblk * p.B * p.Hkv), block(256);
  if (D == 128)
    hipLaunchKernelGGL(mala_bwd_kernel<128>, grid, block, 0, st, p);
  else
    hipLaunchKernelGGL(mala_bwd_kernel<64>, grid, block, 0, st, p);
  return hipGetLastError();
}

}  // namespace mala
