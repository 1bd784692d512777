/*
 * MALA oracle: plain, slow, fp64 CPU reference for causal attention and for the
 * MassAlloc (MALA) allocation rule.  TEST INFRASTRUCTURE ONLY: it is linked by
 * the tests, by the smoke check and by the benchmark's cpu_baseline leg, never by
 * the product library, and it shares no code with the HIP path.
 *
 * Everything here works on ONE attention head (one query head paired with the
 * key/value head it reads).  Arrays are row-major fp64:
 *   q, o, dO : [Nq][D]      k, v : [Nk][D]      lse : [Nq]
 * Scores are s_qk = scale * <q_q, k_k> in fp64 (the paper absorbs the softmax
 * scale into Q; here it is applied to the fp64 dot product, which is the same
 * real number without an extra rounding of Q).  Natural exp/log throughout
 * (Methodology, "Attention as a Compute Allocator").
 *
 * Causal visibility is bottom-right aligned: query row q sees keys
 * k <= q + (Nk - Nq), so L_q = q + 1 + (Nk - Nq).  With Nq == Nk this is the
 * paper's L_q = q + 1; for one decode token it is L_0 = Nk (same section).
 *
 * Parity with the paper, function by function:
 *   oracle_dense_fwd / oracle_dense_bwd : the definition of softmax attention and
 *       of its gradient (the FullAttn limit, Attention Cost section, tau -> 0).
 *   oracle_mala_fwd  : Algorithm 1 (MALA Forward) with the online test of
 *       Eq. (online test) and the empty-state convention of the Online Sparse
 *       Softmax paragraph.
 *   oracle_mala_bwd  : Algorithm 2 (MALA Backward) with the offline test of
 *       Eq. (offline test).
 *   oracle_mala_decode : the split-KV decode of the Fused Execution section and
 *       of the appendix "Fused decoding execution": Algorithm 1's rule applied
 *       per split with B_q = 1 and L = Nk, then the normalizer-aware merge.
 * Pins (see tests/test_oracle_pins.py): brute-force softmax, finite differences,
 * an independent direct-sum implementation of the rule, Proposition 1, support
 * nesting and closed-form special cases.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double dot(const double* a, const double* b, int D) {
  double s = 0.0;
  for (int d = 0; d < D; ++d) s += a[d] * b[d];
  return s;
}

/* number of causally visible keys of query row q (bottom-right aligned) */
static double visible_keys(long q, long Nq, long Nk) { return (double)(q + 1 + Nk - Nq); }
/* is key c visible to query row q */
static int legal(long q, long c, long Nq, long Nk) { return c <= q + (Nk - Nq); }

/* ------------------------------------------------------------------------- */
/* Dense causal attention: the definition.                                    */
/* ------------------------------------------------------------------------- */

/* O_q = sum_k softmax(s_q)_k v_k over visible keys, lse_q = log sum_k exp(s_qk).
 * Rows [r0, r1) only. */
void oracle_dense_fwd(const double* q, const double* k, const double* v, int Nq, int Nk, int D,
                      double scale, int r0, int r1, double* o, double* lse) {
  #pragma omp parallel for schedule(dynamic, 1)
  for (int r = r0; r < r1; ++r) {
    long nvis = (long)r + 1 + Nk - Nq;
    if (nvis > Nk) nvis = Nk;
    double* s = (double*)malloc(sizeof(double) * (nvis > 0 ? nvis : 1));
    double mx = -INFINITY;
    for (long c = 0; c < nvis; ++c) {
      s[c] = scale * dot(q + (long)r * D, k + c * D, D);
      if (s[c] > mx) mx = s[c];
    }
    double z = 0.0;
    for (long c = 0; c < nvis; ++c) z += exp(s[c] - mx);
    double lz = mx + log(z);
    for (int d = 0; d < D; ++d) o[(long)r * D + d] = 0.0;
    for (long c = 0; c < nvis; ++c) {
      double p = exp(s[c] - lz);
      for (int d = 0; d < D; ++d) o[(long)r * D + d] += p * v[c * D + d];
    }
    lse[r] = lz;
    free(s);
  }
}

/* Gradient of <O, dO> for dense causal attention of one head.
 * dq is written for all rows; dk, dv are ACCUMULATED (+=) so that the query
 * heads of a GQA group can be summed into one key/value head. */
void oracle_dense_bwd(const double* q, const double* k, const double* v, const double* dO,
                      int Nq, int Nk, int D, double scale, double* dq, double* dk, double* dv) {
  double* o = (double*)malloc(sizeof(double) * (size_t)Nq * D);
  double* lse = (double*)malloc(sizeof(double) * (size_t)Nq);
  oracle_dense_fwd(q, k, v, Nq, Nk, D, scale, 0, Nq, o, lse);
  for (int r = 0; r < Nq; ++r) {
    double Dr = dot(o + (long)r * D, dO + (long)r * D, D);
    for (int d = 0; d < D; ++d) dq[(long)r * D + d] = 0.0;
    for (long c = 0; c < Nk; ++c) {
      if (!legal(r, c, Nq, Nk)) break;
      double s = scale * dot(q + (long)r * D, k + c * D, D);
      double p = exp(s - lse[r]);
      double dp = dot(dO + (long)r * D, v + c * D, D);
      double ds = p * (dp - Dr);
      for (int d = 0; d < D; ++d) {
        dv[c * D + d] += p * dO[(long)r * D + d];
        dk[c * D + d] += scale * ds * q[(long)r * D + d];
        dq[(long)r * D + d] += scale * ds * k[c * D + d];
      }
    }
  }
  free(o);
  free(lse);
}

/* ------------------------------------------------------------------------- */
/* MALA forward: Algorithm 1.                                                 */
/* ------------------------------------------------------------------------- */

/*
 * Query blocks [i0, i1) of B_q rows; key blocks of B_k keys.
 * Outputs (rows of the processed blocks only):
 *   o[Nq][D], lse[Nq]          the retained-set softmax output and z_q = m + log l
 *   row_tiles[Nq]              number of retained tiles (i, j) in which row q has a legal key
 *   tie_abs[Nq], tie_rel[Nq]   min over the tiles of the row's query block of |T - tau| and
 *                              |T/tau - 1|, where T is the tile's decisive value
 *                              max over voting rows of L_q * exp(rowmax - m - log l)
 *                              (+inf while a voter is still empty); the tile is retained
 *                              iff T >= tau.  Rows whose block saw a tile near tau are the
 *                              ones whose decisions may legitimately differ between two
 *                              finite-precision implementations.
 *   tile_keep (nullable)       [ceil(Nq/Bq)][ceil(Nk/Bk)] int8: 1 retained, 0 skipped,
 *                              -1 not legal/not visited.
 */
void oracle_mala_fwd(const double* q, const double* k, const double* v, int Nq, int Nk, int D,
                     double scale, double tau, int Bq, int Bk, int i0, int i1,
                     double* o, double* lse, int32_t* row_tiles, double* tie_abs,
                     double* tie_rel, int8_t* tile_keep) {
  const int Tc = (Nk + Bk - 1) / Bk;
  #pragma omp parallel for schedule(dynamic, 1)
  for (int i = i0; i < i1; ++i) {
    const int r_lo = i * Bq;
    const int r_hi = (r_lo + Bq < Nq) ? r_lo + Bq : Nq;
    const int nr = r_hi - r_lo;
    double* m = (double*)malloc(sizeof(double) * nr);
    double* l = (double*)malloc(sizeof(double) * nr);
    double* acc = (double*)calloc((size_t)nr * D, sizeof(double));
    double* thr = (double*)malloc(sizeof(double) * nr);
    double* S = (double*)malloc(sizeof(double) * (size_t)nr * Bk);
    double* mt = (double*)malloc(sizeof(double) * nr);
    int* has = (int*)malloc(sizeof(int) * nr);
    int32_t* cnt = (int32_t*)calloc(nr, sizeof(int32_t));
    double best_abs = INFINITY, best_rel = INFINITY;

    /* initialise O_i = 0, l_i = 0, m_i = -inf; per-row visible counts L_i */
    for (int a = 0; a < nr; ++a) {
      m[a] = -INFINITY;
      l[a] = 0.0;
      double L = visible_keys(r_lo + a, Nq, Nk);
      thr[a] = (tau > 0.0) ? log(tau) - log(L) : -INFINITY; /* log(tau / L_q) */
    }
    if (tile_keep)
      for (int j = 0; j < Tc; ++j) tile_keep[(long)i * Tc + j] = -1;

    /* legal key blocks, visited from the diagonal towards earlier keys */
    const long last_key = (long)(r_hi - 1) + (Nk - Nq);
    const int j_top = (int)(last_key / Bk);
    for (int j = j_top; j >= 0; --j) {
      const int c_lo = j * Bk;
      const int c_hi = (c_lo + Bk < Nk) ? c_lo + Bk : Nk;
      /* S_ij = Q_i K_j^T with the causal mask at the boundary; rowmax */
      for (int a = 0; a < nr; ++a) {
        mt[a] = -INFINITY;
        has[a] = 0;
        for (int c = c_lo; c < c_hi; ++c) {
          double s = -INFINITY;
          if (legal(r_lo + a, c, Nq, Nk)) {
            s = scale * dot(q + (long)(r_lo + a) * D, k + (long)c * D, D);
            has[a] = 1;
            if (s > mt[a]) mt[a] = s;
          }
          S[(long)a * Bk + (c - c_lo)] = s;
        }
      }
      /* the online test: skip iff every row with a legal key in the tile has
       * rowmax - m - log l < log(tau / L); an empty row (l = 0) demands retention */
      int retain = 0;
      double T = 0.0;
      for (int a = 0; a < nr; ++a) {
        if (!has[a]) continue; /* rows with no legal key do not constrain */
        if (l[a] == 0.0) {
          retain = 1;
          T = INFINITY;
          continue;
        }
        double g = mt[a] - m[a] - log(l[a]);
        if (g >= thr[a]) retain = 1;
        double Ta = visible_keys(r_lo + a, Nq, Nk) * exp(g);
        if (Ta > T) T = Ta;
      }
      if (isfinite(T) && tau > 0.0) {
        double da = fabs(T - tau), dr = fabs(T / tau - 1.0);
        if (da < best_abs) best_abs = da;
        if (dr < best_rel) best_rel = dr;
      }
      if (tile_keep) tile_keep[(long)i * Tc + j] = (int8_t)retain;
      if (!retain) continue; /* skipped: m, l and O unchanged */

      /* retained: the standard online-softmax update */
      for (int a = 0; a < nr; ++a) {
        if (!has[a]) continue; /* no legal key: its P row is zero, state unchanged */
        cnt[a] += 1;
        double m_new = (mt[a] > m[a]) ? mt[a] : m[a];
        double alpha = exp(m[a] - m_new);
        double rowsum = 0.0;
        for (int d = 0; d < D; ++d) acc[(long)a * D + d] *= alpha;
        for (int c = c_lo; c < c_hi; ++c) {
          double s = S[(long)a * Bk + (c - c_lo)];
          if (s == -INFINITY) continue;
          double p = exp(s - m_new);
          rowsum += p;
          for (int d = 0; d < D; ++d) acc[(long)a * D + d] += p * v[(long)c * D + d];
        }
        l[a] = alpha * l[a] + rowsum;
        m[a] = m_new;
      }
    }
    /* epilogue: O_i <- diag(l)^-1 O_i, l_i <- m_i + log l_i */
    for (int a = 0; a < nr; ++a) {
      const long r = r_lo + a;
      for (int d = 0; d < D; ++d) o[r * D + d] = acc[(long)a * D + d] / l[a];
      lse[r] = m[a] + log(l[a]);
      row_tiles[r] = cnt[a];
      tie_abs[r] = best_abs;
      tie_rel[r] = best_rel;
    }
    free(m); free(l); free(acc); free(thr); free(S); free(mt); free(has); free(cnt);
  }
}

/* ------------------------------------------------------------------------- */
/* MALA backward: Algorithm 2.                                                */
/* ------------------------------------------------------------------------- */

/*
 * The offline test of tile (j, i): retained iff some valid causal entry has
 * s_qk - lse_q >= log(tau / L_q).  Writes the decisive value
 * T = max over valid entries of L_q * exp(s_qk - lse_q).  Returns -1 if the tile
 * has no legal entry.
 */
static int offline_test(const double* q, const double* k, const double* lse, int Nq, int Nk,
                        int D, double scale, double tau, int Bq, int Bk, int i, int j,
                        double* T_out) {
  const int r_lo = i * Bq, r_hi = (r_lo + Bq < Nq) ? r_lo + Bq : Nq;
  const int c_lo = j * Bk, c_hi = (c_lo + Bk < Nk) ? c_lo + Bk : Nk;
  int any = 0, retain = 0;
  double T = 0.0;
  for (int r = r_lo; r < r_hi; ++r) {
    double L = visible_keys(r, Nq, Nk);
    double thr = (tau > 0.0) ? log(tau) - log(L) : -INFINITY;
    for (int c = c_lo; c < c_hi; ++c) {
      if (!legal(r, c, Nq, Nk)) continue;
      any = 1;
      double g = scale * dot(q + (long)r * D, k + (long)c * D, D) - lse[r];
      if (g >= thr) retain = 1;
      double Tv = L * exp(g);
      if (Tv > T) T = Tv;
    }
  }
  *T_out = T;
  return any ? retain : -1;
}

/*
 * Gradients of one (query head, key/value head) pair, given that head's forward
 * output o and saved lse (the MALA forward's own) and dO.
 *   dq rows of query blocks [qi0, qi1) are written (overwritten);
 *   dk, dv rows of key blocks [kj0, kj1) are ACCUMULATED (+=) (GQA groups sum);
 *   row_tiles[Nq]: retained tiles (j, i(q)) in which row q has a legal key,
 *   tie_abs/tie_rel[Nq]: min over the tiles (j, i(q)) of |T - tau|, |T/tau - 1|;
 *   tile_keep (nullable) [Tr][Tc] int8 as in the forward (written by the dq sweep).
 * D_q = rowsum(O_q * dO_q) uses the MALA output O.
 */
void oracle_mala_bwd(const double* q, const double* k, const double* v, const double* o,
                     const double* lse, const double* dO, int Nq, int Nk, int D, double scale,
                     double tau, int Bq, int Bk, int qi0, int qi1, int kj0, int kj1,
                     double* dq, double* dk, double* dv, int32_t* row_tiles, double* tie_abs,
                     double* tie_rel, int8_t* tile_keep) {
  const int Tr = (Nq + Bq - 1) / Bq, Tc = (Nk + Bk - 1) / Bk;
  (void)Tr;
  /* query side: dQ_i = sum over retained (j, i) of scale * dS_ij K_j */
  #pragma omp parallel for schedule(dynamic, 1)
  for (int i = qi0; i < qi1; ++i) {
    const int r_lo = i * Bq, r_hi = (r_lo + Bq < Nq) ? r_lo + Bq : Nq;
    double best_abs = INFINITY, best_rel = INFINITY;
    for (int r = r_lo; r < r_hi; ++r) {
      row_tiles[r] = 0;
      for (int d = 0; d < D; ++d) dq[(long)r * D + d] = 0.0;
    }
    for (int j = 0; j < Tc; ++j) {
      double T;
      int keep = offline_test(q, k, lse, Nq, Nk, D, scale, tau, Bq, Bk, i, j, &T);
      if (tile_keep) tile_keep[(long)i * Tc + j] = (int8_t)keep;
      if (keep < 0) continue;
      if (tau > 0.0) {
        double da = fabs(T - tau), dr = fabs(T / tau - 1.0);
        if (da < best_abs) best_abs = da;
        if (dr < best_rel) best_rel = dr;
      }
      if (keep == 0) continue;
      const int c_lo = j * Bk, c_hi = (c_lo + Bk < Nk) ? c_lo + Bk : Nk;
      for (int r = r_lo; r < r_hi; ++r) {
        if (!legal(r, c_lo, Nq, Nk)) continue; /* no legal key of this row in the tile */
        row_tiles[r] += 1;
        const double Dr = dot(o + (long)r * D, dO + (long)r * D, D);
        for (int c = c_lo; c < c_hi; ++c) {
          if (!legal(r, c, Nq, Nk)) continue;
          double s = scale * dot(q + (long)r * D, k + (long)c * D, D);
          double p = exp(s - lse[r]);
          double dp = dot(dO + (long)r * D, v + (long)c * D, D);
          double ds = p * (dp - Dr);
          for (int d = 0; d < D; ++d) dq[(long)r * D + d] += scale * ds * k[(long)c * D + d];
        }
      }
    }
    for (int r = r_lo; r < r_hi; ++r) {
      tie_abs[r] = best_abs;
      tie_rel[r] = best_rel;
    }
  }
  /* key side: dV_j += P_ji dO_i, dK_j += scale * dS_ji Q_i over retained (j, i) */
  #pragma omp parallel for schedule(dynamic, 1)
  for (int j = kj0; j < kj1; ++j) {
    const int c_lo = j * Bk, c_hi = (c_lo + Bk < Nk) ? c_lo + Bk : Nk;
    const int Tr_ = (Nq + Bq - 1) / Bq;
    for (int i = 0; i < Tr_; ++i) {
      double T;
      int keep = offline_test(q, k, lse, Nq, Nk, D, scale, tau, Bq, Bk, i, j, &T);
      if (keep <= 0) continue;
      const int r_lo = i * Bq, r_hi = (r_lo + Bq < Nq) ? r_lo + Bq : Nq;
      for (int r = r_lo; r < r_hi; ++r) {
        const double Dr = dot(o + (long)r * D, dO + (long)r * D, D);
        for (int c = c_lo; c < c_hi; ++c) {
          if (!legal(r, c, Nq, Nk)) continue;
          double s = scale * dot(q + (long)r * D, k + (long)c * D, D);
          double p = exp(s - lse[r]);
          double dp = dot(dO + (long)r * D, v + (long)c * D, D);
          double ds = p * (dp - Dr);
          for (int d = 0; d < D; ++d) {
            dv[(long)c * D + d] += p * dO[(long)r * D + d];
            dk[(long)c * D + d] += scale * ds * q[(long)r * D + d];
          }
        }
      }
    }
  }
}

/* ------------------------------------------------------------------------- */
/* MALA split-KV decode.                                                      */
/* ------------------------------------------------------------------------- */

/*
 * One query vector q[D] at position Nk - 1 (it sees all Nk cached keys, L = Nk).
 * Key tiles of B_k keys, T = ceil(Nk / B_k); split s owns the contiguous tiles
 * [s * tps, min(T, (s + 1) * tps)) with tps = ceil(T / num_splits).  Each split
 * starts from an empty state and applies the forward rule to its own tiles in
 * descending order against its own partial normalizer, with the threshold
 * log(tau / Nk) of the full context.  Splits are merged by the normalizer-aware
 * (log-sum-exp weighted) reduction.
 * Outputs: o[D], *lse, *tiles (retained tiles summed over splits), *tie_abs,
 * *tie_rel, keep[T] (nullable): per-tile 1 retained / 0 skipped.
 */
void oracle_mala_decode(const double* q, const double* k, const double* v, int Nk, int D,
                        double scale, double tau, int Bk, int num_splits, double* o, double* lse,
                        int32_t* tiles, double* tie_abs, double* tie_rel, int8_t* keep) {
  const int T = (Nk + Bk - 1) / Bk;
  const int tps = (T + num_splits - 1) / num_splits;
  const double thr = (tau > 0.0) ? log(tau) - log((double)Nk) : -INFINITY;
  double* os = (double*)calloc((size_t)num_splits * D, sizeof(double));
  double* lses = (double*)malloc(sizeof(double) * num_splits);
  double* s = (double*)malloc(sizeof(double) * Bk);
  double best_abs = INFINITY, best_rel = INFINITY;
  int32_t count = 0;
  for (int sp = 0; sp < num_splits; ++sp) {
    int t_lo = sp * tps, t_hi = (sp + 1) * tps;
    if (t_hi > T) t_hi = T;
    double m = -INFINITY, l = 0.0;
    double* acc = os + (long)sp * D;
    for (int t = t_hi - 1; t >= t_lo; --t) {
      const int c_lo = t * Bk, c_hi = (c_lo + Bk < Nk) ? c_lo + Bk : Nk;
      double mt = -INFINITY;
      for (int c = c_lo; c < c_hi; ++c) {
        s[c - c_lo] = scale * dot(q, k + (long)c * D, D);
        if (s[c - c_lo] > mt) mt = s[c - c_lo];
      }
      int retain;
      if (l == 0.0) {
        retain = 1;
      } else {
        double g = mt - m - log(l);
        retain = g >= thr;
        if (tau > 0.0) {
          double Tv = (double)Nk * exp(g);
          double da = fabs(Tv - tau), dr = fabs(Tv / tau - 1.0);
          if (da < best_abs) best_abs = da;
          if (dr < best_rel) best_rel = dr;
        }
      }
      if (keep) keep[t] = (int8_t)retain;
      if (!retain) continue;
      count += 1;
      double m_new = (mt > m) ? mt : m;
      double alpha = exp(m - m_new), rowsum = 0.0;
      for (int d = 0; d < D; ++d) acc[d] *= alpha;
      for (int c = c_lo; c < c_hi; ++c) {
        double p = exp(s[c - c_lo] - m_new);
        rowsum += p;
        for (int d = 0; d < D; ++d) acc[d] += p * v[(long)c * D + d];
      }
      l = alpha * l + rowsum;
      m = m_new;
    }
    if (l > 0.0) {
      for (int d = 0; d < D; ++d) acc[d] /= l;
      lses[sp] = m + log(l);
    } else {
      lses[sp] = -INFINITY; /* a split with no tile contributes nothing */
    }
  }
  /* normalizer-aware merge of the split partials */
  double mx = -INFINITY;
  for (int sp = 0; sp < num_splits; ++sp)
    if (lses[sp] > mx) mx = lses[sp];
  double z = 0.0;
  for (int sp = 0; sp < num_splits; ++sp)
    if (lses[sp] > -INFINITY) z += exp(lses[sp] - mx);
  const double LSE = mx + log(z);
  for (int d = 0; d < D; ++d) o[d] = 0.0;
  for (int sp = 0; sp < num_splits; ++sp) {
    if (lses[sp] == -INFINITY) continue;
    double w = exp(lses[sp] - LSE);
    for (int d = 0; d < D; ++d) o[d] += w * os[(long)sp * D + d];
  }
  *lse = LSE;
  *tiles = count;
  *tie_abs = best_abs;
  *tie_rel = best_rel;
  free(os); free(lses); free(s);
}
