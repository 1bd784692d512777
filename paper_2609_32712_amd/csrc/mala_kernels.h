// Kernel parameter blocks and host-side launchers of the MALA kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mala {

// Decision geometry (shared by forward and backward so that the backward
// support nests inside the forward support; decode uses 1 x kDecBk).
constexpr int kBq = 32;      // query rows per decision tile = rows of one wavefront
constexpr int kBk = 32;      // keys per decision tile
constexpr int kDecBk = 32;   // keys per decode decision tile

constexpr int kFwdWaves = 8;                 // wavefronts per forward workgroup (2 per SIMD)
constexpr int kFwdRows = kFwdWaves * kBq;    // 256 query rows per workgroup
constexpr int kDqWaves = 8;                  // wavefronts per dQ workgroup (2 per SIMD)
constexpr int kDqRows = kDqWaves * kBq;      // 256 query rows per workgroup
constexpr int kFwdStage = 64;                // keys per K/V stage in LDS (forward and dQ)
constexpr int kBwdKeys = 128;                // keys per dK/dV workgroup (4 key groups x kBk)
constexpr int kDkdvChunk = 4096;             // sweep iterations the dK/dV kernel compacts at once
// Below kDkdvSplitGroups key-block workgroups (batch x KV heads x key blocks) the
// dK/dV sweeps are split into parts of at least kDkdvPartMin iterations, run by
// workgroups of their own, and summed by a reduction pass (fixed-length batches).
constexpr int kDkdvSplitGroups = 1024;
constexpr int kDkdvPartMin = 512;
// Budgets of the low bf16 term in the backward.  P and dS enter the MFMAs as
// hi + lo (two bf16 terms, 2^-16 relative).  The lo term of a tile is left out of
// dV (P) or dK (dS) while, for every key of the tile, the P mass or the sum of |dS|
// of the tiles run without it stays within a budget, and out of dQ (dS) while the
// same holds for every query row.  Since |lo| <= 2^-8 |hi + lo|, the added error
// of a dV (dK, dQ) element is at most 2^-8 x budget x the largest |dO| (|Q|, |K|,
// times the softmax scale).  For dK and dQ, a tile whose own sum of |dS| for some
// key (row) exceeds 1/16 of the budget always takes the lo term without drawing on
// the budget, which is thereby kept for the many small tiles; the bound holds as
// before.
constexpr float kLoMassDv = 1.0f / 16;      // dV: P mass per key
constexpr float kLoMassDk = 0.25f;          // dK: sum of |dS| per key
constexpr float kLoTileDk = kLoMassDk / 16;  // dK: |dS| of one tile and key, above it lo always
constexpr float kLoMassDq = 1.0f;           // dQ: sum of |dS| per query row
constexpr float kLoTileDq = kLoMassDq / 16;  // dQ: |dS| of one tile and row, above it lo always
// Forward: the lo term of P runs on a tile only if, for some row of the wavefront,
// the tile's mass exceeds this share of the row's retained normalizer (the tile
// included).  The tiles that hold a row's dominant keys then keep ~16 significant
// bits; every other tile adds at most 2^-9 x its share of the row's mass as
// rounding error, and such errors of many small tiles do not line up.
constexpr float kFwdLoShare = 1.0f / 64;
constexpr int kDecStride = 4;                // extra floats per decode partial (lse, count, pad)

// Statistics counters (int64 each; the indices of MALA_CNT_* in mala.h).
constexpr int kNumCounters = 8;
enum {
  kCntLegal = 0, kCntRetained = 1, kCntVTiles = 2, kCntSlots = 3,
  kCntRetainedKV = 4, kCntVNeeded = 5, kCntSetHash = 6, kCntSetHashKV = 7
};

// Fingerprint of one retained decision tile: splitmix64 (Steele, Lea and Flood's
// SplitMix generator, its output mixing function) of the tile's coordinates
// (sequence b, query head h, query tile i, key tile j of the sequence's own
// tiling) packed as b << 52 | h << 40 | i << 20 | j.  A pass sums the fingerprints
// of the tiles it retains modulo 2^64; the sum does not depend on the order of the
// tiles, and two passes that retain different sets of tiles differ in it except
// with probability ~2^-64.  It lets the statistics compare the retained sets of
// two passes (or of a pass and an independent implementation) tile by tile
// without storing them.
__device__ __forceinline__ unsigned long long tile_hash(int b, int h, int i, int j) {
  unsigned long long z = ((unsigned long long)b << 52) | ((unsigned long long)h << 40) |
                         ((unsigned long long)i << 20) | (unsigned long long)j;
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Statistics of one workgroup: its wavefronts add into an LDS copy of the counters
// (blk_add, LDS atomics), then one thread per counter adds the workgroup's sums to
// the global counters (blk_flush).  Same-address global atomics from every
// wavefront of a grid serialise at the L2; one per counter and workgroup keeps
// their count small.  blk_init runs before a barrier that precedes every blk_add;
// every thread of the workgroup calls blk_flush.
__device__ __forceinline__ void blk_init(unsigned long long* s) {
  if (threadIdx.x < kNumCounters) s[threadIdx.x] = 0;
}
__device__ __forceinline__ void blk_add(unsigned long long* s, int i, unsigned long long x) {
  if (x) atomicAdd(&s[i], x);
}
__device__ __forceinline__ void blk_flush(unsigned long long* s, unsigned long long* g) {
  __syncthreads();
  if (threadIdx.x < kNumCounters && s[threadIdx.x]) atomicAdd(&g[threadIdx.x], s[threadIdx.x]);
}

// Batches come in two layouts.  Fixed length: [B, H, N, D], slice (b, h) at rows
// (b H + h) N.  Packed (cu non-null): B sequences along the token axes of
// [Hq, Nq, D] queries and [Hkv, Nk, D] keys (Nq, Nk = the totals, the head
// strides); sequence b holds query rows cu[b] .. cu[b + 1] and key rows
// cu_k[b] .. cu_k[b + 1] (cu_k null: the same as cu), clamped into the totals and
// cut to max_len / max_len_k rows; it is a causal problem of its own (bottom-right
// aligned when it has fewer query rows than keys) tiled from its own first rows.
// A sequence with more query rows than keys is skipped.
struct Seg {
  int Nq, Nk;   // rows of the sequence (queries, keys)
  long qb, kb;  // its first row in head 0 of q (o, lse, ...) and of k (v, dk, dv)
};
template <class P>
__device__ __forceinline__ Seg seq_slice(const P& p, int b) {
  if (p.cu) {
    const int32_t* ck = p.cu_k ? p.cu_k : p.cu;
    const int q0 = min(max(p.cu[b], 0), p.Nq), q1 = min(max(p.cu[b + 1], q0), p.Nq);
    const int k0 = min(max(ck[b], 0), p.Nk), k1 = min(max(ck[b + 1], k0), p.Nk);
    const int nk = min(k1 - k0, p.max_len_k);
    const int nq = min(q1 - q0, p.max_len);
    return Seg{nq <= nk ? nq : 0, nk, (long)q0, (long)k0};
  }
  return Seg{p.Nq, p.Nk, (long)b * p.Hq * p.Nq, (long)b * p.Hkv * p.Nk};
}

struct FwdParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  void* o;             // fp32, or bf16 when o_bf16
  float* lse;
  int32_t* row_tiles;
  unsigned long long* counters;
  int o_bf16;
  const int32_t* cu;   // packed batches: [B + 1] query-row starts, else null
  const int32_t* cu_k; // packed batches: [B + 1] key-row starts, or null (= cu)
  int max_len, max_len_k;   // packed batches: query / key rows per sequence at most
  int B, Hq, Hkv, Nq, Nk;
  float scale2;    // softmax scale * log2(e): scores are kept in base-2 units
  float log2tau;   // log2(tau); -inf for tau == 0
  int nqblk;       // ceil(Nq / kFwdRows) (packed: ceil(max_len / kFwdRows))
};

struct BwdParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* dout;
  const float* lse;
  const float* dvec;   // D_q = rowsum(O_q * dO_q)
  void* dq;            // fp32, or bf16 when grad_bf16 (dk, dv alike)
  void* dk;
  void* dv;
  int grad_bf16;
  int32_t* row_tiles;
  unsigned long long* counters;
  const int32_t* cu;   // packed batches: [B + 1] query-row starts, else null
  const int32_t* cu_k; // packed batches: [B + 1] key-row starts, or null (= cu)
  int max_len, max_len_k;   // packed batches: query / key rows per sequence at most
  int B, Hq, Hkv, Nq, Nk;
  float scale, scale2, log2tau;
  int nkblk;           // ceil(Nk / kBwdKeys) (packed: ceil(max_len_k / kBwdKeys))
  int nqblk;           // ceil(Nq / kDqRows) (packed: ceil(max_len / kDqRows))
  // Tile decisions of the dQ pass for the key-major pass: one byte per (query-tile row,
  // query head, 128-key block) at mask_index, bit j % 4 for the block's key tile j.
  uint8_t* mask;
  int mask_rows;       // query-tile rows: B ceil(Nq / kBq) (packed: total_q / kBq + B)
  // Split key-block sweeps: part p of a block takes iterations [p psize, (p + 1) psize)
  // and, when nparts > 1, writes its fp32 dV and dK sums to part[(2 p + {0, 1}) rows + row]
  // (rows = B Hkv Nk rows of D floats), which the reduction pass adds up in order.
  int psize, nparts;
  float* part;
};

// Iterations of the dK/dV sweep of the key block starting at key kb0 of a sequence
// (Nq query rows, the last aligned with the last of Nk keys): every (query tile, head
// of the GQA group) from the last query tile down to the block's diagonal.
__host__ __device__ inline int dkdv_iterations(int Nq, int Nk, int kb0, int grp) {
  const long first_q = (long)kb0 - ((long)Nk - Nq);
  const int qi_start = first_q <= 0 ? 0 : (int)(first_q / kBq);
  return grp * ((Nq + kBq - 1) / kBq - qi_start);
}

// Byte of the decisions of query-tile row `row` (mask_row0 + query tile), query head
// hq and key block jb: the key blocks of one row and head are contiguous.
__device__ __forceinline__ size_t mask_index(const BwdParams& p, int row, int hq, int jb) {
  return ((size_t)row * p.Hq + hq) * p.nkblk + jb;
}

// First query-tile row of sequence b in the decision bytes: b ceil(Nq / kBq) for the
// fixed-length layout; floor(q0 / kBq) + b for packed sequences starting at row q0
// (disjoint ranges: sequence b has at most ceil(n_b / kBq) tiles).
__device__ __forceinline__ int mask_row0(const BwdParams& p, int b, const Seg& sg) {
  return p.cu ? (int)(sg.qb / kBq) + b : b * ((p.Nq + kBq - 1) / kBq);
}

struct DecParams {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  float* part;         // [B, Hq, S, D + kDecStride]
  unsigned long long* counters;
  const int32_t* lens; // [B] valid cache tokens per sequence, or null (all Nk)
  int B, Hq, Hkv, Nk, S, T, tps;   // T, tps: tiles and tiles per split at length Nk
  int nchunk;          // ceil((Hq / Hkv) / 16): workgroups per (sequence, KV head, split)
  float scale2, thr2;  // thr2 = log2(tau) - log2(Nk)
  float log2tau;       // for the per-sequence thresholds log2(tau) - log2(n_b)
};

hipError_t launch_fill_zero(void* ptr, size_t bytes, hipStream_t st);
hipError_t launch_fwd(const FwdParams& p, int D, hipStream_t st);
hipError_t launch_bwd_preprocess(const void* o, bool o_bf16, const __bf16* dout, float* dvec,
                                 long rows, int D, hipStream_t st);
hipError_t launch_bwd(const BwdParams& p, int D, hipStream_t st);
hipError_t launch_decode(const DecParams& p, int D, hipStream_t st);
hipError_t launch_decode_combine(const float* part, void* o, bool o_bf16, float* lse,
                                 int32_t* head_tiles, int BH, int S, int D, hipStream_t st);

}  // namespace mala
