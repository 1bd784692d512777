/*
 * mala.h — C ABI of the MI355X (gfx950) MALA causal-attention library (libmala.so).
 *
 * MALA ("MassAlloc Attention") computes the QK score tile of EVERY causally legal
 * tile and runs the post-score work of a tile only when the tile's normalized
 * contribution reaches the length-aware tolerance tau / L_q (Methodology,
 * "Attention as a Compute Allocator": L_q is the number of keys visible to query
 * row q).
 *   - forward: Algorithm 1 with the online test (Eq. online test) against the
 *     running max m and normalizer l of the retained tiles; tiles are visited from
 *     the diagonal towards earlier keys; an empty row always retains;
 *   - backward: Algorithm 2 with the offline test (Eq. offline test) against the
 *     saved log-normalizer (LSE);
 *   - decode: the forward rule applied per split of the KV cache with the
 *     threshold of the full context (L = Nk), splits merged by the
 *     normalizer-aware reduction (Fused Execution section and its appendix).
 *
 * Conventions shared by every entry point
 *   - All tensor arguments are DEVICE pointers, owned by the caller, contiguous,
 *     in BHSD layout (batch, head, sequence, head_dim; the packed entry points use
 *     [head, token, head_dim]).  The library never allocates, frees or retains
 *     them.
 *   - Q, K, V, dO, the KV caches and the decode query are bf16 (passed as void*);
 *     O and the gradients are fp32 or bf16 (MALA_OUT_*), LSE is fp32; LSE is the
 *     natural-log normalizer z_q = log sum_{k in R_q} exp(s_qk) of the retained
 *     set R_q.
 *   - scale multiplies Q.K in fp32 (the paper absorbs it into Q; it is never
 *     re-rounded to bf16 here); tau >= 0 (tau = 0 runs every tile: dense
 *     attention through the same kernels).
 *   - GQA: query head h reads key/value head h / (Hq / Hkv).
 *   - Causal masking is bottom-right aligned: row q sees keys k <= q + Nk - Nq, so
 *     L_q = q + 1 + Nk - Nq (L_q = q + 1 when Nq == Nk; L = Nk for decode).
 *   - Decision geometry: the forward and backward share one tile partition
 *     (B_q x B_k, reported by mala_geometry), which the support-nesting property
 *     of the backward needs.  Decode tiles are 1 x B_k per query head.
 *   - Calls validate synchronously, then enqueue kernels on `stream` (a
 *     hipStream_t; NULL = the default stream) and return without waiting.  The
 *     return value reports validation and launch errors only; a device fault is
 *     reported by the caller's next synchronisation.  Calls are re-entrant; the
 *     library keeps no state between calls.
 *   - Statistics pointers (row_tiles, head_tiles, counters) may be NULL.  When
 *     given they are OVERWRITTEN by the call: the counters are cleared first on
 *     the same stream, and per-row / per-head statistics are written for every
 *     row and head the call computes.  No mask or retained-tile index is ever
 *     materialised.
 */
#ifndef MALA_H
#define MALA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes (0 = success, negative = error). */
typedef enum {
  MALA_OK = 0,
  MALA_ERR_INVALID_ARG = -1, /* null required pointer, non-positive size, Hq % Hkv != 0,
                                Nq > Nk, tau < 0 or NaN, scale not finite or <= 0,
                                num_splits < 1, an output type not MALA_OUT_* */
  MALA_ERR_UNSUPPORTED = -2, /* head_dim not in {64, 128}, causal == 0 (the paper's
                                traversal is defined for causal attention only), or a
                                forward/backward K/V slice of 2^32 bytes or more */
  MALA_ERR_WORKSPACE = -3,   /* workspace NULL or smaller than the *_workspace_size query */
  MALA_ERR_HIP = -4          /* a HIP launch/runtime call failed; see mala_last_error() */
} mala_status;

/* Indices into the int64 counters[MALA_NUM_COUNTERS] array that every entry point
 * can fill (a NULL counters pointer skips them; otherwise all eight are cleared on
 * the stream and then written).  "Tile" means a decision tile (B_q x B_k, or 1 x B_k
 * per query head in decode). */
enum {
  MALA_CNT_LEGAL = 0,    /* decision tiles holding at least one legal (causal) entry,
                            per query head */
  MALA_CNT_RETAINED = 1, /* of those, tiles whose post-score path ran (backward: as
                            counted by the query-major dQ pass) */
  MALA_CNT_V_TILES = 2,  /* forward: V tiles of B_k keys staged (a workgroup of 256
                            query rows stages every key tile it visits);
                            backward: dO tiles of B_q rows staged by the key-major pass
                            (a workgroup of 128 keys stages only the query tiles that
                            some of its key tiles retain);
                            decode: V tiles of B_k keys fetched (once per up to 16 query
                            heads of a GQA group, look-ahead fetches included) */
  MALA_CNT_SLOTS = 3,    /* post-score key slots summed over query rows: a retained
                            B_q x B_k tile adds B_k slots to each of its valid rows
                            (Attention Cost section; mean slots per query =
                            counters[3] / number of query rows) */
  MALA_CNT_RETAINED_KV = 4, /* backward only: of the tiles the dQ pass retained, those
                               whose offline test the key-major dK/dV pass, recomputing
                               it, confirms (equal to MALA_CNT_RETAINED when the two
                               passes agree; 0 in forward and decode) */
  MALA_CNT_V_NEEDED = 5, /* the loads of MALA_CNT_V_TILES that a retained tile used:
                            forward: (workgroup, key tile) pairs with a retained tile;
                            backward: (key-major workgroup, query tile) pairs with a
                            retained tile; decode: fetched V tiles that some head of
                            the group retained */
  MALA_CNT_SET_HASH = 6, /* fingerprint of the retained set: the sum modulo 2^64 of
                            splitmix64(b << 52 | h << 40 | i << 20 | j) over the
                            retained tiles (sequence b, query head h, query tile i,
                            key tile j of the sequence's own tiling; decode: i = 0, j =
                            the key tile); backward: of the query-major dQ pass */
  MALA_CNT_SET_HASH_KV = 7, /* backward only: the same fingerprint over the tiles of
                               MALA_CNT_RETAINED_KV (equal to MALA_CNT_SET_HASH when the
                               key-major pass confirms every tile, up to a 2^-64 chance) */
  MALA_NUM_COUNTERS = 8
};

enum { MALA_PASS_FWD = 0, MALA_PASS_BWD = 1, MALA_PASS_DECODE = 2 };

/* Element type of O and of the gradients (the *_dtype arguments).  Outputs are
 * computed in fp32 and either stored as fp32 or rounded once to bf16 (nearest
 * even) at the store; LSE is always fp32.  A bf16 O given to the backward enters
 * D_q = rowsum(O * dO) with its rounding. */
enum { MALA_OUT_F32 = 0, MALA_OUT_BF16 = 1 };

/* Decision tile of a pass: B_q query rows x B_k keys. */
typedef struct {
  int32_t block_q;
  int32_t block_k;
} mala_geometry_t;

/* Decision geometry used by `pass` (MALA_PASS_*) at head_dim (64 or 128).
 * Returns {0, 0} for an unsupported pass or head_dim. */
mala_geometry_t mala_geometry(int head_dim, int pass);

/* Static description of a status code; never NULL. */
const char* mala_strerror(int status);

/* Detail of the last error raised on the calling thread ("" if none). */
const char* mala_last_error(void);

/*
 * MALA forward (Algorithm 1), also the prefill operator.
 *   q:  bf16 [B, Hq,  Nq, D]        k, v: bf16 [B, Hkv, Nk, D]
 *   o:  [B, Hq, Nq, D] out, fp32 or bf16 by out_dtype: softmax output renormalised
 *       over the retained set
 *   lse: fp32 [B, Hq, Nq]    out    natural-log normalizer z_q = m_q + log l_q
 *   row_tiles: int32 [B, Hq, Nq] or NULL   out: retained tiles in which the row has a
 *              legal key
 *   counters:  int64 [MALA_NUM_COUNTERS] or NULL   out: see MALA_CNT_*
 *   causal must be 1.  Requires Nq <= Nk, D in {64, 128} and Nk * D * 2 < 2^32
 *   (Nk below 16M tokens at D = 128); otherwise MALA_ERR_UNSUPPORTED.
 */
int mala_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
             int32_t* row_tiles, int64_t* counters, int B, int Hq, int Hkv, int Nq, int Nk,
             int D, int causal, float scale, float tau, int out_dtype, void* stream);

/* Bytes of device workspace mala_bwd needs for this shape: the per-row
 * D_q = rowsum(O_q * dO_q) vector of Algorithm 2 (B Hq Nq floats) and the tile
 * decisions that the query-major dQ pass hands to the key-major dK/dV pass (one byte
 * per query tile of B_q rows, query head and block of 128 keys: B Hq ceil(Nq / B_q)
 * ceil(Nk / 128) bytes, ~32 MB at B = 1, Hq = 8, Nq = Nk = 131072).  Shapes with
 * fewer than 1024 key blocks in all (B Hkv ceil(Nk / 128)) run each key block's
 * sweep over the query tiles in up to P parts of at least 512 (query tile, head)
 * iterations on workgroups of their own, so that one long sweep does not set the
 * time alone; the workspace then also holds the parts' fp32 dK and dV sums
 * (P x 2 x B Hkv Nk D floats, ~268 MB at B = 1, Hq = 8, Hkv = 2, Nq = Nk = 32768,
 * P = 4), which a last pass adds in part order.  0 for an invalid shape. */
size_t mala_bwd_workspace_size(int B, int Hq, int Hkv, int Nq, int Nk, int D);

/* Bytes of device workspace mala_bwd_varlen needs: Hq total_q floats of D_q and
 * Hq (total_q / B_q + num_seqs) ceil(max_seqlen_k / 128) decision bytes. */
size_t mala_bwd_varlen_workspace_size(int num_seqs, int max_seqlen_k, int total_q, int Hq,
                                      int Hkv, int D);

/*
 * MALA backward (Algorithm 2): gradients of <O, dO> restricted to the tiles that
 * pass the offline test against the saved lse.
 *   q: bf16 [B, Hq, Nq, D]; k, v: bf16 [B, Hkv, Nk, D]; o: [B, Hq, Nq, D] (fp32 or
 *   bf16 by o_dtype) and lse: fp32 [B, Hq, Nq] as returned by mala_fwd; dout: bf16
 *   [B, Hq, Nq, D].
 *   dq: [B, Hq, Nq, D] out; dk, dv: [B, Hkv, Nk, D] out (dK and dV of a KV head
 *       summed over its GQA group); all three fp32 or bf16 by grad_dtype.  No
 *       atomics: all three are bitwise reproducible.  dQ comes from a query-major
 *       pass that takes every tile decision; the key-major dK/dV pass processes
 *       only the query tiles that pass retained for some of its keys;
 *   row_tiles: int32 [B, Hq, Nq] or NULL out; counters: int64 [MALA_NUM_COUNTERS]
 *   or NULL out.
 *   workspace: device memory of at least mala_bwd_workspace_size(...) bytes,
 *   16-byte aligned, owned by the caller, not read by the caller afterwards (its
 *   contents on entry do not matter: every byte the call reads it writes first).
 *   The dQ pass runs first and decides every tile; the key-major pass follows its
 *   decisions, so both use exactly the same tiles.
 *   The shape limits of mala_fwd apply.
 */
int mala_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
             const void* dout, void* dq, void* dk, void* dv, int32_t* row_tiles,
             int64_t* counters, void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv,
             int Nq, int Nk, int D, int causal, float scale, float tau, int o_dtype,
             int grad_dtype, void* stream);

/*
 * Packed variable-length batches (the forward of Algorithm 1 per sequence).
 * num_seqs sequences lie back to back along the token axes: sequence b holds query
 * rows [cu_seqlens_q[b], cu_seqlens_q[b + 1]) and key / value rows
 * [cu_seqlens_k[b], cu_seqlens_k[b + 1]) of every head, attends only to its own
 * keys, causally with bottom-right alignment (with n_q query rows and n_k >= n_q
 * keys, its i-th query row sees its keys 0 .. i + n_k - n_q, L_q = i + 1 + n_k - n_q:
 * n_q = n_k is self-attention, n_q < n_k is prefill against a cache), and is tiled
 * from its own first rows, exactly as a batch of one with Nq = n_q, Nk = n_k.
 *   q: bf16 [Hq, total_q, D]; k, v: bf16 [Hkv, total_k, D] (head-major: the
 *   fixed-length layout with B = 1); o: [Hq, total_q, D] out (out_dtype); lse: fp32
 *   [Hq, total_q] out; row_tiles: int32 [Hq, total_q] or NULL out; counters as mala_fwd.
 *   cu_seqlens_q, cu_seqlens_k: int32 [num_seqs + 1] device arrays, non-decreasing
 *   from 0 to at most total_q / total_k; cu_seqlens_k may be NULL (the same rows as
 *   the queries; then total_k = total_q and max_seqlen_k = max_seqlen_q).
 *   max_seqlen_q / _k: the longest query / key run (the launch is sized by them).
 *   On the device the starts are clamped into the totals and a run longer than its
 *   max_seqlen is cut to its first max_seqlen rows; a sequence with more query rows
 *   than keys is skipped.  Rows that no (cut, not skipped) sequence covers are not
 *   written.  Requires max_seqlen_q <= total_q, max_seqlen_k <= total_k,
 *   total_q <= total_k, D in {64, 128} and total_k * D * 2 < 2^32.
 */
int mala_fwd_varlen(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_q,
                    const int32_t* cu_seqlens_k, void* o, float* lse, int32_t* row_tiles,
                    int64_t* counters, int num_seqs, int max_seqlen_q, int max_seqlen_k,
                    int total_q, int total_k, int Hq, int Hkv, int D, float scale, float tau,
                    int out_dtype, void* stream);

/*
 * Packed variable-length batches: mala_bwd (Algorithm 2) per sequence, on the
 * layout of mala_fwd_varlen (o, lse as it returned them, o of type o_dtype; dout,
 * dq: [Hq, total_q, D]; dk, dv: [Hkv, total_k, D]; gradients of type grad_dtype).
 * workspace: at least mala_bwd_varlen_workspace_size(num_seqs, max_seqlen_k, total_q,
 * Hq, Hkv, D) bytes.  Rows that no sequence covers are not written.
 */
int mala_bwd_varlen(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_q,
                    const int32_t* cu_seqlens_k, const void* o, const float* lse,
                    const void* dout, void* dq, void* dk, void* dv, int32_t* row_tiles,
                    int64_t* counters, void* workspace, size_t workspace_bytes, int num_seqs,
                    int max_seqlen_q, int max_seqlen_k, int total_q, int total_k, int Hq,
                    int Hkv, int D, float scale, float tau, int o_dtype, int grad_dtype,
                    void* stream);

/* Bytes of device workspace mala_decode needs: fp32 split partials
 * [B, Hq, num_splits, D + 4] (O_s / l_s, lse_s, retained count, pad). */
size_t mala_decode_workspace_size(int B, int Hq, int D, int num_splits);

/*
 * MALA split-KV decode of one new query token per (batch, query head) against a
 * KV cache of Nk tokens that already includes the token's own key/value.
 *   q: bf16 [B, Hq, D]; k_cache, v_cache: bf16 [B, Hkv, Nk, D]
 *   cache_lens: int32 [B] device array or NULL: sequence b's cache holds n_b valid
 *       tokens (rows [0, n_b) of k_cache[b] and v_cache[b]; the rest is not read),
 *       its query sees them all (L = n_b) and its ceil(n_b / B_k) key tiles are cut
 *       into the splits as below.  Values are clamped into [0, Nk]; a sequence with
 *       n_b = 0 gets o = 0 and lse = -inf.  NULL means n_b = Nk for every sequence.
 *   o: [B, Hq, D] out (fp32 or bf16 by out_dtype); lse: fp32 [B, Hq] out
 *   head_tiles: int32 [B, Hq] or NULL out (retained tiles summed over splits)
 *   counters: int64 [MALA_NUM_COUNTERS] or NULL out
 *   num_splits >= 1: a sequence's key tiles (T = ceil(n_b / B_k) of them) are cut
 *   into num_splits contiguous ranges of ceil(T / num_splits) tiles; each range
 *   starts from an empty normalizer, so the retained set depends on num_splits.
 *   workspace: at least mala_decode_workspace_size(...) bytes.
 */
int mala_decode(const void* q, const void* k_cache, const void* v_cache,
                const int32_t* cache_lens, void* o, float* lse, int32_t* head_tiles,
                int64_t* counters, int num_splits, void* workspace, size_t workspace_bytes,
                int B, int Hq, int Hkv, int Nk, int D, float scale, float tau, int out_dtype,
                void* stream);

/* Bytes of the decode buffer that libmala.so keeps on every GPU it runs on (see
 * mala_decode_noalloc). */
#define MALA_DECODE_SCRATCH_BYTES (16u << 20)

/*
 * mala_decode for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * computation, arguments and results as mala_decode, without the workspace: the
 * split partials live in a buffer of MALA_DECODE_SCRATCH_BYTES that the library
 * holds on each GPU until the process ends (a file-scope device array, not a
 * hipMalloc).  The call itself allocates and frees nothing; its first call on a
 * device looks up the buffer's address on that device (the device of `stream`, or
 * the current device for the null stream).
 *   Limit: mala_decode_workspace_size(B, Hq, D, num_splits) must not exceed
 *   MALA_DECODE_SCRATCH_BYTES (16 MiB: e.g. 16 sequences x 32 heads x 64 splits at
 *   D = 128 do not fit, x 32 splits do); a larger call returns MALA_ERR_WORKSPACE
 *   and launches nothing.
 *   Sharing: all calls on one GPU use that GPU's one buffer, which keeps the last
 *   call's partials (every partial a call reads is written by the same call, so
 *   nothing needs clearing).  Calls ordered on one stream are safe; calls that may
 *   run at the same time on one GPU (different streams, or different threads
 *   without ordering) race on the buffer and must not be issued.
 */
int mala_decode_noalloc(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* cache_lens, void* o, float* lse, int32_t* head_tiles,
                        int64_t* counters, int num_splits, int B, int Hq, int Hkv, int Nk, int D,
                        float scale, float tau, int out_dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MALA_H */
