// C ABI of libmala.so: argument validation, workspace sizing and kernel launches.
// Declarations and the contract of every entry point are in include/mala.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "mala.h"
#include "mala_device.h"
#include "mala_kernels.h"

namespace {

thread_local char g_err[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return status;
}

int hip_fail(hipError_t e, const char* where) {
  snprintf(g_err, sizeof(g_err), "%s: %s", where, hipGetErrorString(e));
  return MALA_ERR_HIP;
}

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Backward workspace: D_q = rowsum(O_q * dO_q) for every query row, then the dQ pass's
// tile decisions for the key-major pass (one byte per query tile, query head and
// 128-key block; query-tile rows as mask_rows gives them).
size_t dvec_bytes(long rows) { return round_up((size_t)rows * sizeof(float), 256); }
int mask_rows(bool packed, int B, int Nq) {
  return packed ? Nq / mala::kBq + B : B * ((Nq + mala::kBq - 1) / mala::kBq);
}
size_t mask_bytes(bool packed, int B, int Hq, int Nq, int max_k) {
  const size_t nkblk = (size_t)(max_k + mala::kBwdKeys - 1) / mala::kBwdKeys;
  return round_up((size_t)Hq * nkblk * mask_rows(packed, B, Nq), 256);
}
// Parts of the dK/dV sweeps (fixed-length batches): one per sweep when the key
// blocks alone give kDkdvSplitGroups workgroups; otherwise parts of the smallest
// power of two >= kDkdvPartMin iterations that gives at most ~kDkdvSplitGroups
// parts over all sweeps, so that a long sweep (the first key blocks', or one that
// retains every tile) no longer sets the kernel's time alone.
void dkdv_split(int B, int Hq, int Hkv, int Nq, int Nk, int* psize, int* nparts) {
  const int grp = Hq / Hkv, nkblk = (Nk + mala::kBwdKeys - 1) / mala::kBwdKeys;
  *psize = 1 << 30;
  *nparts = 1;
  if ((long)nkblk * B * Hkv >= mala::kDkdvSplitGroups) return;
  long total = 0;
  for (int j = 0; j < nkblk; ++j) total += mala::dkdv_iterations(Nq, Nk, j * mala::kBwdKeys, grp);
  total *= (long)B * Hkv;
  const int longest = mala::dkdv_iterations(Nq, Nk, 0, grp);
  long ps = mala::kDkdvPartMin;
  while (ps * 2 * mala::kDkdvSplitGroups <= total) ps *= 2;
  if (ps >= longest) return;
  *psize = (int)ps;
  *nparts = (int)((longest + ps - 1) / ps);
}
// fp32 partial dV and dK of every part of the split sweeps (fixed-length batches)
size_t part_bytes(int B, int Hq, int Hkv, int Nq, int Nk, int D) {
  int psize, nparts;
  dkdv_split(B, Hq, Hkv, Nq, Nk, &psize, &nparts);
  return nparts > 1 ? round_up((size_t)nparts * 2 * B * Hkv * Nk * D * sizeof(float), 256) : 0;
}
size_t bwd_workspace(bool packed, int B, int Hq, int Hkv, int Nq, int max_k, int D) {
  const long rows = packed ? (long)Hq * Nq : (long)B * Hq * Nq;
  return dvec_bytes(rows) + mask_bytes(packed, B, Hq, Nq, max_k) +
         (packed ? 0 : part_bytes(B, Hq, Hkv, Nq, max_k, D));
}

int check_common(int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal, float scale, float tau) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || Nq <= 0 || Nk <= 0)
    return fail(MALA_ERR_INVALID_ARG, "non-positive size (B, Hq, Hkv, Nq, Nk)");
  if (Hq % Hkv != 0) return fail(MALA_ERR_INVALID_ARG, "Hq (%d) is not a multiple of Hkv (%d)", Hq, Hkv);
  if (Nq > Nk) return fail(MALA_ERR_INVALID_ARG, "Nq (%d) > Nk (%d)", Nq, Nk);
  if (!(tau >= 0.f) || isinf(tau)) return fail(MALA_ERR_INVALID_ARG, "tau must be finite and >= 0");
  if (!(scale > 0.f) || isinf(scale)) return fail(MALA_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (causal != 1) return fail(MALA_ERR_UNSUPPORTED, "only causal attention is supported");
  if (D != 64 && D != 128) return fail(MALA_ERR_UNSUPPORTED, "head_dim %d not in {64, 128}", D);
  return MALA_OK;
}

// The training kernels address one (batch, head) slice from a tile start through
// buffer resources whose range is a 32-bit byte count: Nk x D bf16 values must fit.
int check_slice_range(int Nk, int D) {
  const long long bytes = (long long)Nk * D * 2;
  if (bytes > 0xffffffffLL)
    return fail(MALA_ERR_UNSUPPORTED, "Nk x D x 2 = %lld bytes exceeds the 32-bit slice range", bytes);
  return MALA_OK;
}

float log2_tau(float tau) { return tau > 0.f ? log2f(tau) : -INFINITY; }

}  // namespace

extern "C" {

mala_geometry_t mala_geometry(int head_dim, int pass) {
  mala_geometry_t g = {0, 0};
  if (head_dim != 64 && head_dim != 128) return g;
  if (pass == MALA_PASS_FWD || pass == MALA_PASS_BWD) {
    g.block_q = mala::kBq;
    g.block_k = mala::kBk;
  } else if (pass == MALA_PASS_DECODE) {
    g.block_q = 1;
    g.block_k = mala::kDecBk;
  }
  return g;
}

const char* mala_strerror(int status) {
  switch (status) {
    case MALA_OK: return "success";
    case MALA_ERR_INVALID_ARG: return "invalid argument";
    case MALA_ERR_UNSUPPORTED: return "unsupported configuration";
    case MALA_ERR_WORKSPACE: return "workspace missing or too small";
    case MALA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* mala_last_error(void) { return g_err; }

}  // extern "C"

namespace {

// Packed batches: the query-row / key-row starts of the sequences (cu null for the
// fixed-length layout, cu_k null for the same starts as cu) and their longest
// lengths.
struct Packed {
  const int32_t* cu;
  const int32_t* cu_k;
  int max_q, max_k;
};

// Shared by the fixed-length and packed entry points: B slices (sequences) of
// Nq / Nk rows each (packed: Nq, Nk = the query / key totals, the head strides).
int run_fwd(const void* q, const void* k, const void* v, const Packed& pk,
            void* o, int o_dtype, float* lse, int32_t* row_tiles, int64_t* counters, int B,
            int Hq, int Hkv, int Nq, int Nk, int D, float scale, float tau, hipStream_t s) {
  if (counters) {
    hipError_t e = mala::launch_fill_zero(counters, mala::kNumCounters * sizeof(int64_t), s);
    if (e != hipSuccess) return hip_fail(e, "mala_fwd: clearing counters");
  }
  mala::FwdParams p;
  p.q = (const __bf16*)q;
  p.k = (const __bf16*)k;
  p.v = (const __bf16*)v;
  p.o = o;
  p.o_bf16 = o_dtype == MALA_OUT_BF16;
  p.lse = lse;
  p.row_tiles = row_tiles;
  p.counters = (unsigned long long*)counters;
  p.cu = pk.cu;
  p.cu_k = pk.cu_k;
  p.max_len = pk.cu ? pk.max_q : Nq;
  p.max_len_k = pk.cu ? pk.max_k : Nk;
  p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.Nq = Nq; p.Nk = Nk;
  p.scale2 = scale * mala::kLog2e;
  p.log2tau = log2_tau(tau);
  p.nqblk = (p.max_len + mala::kFwdRows - 1) / mala::kFwdRows;
  hipError_t e = mala::launch_fwd(p, D, s);
  if (e != hipSuccess) return hip_fail(e, "mala_fwd: kernel launch");
  return MALA_OK;
}

int run_bwd(const void* q, const void* k, const void* v, const Packed& pk,
            const void* o, int o_dtype, const float* lse, const void* dout, void* dq, void* dk,
            void* dv, int grad_dtype, int32_t* row_tiles, int64_t* counters, void* workspace,
            int B, int Hq, int Hkv, int Nq, int Nk, int D, float scale, float tau,
            hipStream_t s) {
  hipError_t e;
  // D_q over every row of the q-shaped tensors (packed: all heads x total rows)
  const long rows = pk.cu ? (long)Hq * Nq : (long)B * Hq * Nq;
  if (counters && (e = mala::launch_fill_zero(counters, mala::kNumCounters * sizeof(int64_t), s)) != hipSuccess)
    return hip_fail(e, "mala_bwd: clearing counters");
  float* dvec = (float*)workspace;
  if ((e = mala::launch_bwd_preprocess(o, o_dtype == MALA_OUT_BF16, (const __bf16*)dout, dvec,
                                       rows, D, s)) != hipSuccess)
    return hip_fail(e, "mala_bwd: preprocess launch");
  mala::BwdParams p;
  p.q = (const __bf16*)q;
  p.k = (const __bf16*)k;
  p.v = (const __bf16*)v;
  p.dout = (const __bf16*)dout;
  p.lse = lse;
  p.dvec = dvec;
  p.dq = dq; p.dk = dk; p.dv = dv;
  p.grad_bf16 = grad_dtype == MALA_OUT_BF16;
  p.row_tiles = row_tiles;
  p.counters = (unsigned long long*)counters;
  p.cu = pk.cu;
  p.cu_k = pk.cu_k;
  p.max_len = pk.cu ? pk.max_q : Nq;
  p.max_len_k = pk.cu ? pk.max_k : Nk;
  p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.Nq = Nq; p.Nk = Nk;
  p.scale = scale;
  p.scale2 = scale * mala::kLog2e;
  p.log2tau = log2_tau(tau);
  p.nkblk = (p.max_len_k + mala::kBwdKeys - 1) / mala::kBwdKeys;
  p.nqblk = (p.max_len + mala::kDqRows - 1) / mala::kDqRows;
  p.mask = (uint8_t*)workspace + dvec_bytes(rows);
  p.mask_rows = mask_rows(pk.cu != nullptr, B, Nq);
  p.psize = 1 << 30;
  p.nparts = 1;
  p.part = nullptr;
  if (!pk.cu) {
    dkdv_split(B, Hq, Hkv, Nq, Nk, &p.psize, &p.nparts);
    p.part = (float*)((char*)p.mask + mask_bytes(false, B, Hq, Nq, Nk));
  }
  if ((e = mala::launch_bwd(p, D, s)) != hipSuccess) return hip_fail(e, "mala_bwd: kernel launch");
  return MALA_OK;
}

int check_dtype(int d, const char* what) {
  if (d != MALA_OUT_F32 && d != MALA_OUT_BF16)
    return fail(MALA_ERR_INVALID_ARG, "%s must be MALA_OUT_F32 or MALA_OUT_BF16, got %d", what, d);
  return MALA_OK;
}

int check_varlen(const int32_t* cu_q, const int32_t* cu_k, int num_seqs, int max_q, int max_k,
                 int total_q, int total_k, int Hq, int Hkv, int D, float scale, float tau) {
  if (!cu_q) return fail(MALA_ERR_INVALID_ARG, "null cu_seqlens_q");
  if (num_seqs <= 0 || max_q <= 0 || max_k <= 0 || total_q <= 0 || total_k <= 0)
    return fail(MALA_ERR_INVALID_ARG, "non-positive size (num_seqs, max_seqlen, total)");
  if (max_q > total_q || max_k > total_k)
    return fail(MALA_ERR_INVALID_ARG, "max_seqlen above its total (%d > %d or %d > %d)", max_q,
                total_q, max_k, total_k);
  if (!cu_k && (total_k != total_q || max_k != max_q))
    return fail(MALA_ERR_INVALID_ARG, "without cu_seqlens_k the key totals must equal the query's");
  int st = check_common(1, Hq, Hkv, total_q, total_k, D, 1, scale, tau);
  if (!st) st = check_slice_range(total_k, D);
  return st;
}

int check_decode(const void* q, const void* k_cache, const void* v_cache, const void* o,
                 const float* lse, int num_splits, int B, int Hq, int Hkv, int Nk, int D,
                 float scale, float tau, int out_dtype) {
  if (!q || !k_cache || !v_cache || !o || !lse)
    return fail(MALA_ERR_INVALID_ARG, "null q, k_cache, v_cache, o or lse");
  int st = check_common(B, Hq, Hkv, 1, Nk, D, 1, scale, tau);
  if (!st) st = check_dtype(out_dtype, "out_dtype");
  if (st) return st;
  if (num_splits < 1) return fail(MALA_ERR_INVALID_ARG, "num_splits must be >= 1");
  return MALA_OK;
}

// The split kernel writes every partial [B, Hq, num_splits, D + 4] (also for splits
// without tiles: o = 0, lse = -inf) before the merge kernel reads it, so the buffer
// needs no clearing.
int run_decode(const void* q, const void* k_cache, const void* v_cache, const int32_t* cache_lens,
               void* o, float* lse, int32_t* head_tiles, int64_t* counters, int num_splits,
               float* part, int B, int Hq, int Hkv, int Nk, int D, float scale, float tau,
               int out_dtype, hipStream_t s) {
  hipError_t e;
  if (counters &&
      (e = mala::launch_fill_zero(counters, mala::kNumCounters * sizeof(int64_t), s)) != hipSuccess)
    return hip_fail(e, "mala_decode: clearing counters");
  const int T = (Nk + mala::kDecBk - 1) / mala::kDecBk;
  mala::DecParams p;
  p.q = (const __bf16*)q;
  p.k = (const __bf16*)k_cache;
  p.v = (const __bf16*)v_cache;
  p.lens = cache_lens;
  p.part = part;
  p.counters = (unsigned long long*)counters;
  p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.Nk = Nk;
  p.S = num_splits;
  p.nchunk = (Hq / Hkv + 15) / 16;
  p.T = T;
  p.tps = (T + num_splits - 1) / num_splits;
  p.scale2 = scale * mala::kLog2e;
  p.thr2 = log2_tau(tau) - log2f((float)Nk);
  p.log2tau = log2_tau(tau);
  if ((e = mala::launch_decode(p, D, s)) != hipSuccess) return hip_fail(e, "mala_decode: split launch");
  if ((e = mala::launch_decode_combine(part, o, out_dtype == MALA_OUT_BF16, lse, head_tiles,
                                       B * Hq, num_splits, D, s)) != hipSuccess)
    return hip_fail(e, "mala_decode: combine launch");
  return MALA_OK;
}

// The decode buffer of mala_decode_noalloc: a file-scope device array that every GPU
// the library runs on holds until the process ends.  In host code `scratch` names a
// host-side stand-in, not the array's device address: the address on a device comes
// from hipGetSymbolAddress, looked up once per device (with that device current) and
// kept in g_scratch; only that address is passed to kernels.
constexpr size_t kDecodeScratchBytes = MALA_DECODE_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];

// The device address of `scratch` on the device of stream s (the current device for
// the null stream).
int scratch_address(hipStream_t s, void** out) {
  int dev = 0;
  hipError_t e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "mala_decode_noalloc: device of the stream");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(MALA_ERR_UNSUPPORTED, "mala_decode_noalloc: device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return hip_fail(e, "mala_decode_noalloc: hipGetDevice");
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess)
      return hip_fail(e, "mala_decode_noalloc: hipSetDevice");
    void* ptr = nullptr;
    const hipError_t eg = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev && (e = hipSetDevice(cur)) != hipSuccess)
      return hip_fail(e, "mala_decode_noalloc: restoring the current device");
    if (eg != hipSuccess) return hip_fail(eg, "mala_decode_noalloc: hipGetSymbolAddress");
    if (!ptr) return fail(MALA_ERR_HIP, "mala_decode_noalloc: no device address for the buffer");
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return MALA_OK;
}

}  // namespace

extern "C" {

int mala_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int32_t* row_tiles,
             int64_t* counters, int B, int Hq, int Hkv, int Nq, int Nk, int D, int causal,
             float scale, float tau, int out_dtype, void* stream) {
  g_err[0] = 0;
  if (!q || !k || !v || !o || !lse) return fail(MALA_ERR_INVALID_ARG, "null q, k, v, o or lse");
  int st = check_common(B, Hq, Hkv, Nq, Nk, D, causal, scale, tau);
  if (!st) st = check_slice_range(Nk, D);
  if (!st) st = check_dtype(out_dtype, "out_dtype");
  if (st) return st;
  return run_fwd(q, k, v, Packed{}, o, out_dtype, lse, row_tiles, counters, B, Hq, Hkv, Nq, Nk,
                 D, scale, tau, (hipStream_t)stream);
}

int mala_fwd_varlen(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_q,
                    const int32_t* cu_seqlens_k, void* o, float* lse, int32_t* row_tiles,
                    int64_t* counters, int num_seqs, int max_seqlen_q, int max_seqlen_k,
                    int total_q, int total_k, int Hq, int Hkv, int D, float scale, float tau,
                    int out_dtype, void* stream) {
  g_err[0] = 0;
  if (!q || !k || !v || !o || !lse) return fail(MALA_ERR_INVALID_ARG, "null q, k, v, o or lse");
  int st = check_varlen(cu_seqlens_q, cu_seqlens_k, num_seqs, max_seqlen_q, max_seqlen_k,
                        total_q, total_k, Hq, Hkv, D, scale, tau);
  if (!st) st = check_dtype(out_dtype, "out_dtype");
  if (st) return st;
  return run_fwd(q, k, v, Packed{cu_seqlens_q, cu_seqlens_k, max_seqlen_q, max_seqlen_k}, o,
                 out_dtype, lse, row_tiles, counters, num_seqs, Hq, Hkv, total_q, total_k, D,
                 scale, tau, (hipStream_t)stream);
}

size_t mala_bwd_workspace_size(int B, int Hq, int Hkv, int Nq, int Nk, int D) {
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || Nq <= 0 || Nk <= 0 || Hq % Hkv || Nq > Nk ||
      (D != 64 && D != 128))
    return 0;
  return bwd_workspace(false, B, Hq, Hkv, Nq, Nk, D);
}

size_t mala_bwd_varlen_workspace_size(int num_seqs, int max_seqlen_k, int total_q, int Hq,
                                      int Hkv, int D) {
  if (num_seqs <= 0 || max_seqlen_k <= 0 || total_q <= 0 || Hq <= 0 || Hkv <= 0) return 0;
  return bwd_workspace(true, num_seqs, Hq, Hkv, total_q, max_seqlen_k, D);
}

int mala_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
             const void* dout, void* dq, void* dk, void* dv, int32_t* row_tiles,
             int64_t* counters, void* workspace, size_t workspace_bytes, int B, int Hq, int Hkv,
             int Nq, int Nk, int D, int causal, float scale, float tau, int o_dtype,
             int grad_dtype, void* stream) {
  g_err[0] = 0;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv)
    return fail(MALA_ERR_INVALID_ARG, "null tensor argument");
  int st = check_common(B, Hq, Hkv, Nq, Nk, D, causal, scale, tau);
  if (!st) st = check_slice_range(Nk, D);
  if (!st) st = check_dtype(o_dtype, "o_dtype");
  if (!st) st = check_dtype(grad_dtype, "grad_dtype");
  if (st) return st;
  const size_t need = mala_bwd_workspace_size(B, Hq, Hkv, Nq, Nk, D);
  if (!workspace || workspace_bytes < need)
    return fail(MALA_ERR_WORKSPACE, "mala_bwd needs %zu workspace bytes, got %zu", need, workspace_bytes);
  if (((uintptr_t)workspace) % 16) return fail(MALA_ERR_WORKSPACE, "workspace not 16-byte aligned");
  return run_bwd(q, k, v, Packed{}, o, o_dtype, lse, dout, dq, dk, dv, grad_dtype, row_tiles,
                 counters, workspace, B, Hq, Hkv, Nq, Nk, D, scale, tau, (hipStream_t)stream);
}

int mala_bwd_varlen(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_q,
                    const int32_t* cu_seqlens_k, const void* o, const float* lse,
                    const void* dout, void* dq, void* dk, void* dv, int32_t* row_tiles,
                    int64_t* counters, void* workspace, size_t workspace_bytes, int num_seqs,
                    int max_seqlen_q, int max_seqlen_k, int total_q, int total_k, int Hq,
                    int Hkv, int D, float scale, float tau, int o_dtype, int grad_dtype,
                    void* stream) {
  g_err[0] = 0;
  if (!q || !k || !v || !o || !lse || !dout || !dq || !dk || !dv)
    return fail(MALA_ERR_INVALID_ARG, "null tensor argument");
  int st = check_varlen(cu_seqlens_q, cu_seqlens_k, num_seqs, max_seqlen_q, max_seqlen_k,
                        total_q, total_k, Hq, Hkv, D, scale, tau);
  if (!st) st = check_dtype(o_dtype, "o_dtype");
  if (!st) st = check_dtype(grad_dtype, "grad_dtype");
  if (st) return st;
  const size_t need = mala_bwd_varlen_workspace_size(num_seqs, max_seqlen_k, total_q, Hq, Hkv, D);
  if (!workspace || workspace_bytes < need)
    return fail(MALA_ERR_WORKSPACE, "mala_bwd_varlen needs %zu workspace bytes, got %zu", need,
                workspace_bytes);
  if (((uintptr_t)workspace) % 16) return fail(MALA_ERR_WORKSPACE, "workspace not 16-byte aligned");
  return run_bwd(q, k, v, Packed{cu_seqlens_q, cu_seqlens_k, max_seqlen_q, max_seqlen_k}, o,
                 o_dtype, lse, dout, dq, dk, dv, grad_dtype, row_tiles, counters, workspace,
                 num_seqs, Hq, Hkv, total_q, total_k, D, scale, tau, (hipStream_t)stream);
}

size_t mala_decode_workspace_size(int B, int Hq, int D, int num_splits) {
  if (B <= 0 || Hq <= 0 || num_splits <= 0 || (D != 64 && D != 128)) return 0;
  return round_up((size_t)B * Hq * num_splits * (D + mala::kDecStride) * sizeof(float), 256);
}

int mala_decode(const void* q, const void* k_cache, const void* v_cache,
                const int32_t* cache_lens, void* o, float* lse, int32_t* head_tiles,
                int64_t* counters, int num_splits, void* workspace, size_t workspace_bytes,
                int B, int Hq, int Hkv, int Nk, int D, float scale, float tau, int out_dtype,
                void* stream) {
  g_err[0] = 0;
  int st = check_decode(q, k_cache, v_cache, o, lse, num_splits, B, Hq, Hkv, Nk, D, scale, tau,
                        out_dtype);
  if (st) return st;
  const size_t need = mala_decode_workspace_size(B, Hq, D, num_splits);
  if (!workspace || workspace_bytes < need)
    return fail(MALA_ERR_WORKSPACE, "mala_decode needs %zu workspace bytes, got %zu", need,
                workspace_bytes);
  if (((uintptr_t)workspace) % 16) return fail(MALA_ERR_WORKSPACE, "workspace not 16-byte aligned");
  return run_decode(q, k_cache, v_cache, cache_lens, o, lse, head_tiles, counters, num_splits,
                    (float*)workspace, B, Hq, Hkv, Nk, D, scale, tau, out_dtype,
                    (hipStream_t)stream);
}

int mala_decode_noalloc(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* cache_lens, void* o, float* lse, int32_t* head_tiles,
                        int64_t* counters, int num_splits, int B, int Hq, int Hkv, int Nk, int D,
                        float scale, float tau, int out_dtype, void* stream) {
  g_err[0] = 0;
  int st = check_decode(q, k_cache, v_cache, o, lse, num_splits, B, Hq, Hkv, Nk, D, scale, tau,
                        out_dtype);
  if (st) return st;
  const size_t need = mala_decode_workspace_size(B, Hq, D, num_splits);
  if (need > kDecodeScratchBytes)
    return fail(MALA_ERR_WORKSPACE,
                "mala_decode_noalloc: the split partials need %zu bytes, more than the library's "
                "%zu-byte decode buffer (use mala_decode with a workspace, or fewer splits)",
                need, kDecodeScratchBytes);
  void* part = nullptr;
  hipStream_t s = (hipStream_t)stream;
  if ((st = scratch_address(s, &part)) != MALA_OK) return st;
  return run_decode(q, k_cache, v_cache, cache_lens, o, lse, head_tiles, counters, num_splits,
                    (float*)part, B, Hq, Hkv, Nk, D, scale, tau, out_dtype, s);
}

}  // extern "C"
