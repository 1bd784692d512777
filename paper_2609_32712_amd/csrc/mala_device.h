// Device-side building blocks shared by the MALA kernels (gfx950 / CDNA4 only).
//
// Lane layouts used throughout (wave64; h = lane / 32, c = lane % 32):
//   v_mfma_f32_32x32x16_bf16  C[32x32] += A[32x16] * B[16x32]
//     A: lane holds row c, k = 8h .. 8h+7          (8 bf16)
//     B: lane holds column c, k = 8h .. 8h+7       (8 bf16)
//     C: lane holds column c, rows 8*(r/4) + 4h + r%4, r = 0..15
//   v_mfma_f32_16x16x32_bf16  C[16x16] += A[16x32] * B[32x16]   (g = lane / 16)
//     A: lane holds row lane%16, k = 8g .. 8g+7;  B: column lane%16, same k;
//     C: lane holds column lane%16, rows 4g + r, r = 0..3
//   ds_read_b64_tr_b16: within each group of 16 lanes, lane t receives element
//     t%4 of the 8-byte chunks addressed by lanes 4n + t/4 (n = 0..3).  If lane i
//     of the group addresses row (R + i/4), columns (C0 + 4*(i%4)) .. +3 of a
//     row-major bf16 tile, lane t receives the column C0 + t of rows R .. R+3,
//     i.e. a 4-deep slice along the row dimension: the operand of an MFMA whose
//     contraction runs along the tile's rows.
// Because the contraction index of an MFMA may be permuted freely (as long as A
// and B agree), the probabilities of a 32x32 C tile are fed back as an operand
// without any register shuffle: k-step ks uses C registers 8ks .. 8ks+7, which
// hold the rows {16ks + 4h + 0..3} and {16ks + 8 + 4h + 0..3}.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mala {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Transposed 4x16 LDS read (see the header comment).
__device__ __forceinline__ bf16x4 lds_read_tr(const bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (__attribute__((address_space(3))) bf16x4*)(p));
}
__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Reductions between lane l and lane l ^ 32 (the two halves of a 32x32 C column).
__device__ __forceinline__ float halves_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS layout of a row-major [rows][D] bf16 tile.  Rows are D + 8 elements apart
// (272 bytes at D = 128: consecutive rows start 4 banks apart), and within a row
// the 16-byte chunk L (columns 8L .. 8L+7) is stored at chunk position
// (D / 32) * (L % 4) + L / 4.  With the 64 banks of 4 bytes and the access phases
// of gfx950 (16 lanes per phase for ds_read_b128, 32 for ds_read_b64_tr_b16),
// both access patterns of the kernels are then free of bank conflicts at D = 128:
//   * A / B operand reads: 16 lanes read the same chunk of 16 consecutive rows
//     (row offsets 17 chunks apart cover all 16 positions mod 256 bytes);
//   * transposed reads: 32 lanes read 4 consecutive rows x 32 columns, i.e. chunks
//     {4 db + x, x = 0..3}, stored at positions {4 x + db}, which the 4 rows shift
//     onto 16 distinct positions.
// Both patterns are also affine in the unrolled loop indices (k-step, column block,
// row block), so one base address per lane serves all reads of a tile with
// immediate offsets: rd_base / rd_step and tr_base / tr_step below.
template <int D>
__device__ __forceinline__ int tile_off(int row, int col) {
  const int ch = col >> 3;
  return row * (D + 8) + 8 * ((D / 32) * (ch & 3) + (ch >> 2)) + (col & 7);
}
template <int D>
constexpr int tile_elems(int rows) {
  return rows * (D + 8);
}
// Element (row, 16 kk + 8 h .. +7), the k-step kk operand of an MFMA lane in half h:
// tile_off(row, 16 kk + 8 h) == rd_base(row, h) + rd_step(kk).
template <int D>
__device__ __forceinline__ int rd_base(int row, int h) {
  return row * (D + 8) + (D / 4) * h;
}
template <int D>
constexpr int rd_step(int kk) {
  return (D / 4) * 2 * (kk & 1) + 8 * (kk >> 1);
}
// Transposed read of rows row .. row+3 at columns 32 db + 16 g1 + 4 (t16 % 4) .. +3
// (lane t16 of a 16-lane group, g1 = group % 2):
// tile_off(row + t16 / 4, 32 db + 16 g1 + 4 (t16 % 4)) == tr_base(row + t16 / 4, g1, t16) + tr_step(db).
template <int D>
__device__ __forceinline__ int tr_base(int row, int g1, int t16) {
  return row * (D + 8) + (D / 4) * (2 * g1 + ((t16 >> 1) & 1)) + 4 * (t16 & 1);
}
template <int D>
constexpr int tr_step(int db) {
  return 8 * db;
}

// The LDS address p (a lane base plus a uniform buffer offset), opaque to the
// compiler's reassociation: reads at p + constant then take the constant in the
// instruction's offset field, instead of the compiler keeping one precomputed
// register per read and re-adding the buffer offset to each.
__device__ __forceinline__ const bf16* lds_pin(const bf16* p) {
  auto q = (const __attribute__((address_space(3))) bf16*)p;
  asm volatile("" : "+v"(q));
  return (const bf16*)q;
}

// Loads through a buffer resource (base address, size in bytes): each lane gives a
// byte offset, and offsets at or past the size read as zeros, which covers the
// ragged end of a sequence without a compare or a clamp.  The address arithmetic
// is then one 32-bit lane offset plus scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}
__device__ __forceinline__ float buf_load1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0));
}
// A streaming 16-byte load (cache policy nt, bit 1 of the buffer instruction's
// policy on gfx950), for data read once per call, such as the decode's K and V
// caches.  Measured on MI355X: 1 KB-contiguous streams of such loads reach ~6.8-7.0
// TB/s where ordinary loads of the same pattern reach ~5.8-6.1.
__device__ __forceinline__ bf16x8 buf_load8_stream(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 2));
}

// Buffer loads straight into LDS (buffer_load_dwordx4 ... lds): lane i's 16 bytes
// land at lds_base + 16 i (lds_base uniform over the wavefront; checked by a
// lane-layout probe on gfx950).  Completion is counted by vmcnt.  Two forms:
//  * buf_load_lds16_tracked, the compiler's builtin: the compiler orders every
//    later LDS access of the wavefront after all of its outstanding loads (it
//    cannot tell ring slots apart), i.e. the wavefront waits for the load at its
//    next LDS access;
//  * buf_load_lds16, in assembly: the compiler does not see the LDS write and adds
//    no wait, so the load overlaps the wavefront's compute; the caller waits with
//    wait_vm / wait_vm_keep before the data is read.  M0 (the LDS base) is saved and
//    restored inside the statement, and one wait state separates its write from
//    the load.
__device__ __forceinline__ void buf_load_lds16_tracked(__amdgpu_buffer_rsrc_t r, uint32_t byte_off,
                                                       bf16* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_base,
                                           16, byte_off, 0, 0, 0);
}
typedef int i32x4 __attribute__((ext_vector_type(4)));
// The words of a buffer resource (base, size in bytes, reads past the size return
// zeros), as make_rsrc builds it, for the assembly form.
__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  return i32x4{(int)(uint32_t)a, (int)((uint32_t)(a >> 32) & 0xffffu), (int)bytes, 0x00020000};
}
__device__ __forceinline__ void buf_load_lds16(i32x4 rsrc, uint32_t byte_off, bf16* lds_base) {
  const uint32_t lds = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) bf16*)lds_base);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(byte_off), "s"(rsrc), "s"(lds)
      : "memory");
}
// Byte offset, within a row-major [*][D] bf16 matrix, of the chunk that an
// LDS-DMA lane must fetch so that chunk position pos of a tile slot laid out by
// tile_off holds the right data: rows of D/8 + 1 positions, position
// (D/32)(L % 4) + L / 4 holding logical chunk L; the padding position takes chunk 0.
template <int D>
__device__ __forceinline__ uint32_t dma_lane_offset(int pos) {
  constexpr int RC = D / 8 + 1;
  const int row = pos / RC, pc = pos % RC;
  const int L = pc < D / 8 ? pc / (D / 32) + 4 * (pc % (D / 32)) : 0;
  return (uint32_t)(row * D + 8 * L) * 2u;
}
// Waits until at most N vector-memory loads of this wavefront are outstanding
// (loads, LDS-DMA included, complete in the order they were issued, so this waits
// for all but the N most recent).  Written with the builtin, which the compiler's
// own wait insertion takes into account, so that it adds no later wait for loads
// this one already covered.  The encoding is gfx9's: vmcnt in bits 3:0 and 15:14,
// expcnt (7) and lgkmcnt (15) left at their maxima.
template <int N>
__device__ __forceinline__ void wait_vm_keep() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void wait_vm() { wait_vm_keep<0>(); }

// Hardware base-2 exponential / logarithm (v_exp_f32 / v_log_f32, ~1 ulp on normal
// results).  The softmax arguments are <= 0, so the results lie in [0, 1]; values
// below 2^-126 may flush to zero, which no tolerance here can see.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

__device__ __forceinline__ bool wave_any(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0; }

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (bf16)0.0f;
  return z;
}

__device__ __forceinline__ bf16x8 load8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
__device__ __forceinline__ void store8(bf16* p, bf16x8 v) { *reinterpret_cast<bf16x8*>(p) = v; }

// Four consecutive output values at element index i of an fp32 array, or rounded
// to bf16 (nearest even) into a bf16 array with the same layout.
__device__ __forceinline__ void store_out4(void* base, long i, f32x4 v, bool to_bf16) {
  if (to_bf16) {
    const bf16x2 a = __builtin_convertvector((f32x2{v[0], v[1]}), bf16x2);
    const bf16x2 b = __builtin_convertvector((f32x2{v[2], v[3]}), bf16x2);
    *reinterpret_cast<bf16x4*>(static_cast<bf16*>(base) + i) = bf16x4{a[0], a[1], b[0], b[1]};
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(base) + i) = v;
  }
}

// Two-term bf16 split of fp32 values: x ~= hi + lo with |x - hi - lo| <= 2^-16 |x|.
// The post-score products (P V, P^T dO, dS^T Q, dS K) run as two MFMAs, one per
// term, so the probabilities keep ~16 significant bits instead of bf16's 8.
__device__ __forceinline__ void split_bf16x8(const float* x, bf16x8& hi, bf16x8& lo) {
  // one packed conversion per pair; the high parts come back to fp32 by bit moves
  // (a bf16 is the upper half of an fp32), so x - hi is exact
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 h2 = __builtin_convertvector((f32x2{x[i], x[i + 1]}), bf16x2);
    const uint32_t u = __builtin_bit_cast(uint32_t, h2);
    const float h0 = __uint_as_float(u << 16), h1 = __uint_as_float(u & 0xffff0000u);
    const bf16x2 l2 = __builtin_convertvector((f32x2{x[i] - h0, x[i + 1] - h1}), bf16x2);
    hi[i] = h2[0];
    hi[i + 1] = h2[1];
    lo[i] = l2[0];
    lo[i + 1] = l2[1];
  }
}

// The high bf16 terms only (see split_bf16x8).
__device__ __forceinline__ bf16x8 hi_bf16x8(const float* x) {
  bf16x8 hi;
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 h2 = __builtin_convertvector((f32x2{x[i], x[i + 1]}), bf16x2);
    hi[i] = h2[0];
    hi[i + 1] = h2[1];
  }
  return hi;
}

// The low bf16 terms of x given its high terms hi (as hi_bf16x8 returned them).
__device__ __forceinline__ bf16x8 lo_bf16x8(const float* x, bf16x8 hi) {
  bf16x8 lo;
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const uint32_t u = __builtin_bit_cast(uint32_t, bf16x2{hi[i], hi[i + 1]});
    const float h0 = __uint_as_float(u << 16), h1 = __uint_as_float(u & 0xffff0000u);
    const bf16x2 l2 = __builtin_convertvector((f32x2{x[i] - h0, x[i + 1] - h1}), bf16x2);
    lo[i] = l2[0];
    lo[i + 1] = l2[1];
  }
  return lo;
}

}  // namespace mala
