// Device-side types and helpers shared by the FEM kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fem {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// v_exp_f32 (2^x) and v_log_f32 (log2 x): the hardware transcendental units.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_hw(float x) { return __builtin_amdgcn_logf(x); }

// Round two floats to bf16 (round-to-nearest-even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x2 to_bf16x2(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_convertvector(f, bf16x2);
}

// c + p.x + p.y for a bf16 pair, widened exactly to fp32 by shifts and masks.
// (The packed dot-product instructions would do this in one op, but they wait
// for the matrix pipe, i.e. behind every MFMA another wave of the SIMD issues.)
__device__ __forceinline__ float add_bf16x2(bf16x2 p, float c) {
  const unsigned u = __builtin_bit_cast(unsigned, p);
  return (c + __uint_as_float(u << 16)) + __uint_as_float(u & 0xffff0000u);
}

// Value of lane (l ^ 32) for every lane l (v_permlane32_swap).
__device__ __forceinline__ float other_half(float x) {
  unsigned u = __float_as_uint(x);
  auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  // lanes 0..31: r[1] holds lane l+32; lanes 32..63: r[0] holds lane l-32
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

__device__ __forceinline__ float wave_max(float x) {
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// LDS byte address of a generic pointer into shared memory.
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// Direct global -> LDS loads (lane l's bytes land at dst + l * size; dst is
// the same for the whole wave).  Issued as inline assembly so the compiler
// does not see an LDS write in flight: with one in flight it treats LDS
// reads as completing out of order (every read then waits for all earlier
// ones) and waits for the whole load queue before transposing reads.  The
// caller waits for completion explicitly (s_waitcnt vmcnt(0)) before the
// barrier that publishes the buffer.
//
// The load takes its LDS address from m0.  An SALU write of m0 needs one
// wait state before an LDS-DMA load reads it, and the hazard recognizer
// does not look inside inline assembly, so the block carries its own
// s_nop.  The compiler also treats m0 as reserved and ignores a clobber of
// it, so the block saves m0 into a scratch SGPR and restores it after the
// load has issued (the load reads m0 at issue): whatever the compiler keeps
// in m0 survives the block.
__device__ __forceinline__ void dma16(const void* src, void* dst) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds_addr(dst)))
      : "memory");
}
// The same load with a wave-uniform 64-bit base in SGPRs and a 32-bit lane
// offset: one VGPR per load instead of a 64-bit address pair.  The base is
// the same in every lane; it is read from the first lane so that it sits in
// SGPRs wherever the compiler cannot prove it uniform.
__device__ __forceinline__ void dma16s(const void* base_any, unsigned off, void* dst) {
  // (the builtin returns int: each half is widened as unsigned, never sign-extended)
  const uint64_t b = reinterpret_cast<uint64_t>(base_any);
  const unsigned hi = (unsigned)__builtin_amdgcn_readfirstlane((unsigned)(b >> 32));
  const unsigned lo = (unsigned)__builtin_amdgcn_readfirstlane((unsigned)b);
  const uint64_t base = ((uint64_t)hi << 32) | (uint64_t)lo;
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds_addr(dst)))
      : "memory");
}
// The same load with the LDS byte address given as an integer the caller
// keeps wave-uniform (no pointer conversion per load): with a uniform base
// and address the block is five scalar instructions and the load.
__device__ __forceinline__ void dma16u(const void* base_any, unsigned off, unsigned lds) {
  const uint64_t b = reinterpret_cast<uint64_t>(base_any);
  const unsigned hi = (unsigned)__builtin_amdgcn_readfirstlane((unsigned)(b >> 32));
  const unsigned lo = (unsigned)__builtin_amdgcn_readfirstlane((unsigned)b);
  const uint64_t base = ((uint64_t)hi << 32) | (uint64_t)lo;
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(base), "s"((unsigned)__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}
// Buffer-resource form: rsrc covers [base, base + bytes) (a raw buffer:
// stride 0, 32-bit data format), so a lane whose offset falls past its end
// loads zeros and reads nothing outside the range.  All operands wave-uniform
// except the lane offset.
typedef __attribute__((ext_vector_type(4))) int rsrc_t;
__device__ __forceinline__ rsrc_t buffer_rsrc(const void* base_any, unsigned bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base_any);
  rsrc_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(unsigned)b);
  r[1] = __builtin_amdgcn_readfirstlane((int)(unsigned)(b >> 32)) & 0xffff;  // stride 0
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;  // data format: 32 bits
  return r;
}
__device__ __forceinline__ void dma16b(rsrc_t rsrc, unsigned off, unsigned lds) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(off), "s"(rsrc), "s"((unsigned)__builtin_amdgcn_readfirstlane(lds))
      : "memory");
}
__device__ __forceinline__ void dma4(const void* src, void* dst) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds_addr(dst)))
      : "memory");
}

// ---- permuted contraction order and swizzled tiles ------------------------
//
// Storage position of contraction index r (0..31) in a row whose 32-blocks feed
// MFMA operands against operands taken from a 32x32 accumulator's rows: the
// accumulator holds rows {8(i/4) + 4h + i%4} in lane half h, i.e. bits 2 and 3
// of the row index swapped.
__host__ __device__ constexpr int epos32(int r) {
  return (r & 16) + (((r >> 2) & 1) << 3) + (((r >> 3) & 1) << 2) + (r & 3);
}
__host__ __device__ constexpr int ppos(int x) { return (x & ~31) + epos32(x & 31); }

// A streamed [64][D] bf16 tile sits in LDS unpadded, 16-byte chunk c of row r
// at chunk position c ^ swz(r).  swz makes both read patterns bank-conflict
// free: a row-major MFMA fragment (16 lanes, 16 consecutive rows, one chunk
// each) and a transposing read (4 consecutive rows, 32 consecutive columns).
template <int D>
__host__ __device__ constexpr int swz(int r) {
  return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3))
       : D == 64  ? ((((r >> 1) & 1) << 2) | ((r >> 2) & 3))
                  : ((r >> 2) & 3);
}

template <int D>
__device__ __forceinline__ int swz_off(int row, int chunk) {  // byte offset
  return row * D * 2 + ((chunk ^ swz<D>(row)) << 4);
}

// Row-major MFMA fragment of a swizzled tile: 8 bf16 of row `row`, chunk `chunk`.
template <int D>
__device__ __forceinline__ bf16x8 frag_rows(const bf16* t, int row, int chunk) {
  return *reinterpret_cast<const bf16x8*>(reinterpret_cast<const char*>(t) + swz_off<D>(row, chunk));
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Transposed MFMA A fragment of a swizzled tile: A[m][k] = tile[row(p0 + k)][col0 + m]
// for m < 32, k < 16, with the contraction positions p0 + k in permuted
// order (row(p) = ppos(p)).  Two transposing reads: in each 16-lane group,
// lanes 4r..4r+3 read 4 columns each of row r, and lane c gets column c of
// the 4 rows.  Group g = lane / 16 takes columns col0 + 16 (g & 1) .. and
// positions p0 + 8 (g >> 1) ..: the A layout of v_mfma_f32_32x32x16_bf16.
template <int D>
__device__ __forceinline__ bf16x8 frag_tr(const bf16* t, int col0, int p0) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  const int r = i >> 2, q = i & 3;
  const int col = col0 + 16 * (g & 1) + 4 * q;
  const int p = p0 + 8 * (g >> 1);
  const char* b = reinterpret_cast<const char*>(t);
  const int r0 = ppos(p) + r, r1 = ppos(p + 4) + r;
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)(b + swz_off<D>(r0, col >> 3) + (col & 7) * 2));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)(b + swz_off<D>(r1, col >> 3) + (col & 7) * 2));
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 x = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, x);
}

// Streaming log2-sum-exp2 accumulator: value = m + log2(s).
struct Lse2 {
  float m = -INFINITY;
  float s = 0.f;
  __device__ __forceinline__ void add(float w) {
    if (w > m) {
      s = s * exp2_hw(m - w) + 1.f;
      m = w;
    } else {
      s += exp2_hw(w - m);
    }
  }
  // Combine across the 64 lanes of a wave; every lane gets the total.
  __device__ __forceinline__ float wave_total() const {
    float M = wave_max(m);
    float part = (m == -INFINITY) ? 0.f : s * exp2_hw(m - M);
    float S = wave_sum(part);
    return M + log2_hw(S);
  }
};

}  // namespace fem
