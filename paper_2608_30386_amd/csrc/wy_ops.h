// Device helpers shared by the two chunkwise WY refresh kernels (gfx950): operand
// types, bf16 hi/lo splitting, MFMA wrappers and raw buffer loads.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dasc_wy {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ inline float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

// The lanes of one wave see each other's LDS writes: the wave waits for its LDS accesses
// to finish, and the compiler moves no memory access across the wait.
__device__ inline void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Raw buffer resource over exactly `bytes` bytes: a load whose total offset (vector +
// scalar + immediate) reaches past the end returns zero instead of touching memory.
// Tokens past a window therefore arrive as k = v = 0, g = 0, beta = 0, which are
// identity steps of the recurrence, and no load needs a clamp or a mask.
__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}
__device__ inline float ldf(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
__device__ inline f32x2 ldf2(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

__device__ inline f32x4 ldf4(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// The value of the lane N places below (DPP row_shr:N) or above (row_shl:N) this one
// within its row of 16 lanes; 0 where that lane is outside the row.
template <int N>
__device__ inline float row_shr(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                               0x110 + N, 0xF, 0xF, true));
}
template <int N>
__device__ inline float row_shl(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                               0x100 + N, 0xF, 0xF, true));
}

// (m & a) | (~m & b) on the bits: with m all ones or all zeros per lane, a select that
// stays a single v_bfi_b32 on every lane.
__device__ inline float bsel(uint32_t m, float a, float b) {
  return __uint_as_float((__float_as_uint(a) & m) | (__float_as_uint(b) & ~m));
}

// DPP quad permute: lane k of each group of four takes the value of lane (CTRL >> 2k) & 3
// of its group (0x55 L broadcasts lane L; 0x90 = [0,0,1,2] shifts up by one lane).
template <int CTRL>
__device__ inline float quad_perm(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                               CTRL, 0xF, 0xF, false));
}

// p.x * m.x + p.y * m.y + c on the packed-bf16 dot product (v_dot2c_f32_bf16).  With m
// a unit selector (+-1 in one half, 0 in the other) it reads one bf16 of a packed word
// straight into an fp32 sum: one instruction instead of an unpack and an add.  The
// products are exact, so the result is the fp32 sum c +- p.e rounded once.
__device__ inline float dot2(bf16x2 p, bf16x2 m, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(p, m, c, false);
}
__device__ inline bf16x2 as_bf2(uint32_t w) { return __builtin_bit_cast(bf16x2, w); }
// Selectors -(low half) and -(high half).  The low one carries -0 in its high half: the
// word (-1, +0) is the fp32 inline constant -1.0's low-half image, which the compiler
// encodes as that constant while the hardware reads it as the fp32 word (+0, -1).
// (-1, -0) has no inline encoding, so it goes out as the literal it is; -0 * x adds
// nothing to the sum.
constexpr bf16x2 kNegLo = {(__bf16)-1.0f, (__bf16)-0.0f};
constexpr bf16x2 kNegHi = {(__bf16)0.0f, (__bf16)-1.0f};

__device__ inline void split(float x, __bf16& hi, __bf16& lo) {
  hi = static_cast<__bf16>(x);
  lo = static_cast<__bf16>(x - static_cast<float>(hi));
}

// Eight values split at once: hi = bf16(x) two values per packed conversion, and the
// remainder x - hi (exact in fp32) by one dot2 per value: 2 VALU per value when x dies
// here, 3 when x lives on (the accumulating dot then needs a copy of it first).
__device__ inline void split8(const float* x, bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const bf16x2 hw = __builtin_convertvector(f32x2{x[2 * p], x[2 * p + 1]}, bf16x2);
    const float r0 = dot2(hw, kNegLo, x[2 * p]), r1 = dot2(hw, kNegHi, x[2 * p + 1]);
    h[p] = __builtin_bit_cast(uint32_t, hw);
    l[p] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{r0, r1}, bf16x2));
  }
  hi = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
}

// Two values split at once into packed bf16 words: hi = (bf16(x0), bf16(x1)), lo = the
// remainders (x - hi, exact in fp32) rounded to bf16, as in split8.
__device__ inline void split2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const bf16x2 hw = __builtin_convertvector(f32x2{x0, x1}, bf16x2);
  const float r0 = dot2(hw, kNegLo, x0), r1 = dot2(hw, kNegHi, x1);
  hi = __builtin_bit_cast(uint32_t, hw);
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{r0, r1}, bf16x2));
}

__device__ inline f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// a b with both operands split: a_lo b_hi + a_hi b_lo + a_hi b_hi (small terms first)
__device__ inline f32x4 mma3(bf16x8 ah, bf16x8 al, bf16x8 bh, bf16x8 bl, f32x4 c) {
  c = mma(al, bh, c);
  c = mma(ah, bl, c);
  return mma(ah, bh, c);
}

// 16x16x16 bf16 MFMA on packed words: lane (q, r) holds A[r][4q .. 4q + 3] and
// B[4q .. 4q + 3][r], two bf16 per word
__device__ inline f32x4 mma16(uint2 a, uint2 b, f32x4 c) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                   __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

__device__ inline f32x4 mma32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8 cat(bf16x4 a, bf16x4 b) {
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Operand layout of the register-chained contractions.  One contraction step feeds lane
// (q, r) the index order k(q, e) = 4q + e (e < 4), 16 + 4q + e - 4 (e >= 4) within a group
// of 32.  Operands staged in LDS along that index are stored interleaved: the four entries
// at 4q .. 4q + 3 and the four at 16 + 4q .. 16 + 4q + 3 sit side by side at 8q, so that
// the lane reads its operand in one 16-byte access.  ilv maps a 4-aligned index to its
// stored position; ld16 reads the eight entries at a stored position.
__device__ inline int ilv(int x) { return (x & ~31) | ((x & 15) << 1) | ((x & 16) >> 2); }
__device__ inline bf16x8 ld16(const __bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

}  // namespace dasc_wy
