// Device helpers shared by the VMM kernels for 2-bit planes.
#pragma once

#include "grinqh_internal.h"

namespace grinqh {
namespace vmmdev {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c,
                                false);
}

// The same dot product in its three-address form (v_dot2_f32_f16): the
// builtin is emitted as v_dot2c, whose accumulator must also be its
// destination, and in a loop whose accumulators travel through different
// registers on different paths the compiler then copies each accumulator
// before its dot (measured ~130 extra moves in the batch-1 VMM loop).
__device__ __forceinline__ float dot2r(uint32_t a, uint32_t b, float c) {
  float d;
  asm("v_dot2_f32_f16 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}

// Number of set predicates in lanes below this one, and in the whole wave.
__device__ __forceinline__ int lanes_below(bool pred) {
  const uint64_t m = __ballot(pred);
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
__device__ __forceinline__ int lanes_total(bool pred) { return (int)__popcll(__ballot(pred)); }

// The same over this lane's half wave (lanes 0..31 or 32..63); the low mask
// is zeroed for the upper half, so both counts run unbranched.
__device__ __forceinline__ int half_below(bool pred) {
  const uint64_t m = __ballot(pred);
  const uint32_t lo = (threadIdx.x & 32) ? 0u : (uint32_t)m;
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo(lo, 0u));
}
__device__ __forceinline__ int half_total(bool pred) {
  const uint64_t m = __ballot(pred);
  return (threadIdx.x & 32) ? __popc((uint32_t)(m >> 32)) : __popc((uint32_t)m);
}

// Sixteen outputs of one pair: w1/w2 are the two plane rows' dwords.
template <int NB, int NACC>
__device__ __forceinline__ void consume_pair(uint32_t w1, uint32_t w2, uint32_t m4,
                                             const uint32_t (&xp)[NB], float (&acc)[NB][NACC],
                                             int base) {
  const uint32_t m6 = m4 - 0x08000800u;   // exponent field - 2 in both halves
  const uint32_t m8 = m4 - 0x10001000u;   // exponent field - 4
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t R = __builtin_amdgcn_perm(w2, w1, h ? 0x07060302u : 0x05040100u);
    const uint32_t A = R, Bv = R << 4, C = R >> 6;
    uint32_t f[8];
    f[0] = (Bv & 0x00300030u) | m4;   // field 0: bits 0-1 moved to 4-5
    f[1] = (Bv & 0x00C000C0u) | m6;   // field 1: bits 2-3 -> 6-7
    f[2] = (A & 0x00300030u) | m4;    // field 2: bits 4-5
    f[3] = (A & 0x00C000C0u) | m6;    // field 3: bits 6-7
    f[4] = (A & 0x03000300u) | m8;    // field 4: bits 8-9
    f[5] = (C & 0x00300030u) | m4;    // field 5: bits 10-11 -> 4-5
    f[6] = (C & 0x00C000C0u) | m6;    // field 6: bits 12-13 -> 6-7
    f[7] = (C & 0x03000300u) | m8;    // field 7: bits 14-15 -> 8-9
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[b][base + h * 8 + e] = dot2(f[e], xp[b], acc[b][base + h * 8 + e]);
  }
}

// 2^(4-p) for the field position p used by output e (mod 8) above: the
// output's offset relative to the position-4 offset summed per pair.
__device__ __forceinline__ float offset_factor(int e) {
  const int m = e & 7;
  return (m == 4 || m == 7) ? 0.0625f : ((m == 1 || m == 3 || m == 6) ? 0.25f : 1.0f);
}

// phi_b - 128 in 8-bit code units for a b-bit read of a b_max-bit code: a
// b_max-bit code is the top b_max bits of an 8-bit one, its phi_b is
// 2^(7-b) in those units, and 0 at b = b_max (nothing dropped).
__device__ __forceinline__ float phi_minus_offset(int b, int bmax) {
  return (b < bmax ? (float)(1 << (7 - b)) : 0.0f) - 128.0f;
}

// Sum of a value over the four 16-lane rows of a wave, in every lane.
// v_permlane32_swap exchanges the upper 32 lanes of its first operand with
// the lower 32 of its second, and v_permlane16_swap the odd rows of the first
// with the even rows of the second; both write both registers.  They are
// written as asm with both registers as in/out operands: the compiler's
// builtins for them, given one value twice, have been seen to read back the
// first result in place of the second.  s_nop 1 covers the VALU-write to
// permlane-read hazard of the copy just before.
__device__ __forceinline__ float row_sum4(float v) {
  uint32_t a = __builtin_bit_cast(uint32_t, v), b = a;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
  v = __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);   // rows r and r^2
  a = __builtin_bit_cast(uint32_t, v);
  b = a;
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);  // and r^1
}

// Rotate right by n lanes inside each 16-lane row (DPP row_ror).
template <int n>
__device__ __forceinline__ float row_ror(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                               0x120 + n, 0xF, 0xF, false));
}

// Sum over the whole wave, in every lane: row sums by rotation, then rows.
__device__ __forceinline__ float wave_sum_dpp(float v) {
  v += row_ror<8>(v);
  v += row_ror<4>(v);
  v += row_ror<2>(v);
  v += row_ror<1>(v);
  return row_sum4(v);
}

// Sum over this lane's half wave, in every lane of it: row sums by rotation,
// then rows r and r^1.
__device__ __forceinline__ float half_sum_dpp(float v) {
  v += row_ror<8>(v);
  v += row_ror<4>(v);
  v += row_ror<2>(v);
  v += row_ror<1>(v);
  uint32_t a = __builtin_bit_cast(uint32_t, v), b = a;
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

// Sum over the lane groups of a wave that hold the same outputs: LPR lanes
// cover a plane row, so 64 / LPR lane groups share each output.
template <int LPR>
__device__ __forceinline__ float lane_group_sum(float v) {
  if constexpr (LPR == 16) {
    return row_sum4(v);
  } else if constexpr (LPR == 32) {
    uint32_t a = __builtin_bit_cast(uint32_t, v), b = a;
    asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
    return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
  } else {
    return v;
  }
}

// Bit o of a 16-bit word moved to bit 2o.
__device__ __forceinline__ uint32_t spread_bits(uint32_t v) {
  v = (v | (v << 8)) & 0x00FF00FFu;
  v = (v | (v << 4)) & 0x0F0F0F0Fu;
  v = (v | (v << 2)) & 0x33333333u;
  return (v | (v << 1)) & 0x55555555u;
}

// The codes of 16 outputs from the four 2-bit plane words (output o's field
// at bit 2o, plane 1 most significant): byte i of q[d] is the code of output
// 4i + d.
__device__ __forceinline__ void assemble_codes(uint32_t w1, uint32_t w2, uint32_t w3, uint32_t w4,
                                               uint32_t (&q)[4]) {
  // 4-bit fields of the even (E) and odd (O) outputs: output 2m or 2m+1 at
  // bits 4m..4m+3, the first plane of the pair on top
  const uint32_t E12 = ((w1 << 2) & 0xCCCCCCCCu) | (w2 & 0x33333333u);
  const uint32_t O12 = (w1 & 0xCCCCCCCCu) | ((w2 >> 2) & 0x33333333u);
  const uint32_t E34 = ((w3 << 2) & 0xCCCCCCCCu) | (w4 & 0x33333333u);
  const uint32_t O34 = (w3 & 0xCCCCCCCCu) | ((w4 >> 2) & 0x33333333u);
  q[0] = ((E12 & 0x0F0F0F0Fu) << 4) | (E34 & 0x0F0F0F0Fu);
  q[1] = ((O12 & 0x0F0F0F0Fu) << 4) | (O34 & 0x0F0F0F0Fu);
  q[2] = (E12 & 0xF0F0F0F0u) | ((E34 >> 4) & 0x0F0F0F0Fu);
  q[3] = (O12 & 0xF0F0F0F0u) | ((O34 >> 4) & 0x0F0F0F0Fu);
}

// Buffer loads through a resource that spans one tile's rows (K R bytes from
// the tile's first row).  An offset at or past kNoRow lies outside every
// such resource (K <= 2^20 and R <= 2048, so a tile spans at most 2^31
// bytes), and the hardware returns zero for it without a memory access, so
// a plane word that must read as zero costs an issue slot and no cache
// traffic.  A lane's offset within a plane row (below 64 KB) may be added.
// (The 2-bit list kernels use plain global loads: buffer loads measured 3%
// slower on their launches of more than one workgroup per CU.)
constexpr uint32_t kNoRow = 0xFFFF0000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint8_t* tile, const Layer& L) {
  // the base is the same in every lane; taken from the first one so the
  // compiler keeps the resource in scalar registers (a value it cannot prove
  // uniform would put each load in a loop over the distinct values)
  const uint64_t p = (uint64_t)tile;
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(p >> 32));
  // word 3: 32-bit data format (a zero format would make every access
  // return zero), no swizzle, no stride
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0,
                                           (int)((uint32_t)L.K * (uint32_t)L.RB), 0x00020000);
}

// One dword of a plane row, streamed (non-temporal).
__device__ __forceinline__ uint32_t load_plane(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 2);
}

}  // namespace vmmdev
}  // namespace grinqh
