// The bfloat16 hi + lo split shared by the kernels that feed binary32 data
// to the 16-bit matrix cores as an unevaluated sum of two words.
#pragma once
#include "tcu_device.h"

namespace tcu {

// Two binary32 values as the high ("hi") and remainder ("lo") bfloat16
// words, packed two per 32-bit word: hi = v rounded to nearest even, lo =
// (v - hi) rounded again, so hi + lo is v to 2^-17 |v| or better, and
// exactly v when v has at most 16 significant bits.  The remainder v - hi is
// exact in binary32; it is formed straight from the packed hi word by the
// two-term bfloat16 dot product v_dot2_f32_bf16 (hi . (-1, 0) + v and
// hi . (0, -1) + v), one instruction per value instead of unpacking hi and
// subtracting.
//
// The two constant words are held in scalar registers (an opaque s_mov the
// compiler cannot fold): given the literal 0x0000bf80 it encodes the inline
// constant -1.0, which the instruction reads as the binary32 word
// 0xbf800000, i.e. (0, -1) instead of (-1, 0).
struct SplitConsts {
  unsigned neg_lo, neg_hi;   // bfloat16 pairs (-1, 0) and (0, -1)
};
__device__ __forceinline__ SplitConsts split_consts() {
  SplitConsts c;
  asm("s_mov_b32 %0, 0x0000bf80" : "=s"(c.neg_lo));
  asm("s_mov_b32 %0, 0xbf800000" : "=s"(c.neg_hi));
  return c;
}
__device__ __forceinline__ void split_bf16x2(float v0, float v1, unsigned &hi, unsigned &lo,
                                             SplitConsts c) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  hi = pack_bf16x2(v0, v1);
  const bf16x2 h = bitcast<bf16x2>(hi);
  const float l0 = __builtin_amdgcn_fdot2_f32_bf16(h, bitcast<bf16x2>(c.neg_lo), v0, false);
  const float l1 = __builtin_amdgcn_fdot2_f32_bf16(h, bitcast<bf16x2>(c.neg_hi), v1, false);
  lo = pack_bf16x2(l0, l1);
}

}  // namespace tcu
