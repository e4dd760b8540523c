// Device-side helpers shared by the tall-call and blocked-product kernels
// (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <type_traits>
#include <stdint.h>

#include "tcu.h"

namespace tcu {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Internal element-type code: int8 0/1 inputs, int8 0/1 output formed as
// old OR (sum > 0) -- the update X <- min(X + Y Z, 1) of the transitive
// closure's D function on 0/1 matrices.  Not part of the public tcu_dtype.
constexpr int TCU_I8_BOOL = 16;

// Input element size in bytes for a tcu_dtype.
__host__ __device__ constexpr int in_bytes(int dt) {
  return (dt == TCU_I8_I32 || dt == TCU_I8_BOOL) ? 1 : 2;
}
// Output element size in bytes for a tcu_dtype.
__host__ __device__ constexpr int out_bytes(int dt) {
  return dt == TCU_BF16_BF16 ? 2 : dt == TCU_I8_BOOL ? 1 : 4;
}

template <typename T, typename S>
__device__ __forceinline__ T bitcast(const S &s) {
  static_assert(sizeof(T) == sizeof(S), "bitcast size");
  return __builtin_bit_cast(T, s);
}

// ---------------------------------------------------------------- MFMA
// One 16x16 output block of the unit: D = W * X + D, where the lane layout
// of the 16-row operand W (here always the right matrix B, transposed: the
// unit's resident "weights"), of the 16-column operand X (rows of the tall
// left matrix) and of D is the CDNA matrix-core layout: lane l holds row
// (l % 16) of W and column (l % 16) of X over a contiguous run of the
// contracted index chosen by l / 16, and D rows 4*(l/16) .. 4*(l/16)+3 of
// column (l % 16).  K is 32 (16-bit inputs) or 64 (int8) per instruction.
__device__ __forceinline__ f32x4 mfma_k32(int dt, u32x4 w, u32x4 x, f32x4 d) {
  if (dt == TCU_F16_F32)
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(bitcast<f16x8>(w), bitcast<f16x8>(x), d, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(bitcast<bf16x8>(w), bitcast<bf16x8>(x), d, 0, 0, 0);
}

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

// 32 x 32 output blocks: K = 16 (16-bit inputs) or 32 (int8) per
// instruction, 16 bytes of operand per lane.  Lane l holds row (l % 32) of
// W and column (l % 32) of X over the contracted run selected by l / 32,
// and D rows 8*(j/4) + 4*(l/32) + (j%4), j = 0..15, of column (l % 32).
__device__ __forceinline__ f32x16 mfma32_k16(int dt, u32x4 w, u32x4 x, f32x16 d) {
  if (dt == TCU_F16_F32)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(bitcast<f16x8>(w), bitcast<f16x8>(x), d, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast<bf16x8>(w), bitcast<bf16x8>(x), d, 0, 0, 0);
}
__device__ __forceinline__ i32x16 mfma32_i8_k32(u32x4 w, u32x4 x, i32x16 d) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(bitcast<i32x4>(w), bitcast<i32x4>(x), d, 0, 0, 0);
}

__device__ __forceinline__ i32x4 mfma_i8_k64(u32x4 w, u32x4 x, i32x4 d) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(bitcast<i32x4>(w), bitcast<i32x4>(x), d, 0, 0, 0);
}

// Narrow forms: K = 16 for 16-bit inputs, K = 32 for int8 (8 bytes per lane).
__device__ __forceinline__ f32x4 mfma_k16(int dt, u32x2 w, u32x2 x, f32x4 d) {
  if (dt == TCU_F16_F32)
    return __builtin_amdgcn_mfma_f32_16x16x16f16(bitcast<f16x4>(w), bitcast<f16x4>(x), d, 0, 0, 0);
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(bitcast<i16x4>(w), bitcast<i16x4>(x), d, 0, 0, 0);
}

__device__ __forceinline__ i32x4 mfma_i8_k32(u32x2 w, u32x2 x, i32x4 d) {
  return __builtin_amdgcn_mfma_i32_16x16x32_i8(bitcast<long>(w), bitcast<long>(x), d, 0, 0, 0);
}

// ---------------------------------------------------------------- LDS
#define TCU_LDS(T, p) ((__attribute__((address_space(3))) T *)(p))

// Direct global -> LDS copy of 16 bytes per lane: lane l's bytes land at
// lds_base + 16*l (lds_base must be wave-uniform).
__device__ __forceinline__ void load_lds16(const void *gptr, void *lds_base) {
  __builtin_amdgcn_global_load_lds(gptr, TCU_LDS(void, lds_base), 16, 0, 0);
}

// LDS byte address of a __shared__ object.
__device__ __forceinline__ unsigned lds_addr(const void *p) {
  return (unsigned)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
}

// The same direct copy issued as an instruction the compiler cannot see
// into: it then inserts no waits of its own for it, so a multi-stage ring in
// one LDS array keeps its later stages in flight.  The caller orders it with
// explicit vmcnt waits and barriers.  lds_base: wave-uniform LDS address.
__device__ __forceinline__ void dma_lds16(const void *gptr, unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}

// The same with a wave-uniform 64-bit base and a per-lane 32-bit offset.
__device__ __forceinline__ void dma_lds16_saddr(const void *gbase, unsigned voff,
                                                unsigned lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(gbase), "s"(lds_base)
               : "memory", "m0");
}

// Transposing LDS reads (gfx950).  Within each group of 16 lanes, treat the
// 8-byte segments the lanes point at as rows of a 16 x 4 (16-bit) or 16 x 8
// (8-bit) matrix M.  ds_read_b64_tr_b16 returns to lane j the elements
// M[4e + j/4][j%4], e = 0..3; ds_read_b64_tr_b8 returns M[2e + j/8][j%8],
// e = 0..7.  So if lane s points at row k0 + s/4, columns c0 + 4(s%4) of a
// row-major 16-bit matrix, lane j receives column c0 + j, rows k0 .. k0+3
// (rows k0 .. k0+7 of column c0 + j for 8-bit, lane s pointing at row
// k0 + s/2, columns c0 + 8(s%2)).
__device__ __forceinline__ u32x2 lds_read_tr16(const void *p) {
  return bitcast<u32x2>(__builtin_amdgcn_ds_read_tr16_b64_v4i16(TCU_LDS(i16x4, p)));
}
__device__ __forceinline__ u32x2 lds_read_tr8(const void *p) {
  typedef int i32x2 __attribute__((ext_vector_type(2)));
  return bitcast<u32x2>(__builtin_amdgcn_ds_read_tr8_b64_v2i32(TCU_LDS(i32x2, p)));
}

// Two binary32 values -> two bfloat16 in one word (lo in bits 0-15), round
// to nearest even: one gfx950 v_cvt_pk_bf16_f32.
__device__ __forceinline__ unsigned pack_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return bitcast<unsigned>(__builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// bfloat16 bit pattern -> binary32 (exact).
__device__ __forceinline__ float bf16_to_f32(unsigned bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// One 16-byte chunk of EPC elements of ES bytes at p, of which the first
// `valid` (0..EPC) lie inside the matrix; the others are returned as zero
// (the zero padding of a partial strip or block) and are not read.  kVec:
// p is 16-byte aligned, so a full chunk is one vector load.
template <int ES, bool kVec>
__device__ __forceinline__ u32x4 load_chunk(const unsigned char *p, int valid) {
  constexpr int EPC = 16 / ES;
  if (kVec && valid >= EPC) return *(const u32x4 *)p;
  u32x4 v = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < EPC; ++e) {
    if (e < valid) {
      const unsigned x = ES == 2 ? (unsigned)((const unsigned short *)p)[e] : (unsigned)p[e];
      v[(e * ES) >> 2] |= x << (8 * ((e * ES) & 3));
    }
  }
  return v;
}

// One whole 16-byte chunk at p whose address is a multiple of kAl bytes (16,
// 8, 4, 2 or 1): one vector load, or 16 / kAl naturally aligned narrower
// loads.
template <int kAl>
__device__ __forceinline__ u32x4 load16(const unsigned char *p) {
  static_assert(kAl == 16 || kAl == 8 || kAl == 4 || kAl == 2 || kAl == 1,
                "chunk alignment 16, 8, 4, 2 or 1 bytes");
  if constexpr (kAl == 16) {
    return *(const u32x4 *)p;
  } else if constexpr (kAl == 8) {
    const u32x2 a = *(const u32x2 *)p, b = *(const u32x2 *)(p + 8);
    return u32x4{a[0], a[1], b[0], b[1]};
  } else if constexpr (kAl == 4) {
    const unsigned *q = (const unsigned *)p;
    return u32x4{q[0], q[1], q[2], q[3]};
  } else if constexpr (kAl == 2) {
    const unsigned short *q = (const unsigned short *)p;
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = (unsigned)q[2 * i] | ((unsigned)q[2 * i + 1] << 16);
    return v;
  } else {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      v[i] = (unsigned)p[4 * i] | ((unsigned)p[4 * i + 1] << 8) | ((unsigned)p[4 * i + 2] << 16) |
             ((unsigned)p[4 * i + 3] << 24);
    return v;
  }
}

// Store 4 consecutive output values of one row of C at p (element col of
// the row), of which the first `valid` (0..4) lie inside the matrix.  With
// acc the stored values are read and added first (binary32 or int32 sum,
// one rounding to the output type).  kVec: p is aligned for one vector
// access of the 4 values.
template <int DT, bool kVec, typename Acc>
__device__ __forceinline__ void store_out4(unsigned char *p, Acc v, int valid, bool acc) {
  if constexpr (DT == TCU_I8_BOOL) {
    // 0/1 output: old OR (sum > 0); the accumulate flag is implied.  OR is
    // idempotent, so with no new flag nothing is read or written, and an
    // unchanged word is not written back.
    if (kVec && valid >= 4) {
      unsigned f = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) f |= (unsigned)(v[e] > 0) << (8 * e);
      if (f == 0u) return;
      const unsigned old = *(const unsigned *)p;
      unsigned w = f;
#pragma unroll
      for (int e = 0; e < 4; ++e) w |= (unsigned)(((old >> (8 * e)) & 0xffu) != 0u) << (8 * e);
      if (w != old) *(unsigned *)p = w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < valid) p[e] = (unsigned char)((p[e] != 0) | (v[e] > 0));
    }
  } else if constexpr (DT == TCU_BF16_BF16) {
    unsigned short *q = (unsigned short *)p;
    if (kVec && valid >= 4) {
      if (acc) {
        const u32x2 o = *(const u32x2 *)p;
        v[0] += bf16_to_f32(o[0] & 0xffffu);
        v[1] += bf16_to_f32(o[0] >> 16);
        v[2] += bf16_to_f32(o[1] & 0xffffu);
        v[3] += bf16_to_f32(o[1] >> 16);
      }
      *(u32x2 *)p = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < valid) {
          float x = v[e];
          if (acc) x += bf16_to_f32(q[e]);
          q[e] = (unsigned short)(pack_bf16x2(x, 0.f) & 0xffffu);
        }
      }
    }
  } else {
    // int32 sums are formed as unsigned words: two's-complement wrap-around.
    constexpr bool kInt = (DT == TCU_I8_I32);
    if (kVec && valid >= 4) {
      u32x4 w = bitcast<u32x4>(v);
      if (acc) {
        const u32x4 o = *(const u32x4 *)p;
        if constexpr (kInt)
          w += o;
        else
          w = bitcast<u32x4>(bitcast<f32x4>(w) + bitcast<f32x4>(o));
      }
      *(u32x4 *)p = w;
    } else {
      unsigned *q = (unsigned *)p;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < valid) {
          unsigned w = bitcast<unsigned>(v[e]);
          if (acc) {
            if constexpr (kInt)
              w += q[e];
            else
              w = bitcast<unsigned>(bitcast<float>(w) + bitcast<float>(q[e]));
          }
          q[e] = w;
        }
      }
    }
  }
}

// The accumulating store in two steps, for 4 values of one row that lie
// inside the matrix at an aligned p: load_old4 reads the stored values'
// bits and store_sum4 adds the new values to them and stores the result
// (binary32 or int32 sum, one rounding to the output type), so that a wave
// can have the loads of several blocks in flight before the first sum.
template <int DT>
using Old4 = typename std::conditional<DT == TCU_BF16_BF16, u32x2, u32x4>::type;

template <int DT>
__device__ __forceinline__ Old4<DT> load_old4(const unsigned char *p) {
  return *(const Old4<DT> *)p;
}

template <int DT, typename Acc>
__device__ __forceinline__ void store_sum4(unsigned char *p, Acc v, Old4<DT> o) {
  static_assert(DT != TCU_I8_BOOL, "0/1 outputs are OR-ed, not added");
  if constexpr (DT == TCU_BF16_BF16) {
    v[0] += bf16_to_f32(o[0] & 0xffffu);
    v[1] += bf16_to_f32(o[0] >> 16);
    v[2] += bf16_to_f32(o[1] & 0xffffu);
    v[3] += bf16_to_f32(o[1] >> 16);
    *(u32x2 *)p = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
  } else if constexpr (DT == TCU_I8_I32) {
    *(u32x4 *)p = bitcast<u32x4>(v) + o;
  } else {
    *(u32x4 *)p = bitcast<u32x4>(bitcast<f32x4>(v) + bitcast<f32x4>(o));
  }
}

// Add 4 consecutive partial sums into C at p with device-scope atomic adds
// (binary32 or int32; split-K partial tiles).  Not for bfloat16 outputs,
// which must be rounded once from the whole sum.
template <int DT, typename Acc>
__device__ __forceinline__ void atomic_add_out4(unsigned char *p, Acc v) {
  static_assert(DT == TCU_F16_F32 || DT == TCU_BF16_F32 || DT == TCU_I8_I32,
                "only binary32 and int32 outputs are split");
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if constexpr (DT == TCU_I8_I32)
      __hip_atomic_fetch_add((int *)p + e, (int)v[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      __hip_atomic_fetch_add((float *)p + e, (float)v[e], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
  }
}

}  // namespace tcu
