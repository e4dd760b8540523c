// Closure of a diagonal block of the transitive closure (Section 4.3,
// function A on a 256-vertex pivot band), as a workgroup-wide device
// function: the standalone one-workgroup kernel (1024 threads) and the
// full-tile product kernel's 0/1 instance (512 threads, which closes the
// next band's block right after updating it) share it.
#pragma once

#include "tcu_device.h"

namespace tcu {

constexpr int kDiagBand = 256;                  // vertices per pivot band
constexpr int kDiagWords = kDiagBand / 32;      // 32-bit words per row
constexpr int kTab2Pitch = 8 * 16 + 8;

// 4 bytes holding 0/1 -> 4 bits, and back.
__device__ __forceinline__ unsigned bytes_to_bits4(unsigned x) {
  return (x & 1u) | ((x >> 7) & 2u) | ((x >> 14) & 4u) | ((x >> 21) & 8u);
}
__device__ __forceinline__ unsigned bits4_to_bytes(unsigned b) {
  return (b & 1u) | ((b & 2u) << 7) | ((b & 4u) << 14) | ((b & 8u) << 21);
}

// Value of lane h (wave-uniform) of each group of kTPR consecutive lanes
// (kTPR 2 or 4; DPP quad permutations).
template <int kTPR>
__device__ __forceinline__ unsigned group_broadcast(unsigned v, int h) {
  if constexpr (kTPR == 4) {
    switch (h) {
      case 0: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x00, 0xf, 0xf, false);
      case 1: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0x55, 0xf, 0xf, false);
      case 2: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xaa, 0xf, 0xf, false);
      default: return (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xff, 0xf, 0xf, false);
    }
  } else {
    static_assert(kTPR == 2, "2 or 4 threads per row");
    // quad_perm [0, 0, 2, 2] or [1, 1, 3, 3]
    return h == 0 ? (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xa0, 0xf, 0xf, false)
                  : (unsigned)__builtin_amdgcn_update_dpp(0, (int)v, 0xf5, 0xf, 0xf, false);
  }
}

// LDS of one diagonal closure.
struct DiagShared {
  unsigned krow[32][kDiagWords];                 // the sub-band's published pivot rows
  unsigned tab1[8 * 16];                         // [group][subset]
  unsigned tab2[kDiagWords * kTab2Pitch];        // [word][group][subset]
};

// Close the Bk x Bk diagonal block at D (row pitch ld; entries already 0/1),
// Bk <= 256, with the kThreads threads of the workgroup (512 or 1024; every
// thread must call it: it synchronises the workgroup).  Row i is held as 8
// words of bits by the kThreads / 256 threads of row i (8 / that many words
// each).  The pivots are taken in sub-bands K of 32; for each:
//   * the pivots' current rows are published to LDS;
//   * one wave closes the 32 x 32 block of K's rows and columns (the
//     iterative algorithm on 32 one-word rows, the pivot row broadcast with
//     readlane), giving T*[k]: the pivots reachable from pivot k through K,
//     k included;
//   * every row i (pivot or not) forms R_i, the union of T*[k] over the
//     pivots k it has an edge to, and ORs in the published rows of R_i.
// That is the iterative algorithm's 32 steps over K: a vertex reaches v
// through K exactly when some pivot it reaches through K has an edge to v.
// Both unions over a 32-bit set are taken 4 bits at a time from tables of
// all 16 unions of 4 consecutive pivots' words (8 lookups instead of 32
// masked terms): tab1 over T*, tab2 over each word of the published rows.
// Regions of tab2 kTab2Pitch = 136 words apart start 8 banks further on per
// word, so the lookups of the words a wave touches at once fall on distinct
// bank windows (16 subsets of one region lie in 16 distinct banks).
template <bool kVec, int kThreads>
__device__ __forceinline__ void close_diag_block(unsigned char *D, int64_t ld, int Bk,
                                                 DiagShared &s) {
  constexpr int kTPR = kThreads / kDiagBand;     // threads per row
  constexpr int kWPT = kDiagWords / kTPR;        // words per thread
  const int t = threadIdx.x;
  const int i = t / kTPR;                        // row
  const int w0 = kWPT * (t % kTPR);              // this thread's words w0 .. w0 + kWPT - 1
  unsigned row[kWPT];
  // bytes -> bits (bit b of word w = column 32w + b)
  const unsigned char *src = D + (int64_t)i * ld;
#pragma unroll
  for (int q = 0; q < kWPT; ++q) {
    const int w = w0 + q;
    unsigned word = 0;
    if (i < Bk) {
      if (kVec && 32 * w + 32 <= Bk) {
        const u32x4 a = *(const u32x4 *)(src + 32 * w);
        const u32x4 b = *(const u32x4 *)(src + 32 * w + 16);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          word |= bytes_to_bits4(a[c]) << (4 * c);
          word |= bytes_to_bits4(b[c]) << (16 + 4 * c);
        }
      } else {
        for (int b = 0; b < 32; ++b)
          if (32 * w + b < Bk && src[32 * w + b]) word |= 1u << b;
      }
    }
    row[q] = word;
  }
#pragma unroll
  for (int sb = 0; sb < kDiagWords; ++sb) {
    if (32 * sb >= Bk) break;
    const int nk = Bk - 32 * sb < 32 ? Bk - 32 * sb : 32;   // pivots in this sub-band
    const unsigned kmask = nk == 32 ? ~0u : (1u << nk) - 1u;
    if (i >= 32 * sb && i < 32 * sb + 32) {
#pragma unroll
      for (int q = 0; q < kWPT; ++q) s.krow[i - 32 * sb][w0 + q] = row[q];
    }
    __syncthreads();
    // (Pivots past nk have zero rows and no bits in kmask: they add nothing.)
    if (t < 64) {
      // wave 0: lanes 0..31 close the pivot block; then tab1 from T*.
      unsigned tk = t < 32 ? s.krow[t][sb] & kmask : 0u;
#pragma unroll
      for (int kk = 0; kk < 32; ++kk) {
        const unsigned pivot = (unsigned)__builtin_amdgcn_readlane((int)tk, kk);
        tk |= pivot & (0u - ((tk >> kk) & 1u));
      }
      const unsigned tstar = t < 32 ? (tk | (1u << t)) : 0u;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int e = t + 64 * h, grp = e >> 4, m = e & 15;
        unsigned v = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const unsigned x = (unsigned)__shfl((int)tstar, 4 * grp + b, 64);
          v |= x & (0u - ((unsigned)(m >> b) & 1u));
        }
        s.tab1[e] = v;
      }
    }
    // tab2[w][grp][m] = union of word w of the published rows 4 grp + b, b in m
#pragma unroll
    for (int e0 = 0; e0 < kDiagWords * 128; e0 += kThreads) {
      const int e = e0 + t;
      const int w = e >> 7, grp = (e >> 4) & 7, m = e & 15;
      unsigned v = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) v |= s.krow[4 * grp + b][w] & (0u - ((unsigned)(m >> b) & 1u));
      s.tab2[w * kTab2Pitch + (e & 127)] = v;
    }
    __syncthreads();
    // word sb of row i, from the thread of the row that holds it
    const unsigned wsb = group_broadcast<kTPR>(row[sb % kWPT], sb / kWPT);
    const unsigned edges = wsb & kmask;
    unsigned reach = 0;
#pragma unroll
    for (int grp = 0; grp < 8; ++grp) reach |= s.tab1[16 * grp + ((edges >> (4 * grp)) & 15u)];
    reach &= kmask;
#pragma unroll
    for (int q = 0; q < kWPT; ++q) {
      const unsigned *t2 = s.tab2 + kTab2Pitch * (w0 + q);
      unsigned add = 0;
#pragma unroll
      for (int grp = 0; grp < 8; ++grp) add |= t2[16 * grp + ((reach >> (4 * grp)) & 15u)];
      row[q] |= add;
    }
    __syncthreads();   // krow and the tables are rewritten by the next sub-band
  }
  // bits -> bytes
  if (i < Bk) {
    unsigned char *dst = D + (int64_t)i * ld;
#pragma unroll
    for (int q = 0; q < kWPT; ++q) {
      const int w = w0 + q;
      if (kVec && 32 * w + 32 <= Bk) {
        u32x4 a, b;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          a[c] = bits4_to_bytes(row[q] >> (4 * c));
          b[c] = bits4_to_bytes(row[q] >> (16 + 4 * c));
        }
        *(u32x4 *)(dst + 32 * w) = a;
        *(u32x4 *)(dst + 32 * w + 16) = b;
      } else {
        for (int b = 0; b < 32; ++b)
          if (32 * w + b < Bk) dst[32 * w + b] = (unsigned char)((row[q] >> b) & 1u);
      }
    }
  }
}

}  // namespace tcu
