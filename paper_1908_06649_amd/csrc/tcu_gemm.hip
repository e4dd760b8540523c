// Blocked dense multiplication of Theorem 2 (Section 4.1), fused into one
// launch: C (N x N) = A (N x N) * B (N x N) with unit size s.
//
// Theorem 2 cuts A into N x s vertical strips A_i and B into s x s blocks
// B_{i,j}, issues the (N/s)^2 tensor-unit calls C_{i,j} = A_i * B_{i,j} and
// sums output strip j over i.  Issued literally, every call would re-stream
// its N x s strip from memory, giving about s/2 flops per byte -- far below
// what the matrix cores need.  Here each workgroup owns one BM x BN output
// tile and walks the contracted index: for every strip i it performs the
// calls A_i[rows of the tile] * B_{i,j} for all column blocks j of the tile,
// accumulating sum_i in registers.  So every one of the (N/s)^2 calls is
// executed (restricted to the tile's rows, across the grid), no partial
// product C_{i,j} is ever written, and each staged slab of A_i is reused
// across all the tile's B_{i,j}.
//
// Data flow per K-step of 128 bytes (64 16-bit or 128 int8 elements):
//   HBM/L2 --(16-byte loads)--> registers --> LDS (double-buffered)
//   A rows are stored as they are (the contracted index is contiguous);
//   B is transposed on the way (in registers, with byte permutes) so that
//   LDS holds B^T rows -- the s x s blocks B_{i,j} in the layout the matrix
//   core takes as its resident row operand.  LDS rows are 128 bytes with the
//   16-byte chunks XOR-swizzled so that fragment reads and tile writes hit
//   distinct banks.
// Compute: 4 waves in a 2 x 2 arrangement, each owning a (BM/2) x (BN/2)
// sub-tile of 16 x 16 accumulator blocks, fed by 16x16x32 (16-bit) or
// 16x16x64 (int8) matrix-core instructions.  The product is formed as
// C^T = B^T A^T so each lane holds 4 consecutive columns of one row of C,
// stored as one 16-byte write.
// Workgroup order is XCD-aware: consecutive workgroup ids land on different
// XCDs, so ids are remapped to give each XCD a contiguous, grouped range of
// tiles that share A row-panels and B column-panels in its private L2.
#include "tcu_device.h"
#include "tcu_launch.h"

namespace tcu {
namespace {

constexpr int kBKB = 128;  // bytes of the contracted index per K-step and LDS row

__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row ^ (row >> 3)) & 7); }

// Map a workgroup id to an output tile (tm, tn).
__device__ __forceinline__ void map_tile(int pid, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int total = tiles_m * tiles_n;
  constexpr int kXcds = 8;
  if (total % kXcds == 0) pid = (pid % kXcds) * (total / kXcds) + pid / kXcds;
  constexpr int kGroupM = 8;
  const int per_group = kGroupM * tiles_n;
  const int group = pid / per_group;
  const int first_m = group * kGroupM;
  const int gsz = min(tiles_m - first_m, kGroupM);
  const int in_group = pid % per_group;
  tm = first_m + in_group % gsz;
  tn = in_group / gsz;
}

template <int DT, int BM, int BN, int WM, int WN>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(1, 1))) void
gemm_kernel(const unsigned char *__restrict__ A, const unsigned char *__restrict__ B,
            unsigned char *__restrict__ C, int N, int tiles_m, int tiles_n) {
  constexpr bool kI8 = (DT == TCU_I8_I32);
  constexpr int NT = 64 * WM * WN;
  constexpr int ES = in_bytes(DT);
  constexpr int BK = kBKB / ES;                // contracted elements per K-step
  constexpr int EPC = 16 / ES;                 // elements per 16-byte chunk
  constexpr int CA = BM * 8 / NT;              // A chunks per thread
  static_assert(CA * NT == BM * 8, "A tile must split evenly over threads");
  constexpr int NBW = BN * ES / 16;            // B 8-row blocks across the tile
  constexpr int NBLK = (BK / 8) * NBW;         // B 8-row x 16-byte blocks per K-step
  constexpr int CB = (NBLK + NT - 1) / NT;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave sub-tile
  constexpr int FM = WTM / 16, FN = WTN / 16;
  typedef typename std::conditional<kI8, i32x4, f32x4>::type Acc;

  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * (BM + BN) * kBKB];
  unsigned char *const As = smem;                  // [2][BM][128]
  unsigned char *const Bs = smem + 2 * BM * kBKB;  // [2][BN][128]  (B^T rows)

  int tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int64_t ld = (int64_t)N * ES;  // bytes per row of A and B

  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const int wm = wid / WN, wn = wid % WN;

  Acc acc[FN][FM];
#pragma unroll
  for (int a = 0; a < FN; ++a)
#pragma unroll
    for (int b = 0; b < FM; ++b) acc[a][b] = Acc{0, 0, 0, 0};

  u32x4 ra[CA];
  u32x4 rb[CB][8];
  const u32x4 zero = {0u, 0u, 0u, 0u};

  // ---- global -> registers for the K-step starting at element k0 ----
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int q = tid + NT * i;
      const int row = q >> 3, c = q & 7;
      const bool ok = (m0 + row < N) && (k0 + c * EPC < N);
      ra[i] = ok ? *(const u32x4 *)(A + (int64_t)(m0 + row) * ld + (int64_t)k0 * ES + c * 16) : zero;
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int q = tid + NT * i;
      const int nb = q % NBW, kb = q / NBW;
      const bool okn = (q < NBLK) && (n0 + nb * EPC < N);
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int k = k0 + 8 * kb + rr;
        rb[i][rr] = (okn && k < N)
                        ? *(const u32x4 *)(B + (int64_t)k * ld + (int64_t)n0 * ES + nb * 16)
                        : zero;
      }
    }
  };

  // ---- registers -> LDS buffer `buf` (B transposed on the way) ----
  auto sstore = [&](int buf) {
    unsigned char *as = As + buf * BM * kBKB;
    unsigned char *bs = Bs + buf * BN * kBKB;
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int q = tid + NT * i;
      const int row = q >> 3, c = q & 7;
      *(u32x4 *)(as + row * kBKB + swz(row, c) * 16) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int q = tid + NT * i;
      if (q >= NBLK) break;
      const int nb = q % NBW, kb = q / NBW;
      if constexpr (!kI8) {
        // 8 (k) x 8 (n) block of 16-bit values -> 8 rows of B^T, 16 bytes each
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const unsigned sel = (j & 1) ? 0x07060302u : 0x05040100u;
          u32x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[e] = __builtin_amdgcn_perm(rb[i][2 * e + 1][j >> 1], rb[i][2 * e][j >> 1], sel);
          const int row = 8 * nb + j;
          *(u32x4 *)(bs + row * kBKB + swz(row, kb) * 16) = o;
        }
      } else {
        // 8 (k) x 16 (n) block of bytes -> 16 rows of B^T, 8 bytes each
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          unsigned lo[4], hi[4];
#pragma unroll
          for (int p = 0; p < 4; ++p) {
            const unsigned x = rb[i][2 * p][d], y = rb[i][2 * p + 1][d];
            lo[p] = __builtin_amdgcn_perm(y, x, 0x05010400u);  // n = 4d, 4d+1
            hi[p] = __builtin_amdgcn_perm(y, x, 0x07030602u);  // n = 4d+2, 4d+3
          }
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const unsigned *src = (t < 2) ? lo : hi;
            const unsigned sel = (t & 1) ? 0x07060302u : 0x05040100u;
            u32x2 o = {__builtin_amdgcn_perm(src[1], src[0], sel),
                       __builtin_amdgcn_perm(src[3], src[2], sel)};
            const int row = 16 * nb + 4 * d + t;
            *(u32x2 *)(bs + row * kBKB + swz(row, kb >> 1) * 16 + (kb & 1) * 8) = o;
          }
        }
      }
    }
  };

  // ---- matrix-core work on LDS buffer `buf` ----
  auto compute = [&](int buf) {
    const unsigned char *as = As + buf * BM * kBKB;
    const unsigned char *bs = Bs + buf * BN * kBKB;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      u32x4 xf[FM];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        const int row = wm * WTM + 16 * fm + r;
        xf[fm] = *(const u32x4 *)(as + row * kBKB + swz(row, kk * 4 + g) * 16);
      }
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int row = wn * WTN + 16 * fn + r;
        const u32x4 wf = *(const u32x4 *)(bs + row * kBKB + swz(row, kk * 4 + g) * 16);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          if constexpr (kI8)
            acc[fn][fm] = mfma_i8_k64(wf, xf[fm], acc[fn][fm]);
          else
            acc[fn][fm] = mfma_k32(DT, wf, xf[fm], acc[fn][fm]);
        }
      }
    }
  };

  const int nk = (N + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    compute(cur);
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds C[row][col .. col+3] of every accumulator block ----
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = m0 + wm * WTM + 16 * fm + r;
      const int col = n0 + wn * WTN + 16 * fn + 4 * g;
      if (row < N && col < N) {
        if constexpr (DT == TCU_BF16_BF16) {
          const f32x4 v = acc[fn][fm];
          *(u32x2 *)(C + ((int64_t)row * N + col) * 2) =
              u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        } else {
          *(u32x4 *)(C + ((int64_t)row * N + col) * 4) = bitcast<u32x4>(acc[fn][fm]);
        }
      }
    }
  }
}

template <int DT, int BM, int BN, int WM, int WN>
hipError_t launch_cfg(const void *A, const void *B, void *C, int64_t N, hipStream_t stream) {
  const int tiles_m = (int)((N + BM - 1) / BM), tiles_n = (int)((N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<DT, BM, BN, WM, WN>), dim3(tiles_m * tiles_n), dim3(64 * WM * WN),
                     0, stream, (const unsigned char *)A, (const unsigned char *)B,
                     (unsigned char *)C, (int)N, tiles_m, tiles_n);
  return hipGetLastError();
}

template <int DT>
hipError_t launch_dt(const void *A, const void *B, void *C, int64_t N, hipStream_t stream,
                     int num_cus) {
  // Big tiles when they fill the chip; otherwise smaller tiles for more workgroups.
  const int64_t big_tiles = ((N + 255) / 256) * ((N + 255) / 256);
  if (big_tiles >= num_cus) return launch_cfg<DT, 256, 256, 2, 2>(A, B, C, N, stream);
  return launch_cfg<DT, 128, 128, 2, 2>(A, B, C, N, stream);
}

}  // namespace

hipError_t launch_gemm(int dtype, const void *A, const void *B, void *C, int64_t N,
                       hipStream_t stream, int num_cus) {
  switch (dtype) {
    case TCU_F16_F32: return launch_dt<TCU_F16_F32>(A, B, C, N, stream, num_cus);
    case TCU_BF16_F32: return launch_dt<TCU_BF16_F32>(A, B, C, N, stream, num_cus);
    case TCU_BF16_BF16: return launch_dt<TCU_BF16_BF16>(A, B, C, N, stream, num_cus);
    case TCU_I8_I32: return launch_dt<TCU_I8_I32>(A, B, C, N, stream, num_cus);
  }
  return hipErrorInvalidValue;
}

}  // namespace tcu
