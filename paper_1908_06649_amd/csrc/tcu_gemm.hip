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
// Workgroup order is XCD-aware (see map_tile).
#include "tcu_device.h"
#include "tcu_launch.h"
#include "tcu_tc_diag.h"

namespace tcu {
namespace {

// Tile rows per group of the tile order (map_tile) and LDS ring depth of
// the full-tile kernel, both measured best on the order-8192 products.
constexpr int kGroupM = 2;
constexpr int kRingStages = 5;

constexpr int kBKB = 128;  // bytes of the contracted index per K-step and LDS row


__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row ^ (row >> 3)) & 7); }

// Map a workgroup id to an output tile (tm, tn): groups of kGroupM tile
// rows are walked column by column.  Consecutive workgroup ids are dispatched
// round-robin over the 8 XCDs, so with groups of 2 rows each XCD's concurrent
// workgroups cover a compact block of tiles (shared A row-panels and B
// column-panels in its L2) while all XCDs together sweep a band of full rows
// (B panels shared through the memory-side cache).  Measured best for N=8192
// against larger groups and an explicit per-XCD remap of the ids.
__device__ __forceinline__ void map_tile(int pid, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int per_group = kGroupM * tiles_n;
  const int group = pid / per_group;
  const int first_m = group * kGroupM;
  const int gsz = min(tiles_m - first_m, kGroupM);
  const int in_group = pid % per_group;
  tm = first_m + in_group % gsz;
  tn = in_group / gsz;
}

// C (M x N) = A (M x K) * B (K x N) [+ C when accum], operands with row
// pitches lda, ldb, ldc (elements).  Rows, columns and contracted indices
// beyond M, N, K are zero padding: chunks reaching past an edge are loaded
// element by element with zeros in place of the missing elements, and only
// in-range outputs are stored.  kVec: every pitch is a multiple of 16 bytes
// (full chunks are vector loads, 4-value groups of C vector accesses).
// Otherwise kAl > 0: A's and B's pitches are multiples of kAl (8, 4, 2 or 1)
// bytes, and the whole chunks of interior tiles are loaded as 16 / kAl
// naturally aligned pieces; kAl = 0: every chunk element by element.
template <int DT, int BM, int BN, int WM, int WN, bool kVec, int kAl = 0>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(1, 1))) void
gemm_kernel(const unsigned char *__restrict__ A, const unsigned char *__restrict__ B,
            unsigned char *__restrict__ C, int M, int N, int K, int64_t lda, int64_t ldb,
            int64_t ldc, int accum, int tiles_m, int tiles_n, int band_tm, int skip_m,
            int band_tn, int skip_n) {
  constexpr bool kI8 = (in_bytes(DT) == 1);
  constexpr int NT = 64 * WM * WN;
  constexpr int ES = in_bytes(DT);
  constexpr int OB = out_bytes(DT);
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
  // Tile rows from band_tm on (columns from band_tn on) start skip_m
  // (skip_n) further: the tiles then step over a band of the output that
  // another launch owns (the transitive closure's pivot block row/column).
  const int m0 = tm * BM + (tm >= band_tm ? skip_m : 0);
  const int n0 = tn * BN + (tn >= band_tn ? skip_n : 0);
  const int64_t lda_b = lda * ES, ldb_b = ldb * ES, ldc_b = ldc * OB;  // row pitches in bytes

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

  // ---- global -> registers for the K-step starting at element k0 ----
  // Whole tile inside M x N: only the last K-step can reach past K, and
  // only when K is not a multiple of the step.  Interior steps load whole
  // chunks with no per-element checks.
  constexpr int kLd = kVec ? 16 : kAl;         // alignment of whole-chunk loads
  const bool inside = m0 + BM <= M && n0 + BN <= N;
  const bool interior = kLd > 0 && inside;
  auto gload_full = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int q = tid + NT * i;
      const int row = m0 + (q >> 3), kc = k0 + (q & 7) * EPC;
      ra[i] = load16<kLd ? kLd : 16>(A + (int64_t)row * lda_b + (int64_t)kc * ES);
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int q = tid + NT * i;
      if (CB * NT > NBLK && q >= NBLK) break;
      const int nb = q % NBW, kb = q / NBW;
      const int nc = n0 + nb * EPC;
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int k = k0 + 8 * kb + rr;
        rb[i][rr] = load16<kLd ? kLd : 16>(B + (int64_t)k * ldb_b + (int64_t)nc * ES);
      }
    }
  };
  auto gload_edge = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int q = tid + NT * i;
      const int row = m0 + (q >> 3), kc = k0 + (q & 7) * EPC;
      const int valid = row < M ? min(max(K - kc, 0), EPC) : 0;
      ra[i] = load_chunk<ES, kVec>(A + (int64_t)row * lda_b + (int64_t)kc * ES, valid);
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int q = tid + NT * i;
      const int nb = q % NBW, kb = q / NBW;
      const int nc = n0 + nb * EPC;
      const int nvalid = q < NBLK ? min(max(N - nc, 0), EPC) : 0;
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const int k = k0 + 8 * kb + rr;
        rb[i][rr] = load_chunk<ES, kVec>(B + (int64_t)k * ldb_b + (int64_t)nc * ES,
                                         k < K ? nvalid : 0);
      }
    }
  };
  auto gload = [&](int k0) __attribute__((always_inline)) {
    if (interior && k0 + BK <= K)
      gload_full(k0);
    else
      gload_edge(k0);
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

  const int nk = (K + BK - 1) / BK;
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
      unsigned char *p = C + (int64_t)row * ldc_b + (int64_t)col * OB;
      if (kVec && inside) {
        store_out4<DT, true>(p, acc[fn][fm], 4, accum != 0);
      } else {
        const int valid = row < M ? min(max(N - col, 0), 4) : 0;
        if (valid > 0) store_out4<DT, kVec>(p, acc[fn][fm], valid, accum != 0);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Full-tile kernel (M, N multiples of 256, K a multiple of one stage):
// 256 x 256 output tiles, a persistent grid of one workgroup per CU walking
// the tiles, and a ring of LDS stages, each holding 64 bytes of the
// contracted index (32 16-bit or 64 int8 values: one matrix-core K step, and
// one or two strips A_i of the unit).
//   * Both operands go HBM/L2 -> LDS with direct 16-byte DMA loads
//     (global_load_lds_dwordx4): no register staging, no VALU work.
//   * A stage of A is 256 rows x 64 bytes, kept as 1 KiB blocks of 16 rows
//     stored chunk-major (the DMA lane -> row/chunk assignment does this for
//     free), so every fragment read is a linear ds_read_b128, the access
//     pattern LDS serves at full rate.
//   * A stage of B is kept row-major as it is in memory (k rows of 256
//     columns); the weights operand (B^T) is formed by transposing LDS
//     reads (ds_read_b64_tr_b16 / _tr_b8), chunks XOR-swizzled per row so
//     the 16 lanes of a read group hit distinct banks.
//   * The DMA is issued through an instruction the compiler cannot see
//     into, so it adds no conservative waits; the kernel orders it with
//     explicit vmcnt waits and fence-free barriers.
// ---------------------------------------------------------------------------
constexpr int kFastKB = 64;                     // bytes of K per stage
constexpr int kFastStage = 256 * kFastKB;       // 16 KiB per operand per stage

// B stage, 16-bit: 512-byte rows (32 chunks).
__device__ __forceinline__ int fb16_swz(int k) { return ((k & 3) << 1) | (((k >> 3) & 3) << 3); }
// B stage, int8: 256-byte rows (16 chunks).
__device__ __forceinline__ int fb8_swz(int k) { return (k & 7) | (((k >> 4) & 1) << 3); }

// ---------------------------------------------------------------------------
// The full-tile kernel runs 8 waves, two per SIMD, in two groups.  Group 0 (waves 0-3) owns rows 0-127 of the 256 x 256 tile, group 1
// (waves 4-7) rows 128-255; wave q of a group owns columns 64q .. 64q+63.
// Each K stage is two phases separated by barriers:
//   phase A(t): group 0 runs its matrix-core work of stage t while group 1
//               reads its fragments of stage t and issues DMA loads;
//   phase B(t): group 1 runs its matrix-core work of stage t while group 0
//               reads its fragments of stage t+1 and issues DMA loads.
// The fragment reads go first: they are the phase's critical path (LDS
// reads of four waves take about as long as the 32 products), and queued
// behind the DMA instructions they started later (measured 1.5 % slower).
// A wave stalled on memory (full load queues, late data) therefore never
// idles its SIMD's matrix core: the other wave on that SIMD is computing,
// with raised issue priority.  Group 0 loads the A part of every stage and
// group 1 the B part (4 DMA instructions per wave per stage).
// Ring bookkeeping: the slot of stage t has been read by group 0 (in
// B(t-1)) and by group 1 (in A(t)) once A(t) ends, so it is refilled with
// stage t+kRing in B(t) (A part, group 0) and A(t+1) (B part, group 1).
// Stage t+1 must be complete when A(t) ends, so every wave waits there for
// its own loads of stage t+1 before the barrier.
// ---------------------------------------------------------------------------
// Wait until at most n of this wave's DMA loads are in flight and all its
// LDS reads have returned, then a workgroup barrier.  The barrier is an
// instruction with a memory clobber: the compiler may not move LDS accesses
// across it (the barrier intrinsic alone does not order memory), while no
// memory fence -- which would drain every in-flight DMA -- is emitted.
template <int n>
__device__ __forceinline__ void vm_wait_barrier() {
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (0 << 8) | (((n >> 4) & 3) << 14));
  asm volatile("s_barrier" ::: "memory");
}

// kEdge: C's edge may cut through tiles and K may end inside a stage (the
// ragged shapes); without it every tile and stage is whole.
template <int DT, int kRing, bool kEdge>
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2))) void
gemm_pp_kernel(const unsigned char *__restrict__ A, const unsigned char *__restrict__ B,
               unsigned char *__restrict__ C, int K, int64_t lda, int64_t ldb, int64_t ldc,
               int accum, int tiles_m, int tiles_n, int full, int nsplit, int m_lim,
               int n_lim, TileRemap remap, int diag_pid) {
  constexpr bool kI8 = (in_bytes(DT) == 1);
  constexpr int ES = in_bytes(DT);
  constexpr int OB = out_bytes(DT);
  constexpr int KE = kFastKB / ES;     // contracted elements per stage
  constexpr int BROW = 256 * ES;       // bytes per B row in a stage
  constexpr int FM = 8, FN = 4;        // 16 x 16 blocks per wave (128 x 64)
  constexpr int kDma = 4;              // DMA instructions per wave per stage
  static_assert(kRing - 2 <= 3, "waits cover at most 3 later stages");
  typedef typename std::conditional<kI8, i32x4, f32x4>::type Acc;

  // The ring (A and B parts), then, for 0/1 outputs, the epilogue's 256 x
  // 256 flag tile in LDS of its own, so that the next tile's first stages
  // can be loaded into the ring while the epilogue runs.
  constexpr int kFlagBytes = DT == TCU_I8_BOOL ? 256 * 256 : 0;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * kRing * kFastStage + kFlagBytes];
  unsigned char *const sA = smem;
  unsigned char *const sB = smem + kRing * kFastStage;
  unsigned char *const sF = sB + kRing * kFastStage;

  // Work items: the first `full` tiles (in map_tile order) whole, then the
  // other tiles as (K slice, tile) pairs, slice-major so that the workgroups
  // running at one time share the K range of their A and B panels.  With
  // nsplit > 1 such an item sums one contiguous range of whole stages
  // (about nk_all / nsplit strips A_i of the unit) and adds its partial
  // tile into C atomically.  full = 0 splits every tile; full = tiles (or
  // nsplit = 1) none.
  const int tiles = tiles_m * tiles_n;
  const int tail_tiles = tiles - full;
  const int total = full + tail_tiles * nsplit;
  // Stages of the contracted index; when K is not a whole number of stages
  // the last one holds k_tail < KE elements and is loaded element-wise with
  // zeros past K (the zero padding of a ragged dimension).
  const int nk_all = kEdge ? (K + KE - 1) / KE : K / KE;
  const int k_tail = K - (nk_all - 1) * KE;
  const int64_t lda_b = lda * ES, ldb_b = ldb * ES, ldc_b = ldc * OB;
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int grp = wid >> 2, q = wid & 3;
  const int r = lane & 15, g = lane >> 4;
  // With diag_pid >= 0 (the closure's D update, which also closes the next
  // pivot band's diagonal block -- a tile of this launch): workgroup 0 takes
  // that tile alone and then closes the block (close_diag_block, 512
  // threads) while the others share the remaining tiles, skipping it.
  const bool with_diag = DT == TCU_I8_BOOL && diag_pid >= 0;
  const int stride = with_diag ? (int)gridDim.x - 1 : (int)gridDim.x;
  const int limit = with_diag ? total - 1 : total;
  int item = with_diag ? (int)blockIdx.x - 1 : (int)blockIdx.x;   // -1: the diagonal tile
  int m0, n0, nk;
  int tail_t = -1;   // item-relative index of a partial last stage, if the item holds it
  // This wave's DMA share of a stage: group 0 -> A blocks 4q..4q+3 (16 rows
  // each, stored chunk-major), group 1 -> B blocks 4q..4q+3 (1 KiB each).
  // Wave-uniform 64-bit base + per-lane 32-bit offsets (saddr form).
  const unsigned char *gbase;
  unsigned voff[kDma];
  // Per-lane offsets.  In a tile that crosses the edge of C (rows >= m_lim
  // or columns >= n_lim) a lane past the edge loads the last row of A, or
  // the last 16-byte chunk of B's row, inside it instead: every load stays
  // in the operands, every DMA instruction is issued (the wait counts rely
  // on it), and the products it feeds are never stored.
  auto set_voff = [&]() {
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int blk = q * 4 + i;
      if (grp == 0) {
        int row = blk * 16 + (lane & 15);
        if (kEdge && m0 + row >= m_lim) row = m_lim - 1 - m0;
        voff[i] = (unsigned)(row * lda_b) + 16u * (lane >> 4);
      } else {
        int krow, c;
        if constexpr (!kI8) {
          krow = blk * 2 + (lane >> 5);
          c = (lane & 31) ^ fb16_swz(krow);
        } else {
          krow = blk * 4 + (lane >> 4);
          c = (lane & 15) ^ fb8_swz(krow);
        }
        if constexpr (kEdge) {
          const int c_last = (n_lim - n0) * ES / 16 - 1;
          if (c > c_last) c = c_last;
        }
        voff[i] = (unsigned)(krow * ldb_b) + 16u * c;
      }
    }
  };
  // Split items are few and long, and consecutive workgroup ids go
  // round-robin to the 8 XCDs: their ids are permuted so that each XCD
  // holds a contiguous run of them (one K range, a compact block of tiles),
  // and its concurrent workgroups share their A and B panels in its own L2
  // (measured: 2048 x 65536 x 2048 int8, split 4, 0.261 -> 0.235 ms).  The
  // items past the last multiple of 8 keep their ids.
  const int split_items = nsplit > 1 ? total - full : 0;
  const int xcd_body = split_items - split_items % 8;
  bool split_item = false;   // the current item is a K slice (atomic epilogue)
  auto place = [&](int w) {
    int pid = w, slice = 0;
    if (with_diag) pid = w < 0 ? diag_pid : (w < diag_pid ? w : w + 1);
    split_item = nsplit > 1 && w >= full;
    if (split_item) {
      int v = w - full;
      if (v < xcd_body) v = (v % 8) * (xcd_body / 8) + v / 8;
      slice = v / tail_tiles;
      pid = full + (v - slice * tail_tiles);
    }
    int tm, tn;
    map_tile(pid, tiles_m, tiles_n, tm, tn);
    m0 = remap.m_base + tm * 256 + (tm >= remap.band_m ? remap.skip_m : 0);
    n0 = remap.n_base + tn * 256 + (tn >= remap.band_n ? remap.skip_n : 0);
    const int s_begin = split_item ? (int)((int64_t)nk_all * slice / nsplit) : 0;
    nk = split_item ? (int)((int64_t)nk_all * (slice + 1) / nsplit) - s_begin : nk_all;
    if constexpr (kEdge) tail_t = (k_tail < KE && s_begin + nk == nk_all) ? nk - 1 : -1;
    gbase = grp == 0 ? A + (int64_t)m0 * lda_b + (int64_t)s_begin * kFastKB
                     : B + (int64_t)n0 * ES + (int64_t)s_begin * KE * ldb_b;
    if constexpr (kEdge) set_voff();
  };
  place(item);
  if constexpr (!kEdge) set_voff();    // the same for every tile
  const int64_t gstep = grp == 0 ? (int64_t)kFastKB : (int64_t)KE * ldb_b;
  const unsigned lds0 = (grp == 0 ? lds_addr(sA) : lds_addr(sB)) + q * 4 * 1024;
  // The partial last stage: the same 16 bytes per lane into the same LDS
  // bytes as the DMA would write (lane L of instruction i at 1024 i + 16 L),
  // read with ordinary loads that skip every element past K -- A's columns
  // beyond K (the next row, or past the array) and B's rows beyond K -- and
  // write zeros there.  A wave may take any number of these loads (none when
  // its part lies wholly past K), so the issue ends by waiting for every
  // load of the wave: afterwards no load of this or an older stage is in
  // flight, and the stage waits below (which count kDma loads per later
  // stage in flight) hold trivially until the next tile's stages.
  auto issue_tail = [&](int slot_, int t) {
    const unsigned char *base = gbase + (int64_t)t * gstep;
    unsigned char *dst = (grp == 0 ? sA : sB) + q * 4 * 1024 + slot_ * kFastStage;
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int blk = q * 4 + i;
      u32x4 v = {0u, 0u, 0u, 0u};
      const unsigned char *src = base + voff[i];
      if (grp == 0) {
        const int valid = k_tail - (lane >> 4) * (16 / ES);   // elements of this chunk in K
        if (valid >= 16 / ES) {
          v = *(const u32x4 *)src;
        } else if (valid > 0) {
          unsigned w[4] = {0u, 0u, 0u, 0u};
          for (int e = 0; e < valid; ++e) {
            const unsigned x = ES == 2 ? (unsigned)((const unsigned short *)src)[e]
                                       : (unsigned)src[e];
            w[(e * ES) >> 2] |= x << (8 * ((e * ES) & 3));
          }
          v = u32x4{w[0], w[1], w[2], w[3]};
        }
      } else {
        const int krow = kI8 ? blk * 4 + (lane >> 4) : blk * 2 + (lane >> 5);
        if (krow < k_tail) v = *(const u32x4 *)src;
      }
      *(u32x4 *)(dst + i * 1024 + 16 * lane) = v;
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  };
  auto issue = [&](int slot_, int t) {
    if constexpr (kEdge) {
      if (t == tail_t) {
        issue_tail(slot_, t);
        return;
      }
    }
    const unsigned char *base = gbase + (int64_t)t * gstep;
#pragma unroll
    for (int i = 0; i < kDma; ++i) dma_lds16_saddr(base, voff[i], lds0 + slot_ * kFastStage + i * 1024);
  };

  // Fragment offsets (stage 0): rows 128*grp.. of A, columns 64q.. of B^T.
  const int x_off = grp * 8 * 1024 + 16 * lane;
  int w_off[FN];
#pragma unroll
  for (int fn = 0; fn < FN; ++fn) {
    const int nbase = q * 64 + fn * 16;
    if constexpr (!kI8) {
      const int n = nbase + 4 * (r & 3);
      const int k0 = 8 * g + (r >> 2);
      w_off[fn] = k0 * BROW + 16 * ((n >> 3) ^ fb16_swz(k0)) + ((2 * n) & 15);
    } else {
      const int n = nbase + 8 * (r & 1);
      const int k0 = 16 * g + (r >> 1);
      w_off[fn] = k0 * BROW + 16 * ((n >> 4) ^ fb8_swz(k0)) + (n & 15);
    }
  }
  constexpr int kW1 = (kI8 ? 8 : 4) * BROW;

  Acc acc[FN][FM];
  u32x4 xf[FM], wf[FN];
  auto read_frags = [&](int slot_) {
    const unsigned char *sa = sA + slot_ * kFastStage;
    const unsigned char *sb = sB + slot_ * kFastStage;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) xf[fm] = *(const u32x4 *)(sa + x_off + fm * 1024);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      u32x2 w0, w1;
      if constexpr (!kI8) {
        w0 = lds_read_tr16(sb + w_off[fn]);
        w1 = lds_read_tr16(sb + w_off[fn] + kW1);
      } else {
        w0 = lds_read_tr8(sb + w_off[fn]);
        w1 = lds_read_tr8(sb + w_off[fn] + kW1);
      }
      wf[fn] = u32x4{w0[0], w0[1], w1[0], w1[1]};
    }
  };
  auto mfmas = [&]() {
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        if constexpr (kI8)
          acc[fn][fm] = mfma_i8_k64(wf[fn], xf[fm], acc[fn][fm]);
        else
          acc[fn][fm] = mfma_k32(DT, wf[fn], xf[fm], acc[fn][fm]);
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };
  auto next_slot = [](int s0) { return s0 + 1 == kRing ? 0 : s0 + 1; };
  auto prev_slot = [](int s0) { return s0 == 0 ? kRing - 1 : s0 - 1; };
  // Wait until this wave's loads of a stage are complete while `later` of
  // its loads of later stages stay in flight, then barrier.
  auto wait_stage = [&](int later) {
    if (later >= 3)
      vm_wait_barrier<3 * kDma>();
    else if (later == 2)
      vm_wait_barrier<2 * kDma>();
    else if (later == 1)
      vm_wait_barrier<kDma>();
    else
      vm_wait_barrier<0>();
  };
  auto later_after = [&](int t) {   // loads of stages after t+1 in flight at the end of A(t)
    const int l = nk - 2 - t;
    return l < kRing - 2 ? l : kRing - 2;
  };

  for (int s0 = 0; s0 < kRing; ++s0)
    if (s0 < nk) issue(s0, s0);
  // Persistent loop over output tiles: after a tile's epilogue stores, the
  // first stages of the next tile are issued at once, so their loads overlap
  // the stores' drain instead of waiting for a new workgroup.
  for (;;) {
#pragma unroll
    for (int a = 0; a < FN; ++a)
#pragma unroll
      for (int b = 0; b < FM; ++b) acc[a][b] = Acc{0, 0, 0, 0};
    wait_stage(nk - 1 < kRing - 1 ? nk - 1 : kRing - 1);
    int slot = 0;
    if (grp == 0) {
      read_frags(0);
      for (int t = 0; t < nk; ++t) {
        mfmas();                                            // A(t): compute stage t
        wait_stage(later_after(t));
        if (t + 1 < nk) read_frags(next_slot(slot));       // B(t): read t+1, refill
        if (t + kRing < nk) issue(slot, t + kRing);
        vm_wait_barrier<63>();
        slot = next_slot(slot);
      }
    } else {
      for (int t = 0; t < nk; ++t) {
        read_frags(slot);                                   // A(t): read t, refill
        if (t >= 1 && t - 1 + kRing < nk) issue(prev_slot(slot), t - 1 + kRing);
        wait_stage(later_after(t));
        mfmas();                                            // B(t): compute stage t
        vm_wait_barrier<63>();
        slot = next_slot(slot);
      }
    }

    bool next_issued = false;   // the next tile's first stages are already in flight
    if constexpr (DT == TCU_I8_BOOL) {
      // 0/1 output (a quarter of the bytes of a binary32 tile): the flags
      // (sum > 0) go through LDS so that the read-modify-write of C is done
      // in whole 16-byte row chunks, consecutive threads on consecutive
      // chunks.  The flags have LDS of their own, so the next tile's first
      // stages are issued first (the ring is free after the loop's last
      // barrier) and load while this epilogue runs; the K loop is short here
      // (one pivot band), so that latency would otherwise be paid per tile.
      // Flag rows are 256 bytes with the 16-byte chunks XOR-swizzled by the
      // row: the 16 rows one store instruction touches land in distinct
      // banks, and a row's chunks are still one 256-byte row.
      const int em0 = m0, en0 = n0;
      if (item >= 0 && item + stride < limit) {
        item += stride;
        place(item);
        for (int s0 = 0; s0 < kRing; ++s0)
          if (s0 < nk) issue(s0, s0);
        next_issued = true;
      }
      auto flag_at = [&](int row, int byte) {
        return sF + row * 256 + (((byte >> 4) ^ (row & 15)) << 4) + (byte & 15);
      };
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          const int row = grp * 128 + fm * 16 + r;
          const int col = q * 64 + fn * 16 + 4 * g;
          unsigned w = 0;
#pragma unroll
          for (int e = 0; e < 4; ++e) w |= (unsigned)(acc[fn][fm][e] > 0) << (8 * e);
          *(unsigned *)flag_at(row, col) = w;
        }
      }
      __syncthreads();
      // OR is idempotent: a chunk with no new flag is neither read nor
      // written, and a chunk whose OR changes nothing is not written back
      // (once the closure fills in, most of a band's update is such a no-op).
      // The flags are read first so that all of a thread's C loads are in
      // flight together.
      constexpr int kChunks = 256 * 16 / 512;   // 16-byte chunks per thread
      u32x4 f[kChunks], old[kChunks];
#pragma unroll
      for (int j = 0; j < kChunks; ++j) {
        const int c = threadIdx.x + 512 * j, row = c >> 4, cc = c & 15;
        f[j] = *(const u32x4 *)flag_at(row, 16 * cc);
      }
#pragma unroll
      for (int j = 0; j < kChunks; ++j) {
        const int c = threadIdx.x + 512 * j, row = c >> 4, cc = c & 15;
        old[j] = u32x4{0u, 0u, 0u, 0u};
        if ((f[j][0] | f[j][1] | f[j][2] | f[j][3]) != 0u)
          old[j] = *(const u32x4 *)(C + (int64_t)(em0 + row) * ldc_b + en0 + 16 * cc);
      }
#pragma unroll
      for (int j = 0; j < kChunks; ++j) {
        const int c = threadIdx.x + 512 * j, row = c >> 4, cc = c & 15;
        const u32x4 nw = old[j] | f[j];
        const u32x4 d = nw ^ old[j];
        if ((d[0] | d[1] | d[2] | d[3]) != 0u)
          *(u32x4 *)(C + (int64_t)(em0 + row) * ldc_b + en0 + 16 * cc) = nw;
      }
      __syncthreads();   // flag reads done before the next tile's epilogue rewrites them
    } else {
      // Epilogue: lane holds C[row][col .. col+3] of every accumulator block.
      auto out_ptr = [&](int fn, int fm) {
        const int row = m0 + grp * 128 + fm * 16 + r;
        const int col = n0 + q * 64 + fn * 16 + 4 * g;
        return C + (int64_t)row * ldc_b + (int64_t)col * OB;
      };
      // The lane's 4 columns lie wholly inside or wholly outside C (n_lim is
      // a multiple of 4).
      auto in_c = [&](int fn, int fm) {
        return !kEdge ||
               (m0 + grp * 128 + fm * 16 + r < m_lim && n0 + q * 64 + fn * 16 + 4 * g < n_lim);
      };
      constexpr bool kSplittable = DT == TCU_F16_F32 || DT == TCU_BF16_F32 || DT == TCU_I8_I32;
      if (kSplittable && split_item) {
        // Partial tiles are added into C atomically.  In the accumulator
        // layout one atomic instruction would touch one element in each of
        // 16 rows, so every 64-byte line gets four separate requests; the
        // wave's 128 x 64 sub-tile goes through LDS instead (the ring is
        // free after the loop's last barrier), 64 rows at a time, and each
        // atomic instruction then adds 64 consecutive elements of one row.
        // Row stride 272 bytes: the 16 rows one 16-byte store instruction
        // touches land in distinct banks.
        if constexpr (kSplittable) {
          constexpr int kStride = 272;
          unsigned char *stage = (grp == 0 ? sA : sB) + q * 64 * kStride;
          const int col = n0 + q * 64 + lane;
#pragma unroll
          for (int h = 0; h < FM / 4; ++h) {
#pragma unroll
            for (int fn = 0; fn < FN; ++fn)
#pragma unroll
              for (int fm = 0; fm < 4; ++fm)
                *(Acc *)(stage + (fm * 16 + r) * kStride + (fn * 16 + 4 * g) * 4) =
                    acc[fn][h * 4 + fm];
            __syncthreads();
            const int row0 = m0 + grp * 128 + h * 64;
#pragma unroll 8
            for (int i = 0; i < 64; ++i) {
              if (kEdge && (row0 + i >= m_lim || col >= n_lim)) continue;
              unsigned char *p = C + (int64_t)(row0 + i) * ldc_b + (int64_t)col * OB;
              if constexpr (DT == TCU_I8_I32)
                __hip_atomic_fetch_add((int *)p, *(const int *)(stage + i * kStride + 4 * lane),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              else
                __hip_atomic_fetch_add((float *)p, *(const float *)(stage + i * kStride + 4 * lane),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __syncthreads();   // reads done before the next half (or the ring) overwrites
          }
        }
      } else {
        // Blocks fn and fn + 1 hold the two 64-byte halves of 128-byte rows
        // of C, so they are stored back to back: a half-written line left
        // in L2 while other stores intervene is written to memory twice
        // (measured: 1.37x the output bytes with fn outermost, 1.006x here).
        if (accum) {
          // C <- C + tile: the old values of two block rows (8 blocks) are
          // loaded together, then summed and stored -- one memory round trip
          // per 8 blocks instead of one per block.
#pragma unroll
          for (int fm0 = 0; fm0 < FM; fm0 += 2) {
            Old4<DT> old[2][FN];
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int fn = 0; fn < FN; ++fn)
                old[j][fn] = in_c(fn, fm0 + j) ? load_old4<DT>(out_ptr(fn, fm0 + j)) : Old4<DT>{};
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int fn = 0; fn < FN; ++fn)
                if (in_c(fn, fm0 + j))
                  store_sum4<DT>(out_ptr(fn, fm0 + j), acc[fn][fm0 + j], old[j][fn]);
          }
        } else {
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
#pragma unroll
            for (int fn = 0; fn < FN; ++fn)
              if (in_c(fn, fm)) store_out4<DT, true>(out_ptr(fn, fm), acc[fn][fm], 4, false);
        }
      }
    }
    // Every wave finished reading the ring at the last barrier of the loop.
    if (next_issued) continue;
    if constexpr (DT == TCU_I8_BOOL) {
      if (with_diag && item < 0) {
        // The block's update is stored (the epilogue ends with a workgroup
        // barrier, which orders the stores before the loads below); the ring
        // is free.
        close_diag_block<true, 512>(C + (int64_t)m0 * ldc_b + n0, ldc_b, kDiagBand,
                                    *reinterpret_cast<DiagShared *>(smem));
        break;
      }
    }
    item += stride;
    if (item >= limit) break;
    place(item);
    for (int s0 = 0; s0 < kRing; ++s0)
      if (s0 < nk) issue(s0, s0);
  }
}

// ---------------------------------------------------------------------------
// Small-tile kernel for 16-bit inputs (M, N multiples of 64, K a multiple of
// one 128-byte stage): 64 x 64 output tiles, 4 waves of 32 x 32, and a ring
// of kStages LDS stages filled by direct DMA loads kStages - 1 stages ahead.
// Products with few tiles and a long K per tile (N = 1024: 256 tiles with
// K = 1024 each) are latency-bound on a register-staged double buffer, which
// exposes one L2 round trip per K step; the ring keeps kStages - 1 stages of
// every workgroup in flight instead.
//   * A stage of A: 64 rows x 128 bytes as four 2 KiB blocks of 16 rows,
//     chunk-major, so a fragment read is a linear ds_read_b128.
//   * A stage of B: 64 k-rows x 128 bytes (64 columns), row-major, 16-byte
//     chunks XOR-swizzled by bits 1 and 3 of the row, so that the 32 lanes
//     of one ds_read_b64_tr_b16 pass (8 rows, 32 bytes each) hit distinct
//     banks.
//   * Wave w loads A block w and B rows 16w .. 16w+15 of every stage (four
//     1 KiB DMA instructions), and computes rows 32(w/2) .., columns
//     32(w%2) .. of the tile.
// ---------------------------------------------------------------------------
constexpr int kRingKB = 128;                    // bytes of K per stage
constexpr int kRingHalf = 64 * kRingKB;         // 8 KiB per operand per stage

__device__ __forceinline__ int ring_b_swz(int k) {
  return (((k >> 1) & 1) << 1) | (((k >> 3) & 1) << 2);
}

// Wait until at most 4 * min(later, kMax) of this wave's DMA loads are in
// flight (and its LDS reads returned), then barrier.
template <int kMax>
__device__ __forceinline__ void ring_wait(int later) {
  if constexpr (kMax == 0) {
    vm_wait_barrier<0>();
  } else {
    if (later >= kMax)
      vm_wait_barrier<4 * kMax>();
    else
      ring_wait<kMax - 1>(later);
  }
}

template <int DT, int kStages>
__global__ __launch_bounds__(256) void gemm_ring_kernel(
    const unsigned char *__restrict__ A, const unsigned char *__restrict__ B,
    unsigned char *__restrict__ C, int K, int64_t lda, int64_t ldb, int64_t ldc, int accum,
    int tiles_m, int tiles_n) {
  static_assert(in_bytes(DT) == 2, "16-bit inputs");
  static_assert(kStages >= 2 && 4 * (kStages - 2) <= 63, "vmcnt range");
  constexpr int OB = out_bytes(DT);
  constexpr int KE = kRingKB / 2;               // contracted elements per stage
  __shared__ __attribute__((aligned(1024))) unsigned char sA[kStages * kRingHalf];
  __shared__ __attribute__((aligned(1024))) unsigned char sB[kStages * kRingHalf];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int r = lane & 15, g = lane >> 4;
  int tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * 64, n0 = tn * 64;
  const int64_t lda_b = lda * 2, ldb_b = ldb * 2, ldc_b = ldc * OB;
  const int nk = K / KE;

  // DMA share of wave w (wave-uniform bases, per-lane 32-bit offsets).
  const unsigned char *abase = A + (int64_t)(m0 + 16 * w) * lda_b;
  const unsigned char *bbase = B + (int64_t)(16 * w) * ldb_b + (int64_t)n0 * 2;
  unsigned aoff[2], boff[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    aoff[h] = (unsigned)((lane & 15) * lda_b) + 16u * (4 * h + (lane >> 4));
    const int krow = 8 * h + (lane >> 3);
    boff[h] = (unsigned)(krow * ldb_b) + 16u * ((lane & 7) ^ ring_b_swz(16 * w + krow));
  }
  const unsigned a_lds = lds_addr(sA) + w * 2048, b_lds = lds_addr(sB) + w * 2048;
  auto issue = [&](int slot, int t) {
    const unsigned char *ga = abase + (int64_t)t * kRingKB;
    const unsigned char *gb = bbase + (int64_t)t * KE * ldb_b;
#pragma unroll
    for (int h = 0; h < 2; ++h) dma_lds16_saddr(ga, aoff[h], a_lds + slot * kRingHalf + h * 1024);
#pragma unroll
    for (int h = 0; h < 2; ++h) dma_lds16_saddr(gb, boff[h], b_lds + slot * kRingHalf + h * 1024);
  };

  // Fragment offsets within a stage: A rows 32 wm .., B^T columns 32 wn ..
  const int x_off = wm * 2 * 2048 + 16 * lane;
  int w_off[2];
#pragma unroll
  for (int fn = 0; fn < 2; ++fn) {
    const int n = wn * 32 + fn * 16 + 4 * (r & 3);
    const int k0 = 8 * g + (r >> 2);
    w_off[fn] = k0 * kRingKB + 16 * ((n >> 3) ^ ring_b_swz(k0)) + ((2 * n) & 15);
  }

  f32x4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int s0 = 0; s0 < kStages - 1; ++s0)
    if (s0 < nk) issue(s0, s0);
  int slot = 0;
  for (int t = 0; t < nk; ++t) {
    // This wave's loads of stage t done (those of the stages after it may
    // stay in flight); the barrier makes every wave's share visible and
    // ensures all waves finished reading stage t-1, whose slot is refilled.
    const int later = nk - 1 - t < kStages - 2 ? nk - 1 - t : kStages - 2;
    ring_wait<kStages - 2>(later);
    const int refill = t + kStages - 1;
    if (refill < nk) issue(slot == 0 ? kStages - 1 : slot - 1, refill);
    const unsigned char *sa = sA + slot * kRingHalf;
    const unsigned char *sb = sB + slot * kRingHalf;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      u32x4 xf[2], wf[2];
#pragma unroll
      for (int fm = 0; fm < 2; ++fm) xf[fm] = *(const u32x4 *)(sa + x_off + fm * 2048 + kk * 1024);
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const u32x2 w0 = lds_read_tr16(sb + w_off[fn] + kk * 32 * kRingKB);
        const u32x2 w1 = lds_read_tr16(sb + w_off[fn] + kk * 32 * kRingKB + 4 * kRingKB);
        wf[fn] = u32x4{w0[0], w0[1], w1[0], w1[1]};
      }
#pragma unroll
      for (int fn = 0; fn < 2; ++fn)
#pragma unroll
        for (int fm = 0; fm < 2; ++fm) acc[fn][fm] = mfma_k32(DT, wf[fn], xf[fm], acc[fn][fm]);
    }
    slot = slot + 1 == kStages ? 0 : slot + 1;
  }

  // Epilogue: lane holds C[row][col .. col+3] of every accumulator block.
#pragma unroll
  for (int fn = 0; fn < 2; ++fn) {
#pragma unroll
    for (int fm = 0; fm < 2; ++fm) {
      const int row = m0 + wm * 32 + fm * 16 + r;
      const int col = n0 + wn * 32 + fn * 16 + 4 * g;
      store_out4<DT, true>(C + (int64_t)row * ldc_b + (int64_t)col * OB, acc[fn][fm], 4,
                           accum != 0);
    }
  }
}

// Zero the rows x row_bytes view at C (row pitch ldc_b bytes; row_bytes and
// ldc_b multiples of 16): the starting value of a split-K product that
// overwrites C.
__global__ __launch_bounds__(256) void zero_fill_kernel(unsigned char *__restrict__ C, int64_t rows,
                                                        int64_t row_bytes, int64_t ldc_b) {
  const int64_t per_row = row_bytes / 16;
  const int64_t total = rows * per_row;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t rr = i / per_row;
    *(u32x4 *)(C + rr * ldc_b + (i - rr * per_row) * 16) = u32x4{0u, 0u, 0u, 0u};
  }
}

// Zero the output tiles pid in [first, first + count) of a tiles_m x
// tiles_n grid of 256 x 256 tiles of 4-byte values (placed by map_tile),
// clipped to rows < m_lim and to the first row_bytes bytes of each row (a
// multiple of 16): the starting value of the split tail tiles of a product
// that overwrites C.
__global__ __launch_bounds__(256) void zero_tiles_kernel(unsigned char *__restrict__ C,
                                                         int64_t ldc_b, int tiles_m, int tiles_n,
                                                         int first, int count, int m_lim,
                                                         int64_t row_bytes) {
  constexpr int kChunks = 256 * 4 / 16;   // 16-byte chunks per tile row
  const int64_t total = (int64_t)count * 256 * kChunks;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int t = (int)(i / (256 * kChunks));
    const int rem = (int)(i - (int64_t)t * 256 * kChunks);
    int tm, tn;
    map_tile(first + t, tiles_m, tiles_n, tm, tn);
    const int row = tm * 256 + rem / kChunks;
    const int64_t cb = (int64_t)tn * 1024 + 16 * (rem % kChunks);
    if (row < m_lim && cb < row_bytes)
      *(u32x4 *)(C + (int64_t)row * ldc_b + cb) = u32x4{0u, 0u, 0u, 0u};
  }
}

// The tail split: when a persistent grid of `grid` workgroups walks `tiles`
// whole tiles and the last round holds only tiles % grid of them, most CUs
// would idle through it.  Those tail tiles are cut into nsplit K ranges
// instead (at least kMinStages stages each, at most grid / tail of them),
// added into C atomically, so the last round is about 1 / nsplit as long.
// binary32 and int32 outputs only (a bfloat16 output is rounded once from
// the whole sum).  The test override TCU_KNOB_TAIL_SPLIT = n > 0 forces n
// ranges (1: none).  Returns
// nsplit (1: no tail split) and sets *full to the number of whole tiles.
template <int DT>
int tail_split(int tiles, int grid, int64_t stages, int kMinStages, int *full) {
  *full = tiles;
  if (DT == TCU_BF16_BF16 || tiles <= grid || tiles % grid == 0) return 1;
  const int tail = tiles % grid;
  int64_t ns = grid / tail;
  const int64_t cap = stages / kMinStages;
  if (ns > cap) ns = cap;
  const int forced = knob(TCU_KNOB_TAIL_SPLIT);
  if (forced > 0) ns = forced < stages ? forced : stages;
  if (ns < 2) return 1;
  *full = tiles - tail;
  return (int)ns;
}

// Zero the tail tiles [full, tiles) of an overwriting product split by
// tail_split (C of 4-byte values, row pitch ldc_b bytes).
hipError_t zero_tail(unsigned char *C, int64_t ldc_b, int tm, int tn, int full, int m_lim,
                     int64_t row_bytes, hipStream_t stream, int num_cus) {
  hipLaunchKernelGGL(zero_tiles_kernel, dim3(num_cus * 4), dim3(256), 0, stream, C, ldc_b, tm,
                     tn, full, tm * tn - full, m_lim, row_bytes);
  return hipGetLastError();
}

template <int DT, int BM, int BN, int WM, int WN, bool kVec, int kAl = 0>
hipError_t launch_cfg(const RectArgs &a, hipStream_t stream) {
  const int tiles_m = (int)((a.M + BM - 1) / BM), tiles_n = (int)((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_kernel<DT, BM, BN, WM, WN, kVec, kAl>), dim3(tiles_m * tiles_n),
                     dim3(64 * WM * WN), 0, stream, (const unsigned char *)a.A,
                     (const unsigned char *)a.B, (unsigned char *)a.C, (int)a.M, (int)a.N,
                     (int)a.K, a.lda, a.ldb, a.ldc, a.accum ? 1 : 0, tiles_m, tiles_n,
                     kNoBand, 0, kNoBand, 0);
  return hipGetLastError();
}

// Boolean rank-Bk update of the transitive closure on 0/1 int8 data:
// C[rows, cols] <- C OR (A[rows, 0:Bk] B[0:Bk, cols] > 0), the tile grid
// skipping the pivot band [k0, k0 + Bk) in rows and/or columns.
// rows_skip / cols_skip: whether the row / column range of C steps over the
// band (then M / N is the matrix order n and the band starts at k0).
template <int BM, int BN, bool kVec>
hipError_t launch_bool(const unsigned char *A, const unsigned char *B, unsigned char *C,
                       int64_t ld, int M, int N, int Bk, int k0, bool rows_skip, bool cols_skip,
                       hipStream_t stream) {
  const int rows = rows_skip ? M - Bk : M, cols = cols_skip ? N - Bk : N;
  const int tiles_m = (rows + BM - 1) / BM, tiles_n = (cols + BN - 1) / BN;
  if (tiles_m <= 0 || tiles_n <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<TCU_I8_BOOL, BM, BN, 2, 2, kVec>), dim3(tiles_m * tiles_n),
                     dim3(256), 0, stream, A, B, C, M, N, Bk, ld, ld, ld, 1, tiles_m, tiles_n,
                     rows_skip ? k0 / BM : kNoBand, rows_skip ? Bk : 0,
                     cols_skip ? k0 / BN : kNoBand, cols_skip ? Bk : 0);
  return hipGetLastError();
}

// Kernel selection by size; the test override TCU_KNOB_GEMM_KERNEL forces
// the full-tile (ping-pong) kernel wherever its shape conditions hold, the
// general kernel, or the small-tile ring kernel.
enum class GemmPath { kAuto, kFast, kGeneral, kRing };
GemmPath gemm_path() {
  switch (knob(TCU_KNOB_GEMM_KERNEL)) {
    case TCU_PATH_FULL_TILE: return GemmPath::kFast;
    case TCU_PATH_GENERAL: return GemmPath::kGeneral;
    case TCU_PATH_RING: return GemmPath::kRing;
  }
  return GemmPath::kAuto;
}

// The general and small-tile kernels: the product on shapes the full-tile
// kernel does not take.
template <int DT>
hipError_t launch_general(const RectArgs &a, GemmPath path, bool vec, hipStream_t stream,
                          int num_cus) {
  constexpr int ES = in_bytes(DT);
  const int64_t big_tiles = ((a.M + 255) / 256) * ((a.N + 255) / 256);
  const int64_t mid_tiles = ((a.M + 127) / 128) * ((a.N + 127) / 128);
  // Pitches not all multiples of 16 bytes: whole chunks of A and B (interior
  // tiles, full K steps) in the widest naturally aligned pieces both pitches
  // allow (8, 4, 2 or 1 bytes), edges element by element; C element by
  // element.  128 x 128 tiles where they still give every CU a workgroup.
  if (!vec) {
    const int64_t pa = a.lda * ES, pb = a.ldb * ES;
    const int al = pa % 8 == 0 && pb % 8 == 0   ? 8
                   : pa % 4 == 0 && pb % 4 == 0 ? 4
                   : pa % 2 == 0 && pb % 2 == 0 ? 2
                                                : 1;
    if (mid_tiles >= num_cus) {
      if (al == 8) return launch_cfg<DT, 128, 128, 2, 2, false, 8>(a, stream);
      if (al == 4) return launch_cfg<DT, 128, 128, 2, 2, false, 4>(a, stream);
      if (ES == 2 || al == 2) return launch_cfg<DT, 128, 128, 2, 2, false, 2>(a, stream);
      return launch_cfg<DT, 128, 128, 2, 2, false, 1>(a, stream);
    }
    if (al == 8) return launch_cfg<DT, 64, 64, 2, 2, false, 8>(a, stream);
    if (al == 4) return launch_cfg<DT, 64, 64, 2, 2, false, 4>(a, stream);
    if (ES == 2 || al == 2) return launch_cfg<DT, 64, 64, 2, 2, false, 2>(a, stream);
    return launch_cfg<DT, 64, 64, 2, 2, false, 1>(a, stream);
  }
  // The small-tile ring kernel: 16-bit inputs, whole 64 x 64 tiles and
  // 128-byte K stages, where the general kernel would take 64 x 64 tiles
  // (or where forced by the test override).
  if constexpr (ES == 2) {
    const bool ring_ok = path != GemmPath::kGeneral && path != GemmPath::kFast &&
                         a.M % 64 == 0 && a.N % 64 == 0 && a.K % 64 == 0 && a.K > 0 &&
                         16 * a.lda * ES < ((int64_t)1 << 32) &&
                         16 * a.ldb * ES < ((int64_t)1 << 32);
    if (ring_ok && (path == GemmPath::kRing || mid_tiles < num_cus)) {
      const int tm = (int)(a.M / 64), tn = (int)(a.N / 64);
      hipLaunchKernelGGL((gemm_ring_kernel<DT, 8>), dim3(tm * tn), dim3(256), 0, stream,
                         (const unsigned char *)a.A, (const unsigned char *)a.B,
                         (unsigned char *)a.C, (int)a.K, a.lda, a.ldb, a.ldc, a.accum ? 1 : 0,
                         tm, tn);
      return hipGetLastError();
    }
  }
  // Otherwise the largest tiles that still give every CU a workgroup.
  if (big_tiles >= num_cus) return launch_cfg<DT, 256, 256, 2, 2, true>(a, stream);
  if (mid_tiles >= num_cus) return launch_cfg<DT, 128, 128, 2, 2, true>(a, stream);
  return launch_cfg<DT, 64, 64, 2, 2, true>(a, stream);
}

template <int DT>
hipError_t launch_dt(const RectArgs &a, hipStream_t stream, int num_cus) {
  constexpr int ES = in_bytes(DT), OB = out_bytes(DT);
  constexpr int KE = kFastKB / ES;
  const bool vec = (a.lda * ES) % 16 == 0 && (a.ldb * ES) % 16 == 0 && (a.ldc * OB) % 16 == 0;
  const int64_t big_tiles = ((a.M + 255) / 256) * ((a.N + 255) / 256);
  const GemmPath path = gemm_path();
  // The full-tile kernel: whole 256 x 256 tiles, whole K stages, and the
  // per-lane 32-bit DMA offsets within a stage in range.
  const bool fast_ok = path != GemmPath::kGeneral && vec && a.M % 256 == 0 && a.N % 256 == 0 &&
                       a.K % KE == 0 && a.K > 0 && 256 * a.lda * ES < ((int64_t)1 << 32) &&
                       KE * a.ldb * ES < ((int64_t)1 << 32);
  // Split-K: when the full-tile kernel has fewer tiles than CUs and a long
  // K, the stages are cut into nsplit ranges processed by separate work
  // items whose partial tiles are added into C atomically (binary32 or
  // int32 outputs only: a bfloat16 output is rounded once from the whole
  // sum).  Each range keeps at least kMinSplitStages stages.
  constexpr int kMinSplitStages = 32;
  int nsplit = 1;
  if (fast_ok && DT != TCU_BF16_BF16 && big_tiles < num_cus) {
    const int64_t want = (num_cus + big_tiles - 1) / big_tiles;
    const int64_t cap = (a.K / KE) / kMinSplitStages;
    nsplit = (int)(want < cap ? want : cap);
    if (nsplit < 1) nsplit = 1;
  }
  const int forced_split = knob(TCU_KNOB_SPLIT_K);   // test override of the count
  if (forced_split > 0 && fast_ok && DT != TCU_BF16_BF16) {
    nsplit = forced_split;
    if (nsplit > a.K / KE) nsplit = (int)(a.K / KE);
  }
  if (fast_ok && (path == GemmPath::kFast || nsplit > 1 ||
                  (path == GemmPath::kAuto && big_tiles >= num_cus))) {
    const int tm = (int)(a.M / 256), tn = (int)(a.N / 256);
    if (nsplit > 1 && !a.accum) {
      hipLaunchKernelGGL(zero_fill_kernel, dim3(num_cus * 4), dim3(256), 0, stream,
                         (unsigned char *)a.C, a.M, a.N * OB, a.ldc * OB);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    // Persistent grid: one workgroup per CU (the LDS ring admits one), each
    // walking tiles blockIdx, blockIdx + grid, ...  The test override
    // TCU_KNOB_PP_GRID sets the grid size instead (a tiny grid gives every
    // workgroup many tiles).
    const int want = knob(TCU_KNOB_PP_GRID) > 0 ? knob(TCU_KNOB_PP_GRID) : num_cus;
    int full = 0;
    if (nsplit == 1) {
      const int g0 = want < tm * tn ? want : tm * tn;
      nsplit = tail_split<DT>(tm * tn, g0, a.K / KE, kMinSplitStages, &full);
      if (nsplit > 1 && !a.accum) {
        const hipError_t e = zero_tail((unsigned char *)a.C, a.ldc * OB, tm, tn, full,
                                       (int)a.M, a.N * OB, stream, num_cus);
        if (e != hipSuccess) return e;
      }
    }
    const int items = full + (tm * tn - full) * nsplit;
    const int grid = want < items ? want : items;
    hipLaunchKernelGGL((gemm_pp_kernel<DT, kRingStages, false>), dim3(grid), dim3(512), 0, stream,
                       (const unsigned char *)a.A, (const unsigned char *)a.B,
                       (unsigned char *)a.C, (int)a.K, a.lda, a.ldb, a.ldc, a.accum ? 1 : 0,
                       tm, tn, full, nsplit, (int)a.M, (int)a.N, TileRemap{}, -1);
    return hipGetLastError();
  }
  // Ragged shapes (dimensions that are not multiples of the tile or of a
  // stage, zero-padded), large enough to give every CU a 256 x 256 tile:
  //   * N a whole number of 16-byte chunks: the full-tile kernel alone, its
  //     edge tiles loading clamped rows and chunks and storing only inside
  //     C, the contracted index's partial last stage zero-padded;
  //   * otherwise the full-tile kernel takes the 256-aligned interior --
  //     rows [0, M0) and columns [0, N0) over the whole K -- and the
  //     general kernel the bottom rows [M0, M) (all columns) and the right
  //     columns [N0, N) of rows [0, M0).
  // Every output element is formed by one launch over the whole K, so a
  // bfloat16 output is still rounded once.
  const int64_t M0 = a.M / 256 * 256, N0 = a.N / 256 * 256;
  const bool edges_in_kernel = (a.N * ES) % 16 == 0;
  const int64_t tm_all = edges_in_kernel ? (a.M + 255) / 256 : M0 / 256;
  const int64_t tn_all = edges_in_kernel ? (a.N + 255) / 256 : N0 / 256;
  const bool ragged_ok = path == GemmPath::kAuto && vec && a.K >= KE && tm_all >= 1 &&
                         tn_all >= 1 && tm_all * tn_all >= num_cus &&
                         256 * a.lda * ES < ((int64_t)1 << 32) &&
                         KE * a.ldb * ES < ((int64_t)1 << 32);
  if (ragged_ok) {
    const int tm = (int)tm_all, tn = (int)tn_all;
    const int grid = num_cus < tm * tn ? num_cus : tm * tn;
    // The tail tiles' zeroing is clipped to the kernel's part of C: all of
    // it (N * OB is then a multiple of 16 bytes) or the 256-aligned interior.
    int full = tm * tn;
    const int nsplit = tail_split<DT>(tm * tn, grid, (a.K + KE - 1) / KE, kMinSplitStages, &full);
    if (nsplit > 1 && !a.accum) {
      hipError_t e = zero_tail((unsigned char *)a.C, a.ldc * OB, tm, tn, full,
                               (int)(edges_in_kernel ? a.M : M0),
                               (edges_in_kernel ? a.N : N0) * OB, stream, num_cus);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((gemm_pp_kernel<DT, kRingStages, true>), dim3(grid), dim3(512), 0, stream,
                       (const unsigned char *)a.A, (const unsigned char *)a.B,
                       (unsigned char *)a.C, (int)a.K, a.lda, a.ldb, a.ldc, a.accum ? 1 : 0,
                       tm, tn, full, nsplit, (int)a.M, (int)a.N, TileRemap{}, -1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || edges_in_kernel) return e;
    if (a.M > M0) {
      RectArgs b = a;
      b.A = (const unsigned char *)a.A + M0 * a.lda * ES;
      b.C = (unsigned char *)a.C + M0 * a.ldc * OB;
      b.M = a.M - M0;
      e = launch_general<DT>(b, path, vec, stream, num_cus);
      if (e != hipSuccess) return e;
    }
    if (a.N > N0) {
      RectArgs r = a;
      r.B = (const unsigned char *)a.B + N0 * ES;
      r.C = (unsigned char *)a.C + N0 * OB;
      r.M = M0;
      r.N = a.N - N0;
      e = launch_general<DT>(r, path, vec, stream, num_cus);
    }
    return e;
  }
  return launch_general<DT>(a, path, vec, stream, num_cus);
}

}  // namespace

// The transitive closure's matrix-core phases for the pivot band
// [k0, k0 + Bk), Y = X[band, band] already closed.  Every phase is the D
// formula X[I, J] |= X[I, band] X[band, J] over a set of tiles, computed in
// place.  Tiles may read operand blocks that other tiles of the same launch
// are rewriting; that is harmless because every value only grows (0 -> 1)
// and stays between its value before the phase and the closure: with one
// operand final (Y, or a panel finished by an earlier launch), any mix of
// old and new values in the other gives exactly the final product.
//   * column panel: X[I, band] |= X[I, band] Y for I outside the band;
//   * then, in one launch, the row panel X[band, J] |= Y X[band, J] and the
//     rest X[I, J] |= X[I, band] X[band, J]: all tiles with J outside the
//     band (the column panel is final, so the rows I = band and I outside
//     it take the same formula).
hipError_t launch_tc_panels(unsigned char *X, int64_t ld, int n, int k0, int Bk,
                            hipStream_t stream) {
  unsigned char *band_col = X + k0;
  const unsigned char *Y = X + (int64_t)k0 * ld + k0;
  // Column panel tiles of 32 rows x the band: the panel's work is small and
  // latency-bound, so twice the workgroups of 64-row tiles finish sooner
  // (n = 8192: 9.1 -> 6.7 us per band; 32 x 128 and 64 x 128 were slower).
  if (ld % 16 == 0)
    return launch_bool<32, 256, true>(band_col, Y, band_col, ld, n, Bk, Bk, k0, true, false,
                                      stream);
  return launch_bool<32, 256, false>(band_col, Y, band_col, ld, n, Bk, Bk, k0, true, false,
                                     stream);
}

hipError_t launch_tc_rest(unsigned char *X, int64_t ld, int n, int k0, int Bk,
                          hipStream_t stream, int num_cus, bool close_next) {
  const unsigned char *L = X + k0;
  const unsigned char *R = X + (int64_t)k0 * ld;
  // Whole 256-wide bands and 16-byte rows: the full-tile kernel over
  // n/256 x (n/256 - 1) tiles, stepping over the band's tile column.
  if (tc_full_tiles(n, Bk, ld)) {
    TileRemap rm;
    rm.band_n = k0 / 256;
    rm.skip_n = 256;
    const int tiles_m = n / 256, tiles_n = n / 256 - 1;
    int diag_pid = -1;
    if (close_next) {
      // The next band's diagonal tile: tile row b + 1 and, the band's column
      // b being skipped, grid column b; its index in map_tile's order.
      const int tm = k0 / 256 + 1, tn = k0 / 256;
      const int first_m = tm / kGroupM * kGroupM;
      const int gsz = tiles_m - first_m < kGroupM ? tiles_m - first_m : kGroupM;
      diag_pid = first_m * tiles_n + tn * gsz + (tm - first_m);
    }
    return launch_tc_tiles(X, ld, n, k0, tiles_m, tiles_n, rm, stream, num_cus, diag_pid);
  }
  if (ld % 16 == 0)
    return launch_bool<128, 128, true>(L, R, X, ld, n, n, Bk, k0, false, true, stream);
  return launch_bool<128, 128, false>(L, R, X, ld, n, n, Bk, k0, false, true, stream);
}

bool tc_full_tiles(int64_t n, int Bk, int64_t ld) {
  return n % 256 == 0 && Bk == 256 && ld % 16 == 0 && 256 * ld < ((int64_t)1 << 32);
}

hipError_t launch_tc_tiles(unsigned char *X, int64_t ld, int n, int k0, int tiles_m,
                           int tiles_n, const TileRemap &remap, hipStream_t stream,
                           int num_cus, int diag_pid) {
  // The D formula X[I, J] |= X[I, band] X[band, J] (band = [k0, k0 + 256))
  // on a tiles_m x tiles_n grid of 256 x 256 tiles placed by remap, by at
  // most num_cus persistent workgroups.
  const int items = tiles_m * tiles_n;
  if (items <= 0) return hipSuccess;
  const int grid = num_cus < items ? num_cus : items;
  hipLaunchKernelGGL((gemm_pp_kernel<TCU_I8_BOOL, 3, false>), dim3(grid), dim3(512), 0,
                     stream,
                     X + k0, X + (int64_t)k0 * ld, X, 256, ld, ld, ld, 1, tiles_m, tiles_n,
                     tiles_m * tiles_n, 1, n, n, remap, diag_pid);
  return hipGetLastError();
}

hipError_t launch_rect(int dtype, int s, const RectArgs &a, hipStream_t stream, int num_cus) {
  // A single contiguous strip times a single block is one native call.
  if (a.K == s && a.N == s && a.lda == s && a.ldb == s && a.ldc == s)
    return launch_tall(dtype, s, a.A, a.M, a.B, a.C, a.accum, stream, num_cus);
  switch (dtype) {
    case TCU_F16_F32: return launch_dt<TCU_F16_F32>(a, stream, num_cus);
    case TCU_BF16_F32: return launch_dt<TCU_BF16_F32>(a, stream, num_cus);
    case TCU_BF16_BF16: return launch_dt<TCU_BF16_BF16>(a, stream, num_cus);
    case TCU_I8_I32: return launch_dt<TCU_I8_I32>(a, stream, num_cus);
  }
  return hipErrorInvalidValue;
}

}  // namespace tcu
