// Persistent "NT" GEMM on the gfx950 matrix cores: C[M, N] = A[M, K] * B[N, K]^T,
// both operands K-contiguous (the bf16 kernel can also read A transposed from
// its stage-tiled storage), fp32 accumulation, with a fused epilogue functor.
//
// Block tile 256 x 256, 4 waves in a 2 x 2 arrangement, each wave owning a
// 128 x 128 sub-tile as 4 x 4 blocks of 32 x 32 MFMA accumulators
// (v_mfma_f32_32x32x16_bf16 for bf16, v_mfma_f32_32x32x2_f32 for fp32), or, in
// the bf16 kernel's 16 x 16 mode, as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16
// accumulators (half the accumulator traffic per flop: under the board power
// limit the chip then holds a higher clock).
// Each K stage moves 128 bytes of every tile row (64 bf16 or 32 fp32) from
// global memory straight into LDS (no register staging), double-buffered (one
// barrier per stage in the 32 x 32 loops; in the 16 x 16 loop a second one in
// the middle of the stage, so that a stage's copies have until then to land).
// The 16-byte chunk c of tile row r is stored at chunk
// c ^ ((r >> 1) & 7): a 128-bit LDS read serves 16 lanes per pass from a
// 256-byte window (two 128-byte rows), and this places the 16 rows such a pass
// touches in 16 distinct bank groups.
//
// The grid is persistent (about one workgroup per compute unit, since a block
// holds 128 KiB of LDS).  The row counts M and N and the K extent may be read
// from device memory, so a launch sized for an upper bound does only the work
// the data needs without a host round trip.  Tile order: workgroups are dealt to
// the 8 XCDs round-robin, so each full round of tiles is renumbered to give
// every XCD a contiguous run, and runs are laid out group_m row-tiles deep so
// the 32 workgroups of an XCD share A and B panels in its L2.
#pragma once
#include <type_traits>
#include <utility>

#include "common.hpp"

namespace agrl {

constexpr int GBM = 256;
constexpr int GBN = 256;
constexpr int LDS_ROW = 128;                            // bytes per tile row per stage
constexpr int STAGE_BYTES = (GBM + GBN) * LDS_ROW;      // 64 KiB
constexpr int GEMM_LDS = 2 * STAGE_BYTES;               // 128 KiB of stage buffers
// bf16 logit-gradient epilogue (two passes of 128 tile rows): G rows staged
// row-major with 528-byte pitch (the two half-waves of a 16-bit store land in
// different banks); three 256-entry per-row arrays at EPI_META, above both the
// stage buffers and the store epilogue's 132 KiB staging of a pass
constexpr int EPI_G_ROW = 528;
constexpr int EPI_GS = 0;
// fp32 store epilogue of the 16 x 16 layout: a pass of 128 tile rows staged
// column-major, 132 floats per column (see EpiStore::tile16)
constexpr int EPI_COL = 132;
constexpr int EPI_COLS_LDS = 256 * EPI_COL * 4;             // 135168
constexpr int EPI_META = EPI_COLS_LDS > GEMM_LDS ? EPI_COLS_LDS : GEMM_LDS;
constexpr int EPI_STAGE_LDS = EPI_META + 3 * 1024;          // 138240 B
static_assert(EPI_GS + 128 * EPI_G_ROW <= EPI_META, "G staging below the per-row arrays");
constexpr int BF16_KERNEL_LDS = EPI_STAGE_LDS > GEMM_LDS ? EPI_STAGE_LDS : GEMM_LDS;
constexpr int GEMM_THREADS = 256;

template <typename T>
struct KStage;
template <>
struct KStage<__bf16> {
  static constexpr int BK = 64;
};
template <>
struct KStage<float> {
  static constexpr int BK = 32;
};

struct GemmShape {
  const void* A;
  int64_t lda;             // elements
  const void* B;
  int64_t ldb;
  int32_t M;               // rows of A (used when m_dev == nullptr)
  const int32_t* m_dev;    // rows of A read on the device
  int32_t N;               // rows of B (used when n_dev == nullptr)
  const int32_t* n_dev;    // rows of B read on the device
  int32_t K;               // multiple of BK (used when k_dev == nullptr)
  const int32_t* k_dev;    // K read on the device, rounded up to BK
  int32_t group_m;         // row-tiles per tile-order group
  // bf16 kernel only.  a_tiled / b_tiled: the operand is stored stage-tiled,
  // 1 in row-block order (tiled_index; lda / ldb = its padded K extent, a
  // multiple of 64), 2 in column-block order (tiled_cm_index; lda / ldb = its
  // padded row count, a multiple of 256).  a_trans: A is read transposed out
  // of a column-block tiled matrix whose rows are the product's K and whose
  // columns are the product's rows (lda = its padded row count).
  int32_t a_tiled, b_tiled, a_trans;
  // bf16 kernel only: 1 makes the tile-order groups run over column tiles
  // (group_m column tiles deep, sweeping every row tile) instead of row tiles
  int32_t group_cols;
};

// Stage-tiled bf16 layout of a matrix with rows r and K-columns k (K padded to
// k_pad, a multiple of 64; rows padded to a multiple of 256): the 256 x 64
// block (r / 256, k / 64) is 32 KiB contiguous, row-major with 128-byte rows,
// and 16-byte chunk c of a block row rr sits at chunk c ^ ((rr >> 1) & 7), the
// LDS swizzle of the kernel below.  One K stage of a 256-row tile is then one
// contiguous 32 KiB block that copies into LDS unchanged (every copy moves
// 1 KiB of consecutive bytes), and a stage's rows share DRAM pages.
__host__ __device__ __forceinline__ int64_t tiled_index(int64_t r, int64_t k, int64_t k_pad) {
  return (((r >> 8) * (k_pad >> 6) + (k >> 6)) << 14) + ((r & 255) << 6) +
         ((((k & 63) >> 3) ^ ((r >> 1) & 7)) << 3) + (k & 7);
}

// The same blocks in column-block order: block (r / 256, k / 64) at index
// (k / 64) * (r_pad / 256) + r / 256.  This is the layout of the backward's
// logit gradient G (r = token, k = vocabulary entry).  dH reads it with K =
// vocabulary (the stages of a 256-token tile are r_pad / 256 blocks apart); dW
// reads it transposed with K = tokens (a 64-token stage lies 8 KiB further in
// each of the tile's four block columns).  Both are uniform strides.
__host__ __device__ __forceinline__ int64_t tiled_cm_index(int64_t r, int64_t k, int64_t r_pad) {
  return (((k >> 6) * (r_pad >> 8) + (r >> 8)) << 14) + ((r & 255) << 6) +
         ((((k & 63) >> 3) ^ ((r >> 1) & 7)) << 3) + (k & 7);
}

// Accumulator element (i, j, r) of a wave sits at
//   row = wm*128 + i*32 + 8*(r/4) + 4*(lane/32) + r%4,  col = wn*128 + j*32 + lane%32.
__device__ __forceinline__ int acc_row(int wm, int i, int r, int lane) {
  return wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
__device__ __forceinline__ int acc_col(int wn, int j, int lane) {
  return wn * 128 + j * 32 + (lane & 31);
}

__device__ __forceinline__ void map_tile(int t, int grid, int total, int tiles_m, int tiles_n,
                                         int group_m, int& tm, int& tn) {
  int L = t;
  const int round = t / grid;
  if ((grid & 7) == 0 && (round + 1) * grid <= total) {
    const int b = t - round * grid;
    L = round * grid + (b & 7) * (grid >> 3) + (b >> 3);
  }
  const int width = group_m * tiles_n;
  const int grp = L / width;
  const int first = grp * group_m;
  const int gsz = min(tiles_m - first, group_m);
  const int rem = L - grp * width;
  tm = first + rem % gsz;
  tn = rem / gsz;
}

// Swizzle of a tile row: the chunk offset XORed into its 16-byte chunks.
__device__ __forceinline__ int row_swizzle(int r) { return (r >> 1) & 7; }

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// One K stage as direct global -> LDS copies (global_load_lds_dwordx4): each
// instruction moves 8 tile rows (1 KiB) and writes LDS contiguously, lane i at
// byte 16 * i.  Lane i therefore fetches logical chunk (i & 7) ^ row_swizzle(row)
// of row i / 8, which lands it at the swizzled position.  Wave w copies rows
// [64 w, 64 w + 64) of both the A and the B tile.  Rows past M or N are clamped
// to the last valid row (their products are discarded by the epilogue).
__device__ __forceinline__ void dma_stage(uint8_t* st, const uint8_t* A, int64_t lda_b, int m0,
                                          int M, const uint8_t* B, int64_t ldb_b, int n0, int N,
                                          int64_t k0_b, int wave, int lane) {
  const int rl = lane >> 3;
#pragma unroll
  for (int b = 0; b < 8; ++b) {
    const int r0 = wave * 64 + b * 8;
    const int c = (lane & 7) ^ row_swizzle(r0 + rl);
    const int64_t ra = min(m0 + r0 + rl, M - 1);
    const int64_t rb = min(n0 + r0 + rl, N - 1);
    __builtin_amdgcn_global_load_lds((glb_void_t*)(A + ra * lda_b + k0_b + c * 16),
                                     (lds_void_t*)(st + r0 * LDS_ROW), 16, 0, 0);
    __builtin_amdgcn_global_load_lds((glb_void_t*)(B + rb * ldb_b + k0_b + c * 16),
                                     (lds_void_t*)(st + GBM * LDS_ROW + r0 * LDS_ROW), 16, 0, 0);
  }
}

template <typename T>
__device__ __forceinline__ void compute_stage(const uint8_t* st, f32x16 (&acc)[4][4], int wm,
                                              int wn, int lane);

// bf16: four 16-deep k slices per stage.  Each slice runs half of its 16
// MFMAs, then issues the LDS reads of the next slice, then the other half, so
// the wait before a slice only covers reads issued about 256 cycles earlier.
// (sched_barrier pins that order; the scheduler would otherwise sink every
// read next to its first use.)
template <>
__device__ __forceinline__ void compute_stage<__bf16>(const uint8_t* st, f32x16 (&acc)[4][4],
                                                      int wm, int wn, int lane) {
  const int sw = row_swizzle(lane & 31);   // fragment rows start at multiples of 32
  const uint8_t* As = st + (wm * 128 + (lane & 31)) * LDS_ROW;
  const uint8_t* Bs = st + GBM * LDS_ROW + (wn * 128 + (lane & 31)) * LDS_ROW;
  bf16x8 a[2][4], b[2][4];
  auto load = [&](int kk, bf16x8(&fa)[4], bf16x8(&fb)[4]) {
    const int chunk = ((kk * 2 + (lane >> 5)) ^ sw) << 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = *(const bf16x8*)(As + i * 32 * LDS_ROW + chunk);
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = *(const bf16x8*)(Bs + j * 32 * LDS_ROW + chunk);
  };
  auto mfma_rows = [&](int kk, int i0) {
#pragma unroll
    for (int i = i0; i < i0 + 2; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk & 1][i], b[kk & 1][j], acc[i][j],
                                                            0, 0, 0);
  };
  load(0, a[0], b[0]);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    mfma_rows(kk, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (kk < 3) load(kk + 1, a[(kk + 1) & 1], b[(kk + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);
    mfma_rows(kk, 2);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <>
__device__ __forceinline__ void compute_stage<float>(const uint8_t* st, f32x16 (&acc)[4][4],
                                                     int wm, int wn, int lane) {
  const int sw = row_swizzle(lane & 31);   // fragment rows start at multiples of 32
  const uint8_t* As = st + (wm * 128 + (lane & 31)) * LDS_ROW;
  const uint8_t* Bs = st + GBM * LDS_ROW + (wn * 128 + (lane & 31)) * LDS_ROW;
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const int c0 = ((kk * 4 + (lane >> 5) * 2) ^ sw) << 4;
    const int c1 = ((kk * 4 + (lane >> 5) * 2 + 1) ^ sw) << 4;
    f32x4 a[4][2], b[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i][0] = *(const f32x4*)(As + i * 32 * LDS_ROW + c0);
      a[i][1] = *(const f32x4*)(As + i * 32 * LDS_ROW + c1);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      b[j][0] = *(const f32x4*)(Bs + j * 32 * LDS_ROW + c0);
      b[j][1] = *(const f32x4*)(Bs + j * 32 * LDS_ROW + c1);
    }
    // Lane l holds k = (l/32)*8 + e of this 16-wide slice in element e; MFMA e
    // pairs element e of both operands, so the 8 MFMAs cover all 16 k once.
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i][e >> 2][e & 3], b[j][e >> 2][e & 3],
                                                           acc[i][j], 0, 0, 0);
  }
}

template <typename T, class Epi>
__global__ void __launch_bounds__(GEMM_THREADS)
    __attribute__((amdgpu_waves_per_eu(1, 1))) gemm_nt_kernel(GemmShape g, Epi epi) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[GEMM_LDS];
  constexpr int BK = KStage<T>::BK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = g.m_dev ? *g.m_dev : g.M;
  const int N = g.n_dev ? *g.n_dev : g.N;
  const int K = g.k_dev ? cdiv(*g.k_dev, BK) * BK : g.K;
  if (M <= 0 || N <= 0) return;
  const int tiles_m = cdiv(M, GBM), tiles_n = cdiv(N, GBN);
  const int total = tiles_m * tiles_n;
  const int nk = K / BK;
  const uint8_t* A = (const uint8_t*)g.A;
  const uint8_t* B = (const uint8_t*)g.B;
  const int64_t lda_b = g.lda * (int64_t)sizeof(T), ldb_b = g.ldb * (int64_t)sizeof(T);

  for (int t = blockIdx.x; t < total; t += gridDim.x) {
    int tm, tn;
    map_tile(t, gridDim.x, total, tiles_m, tiles_n, g.group_m, tm, tn);
    const int m0 = tm * GBM, n0 = tn * GBN;
    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    if (nk > 0) {
      dma_stage(smem, A, lda_b, m0, M, B, ldb_b, n0, N, 0, wave, lane);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      for (int kt = 0; kt < nk; ++kt) {
        const uint8_t* cur = smem + (kt & 1) * STAGE_BYTES;
        if (kt + 1 < nk)
          dma_stage(smem + ((kt + 1) & 1) * STAGE_BYTES, A, lda_b, m0, M, B, ldb_b, n0, N,
                    (int64_t)(kt + 1) * BK * (int64_t)sizeof(T), wave, lane);
        compute_stage<T>(cur, acc, wm, wn, lane);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
      }
    }
    epi(acc, m0, n0, tn, M, N, smem, wm, wn, lane, tid);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// bf16 kernel.  Same tile, waves and swizzle as above, with a software
// pipeline tuned for one wave per SIMD:
//   * the per-lane global offsets of the stage copies are computed once per
//     tile (32-bit, relative to the tile's first row); each stage only moves a
//     scalar base, so a copy costs one instruction;
//   * every MFMA of a slice is paired with at most one LDS fragment read or
//     one stage copy (sched_barrier keeps that order), so the matrix pipe is
//     never left waiting behind a burst of memory instructions;
//   * (32 x 32 loop) the barrier of stage kt sits before its last 16-deep
//     slice: by then the slice's fragments are in registers, stage kt+1 has
//     landed and stage kt's buffer is free, so the last slice's MFMAs cover
//     the barrier, the reads of stage kt+1's first slice and the copies of
//     stage kt+2 into the freed buffer.  __syncthreads() is avoided because
//     it would also wait for the copies still in flight.
namespace bf16k {
constexpr int SK = 64;                        // k per stage
constexpr int ROW = SK * 2;                   // bytes per tile row per stage
constexpr int STAGE = (GBM + GBN) * ROW;      // 64 KiB
constexpr int HALF = GBM * ROW;               // one operand's part of a stage (32 KiB)
constexpr int NB = 2;                         // stage buffers
constexpr int KK = SK / 16;                   // 16-deep slices per stage
constexpr int RPI = 1024 / ROW;               // tile rows per copy instruction (8)
constexpr int IPW = 64 / RPI;                 // copy instructions per wave per operand (8)
constexpr int NCOPY = 2 * IPW;                // per wave per stage (16)
static_assert(NB * STAGE <= GEMM_LDS, "LDS");
static_assert((NB - 1) * HALF + 3 * 32 * ROW < 65536, "fragment offsets fit a DS immediate");
static_assert(NCOPY == 16, "one copy per MFMA of the last slice");
// Transposed A (a_trans).  The stage's A half holds 64 k-rows of the tile's 256
// rows of A, 512 bytes per k-row: the 64-byte window w (rows 32 w .. 32 w + 31)
// of k-row k sits at window w ^ (k & 3).  A fragment (rows 32-block i, k slice
// kk) is two transposing reads (ds_read_b64_tr_b16): within each 16-lane
// group, lane s supplies k-row (s >> 2) and rows 4 (s & 3) .. + 3, and lane
// 4a + b receives row 4a + b of k-rows 0..3 — in a 32-lane half the four k-rows
// land in four distinct 64-byte bank windows.
constexpr int TR_KROW = GBM * 2;                // bytes per k-row (512)
static_assert((NB - 1) * HALF + (KK - 1) * 16 * TR_KROW + 4 * TR_KROW < 65536,
              "transposed fragment offsets fit a DS immediate");
// Copy schedule.  The 16 copies of stage s are spread over the MFMAs that
// follow the barrier freeing their buffer: MFMA slot 0..15 is the last slice
// of stage s - 2, slots 16..63 are slices 0..2 of stage s - 1, and copy c
// (B rows first, then A rows) goes to slot c * CSTRIDE.  Issuing all 16
// copies of a wave against 16 MFMAs stalls issue when the memory pipeline is
// backed up, and a stalled wave leaves its matrix pipe idle; copies issued
// later have less time to land before stage s - 1's barrier.
constexpr int CSTRIDE = 2;
static_assert(CSTRIDE >= 1 && 15 * CSTRIDE < 48, "copy schedule");
__device__ __forceinline__ constexpr int copy_order(int c) { return (c + IPW) % NCOPY; }
constexpr int NEARLY = (15 / CSTRIDE) + 1;      // copies issued in slot 0..15
static_assert(NB == 2, "the vmcnt waits assume two stage buffers");

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// One 1 KiB global -> LDS copy (16 bytes per lane, LDS written contiguously
// from the wave-uniform byte address `lds`).  Issued as inline assembly on
// purpose: the compiler then does not see an in-flight LDS write, so it does
// not wait for the copy before later LDS reads of the other stage buffer
// (its alias analysis cannot tell the buffers apart and would serialise the
// prefetch).  The kernel orders copies and reads itself: vmcnt wait + barrier
// before a buffer is read, barrier before it is refilled.  Nothing else in
// these kernels uses M0.
template <uint32_t LDS_OFF>
__device__ __forceinline__ void copy16(const void* base, uint32_t off, uint32_t lds) {
  // scalar base + 32-bit per-lane offset: no 64-bit address arithmetic per copy;
  // M0 = lds + LDS_OFF in one scalar add
  asm volatile("s_add_u32 m0, %2, %3\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base),
               "s"(lds), "n"(LDS_OFF)
               : "memory");
}

// 16 x 16 x 32 loop: what rides along with MFMA slot q of a stage (slot
// q = 16 i + 2 j + kk is block (i, j), slice kk).  Copy c of the stage after
// next in slot CS c (even slots, spread over the stage: a burst of copies
// stalls issue when the memory pipeline is backed up, and the wave's matrix
// pipe waits with it).  The next stage's fragments are read in the odd slots
// of the second half only: a wait for the copies of the next stage and a
// barrier sit before slot 64, so a copy has until the middle of the stage
// after the one that issued it to land.  A rows 4..6 are replaced in place,
// two slots after row i's last MFMA; the other odd slots from 65 on carry the
// 16 B fragments, then A rows 0..3, then row 7 (into the spare set).
constexpr int MF16_NONE = -1, MF16_COPY = 0, MF16_BREAD = 16, MF16_AREAD = 32;
constexpr int MF16_MID = 64;   // slot of the mid-stage wait and barrier
__device__ __forceinline__ constexpr bool mf16_inplace_slot(int q) {
  return (q & 1) == 1 && q >= 81 && (q - 81) % 16 < 4 && (q - 81) / 16 < 3;
}
// rank of odd slot q >= 65 among those not taken by the in-place rows (-1: none)
__device__ __forceinline__ constexpr int mf16_late_rank(int q) {
  if ((q & 1) == 0 || q <= MF16_MID || mf16_inplace_slot(q)) return -1;
  int n = 0;
  for (int p = MF16_MID + 1; p < q; p += 2)
    if (!mf16_inplace_slot(p)) ++n;
  return n;
}
// SPLIT (transposed A, whose fragments take two LDS reads each): the B
// fragments come first, in the odd slots 33..63 behind a wait for the next
// stage's B copies (a stage issues B's copies before A's) at slot 32, so that
// the second half carries only A's reads.
constexpr int MF16_MID_B = 32;   // slot of the wait for B's copies (SPLIT)
// CS: slots between two copies (even, so that copies never share a slot with
// a fragment read)
template <int CS, bool SPLIT = false>
__device__ __forceinline__ constexpr int mf16_slot(int q) {
  static_assert(CS % 2 == 0 && 15 * CS < 128, "copy spacing");
  if (q < 16 * CS && q % CS == 0) return MF16_COPY + q / CS;
  if (mf16_inplace_slot(q)) return MF16_AREAD + 8 + 2 * ((q - 81) / 16) + ((q - 81) % 16) / 2;
  if (SPLIT) {
    if ((q & 1) == 1 && q > MF16_MID_B && q < MF16_MID) return MF16_BREAD + (q - MF16_MID_B) / 2;
    const int r = mf16_late_rank(q);
    if (r >= 0 && r < 8) return MF16_AREAD + r;
    if (r >= 8 && r < 10) return MF16_AREAD + 14 + (r - 8);
    return MF16_NONE;
  }
  const int r = mf16_late_rank(q);
  if (r >= 0 && r < 16) return MF16_BREAD + r;
  if (r >= 16 && r < 24) return MF16_AREAD + (r - 16);
  if (r >= 24 && r < 26) return MF16_AREAD + 14 + (r - 24);
  return MF16_NONE;
}
// copies a wave issues in a stage before slot q
template <int CS>
__device__ __forceinline__ constexpr int mf16_copies_before(int q) {
  return (q - 1) / CS + 1 < 16 ? (q - 1) / CS + 1 : 16;
}
// every fragment of the next stage is read exactly once, after the wait for
// its copies
template <int CS, bool SPLIT = false>
__device__ __forceinline__ constexpr bool mf16_schedule_ok() {
  int reads[32] = {}, copies[16] = {};
  for (int q = 0; q < 128; ++q) {
    const int op = mf16_slot<CS, SPLIT>(q);
    if (op >= MF16_COPY && op < MF16_COPY + 16) ++copies[op - MF16_COPY];
    if (op >= MF16_BREAD && op < MF16_AREAD + 16) {
      if (q <= (SPLIT && op < MF16_AREAD ? MF16_MID_B : MF16_MID)) return false;
      ++reads[op - MF16_BREAD];
    }
    // an in-place A row only after the last MFMA of that row
    if (op >= MF16_AREAD && op < MF16_AREAD + 14 && q < 16 * ((op - MF16_AREAD) >> 1) + 17) return false;
  }
  for (int n = 0; n < 32; ++n)
    if (reads[n] != 1) return false;
  for (int n = 0; n < 16; ++n)
    if (copies[n] != 1) return false;
  return true;
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
__device__ __forceinline__ bf16x4 read_tr(const uint8_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
}

}  // namespace bf16k

// f(std::integral_constant<int, 0>{}), ..., f(std::integral_constant<int, N - 1>{})
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// The lane index computed afresh (from the exec mask, not from threadIdx.x), so
// that quantities derived from it are formed where they are used instead of
// being hoisted out of loops into spill slots
__device__ __forceinline__ int fresh_lane() {
  int v;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(v));
  return v;
}

// Barrier that orders LDS accesses only: unlike __syncthreads() it does not
// wait for this wave's global stores to complete.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Up to two independent problems in one launch (the backward's dH and dW).
template <class Epi>
struct GemmBatch {
  GemmShape g[2];
  Epi e[2];
  int32_t n;          // number of problems
  int32_t* queue;     // 8 tile counters, then 8 finished-tile counters, zero at launch
};

// Copy schedule of the 16 x 16 loop, per epilogue (measured on the 32B-shaped
// workload): MFMA slots between two stage copies, whether A's copies go before
// B's, and whether odd rounds of tiles sweep K backwards (a round then starts
// on the operand chunks the previous round of its XCD read last: 2% faster for
// the long-K dH + dW tiles, while the forward and recompute gained nothing and
// their L2 hit rate dropped).
struct EpiLseCols;
struct EpiStore;
template <class Epi>
struct CopySched {
  static constexpr int spacing = 6;
  static constexpr bool a_first = false;
  static constexpr bool serpentine = false;
  static constexpr bool round_sync = false;
};
template <>
struct CopySched<EpiLseCols> {
  static constexpr int spacing = 8;
  static constexpr bool a_first = false;
  static constexpr bool serpentine = false;
  static constexpr bool round_sync = false;
};
template <>
struct CopySched<EpiStore> {
  static constexpr int spacing = 8;
  static constexpr bool a_first = false;
  static constexpr bool serpentine = true;
  static constexpr bool round_sync = true;
};
constexpr int ROUND_SLACK = 2;   // tiles of the earlier rounds that may still run
constexpr int ROUND_SPIN = 32;   // polls of the finished-tile counter (~0.3 us apart)

// Tile scheduling.  Workgroups are dealt round-robin to the 8 XCDs, so
// workgroup b serves queue b % nq (nq = 8, fewer for a small grid).  A
// problem's tiles are ordered 8 row tiles deep, column-major inside a group,
// and cut into rounds of 32 nq tiles; queue q owns slots [32 q, 32 q + 32) of
// every round (the final partial round is dealt round-robin).  So at any time
// all XCDs work on the same few row panels (shared through the Infinity
// Cache) and each XCD on a compact 8 x 4 block of tiles (shared through its
// L2), while the workgroups of a queue take its tiles with an atomic counter
// and balance tiles of unequal length.  Problem 0's tiles come first.  A
// workgroup whose queue is empty takes the remaining tiles of the others.
__device__ __forceinline__ void grouped_tile(int L, int tiles_m, int tiles_n, int group_m,
                                             int& tm, int& tn) {
  const int width = group_m * tiles_n;
  const int grp = L / width;
  const int first = grp * group_m;
  const int gsz = min(tiles_m - first, group_m);
  const int rem = L - grp * width;
  tm = first + rem % gsz;
  tn = rem / gsz;
}

struct QueueShare {
  int full;     // tiles of this queue in the full rounds
  int len;      // all tiles of this queue
};

__device__ __forceinline__ QueueShare queue_share(int total, int q, int nq) {
  const int round = 32 * nq;
  const int rounds = total / round;
  const int tail = total - rounds * round;
  QueueShare s;
  s.full = 32 * rounds;
  s.len = s.full + (tail > q ? (tail - q + nq - 1) / nq : 0);
  return s;
}

// k-th tile of queue q -> tile index in the problem's order
__device__ __forceinline__ int queue_tile(int k, const QueueShare& s, int q, int nq) {
  if (k < s.full) return (k >> 5) * (32 * nq) + 32 * q + (k & 31);
  return (s.full / 32) * (32 * nq) + (k - s.full) * nq + q;
}

// EVEN: every problem's K is a multiple of 2 stages (a device-read K is rounded
// up to one, the operands being zero-padded that far); such launches run the
// 16 x 16 loop (MF16), whose stage pairs know their buffers at compile time, so
// every LDS address of the loop is a base register plus an immediate.  Other
// launches (a hidden size that is not a multiple of 128) run the 32 x 32 loop on
// row-major operands.  ATR: a problem may read A transposed out of stage-tiled
// storage (GemmShape::a_trans; 16 x 16 loop only).
template <class Epi, bool EVEN, bool ATR, bool MF16 = false>
__global__ void __launch_bounds__(GEMM_THREADS)
    __attribute__((amdgpu_waves_per_eu(1, 1))) gemm_bf16_kernel(GemmBatch<Epi> bat) {
  static_assert(MF16 == EVEN, "stage-pair launches run the 16 x 16 loop, the others the 32 x 32 loop");
  static_assert(!ATR || MF16, "transposed A in the 16 x 16 loop only");
  using namespace bf16k;
  __shared__ __attribute__((aligned(16))) uint8_t smem[BF16_KERNEL_LDS];
  __shared__ int s_tile[2];   // claimed tile (-1: none left) and its queue
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int nq = min(8, (int)gridDim.x);
  const int qi = blockIdx.x % nq;
  int Mp[2], Np[2], Kp[2], tmp[2], tnp[2], totp[2];
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const GemmShape& gp = bat.g[p];
    // device-read sizes are the same in every lane; keep them scalar (see below)
    Mp[p] = __builtin_amdgcn_readfirstlane(gp.m_dev ? *gp.m_dev : gp.M);
    Np[p] = __builtin_amdgcn_readfirstlane(gp.n_dev ? *gp.n_dev : gp.N);
    constexpr int KR = EVEN ? 2 * SK : SK;
    Kp[p] = __builtin_amdgcn_readfirstlane(gp.k_dev ? cdiv(*gp.k_dev, KR) * KR : gp.K);
    tmp[p] = cdiv(Mp[p], GBM);
    tnp[p] = cdiv(Np[p], GBN);
    totp[p] = (p < bat.n && Mp[p] > 0 && Np[p] > 0) ? tmp[p] * tnp[p] : 0;
  }

  // fragment reads: lane l reads row (l & 31) of each 32-row block, chunk
  // 2 kk + l / 32 of slice kk.  LDS holds the A halves of the two stage buffers
  // first, then the B halves, so a read's buffer and block are an offset of at
  // most 45 KiB from a per-slice base.
  const int frow = lane & 31;
  const int fsw = row_swizzle(frow);
  int ra[KK], rb[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const int chk = ((kk * 2 + (lane >> 5)) ^ fsw) << 4;
    ra[kk] = (wm * 128 + frow) * ROW + chk;
    rb[kk] = NB * HALF + (wn * 128 + frow) * ROW + chk;
  }
  // LDS byte address of the stage buffers
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void_t*)smem);

  // Tiles come from the queue of this workgroup's XCD until it runs dry, then
  // from the other queues in turn (cq: the first queue the next claim tries).
  // The XCDs do not run at one clock under the power limit (up to 9% apart on
  // one chip), so without this the slowest XCD's share sets the launch time.
  // A counter only grows, so a queue found empty stays empty, and a workgroup
  // leaves after one claim per queue has come back empty.
  int cq = qi, done_q = -1;
  for (;;) {
    if (wave == 0 && fresh_lane() == 0) {
      if (CopySched<Epi>::round_sync && done_q >= 0) atomicAdd(bat.queue + 8 + done_q, 1);
      int q = cq, k = -1;
      for (int n = 0; n < nq; ++n) {
        const int len = queue_share(totp[0], q, nq).len + queue_share(totp[1], q, nq).len;
        const int c = atomicAdd(bat.queue + q, 1);
        if (c < len) {
          k = c;
          break;
        }
        q = q + 1 == nq ? 0 : q + 1;
      }
      if constexpr (CopySched<Epi>::round_sync) {
        // a tile of a full round starts once all but a few tiles of the queue's
        // earlier rounds of the same problem have finished (bounded wait)
        if (k >= 0) {
          const QueueShare s0 = queue_share(totp[0], q, nq), s1 = queue_share(totp[1], q, nq);
          int target = 0;
          if (k < s0.full)
            target = k & ~31;
          else if (k >= s0.len && k - s0.len < s1.full)
            target = s0.full + ((k - s0.len) & ~31);
          target -= ROUND_SLACK;
          for (int it = 0; it < ROUND_SPIN && target > 0 &&
                           __hip_atomic_load(bat.queue + 8 + q, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT) < target;
               ++it)
            __builtin_amdgcn_s_sleep(8);
        }
      }
      s_tile[0] = k;
      s_tile[1] = q;
    }
    __syncthreads();
    // the same value in every lane: make it a scalar, otherwise every quantity
    // derived from it (loop bounds, the copies' LDS base in M0) is treated as
    // divergent and each copy becomes a waterfall loop
    const int t = __builtin_amdgcn_readfirstlane(s_tile[0]);
    if (t < 0) break;
    cq = __builtin_amdgcn_readfirstlane(s_tile[1]);
    done_q = cq;
    QueueShare sh[2];
    sh[0] = queue_share(totp[0], cq, nq);
    sh[1] = queue_share(totp[1], cq, nq);
    const int p = t < sh[0].len ? 0 : 1;
    const GemmShape g = p ? bat.g[1] : bat.g[0];
    const Epi epi = p ? bat.e[1] : bat.e[0];
    const int M = p ? Mp[1] : Mp[0];
    const int N = p ? Np[1] : Np[0];
    const int nk = (p ? Kp[1] : Kp[0]) / SK;
    int tm, tn;
    const int L = p ? queue_tile(t - sh[0].len, sh[1], cq, nq) : queue_tile(t, sh[0], cq, nq);
    if (g.group_cols)
      grouped_tile(L, p ? tnp[1] : tnp[0], p ? tmp[1] : tmp[0], g.group_m, tn, tm);
    else
      grouped_tile(L, p ? tmp[1] : tmp[0], p ? tnp[1] : tnp[0], g.group_m, tm, tn);
    const int64_t lda_b = g.lda * 2, ldb_b = g.ldb * 2;
    const int m0 = tm * GBM, n0 = tn * GBN;
    const bool atr = ATR && g.a_trans;
    // where a tile starts and how far a stage advances.  Row-major: the tile's
    // first row, 128 bytes.  Stage-tiled, row-block order: the tile's first
    // 32 KiB block, one block.  Column-block order: the same, ld / 256 blocks.
    // Transposed A: the tile's first block column, 64 k-rows of 128 bytes.
    auto place = [&](int tiled, int64_t ld, int64_t ld_b, int t, int r0, int64_t& off,
                     int64_t& ks) {
      if (tiled == 2) {
        off = (int64_t)t * HALF;
        ks = (ld >> 8) * HALF;
      } else if (tiled) {
        off = (int64_t)t * (ld >> 6) * HALF;
        ks = HALF;
      } else {
        off = (int64_t)r0 * ld_b;
        ks = ROW;
      }
    };
    int64_t a_off, a_ks, b_off, b_ks;
    if (atr) {
      a_off = (int64_t)tm * 4 * (g.lda >> 8) * HALF;
      a_ks = SK * ROW;
    } else {
      place(g.a_tiled, g.lda, lda_b, tm, m0, a_off, a_ks);
    }
    place(g.b_tiled, g.ldb, ldb_b, tn, n0, b_off, b_ks);
    // serpentine K (16 x 16 loop): odd rounds of the problem's tile order copy
    // the stages last to first
    if (MF16 && CopySched<Epi>::serpentine && ((L / (32 * nq)) & 1)) {
      a_off += (int64_t)(nk - 1) * a_ks;
      b_off += (int64_t)(nk - 1) * b_ks;
      a_ks = -a_ks;
      b_ks = -b_ks;
    }
    const uint8_t* a_base = (const uint8_t*)g.A + a_off;
    const uint8_t* b_base = (const uint8_t*)g.B + b_off;
    // copy q < 8 moves A rows [64 wave + 8 q, +8), q >= 8 the same rows of B;
    // lane i fetches chunk (i & 7) ^ swizzle(row) of row i / 8 (row-major: clamped
    // to the last valid row, those products are discarded by the epilogue;
    // stage-tiled: the chunk is already in place, the copy is 1 KiB contiguous)
    // (the lane index is re-read here: lane-derived constants hoisted out of the
    // tile loop end up in spill slots, and every reload is a round trip to memory
    // that the streaming operands have evicted from the caches)
    const int ln = fresh_lane();
    uint32_t offa[IPW], offb[IPW];
#pragma unroll
    for (int b = 0; b < IPW; ++b) {
      const int row = wave * 64 + b * RPI + (ln >> 3);
      const int ch = ((ln & 7) ^ row_swizzle(row)) << 4;
      offa[b] = g.a_tiled ? (uint32_t)(row * ROW + (ln & 7) * 16)
                          : (uint32_t)(min(row, M - 1 - m0) * lda_b + ch);
      offb[b] = g.b_tiled ? (uint32_t)(row * ROW + (ln & 7) * 16)
                          : (uint32_t)(min(row, N - 1 - n0) * ldb_b + ch);
    }
    if (atr) {
      // transposed A: copy b of a wave fills k-rows 16 wave + 2 b, + 1 (the
      // same LDS bytes as above); lane i lands in physical 16-byte chunk i & 31
      // of its k-row, which holds rows 32 w + 8 (i & 3) .. + 7 of window
      // w = ((i & 31) >> 2) ^ (k-row & 3).  In the source those rows are a
      // 16-byte chunk of k-row (token) 64 s + kr of block column w / 2.
#pragma unroll
      for (int b = 0; b < IPW; ++b) {
        const int kr = wave * 16 + 2 * b + (ln >> 5);
        const int p = ln & 31;
        const int w = (p >> 2) ^ (kr & 3);
        // the 32-byte halves of a window are swapped when bit 3 of the k-row is
        // set, so lane i holds rows 32 w + 16 hf + 8 (i & 1) .. + 7
        const int c16 = (w & 1) * 4 + ((((p >> 1) & 1) ^ ((kr >> 3) & 1)) << 1) + (p & 1);
        // (lda <= 2^23 rows: at most 3 * 2^15 blocks of 32 KiB, within 32 bits)
        offa[b] = (uint32_t)((w >> 1) * (uint32_t)((g.lda >> 8) * HALF) + kr * ROW +
                             ((c16 ^ ((kr >> 1) & 7)) << 4));
      }
    }

    // (the LDS address is formed from scalars only, so it stays in SGPRs)
    // copy Q of stage s into stage buffer BUF (or buf when BUF < 0): the LDS
    // address is a scalar base plus a constant of the copy site
    const uint32_t lds_w = lds0 + (uint32_t)(wave * 64 * ROW);
    auto copy = [&](int s, auto q_c, auto buf_c, int buf) {
      constexpr int Q = decltype(q_c)::value;
      constexpr int BUF = decltype(buf_c)::value;
      constexpr uint32_t b = Q % IPW;
      constexpr uint32_t fixed = BUF >= 0 ? (uint32_t)BUF * HALF : 0u;
      const uint32_t base = BUF >= 0 ? lds_w : lds_w + (uint32_t)(buf * HALF);
      if constexpr (Q < IPW)
        copy16<fixed + b * RPI * ROW>(a_base + s * a_ks, offa[b], base);
      else
        copy16<NB * HALF + fixed + b * RPI * ROW>(b_base + s * b_ks, offb[b], base);
    };
    // q is a constant at every call site once the loops are unrolled
    auto copy_q = [&](int s, int q, auto buf_c, int buf) {
      static_assert(NCOPY == 16, "one case per copy");
      switch (q) {
        case 0: copy(s, std::integral_constant<int, 0>{}, buf_c, buf); break;
        case 1: copy(s, std::integral_constant<int, 1>{}, buf_c, buf); break;
        case 2: copy(s, std::integral_constant<int, 2>{}, buf_c, buf); break;
        case 3: copy(s, std::integral_constant<int, 3>{}, buf_c, buf); break;
        case 4: copy(s, std::integral_constant<int, 4>{}, buf_c, buf); break;
        case 5: copy(s, std::integral_constant<int, 5>{}, buf_c, buf); break;
        case 6: copy(s, std::integral_constant<int, 6>{}, buf_c, buf); break;
        case 7: copy(s, std::integral_constant<int, 7>{}, buf_c, buf); break;
        case 8: copy(s, std::integral_constant<int, 8>{}, buf_c, buf); break;
        case 9: copy(s, std::integral_constant<int, 9>{}, buf_c, buf); break;
        case 10: copy(s, std::integral_constant<int, 10>{}, buf_c, buf); break;
        case 11: copy(s, std::integral_constant<int, 11>{}, buf_c, buf); break;
        case 12: copy(s, std::integral_constant<int, 12>{}, buf_c, buf); break;
        case 13: copy(s, std::integral_constant<int, 13>{}, buf_c, buf); break;
        case 14: copy(s, std::integral_constant<int, 14>{}, buf_c, buf); break;
        case 15: copy(s, std::integral_constant<int, 15>{}, buf_c, buf); break;
        default: break;
      }
    };
    using BUF_RT = std::integral_constant<int, -1>;

    if constexpr (MF16) {
      // 16 x 16 x 32 loop.  acc[i][j] is the 16 x 16 block (i, j) of the wave's
      // 128 x 128 sub-tile: lane l holds column 16 j + (l & 15), rows 16 i +
      // 4 (l >> 4) .. + 3.  A stage is two 32-deep slices; the MFMAs of a stage
      // run rows i = 0..7, columns j = 0..7, and the two slices of block (i, j)
      // back to back (the second accumulates onto the first).  The stage's
      // fragments are in registers before it starts: fa[i][kk] (A, replaced in
      // place by the next stage's row i once row i's MFMAs are issued; row 7 of
      // odd stages lives in fa7) and fb[P][j][kk] (B, two sets by stage parity).
      // Two barriers per stage: at its start every wave is done reading this
      // stage's buffer, which the copies of the stage after next then refill;
      // before slot 64 the next stage has landed, and its fragments are read
      // in the second half.
      // one accumulator set and one epilogue for both operand modes (TR: A
      // read transposed); only the main loop is instantiated per mode
      f32x4 acc[8][8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      auto loop16 = [&](auto tr_c) {
      constexpr bool TR = decltype(tr_c)::value;
      {
        // lane l reads row l & 15 of each 16-row block, 16-byte chunk
        // 4 kk + (l >> 4) of slice kk; the row swizzle depends on the row within
        // the block only, so a block is an immediate offset of 2 KiB.
        // Transposed A: the stage's A half holds 64 k-rows of 512 bytes; the
        // 64-byte window w (rows 32 w .. + 31) of k-row k sits at w ^ (k & 3)
        // and its 32-byte halves are swapped when bit 3 of k is set.  Block i
        // of slice kk is two transposing reads (ds_read_b64_tr_b16): in 16-lane
        // group g, lane s supplies k-row 32 kk + 8 g + (s >> 2) (+ 4 for the
        // second read) and rows 4 (s & 3) .. + 3 of the block, and lane s
        // receives row s of those 4 k-rows.  A 32-lane half touches 8 k-rows,
        // spread over 4 bank windows by (k & 3) and 2 halves by bit 3 of k.
        const int l16 = fresh_lane();
        const int fr = l16 & 15;
        int ra16[2], rb16[2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int chk = ((kk * 4 + (l16 >> 4)) ^ row_swizzle(fr)) << 4;
          ra16[kk] = (wm * 128 + fr) * ROW + chk;
          rb16[kk] = NB * HALF + (wn * 128 + fr) * ROW + chk;
        }
        // block i's transposed read: ta16 ^ (64 (i >> 1) + 32 (i & 1)) (the
        // window and half bits of ta16 hold the lane's XOR pattern; the block's
        // bits go in by one XOR per read instead of eight live addresses)
        int ta16 = 0;
        if constexpr (TR) {
          const int g = l16 >> 4, q4 = (l16 >> 2) & 3;
          ta16 = (8 * g + q4) * TR_KROW + 4 * wm * 64 + (q4 << 6) + ((g & 1) << 5) + 8 * (l16 & 3);
        }
        auto rd_a = [&](int i, int kk, int buf) {
          if constexpr (TR) {
            const uint8_t* p = smem + (ta16 ^ ((i >> 1) << 6 | (i & 1) << 5)) + buf * HALF +
                               kk * 32 * TR_KROW;
            bf16x8 v;
            v.lo = read_tr(p);
            v.hi = read_tr(p + 4 * TR_KROW);
            return v;
          } else {
            return *(const bf16x8*)(smem + ra16[kk] + buf * HALF + i * 16 * ROW);
          }
        };
        auto rd_b = [&](int j, int kk, int buf) {
          return *(const bf16x8*)(smem + rb16[kk] + buf * HALF + j * 16 * ROW);
        };
        // stages 0 and 1 whole (stage 1 in the loop's copy order, which the
        // first stage's waits assume)
#pragma unroll
        for (int q = 0; q < NCOPY; ++q) copy_q(0, q, std::integral_constant<int, 0>{}, 0);
#pragma unroll
        for (int q = 0; q < NCOPY; ++q)
          copy_q(1, CopySched<Epi>::a_first ? q : copy_order(q), std::integral_constant<int, 1>{}, 1);
        wait_vmcnt<NCOPY>();        // stage 0 landed (stage pairs: nk >= 2)
        __builtin_amdgcn_s_barrier();
        using P0 = std::integral_constant<int, 0>;
        using P1 = std::integral_constant<int, 1>;
        // stage 0's fragments
        bf16x8 fa[8][2], fa7[2], fb[2][8][2];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk) {
            fa[i][kk] = rd_a(i, kk, 0);
            fb[0][i][kk] = rd_b(i, kk, 0);
          }
        // Every stage runs the same code (one register assignment for the whole
        // loop): the last two stages copy the last stage again into the buffer
        // they free (its data is in registers already, nothing reads it again),
        // and the last stage reads stale fragments of a stage that does not
        // exist; both stay within the operands and the LDS.
        auto stage16 = [&](int kt, auto par_c) {
          constexpr int P = decltype(par_c)::value;            // kt % 2
          using PC = std::integral_constant<int, P>;
          constexpr int CS = CopySched<Epi>::spacing;
          constexpr bool SPLIT = TR;
          static_assert(mf16_schedule_ok<CS, SPLIT>(), "16 x 16 slot schedule");
          static_assert(!SPLIT || !CopySched<Epi>::a_first, "B's copies go first");
          const int kc = min(kt + 2, nk - 1);                  // stage to copy
          // every wave has read its fragments of this stage's buffer, which the
          // copies below refill
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
          // (every index below is a compile-time constant, so that the
          // fragment and accumulator arrays stay in registers)
          static_for<128>([&](auto q_c) {
            constexpr int q = decltype(q_c)::value;
            constexpr int i = q >> 4, j = (q >> 1) & 7, kk = q & 1;
            constexpr int op = mf16_slot<CS, SPLIT>(q);
            if constexpr (SPLIT && q == MF16_MID_B) {
              // stage kt + 1's B half landed: this wave's first 8 copies of the
              // previous stage, before its 8 A copies and this stage's copies
              wait_vmcnt<8 + mf16_copies_before<CS>(MF16_MID_B)>();
              __builtin_amdgcn_s_barrier();
              __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (q == MF16_MID) {
              // stage kt + 1 landed: this wave's copies of it are all but the
              // ones issued so far in this stage, then the other waves'
              wait_vmcnt<mf16_copies_before<CS>(MF16_MID)>();
              __builtin_amdgcn_s_barrier();
              __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (i == 7 && P == 1)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa7[kk], fb[P][j][kk], acc[i][j],
                                                                  0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i][kk], fb[P][j][kk],
                                                                  acc[i][j], 0, 0, 0);
            if constexpr (op >= MF16_COPY && op < MF16_COPY + 16) {
              constexpr int c = op - MF16_COPY;
              copy_q(kc, CopySched<Epi>::a_first ? c : copy_order(c), PC{}, P);
            } else if constexpr (op >= MF16_BREAD && op < MF16_BREAD + 16) {
              constexpr int n = op - MF16_BREAD;
              fb[P ^ 1][n >> 1][n & 1] = rd_b(n >> 1, n & 1, P ^ 1);
            } else if constexpr (op >= MF16_AREAD && op < MF16_AREAD + 16) {
              constexpr int n = op - MF16_AREAD, ia = n >> 1, ka = n & 1;
              // the next stage's row 7 goes to the set this stage does not use
              if constexpr (ia == 7 && P == 0)
                fa7[ka] = rd_a(7, ka, P ^ 1);
              else
                fa[ia][ka] = rd_a(ia, ka, P ^ 1);
            }
            __builtin_amdgcn_sched_barrier(0);
          });
        };
        for (int kt = 0; kt < nk; kt += 2) {
          stage16(kt, P0{});
          stage16(kt + 1, P1{});
        }
      }
      };
      if (nk > 0) {
        if constexpr (ATR) {
          if (atr)
            loop16(std::true_type{});
          else
            loop16(std::false_type{});
        } else {
          loop16(std::false_type{});
        }
      }
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      __syncthreads();
      {
        const int lane_e = fresh_lane();
        epi.tile16(acc, m0, n0, tn, M, N, smem, wm, wn, lane_e, wave * 64 + lane_e);
      }
    } else {
      f32x16 acc[4][4];
  #pragma unroll
      for (int i = 0; i < 4; ++i)
  #pragma unroll
        for (int j = 0; j < 4; ++j)
  #pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

      if (nk > 0) {
        // stage 0 whole; stage 1's slot 0..15 copies (stage 0 issues the rest)
  #pragma unroll
        for (int q = 0; q < NCOPY; ++q) copy_q(0, q, std::integral_constant<int, 0>{}, 0);
        if (nk > 1) {
  #pragma unroll
          for (int c = 0; c < NEARLY; ++c)
            copy_q(1, copy_order(c), std::integral_constant<int, 1>{}, 1);
          wait_vmcnt<NEARLY>();      // stage 0 landed
        } else {
          wait_vmcnt<0>();
        }
        __builtin_amdgcn_s_barrier();
        // the fragment read paired with MFMA q of a slice (slice kn, buffer
        // offset off): A blocks first, then B
        auto frag = [&](int q, int kn, int off, bf16x8 (&fan)[4], bf16x8 (&fbn)[4]) {
          if (q < 4)
            fan[q] = *(const bf16x8*)(smem + ra[kn] + off + q * 32 * ROW);
          else if (q < 8)
            fbn[q - 4] = *(const bf16x8*)(smem + rb[kn] + off + (q - 4) * 32 * ROW);
        };
        bf16x8 fa[2][4], fb[2][4];
  #pragma unroll
        for (int q = 0; q < 16; ++q) frag(q, 0, 0, fa[0], fb[0]);

        // stage kt reads buffer kt % NB
        auto stage = [&](int kt, auto refill_c, auto more_c) {
          constexpr bool REFILL = decltype(refill_c)::value;   // copy stage kt + NB
          constexpr bool MORE = decltype(more_c)::value;       // stage kt + 1 exists
          const int pr = kt % NB;
          const int cur_off = pr * HALF, nxt_off = (pr ^ 1) * HALF;
          __builtin_amdgcn_sched_barrier(0);
  #pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            const int cur = kk & 1, nxt = cur ^ 1;
            if (kk == KK - 1) {
              if constexpr (MORE) {
                // stage kt+1 landed (its copies are the only ones in flight)
                wait_vmcnt<0>();
              }
              asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
              __builtin_amdgcn_s_barrier();
              __builtin_amdgcn_sched_barrier(0);
            }
  #pragma unroll
            for (int q = 0; q < 16; ++q) {
              const int i = q >> 2, j = q & 3;
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[cur][i], fb[cur][j], acc[i][j],
                                                                  0, 0, 0);
              if (kk < KK - 1) {
                frag(q, kk + 1, cur_off, fa[nxt], fb[nxt]);
                if constexpr (MORE) {
                  const int slot = 16 * (kk + 1) + q;
                  if (slot % CSTRIDE == 0 && slot / CSTRIDE < NCOPY)
                    copy_q(kt + 1, copy_order(slot / CSTRIDE), BUF_RT{}, pr ^ 1);
                }
              } else {
                if constexpr (MORE) frag(q, 0, nxt_off, fa[nxt], fb[nxt]);
                if constexpr (REFILL) {
                  if (q % CSTRIDE == 0) copy_q(kt + NB, copy_order(q / CSTRIDE), BUF_RT{}, pr);
                }
              }
              __builtin_amdgcn_sched_barrier(0);
            }
          }
        };
        using T_ = std::true_type;
        using F_ = std::false_type;
        int kt = 0;
        for (; kt + NB < nk; ++kt) stage(kt, T_{}, T_{});
        for (; kt + 1 < nk; ++kt) stage(kt, F_{}, T_{});
        stage(kt, F_{}, F_{});
      }
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
      __syncthreads();
      {
        const int lane_e = fresh_lane();
        epi.tile(acc, m0, n0, tn, M, N, smem, wm, wn, lane_e, wave * 64 + lane_e);
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Epilogues.  Each receives the finished accumulators of one tile.

// Reductions over the 32 lanes of a half-wave (lanes l and l ^ 16, l ^ 8, ...):
// four DPP steps inside each 16-lane row (xor 1, xor 2 by quad permutes, then
// the half-row and row mirrors, which pair lanes whose partial results are
// already uniform within their quad / half-row), then one swizzle across the
// two rows.  Every lane of the half-wave ends with the result.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                0xF, 0xF, false));
}
__device__ __forceinline__ float swz_xor16(float v) {
  // ds_swizzle bit mode, 32-lane groups: and 0x1F, or 0, xor 0x10
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}
__device__ __forceinline__ float half_wave_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));    // quad_perm(1,0,3,2): lane ^ 1
  v = fmaxf(v, dpp<0x4E>(v));    // quad_perm(2,3,0,1): lane ^ 2
  v = fmaxf(v, dpp<0x141>(v));   // row_half_mirror: lane i <-> 7 - i within 8
  v = fmaxf(v, dpp<0x140>(v));   // row_mirror: lane i <-> 15 - i within 16
  return fmaxf(v, swz_xor16(v));
}
__device__ __forceinline__ float half_wave_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  return v + swz_xor16(v);
}

// Forward: per row of the tile, the max and the sum of exp(z - max) over the
// tile's vocabulary columns (z = acc / temperature), plus the target logit.
// A wave reduces its 128 columns for the 16 rows of one accumulator block at
// a time: 16 independent reduction chains keep the DPP steps free of
// read-after-write stalls.  With scale > 0, max z = scale * max acc and
// exp(z - m) = exp2(acc * scale * log2(e) - max acc * scale * log2(e)).
struct EpiLsePartial {
  const int32_t* y;      // [rows] target id of each compacted row
  f32x2* part;           // [tiles_n][ld_part] (max, sum exp) per row and vocabulary tile
  int64_t ld_part;
  float* zy;             // [rows] logit of the target token
  float scale;           // 1 / temperature

  template <bool FULL, int i>
  __device__ __forceinline__ void block(const f32x16 (&acc)[4][4], int n0, int N,
                                        const int* sy, f32x2* red, int m0, int wm, int wn,
                                        int lane) const {
    const float k1 = scale * 1.44269504088896341f;
    bool ok[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) ok[j] = FULL || n0 + acc_col(wn, j, lane) < N;
    float mx[16], sm[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float a[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) a[j] = ok[j] ? acc[i][j][r] : -INFINITY;
      mx[r] = fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], dpp<0xB1>(mx[r]));
#pragma unroll
    for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], dpp<0x4E>(mx[r]));
#pragma unroll
    for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], dpp<0x141>(mx[r]));
#pragma unroll
    for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], dpp<0x140>(mx[r]));
#pragma unroll
    for (int r = 0; r < 16; ++r) mx[r] = fmaxf(mx[r], swz_xor16(mx[r]));
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      // a half-row beyond the vocabulary has max -inf: its sum is 0
      const float mk = FULL || mx[r] != -INFINITY ? -mx[r] * k1 : 0.0f;
      float t = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float e = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], k1, mk));
        t += FULL || ok[j] ? e : 0.0f;
      }
      sm[r] = t;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) sm[r] += dpp<0xB1>(sm[r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) sm[r] += dpp<0x4E>(sm[r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) sm[r] += dpp<0x141>(sm[r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) sm[r] += dpp<0x140>(sm[r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) sm[r] += swz_xor16(sm[r]);
    if ((lane & 31) == 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[wn * GBM + acc_row(wm, i, r, lane)] = f32x2{mx[r] * scale, sm[r]};
    }
    // target logit: the lane holding the row's target column (if it is one of
    // this wave's columns) stores it
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int rl = acc_row(wm, i, r, lane);
      const int tw = sy[rl] - wn * 128 - (lane & 31);    // 32 * block index if held here
      float v = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) v = tw == 32 * j ? acc[i][j][r] : v;
      if ((unsigned)tw < 128u && (tw & 31) == 0) zy[m0 + rl] = v * scale;
    }
  }

  // the block index must be a compile-time constant: a runtime index into
  // the accumulator array would move it to scratch memory
  template <bool FULL>
  __device__ __forceinline__ void blocks(const f32x16 (&acc)[4][4], int n0, int N,
                                         const int* sy, f32x2* red, int m0, int wm, int wn,
                                         int lane) const {
    block<FULL, 0>(acc, n0, N, sy, red, m0, wm, wn, lane);
    __builtin_amdgcn_sched_barrier(0);
    block<FULL, 1>(acc, n0, N, sy, red, m0, wm, wn, lane);
    __builtin_amdgcn_sched_barrier(0);
    block<FULL, 2>(acc, n0, N, sy, red, m0, wm, wn, lane);
    __builtin_amdgcn_sched_barrier(0);
    block<FULL, 3>(acc, n0, N, sy, red, m0, wm, wn, lane);
  }

  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int m0, int n0, int tn, int M,
                                             int N, uint8_t* smem, int wm, int wn, int lane,
                                             int tid) const {
    int* sy = (int*)smem;
    f32x2* red = (f32x2*)(smem + 1024);
    // target column relative to the tile (-1: dead row; a target outside the
    // tile matches no column)
    sy[tid] = (m0 + tid < M) ? y[m0 + tid] - n0 : -1;
    __syncthreads();
    if (n0 + GBN <= N)
      blocks<true>(acc, n0, N, sy, red, m0, wm, wn, lane);
    else
      blocks<false>(acc, n0, N, sy, red, m0, wm, wn, lane);
    __syncthreads();
    const int row = m0 + tid;
    if (row < M) {
      const f32x2 a = red[tid], b = red[GBM + tid];
      const float m = fmaxf(a.x, b.x);
      const float s = (a.y > 0.0f ? a.y * __expf(a.x - m) : 0.0f) +
                      (b.y > 0.0f ? b.y * __expf(b.x - m) : 0.0f);
      part[(int64_t)tn * ld_part + row] = f32x2{m, s};
    }
  }
};

// Forward partial log-sum-exp on a transposed tile: rows are vocabulary
// entries (A = W), columns are compacted tokens (B = H_act).  The accumulator
// layout gives every lane 64 rows of each of its 4 token columns, so the
// reduction over the tile's vocabulary is lane-local except for one exchange
// between lanes l and l ^ 32 (the two 4-row halves) and one merge of the two
// row waves through LDS.  Same outputs as EpiLsePartial: (max, sum exp) per
// token and vocabulary tile, and the target logit.
struct EpiLseCols {
  const int32_t* y;      // [tokens] target id of each compacted row
  f32x2* part;           // [tiles_v][ld_part] (max, sum exp) per token and vocabulary tile
  int64_t ld_part;
  float* zy;             // [tokens] logit of the target token
  float scale;           // 1 / temperature

  template <bool FULL>
  __device__ __forceinline__ void cols(const f32x16 (&acc)[4][4], int m0, int n0, int M,
                                       const int* sy, f32x2* red, int wm, int wn,
                                       int lane) const {
    const float k1 = scale * 1.44269504088896341f;
    // this lane's rows are wm * 128 + hb + o with o = 32 i + 8 (r >> 2) + (r & 3)
    const int hb = 4 * (lane >> 5);
    const int lim = M - m0 - wm * 128 - hb;     // rows o >= lim are beyond the vocabulary
    auto live = [&](int i, int r) { return FULL || 32 * i + 8 * (r >> 2) + (r & 3) < lim; };
    float mx[4], sm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) mx[j] = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) mx[j] = fmaxf(mx[j], live(i, r) ? acc[i][j][r] : -INFINITY);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      mx[j] = fmaxf(mx[j], __shfl_xor(mx[j], 32));
      sm[j] = 0.0f;
    }
    float mk[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) mk[j] = FULL || mx[j] != -INFINITY ? -mx[j] * k1 : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float e = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], k1, mk[j]));
          sm[j] += live(i, r) ? e : 0.0f;
        }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sm[j] += __shfl_xor(sm[j], 32);
      const int c = wn * 128 + j * 32 + (lane & 31);
      if (lane < 32) red[wm * GBN + c] = f32x2{mx[j] * scale, sm[j]};
      // target logit: local row o of the target, held here iff 0 <= o < 128 and
      // bit 2 of o is clear; the register is picked by a select tree over o's bits
      const int o = sy[c] - wm * 128 - hb;
      float v[64];
#pragma unroll
      for (int q = 0; q < 64; ++q) v[q] = acc[q >> 4][j][q & 15];
      const int idx = ((o >> 5) << 4) | (((o >> 3) & 3) << 2) | (o & 3);
#pragma unroll
      for (int b = 0, w = 32; b < 6; ++b, w >>= 1) {
        const bool hi = (idx >> b) & 1;
#pragma unroll
        for (int q = 0; q < w; ++q) v[q] = hi ? v[2 * q + 1] : v[2 * q];
      }
      if ((unsigned)o < 128u && (o & 4) == 0) zy[n0 + c] = v[0] * scale;
    }
  }

  __device__ __forceinline__ void tile(f32x16 (&acc)[4][4], int m0, int n0, int tn, int M,
                                       int N, uint8_t* smem, int wm, int wn, int lane,
                                       int tid) const {
    int* sy = (int*)smem;
    f32x2* red = (f32x2*)(smem + 1024);
    // target row relative to the tile (-1: dead column; a target outside the
    // tile matches no row)
    sy[tid] = (n0 + tid < N) ? y[n0 + tid] - m0 : -1;
    __syncthreads();
    if (m0 + GBM <= M)
      cols<true>(acc, m0, n0, M, sy, red, wm, wn, lane);
    else
      cols<false>(acc, m0, n0, M, sy, red, wm, wn, lane);
    __syncthreads();
    const int col = n0 + tid;
    if (col < N) {
      const f32x2 a = red[tid], b = red[GBN + tid];
      const float m = fmaxf(a.x, b.x);
      const float s = (a.y > 0.0f ? a.y * __expf(a.x - m) : 0.0f) +
                      (b.y > 0.0f ? b.y * __expf(b.x - m) : 0.0f);
      part[(int64_t)(m0 / GBM) * ld_part + col] = f32x2{m, s};
    }
  }

  // The same on the 16 x 16 accumulator layout: lane l holds 8 token columns
  // (16 j + (l & 15)) and 32 vocabulary rows of each (16 i + 4 (l >> 4) + r),
  // the other 96 rows of the wave's half sit in lanes l ^ 16, l ^ 32, l ^ 48.
  template <bool FULL>
  __device__ __forceinline__ void cols16(const f32x4 (&acc)[8][8], int m0, int n0, int M,
                                         const int* sy, f32x2* red, int wm, int wn,
                                         int lane) const {
    const float k1 = scale * 1.44269504088896341f;
    const int g4 = 4 * (lane >> 4);
    const int lim = M - m0 - wm * 128 - g4;     // rows 16 i + r >= lim are beyond the vocabulary
    auto live = [&](int i, int r) { return FULL || 16 * i + r < lim; };
    float mx[8], sm[8], mk[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      mx[j] = -INFINITY;
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx[j] = fmaxf(mx[j], live(i, r) ? acc[i][j][r] : -INFINITY);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) mx[j] = fmaxf(mx[j], __shfl_xor(mx[j], 16));
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      mx[j] = fmaxf(mx[j], __shfl_xor(mx[j], 32));
      mk[j] = FULL || mx[j] != -INFINITY ? -mx[j] * k1 : 0.0f;
      sm[j] = 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float e = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], k1, mk[j]));
          sm[j] += live(i, r) ? e : 0.0f;
        }
#pragma unroll
    for (int j = 0; j < 8; ++j) sm[j] += __shfl_xor(sm[j], 16);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      sm[j] += __shfl_xor(sm[j], 32);
      const int c = wn * 128 + j * 16 + (lane & 15);
      if (lane < 16) red[wm * GBN + c] = f32x2{mx[j] * scale, sm[j]};
      // target logit: local row o of the target, held here iff 0 <= o < 128 and
      // bits 2..3 of o equal lane / 16; the register is picked by a select tree
      // over o's block (bits 4..6) and row (bits 0..1)
      const int o = sy[c] - wm * 128;
      float v[32];
#pragma unroll
      for (int q = 0; q < 32; ++q) v[q] = acc[q >> 2][j][q & 3];
      const int idx = ((o >> 4) << 2) | (o & 3);
#pragma unroll
      for (int b = 0, w = 16; b < 5; ++b, w >>= 1) {
        const bool hi = (idx >> b) & 1;
#pragma unroll
        for (int q = 0; q < w; ++q) v[q] = hi ? v[2 * q + 1] : v[2 * q];
      }
      if ((unsigned)o < 128u && (o & 12) == g4) zy[n0 + c] = v[0] * scale;
    }
  }

  __device__ __forceinline__ void tile16(f32x4 (&acc)[8][8], int m0, int n0, int tn, int M,
                                         int N, uint8_t* smem, int wm, int wn, int lane,
                                         int tid) const {
    int* sy = (int*)smem;
    f32x2* red = (f32x2*)(smem + 1024);
    sy[tid] = (n0 + tid < N) ? y[n0 + tid] - m0 : -1;
    __syncthreads();
    if (m0 + GBM <= M)
      cols16<true>(acc, m0, n0, M, sy, red, wm, wn, lane);
    else
      cols16<false>(acc, m0, n0, M, sy, red, wm, wn, lane);
    __syncthreads();
    const int col = n0 + tid;
    if (col < N) {
      const f32x2 a = red[tid], b = red[GBN + tid];
      const float m = fmaxf(a.x, b.x);
      const float s = (a.y > 0.0f ? a.y * __expf(a.x - m) : 0.0f) +
                      (b.y > 0.0f ? b.y * __expf(b.x - m) : 0.0f);
      part[(int64_t)(m0 / GBM) * ld_part + col] = f32x2{m, s};
    }
  }
};

template <typename T>
__device__ __forceinline__ T to_store(float v);
template <>
__device__ __forceinline__ __bf16 to_store<__bf16>(float v) {
  return __builtin_bit_cast(__bf16, f32_to_bf16_bits(v));
}
template <>
__device__ __forceinline__ float to_store<float>(float v) {
  return v;
}

// Backward recompute: G = gs_n * (1[v == y_n] - exp(z - lse_n)), rounded to T.
// fp32 writes it as G[row][col] and transposed as Gt[col][row]; bf16 writes G
// only (stage-tiled).  Rows >= M and columns >= N are written as 0 (they pad
// the K extent of the next products).
template <typename T>
struct LogitGradArgs {
  const int32_t* y;
  const float* lse;
  const float* gs;       // dL/dlogp / temperature, per compacted row
  T* G;                  // fp32: row-major [rows][ldg]; bf16: column-block stage-tiled
  int64_t ldg;           // fp32: row pitch; bf16: G's padded row count
  T* Gt;                 // fp32 only: G transposed, row-major [cols][ldgt]
  int64_t ldgt;
  float scale;
  int32_t col0;          // vocabulary index of this chunk's column 0
};

template <typename T>
struct EpiLogitGrad;

// fp32 (simple kernel): direct stores from the accumulator layout.
template <>
struct EpiLogitGrad<float> : LogitGradArgs<float> {
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int m0, int n0, int tn, int M,
                                             int N, uint8_t* smem, int wm, int wn, int lane,
                                             int tid) const {
    int* sy = (int*)smem;
    float* sl = (float*)(smem + 1024);
    float* sg = (float*)(smem + 2048);
    const bool live = m0 + tid < M;
    sy[tid] = live ? y[m0 + tid] - col0 : -1;
    sl[tid] = live ? lse[m0 + tid] : INFINITY;
    sg[tid] = live ? gs[m0 + tid] : 0.0f;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = n0 + acc_col(wn, j, lane);
          float vals[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int rl = acc_row(wm, i, r4 * 4 + q, lane);
            const float p = __expf(acc[i][j][r4 * 4 + q] * scale - sl[rl]);
            const float g = sg[rl] * ((c == sy[rl] ? 1.0f : 0.0f) - p);
            vals[q] = c < N ? g : 0.0f;
            G[(int64_t)(m0 + rl) * ldg + c] = vals[q];
          }
          const int rl0 = acc_row(wm, i, r4 * 4, lane);
          *(f32x4*)(Gt + (int64_t)c * ldgt + m0 + rl0) = f32x4{vals[0], vals[1], vals[2], vals[3]};
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
};

// bf16 (pipelined kernel).  The tile is finished in two passes of 128 rows
// (accumulator blocks i = 2h and 2h + 1 of both wave rows).  A pass stages its
// G rows row-major in LDS, then they leave as full 128-byte lines of G's
// column-block stage-tiled layout (dW reads the same G transposed, so no
// transposed copy is written).  The exponent is evaluated in base 2 with the
// scale folded in: exp(z - lse) = exp2(acc * scale * log2(e) - lse * log2(e)).
template <>
struct EpiLogitGrad<__bf16> : LogitGradArgs<__bf16> {
  template <bool FULL, int h>
  __device__ __forceinline__ void stage_pass(const f32x16 (&acc)[4][4], int n0, int N,
                                             uint8_t* smem, int wm, int wn, int lane) const {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    const float k1 = scale * 1.44269504088896341f;
#pragma unroll
    for (int ii = 0; ii < 2; ++ii) {
      const int i = 2 * h + ii;
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int rt = acc_row(wm, i, r4 * 4, lane);      // tile row of element q = 0
        const i32x4 ry = *(const i32x4*)(smem + EPI_META + 4 * rt);
        const f32x4 rn = *(const f32x4*)(smem + EPI_META + 1024 + 4 * rt);
        const f32x4 rg = *(const f32x4*)(smem + EPI_META + 2048 + 4 * rt);
        const int lr = wm * 64 + ii * 32 + 8 * r4 + 4 * (lane >> 5);   // pass-local row
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int cl = acc_col(wn, j, lane);
          float gv[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float p = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r4 * 4 + q], k1, rn[q]));
            gv[q] = fmaf(-rg[q], p, cl == ry[q] ? rg[q] : 0.0f);
            if constexpr (!FULL) gv[q] = n0 + cl < N ? gv[q] : 0.0f;
          }
          const uint32_t p01 = __builtin_bit_cast(
              uint32_t, __builtin_convertvector(f32x2{gv[0], gv[1]}, bf16x2_t));
          const uint32_t p23 = __builtin_bit_cast(
              uint32_t, __builtin_convertvector(f32x2{gv[2], gv[3]}, bf16x2_t));
          uint8_t* gs_at = smem + EPI_GS + lr * EPI_G_ROW + cl * 2;
          *(uint16_t*)(gs_at) = (uint16_t)p01;
          *(uint16_t*)(gs_at + EPI_G_ROW) = (uint16_t)(p01 >> 16);
          *(uint16_t*)(gs_at + 2 * EPI_G_ROW) = (uint16_t)p23;
          *(uint16_t*)(gs_at + 3 * EPI_G_ROW) = (uint16_t)(p23 >> 16);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  // per tile row: target column relative to the tile, -lse * log2(e) (-inf on
  // dead rows, so their exponentials are 0 and G is +0 there), dL/dlogp
  __device__ __forceinline__ void meta(int m0, int n0, int M, uint8_t* smem, int tid) const {
    const bool live = m0 + tid < M;
    ((int*)(smem + EPI_META))[tid] = live ? y[m0 + tid] - col0 - n0 : -1;
    ((float*)(smem + EPI_META + 1024))[tid] =
        live ? -lse[m0 + tid] * 1.44269504088896341f : -INFINITY;
    ((float*)(smem + EPI_META + 2048))[tid] = live ? gs[m0 + tid] : 0.0f;
  }

  __device__ __forceinline__ void tile(f32x16 (&acc)[4][4], int m0, int n0, int tn, int M,
                                       int N, uint8_t* smem, int wm, int wn, int lane,
                                       int tid) const {
    meta(m0, n0, M, smem, tid);
    __syncthreads();
    const bool full = n0 + GBN <= N;
    pass<0>(acc, full, m0, n0, N, smem, wm, wn, lane, tid);
    __syncthreads();
    pass<1>(acc, full, m0, n0, N, smem, wm, wn, lane, tid);
  }

  // 16 x 16 accumulator layout: pass h takes blocks i = 4 h .. 4 h + 3 of both
  // wave rows (the same tile rows as the 32 x 32 layout's pass h); lane l holds
  // 4 consecutive rows 16 i + 4 (l >> 4) + r of column 16 j + (l & 15).
  template <bool FULL, int h>
  __device__ __forceinline__ void stage_pass16(const f32x4 (&acc)[8][8], int n0, int N,
                                               uint8_t* smem, int wm, int wn, int lane) const {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    const float k1 = scale * 1.44269504088896341f;
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int i = 4 * h + ii;
      const int rt = wm * 128 + 16 * i + 4 * (lane >> 4);      // tile row of r = 0
      const i32x4 ry = *(const i32x4*)(smem + EPI_META + 4 * rt);
      const f32x4 rn = *(const f32x4*)(smem + EPI_META + 1024 + 4 * rt);
      const f32x4 rg = *(const f32x4*)(smem + EPI_META + 2048 + 4 * rt);
      const int lr = wm * 64 + 16 * ii + 4 * (lane >> 4);       // pass-local row
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int cl = wn * 128 + 16 * j + (lane & 15);
        float gv[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float p = __builtin_amdgcn_exp2f(fmaf(acc[i][j][q], k1, rn[q]));
          gv[q] = fmaf(-rg[q], p, cl == ry[q] ? rg[q] : 0.0f);
          if constexpr (!FULL) gv[q] = n0 + cl < N ? gv[q] : 0.0f;
        }
        const uint32_t p01 = __builtin_bit_cast(
            uint32_t, __builtin_convertvector(f32x2{gv[0], gv[1]}, bf16x2_t));
        const uint32_t p23 = __builtin_bit_cast(
            uint32_t, __builtin_convertvector(f32x2{gv[2], gv[3]}, bf16x2_t));
        uint8_t* gs_at = smem + EPI_GS + lr * EPI_G_ROW + cl * 2;
        *(uint16_t*)(gs_at) = (uint16_t)p01;
        *(uint16_t*)(gs_at + EPI_G_ROW) = (uint16_t)(p01 >> 16);
        *(uint16_t*)(gs_at + 2 * EPI_G_ROW) = (uint16_t)p23;
        *(uint16_t*)(gs_at + 3 * EPI_G_ROW) = (uint16_t)(p23 >> 16);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  __device__ __forceinline__ void tile16(f32x4 (&acc)[8][8], int m0, int n0, int tn, int M,
                                         int N, uint8_t* smem, int wm, int wn, int lane,
                                         int tid) const {
    meta(m0, n0, M, smem, tid);
    __syncthreads();
    const bool full = n0 + GBN <= N;
    if (full)
      stage_pass16<true, 0>(acc, n0, N, smem, wm, wn, lane);
    else
      stage_pass16<false, 0>(acc, n0, N, smem, wm, wn, lane);
    __syncthreads();
    copy_out<0>(m0, n0, smem, tid);
    __syncthreads();
    if (full)
      stage_pass16<true, 1>(acc, n0, N, smem, wm, wn, lane);
    else
      stage_pass16<false, 1>(acc, n0, N, smem, wm, wn, lane);
    __syncthreads();
    copy_out<1>(m0, n0, smem, tid);
  }

  template <int h>
  __device__ __forceinline__ void pass(const f32x16 (&acc)[4][4], bool full, int m0, int n0,
                                       int N, uint8_t* smem, int wm, int wn, int lane,
                                       int tid) const {
    {
      if (full)
        stage_pass<true, h>(acc, n0, N, smem, wm, wn, lane);
      else
        stage_pass<false, h>(acc, n0, N, smem, wm, wn, lane);
      __syncthreads();
      copy_out<h>(m0, n0, smem, tid);
    }
  }

  // G: 128 rows of 512 bytes staged in LDS by pass h; pass rows 0..63 are tile
  // rows 64h + r, rows 64..127 are tile rows 128 + 64h + (r - 64).
  // Column-block stage-tiled addresses: m0 and n0 are multiples of 256, so a
  // thread's block and chunk are fixed and only the row within the block
  // changes from store to store.  The loop reads all its LDS chunks before
  // the first store, so the reads overlap.  The stores are non-temporal: G is
  // read back only by the next launch, and a round of tiles writes as much G
  // as an XCD's L2 holds, which would otherwise evict the operand panels the
  // running tiles share.
  template <int h>
  __device__ __forceinline__ void copy_out(int m0, int n0, uint8_t* smem, int tid) const {
    const int c16 = tid & 31;
    __bf16* base = G + (((int64_t)((n0 >> 6) + (c16 >> 3)) * (ldg >> 8) + (m0 >> 8)) << 14);
    u32x4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k)
      v[k] = *(const u32x4*)(smem + EPI_GS + ((tid >> 5) + 8 * k) * EPI_G_ROW + c16 * 16);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int row = (tid >> 5) + 8 * k;
      const int trow = 64 * h + (row < 64 ? row : row + 64);
      __builtin_nontemporal_store(
          v[k], (u32x4*)(base + ((trow << 6) + (((c16 & 7) ^ ((trow >> 1) & 7)) << 3))));
    }
  }
};

// Plain fp32 store (or accumulate) of the tile, rows optionally remapped.
struct EpiStore {
  float* out;
  int64_t ldo;
  const int32_t* row_map;   // nullable: output row of each tile row
  int32_t accumulate;

  // simple kernel: direct stores from the accumulator layout
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int m0, int n0, int tn, int M,
                                             int N, uint8_t* smem, int wm, int wn, int lane,
                                             int tid) const {
    int* sr = (int*)smem;
    if (row_map) {
      sr[tid] = (m0 + tid < M) ? row_map[m0 + tid] : 0;
      __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = acc_row(wm, i, r, lane);
        if (m0 + rl < M) {
          const int64_t orow = row_map ? (int64_t)sr[rl] : (int64_t)(m0 + rl);
          float* dst = out + orow * ldo;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int c = n0 + acc_col(wn, j, lane);
            if (c < N) dst[c] = accumulate ? dst[c] + acc[i][j][r] : acc[i][j][r];
          }
        }
        if ((r & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
  }

  // 16 x 16 accumulator layout.  Pass h stages blocks i = 4 h .. 4 h + 3 of both
  // wave rows (the same tile rows as the 32 x 32 layout's pass h), each block
  // as whole accumulators: a lane's f32x4 (4 consecutive rows of one column)
  // is one 16-byte LDS write into a column-major staging area (128 rows per
  // column, padded to EPI_COL floats so that the 16 columns of a write are 16
  // distinct bank groups).  (Writing the accumulators element by element
  // makes the register allocator shuffle them through VGPRs inside the main
  // loop.)  The write-out takes one staged row per wave at a time, lane l
  // holding columns l, l + 64, l + 128, l + 192: every store instruction
  // covers 256 consecutive bytes of an output row.
  __device__ __forceinline__ void tile16(f32x4 (&acc)[8][8], int m0, int n0, int tn, int M, int N,
                                         uint8_t* smem, int wm, int wn, int lane, int tid) const {
    int* sr = (int*)(smem + EPI_META);
    if (row_map) sr[tid] = (m0 + tid < M) ? row_map[m0 + tid] : 0;
    float* st = (float*)smem;
    if (accumulate)
      out16<true>(acc, m0, n0, M, N, st, sr, wm, wn, lane);
    else
      out16<false>(acc, m0, n0, M, N, st, sr, wm, wn, lane);
  }

  template <bool ACC>
  __device__ __forceinline__ void out16(const f32x4 (&acc)[8][8], int m0, int n0, int M, int N,
                                        float* st, const int* sr, int wm, int wn, int lane) const {
    const int wave = wm * 2 + wn;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h) lds_barrier();                        // pass 0's rows have been read
#pragma unroll
      for (int ii = 0; ii < 4; ++ii)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          *(f32x4*)(st + (wn * 128 + 16 * j + (lane & 15)) * EPI_COL + wm * 64 + 16 * ii +
                    4 * (lane >> 4)) = acc[4 * h + ii][j];
      lds_barrier();                               // rows staged (and sr written)
      // staged row pr is tile row 64 h + pr (pr < 64) or 128 + 64 h + (pr - 64);
      // wave w writes rows w, w + 4, ..., 8 rows at a time
#pragma unroll
      for (int k0 = 0; k0 < 32; k0 += 8) {
        float* dst[8];
        float old[8][4];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int pr = wave + 4 * (k0 + k);
          const int tr = 64 * h + (pr < 64 ? pr : pr + 64);
          const int64_t orow = row_map ? (int64_t)sr[tr] : (int64_t)(m0 + tr);
          dst[k] = m0 + tr < M ? out + orow * ldo + n0 : nullptr;
          if constexpr (ACC) {
#pragma unroll
            for (int m = 0; m < 4; ++m)
              old[k][m] = dst[k] && n0 + lane + 64 * m < N ? dst[k][lane + 64 * m] : 0.0f;
          }
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int pr = wave + 4 * (k0 + k);
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            float v = st[(lane + 64 * m) * EPI_COL + pr];
            if constexpr (ACC) v += old[k][m];
            if (dst[k] && n0 + lane + 64 * m < N) dst[k][lane + 64 * m] = v;
          }
        }
      }
    }
  }
};

}  // namespace agrl
