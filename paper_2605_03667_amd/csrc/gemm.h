// Tiled MFMA GEMM for gfx950 (CDNA4): C = A * B with bf16 operands and fp32
// accumulation, one template covering every product of the ELAS low-rank FFN
// (forward and backward).
//
// Tiling: a workgroup of WAVES_M x WAVES_N wave64s owns a BM x BN tile of C.
// The contraction runs in steps of BK (64 dense, or 128 dense = 64 kept
// values for the 2:4 operand).  Both operands are staged in LDS in
// "K-contiguous rows": row r of a tile holds BK (or 128) contraction elements
// as 16-byte chunks, XOR-swizzled (see swz) so that reads and writes of one
// chunk position across 8 rows hit 8 different bank groups.
//
// Staging.  Dense operands go straight from global memory to LDS with
// global_load_lds_dwordx4 (no registers on the way), through STAGES LDS
// buffers: the loads of step s + STAGES - 1 are issued while step s computes,
// and each wave waits only for its own loads of step s (an exact vmcnt)
// before a plain s_barrier.  Lanes whose chunk lies outside the matrix load
// from a zero block.  K-contiguous operands land in K-contiguous LDS rows;
// K-major operands ([K x rows] in memory) land K-major and their MFMA
// fragments are read with the transposing ds_read_b64_tr_b16.  The 2:4
// operand read along its rows (S^T, dH^T) is expanded in registers and
// written K-major after the current step's MFMAs.  One barrier per step.
//
// Operand modes:
//   OP_K    operand stored [rows x K] row-major (K contiguous): 16-byte copies.
//   OP_T    operand stored [K x rows] (rows contiguous): DMA to a K-major LDS
//           tile, fragments by transposing LDS reads.
//   OP_SP   (A only) 2:4 compressed along K: kept values [rows x K/2] plus
//           metadata [rows x K/8]; consumed by v_smfmac_f32_32x32x32_bf16.
//   OP_TSP  (A only) 2:4 compressed along the row dimension of a [K x rows]
//           matrix (S^T or dH^T read from the compressed activation): each
//           thread expands 16 features of one contraction row from kept values
//           + metadata into the K-major LDS tile.
//
// MFMA layouts (pinned on gfx950 by a probe against a CPU product):
//   v_mfma_f32_32x32x16_bf16: lane l holds A[row l%32][k 8(l/32)..+8] and
//     B[k 8(l/32)..+8][col l%32]; accumulator i of lane l is
//     C[row 8(i/4) + 4(l/32) + i%4][col l%32].
//   v_smfmac_f32_32x32x32_bf16: the 16 index bits of a lane (bits 16*ABID..)
//     hold 2 bits per kept value in slot order; kept slot j of lane l is row
//     l%32, hardware K position 16(q/2) + 8(l/32) + 4(q%2) + idx_j with
//     q = j/2; B lane l holds hardware K 16(l/32)..+16 of column l%32.
//     Permuting the memory K order so that lane half h owns memory groups
//     4h..4h+3 of each 32-wide step makes its 8 kept values one contiguous
//     16-byte chunk whose 16 index bits are the canonical metadata shifted by
//     16h; B lane half c then takes memory K [8c, 8c+8) and [16+8c, 16+8c+8).
#pragma once

#include <type_traits>

#include "device.h"

namespace elas {
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

enum OpMode { OP_K = 0, OP_T = 1, OP_SP = 2, OP_TSP = 3 };
enum EpiMode {
  EPI_BF16 = 0,       // C bf16
  EPI_F32 = 1,        // fp32 split-K partials
  EPI_SPARSIFY = 2,   // ReLU^2 + top-2 of 4 + compressed write (C = H^T)
  EPI_DH = 3,         // dH = dS * mask * 2 relu(h), compressed (C = dS^T)
  EPI_ACT_DENSE = 4,  // dense activation: relu(h)^2 (act_square) or relu(h) (C = H^T)
  EPI_DH_DENSE = 5,   // dense dH = dS * 2 r, r from a dense activation (C = dS^T)
  EPI_DH_STE = 6,     // dense dH = dS * 2 relu(h), h = A B^T of the first operand pair (C = dS^T)
};

struct GemmArgs {
  const uint16_t* A;   // OP_K [M x K], OP_T [K x M], OP_SP vals [M x K/2], OP_TSP vals [K x M/2]
  int64_t lda;         // element pitch of A (or of its kept values)
  const uint8_t* Am;   // OP_SP / OP_TSP metadata
  int64_t ldam;        // byte pitch of the metadata
  const uint16_t* B;   // OP_K [N x K], OP_T [K x N]
  int64_t ldb;
  // b_nsk > 0: B (OP_K) is blocked (blocked_index below) with b_nsk K blocks
  // per row panel, zero-padded, and ldb is 64; every B load is unchecked.
  int64_t b_nsk;
  // EPI_DH_STE: the second operand pair (same shapes and pitches as A, B).
  // The tile's contraction runs over (A, B) first, whose product is H^T, then
  // over (A2, B2), whose product is dS^T.
  const uint16_t* A2;
  const uint16_t* B2;
  int64_t M, N, K;     // C is M x N; contraction length K (dense count)
  int64_t m_valid;     // rows of A that exist in memory (rows >= m_valid read as 0)
  int64_t ka_valid;    // contraction entries of A that exist (>= read as 0)
  int64_t kb_valid;    // contraction entries of B that exist
  int64_t k_split;     // contraction length per split (multiple of the K step)
  void* C;             // EPI_BF16: bf16 [M x N] pitch ldc; EPI_F32: float [splits][M][N]
  int64_t ldc;
  // EPI_SPARSIFY / EPI_DH: C rows are features f (M), columns are tokens t (N).
  // The compressed tensors are tiled (tiled_index) with tok = N rows.
  uint16_t* sv;        // kept values of S (N rows, pitch ldv): written (SPARSIFY) / read (DH)
  uint8_t* sm;         // metadata of S (N rows, pitch ldm)
  int64_t ldv, ldm;
  uint16_t* dv;        // EPI_DH: kept values of dH (N rows, pitch ldv), written
  // EPI_ACT_DENSE / EPI_DH_DENSE: dense [N x ld_act] activations (tokens as
  // rows), features f < f_valid only.
  uint16_t* act;       // ACT_DENSE: written; DH_DENSE: read (r = bf16(sqrt(a)) if act_square, else a)
  uint16_t* dact;      // DH_DENSE: dense dH, written (pitch ld_act)
  int64_t ld_act;
  int64_t f_valid;
  int act_square;
  int tiles_m, tiles_n;
  // M-fast direct kernels: when > 1, the XCDs split the M tiles into this many
  // contiguous panels (XCD x takes panel x % m_groups and a share of the N
  // tiles), so that the A rows a panel needs stay resident in the XCD's L2.
  int m_groups;
  // Stream-K (register-staged path, EPI_F32): when stream_steps > 0, the
  // gridDim.x workgroups split the tiles x stream_steps K steps into equal
  // contiguous ranges; workgroup w writes the partial tile of the j-th tile
  // its range touches to C + (w * stream_segs + j) * BM * BN (row-major).
  int64_t stream_steps;
  int stream_segs;
  // Compressed 2:4 tensors in the tiled layout (tiled_index below): the 2:4
  // operand of OP_SP when a_tiled is set (OP_TSP and the staged epilogues
  // always), with tok token rows.
  int a_tiled;
  int64_t tok;
};

// Tiled layout of a compressed 2:4 tensor with tok rows (tokens) and row pitch
// ld (values, or metadata bytes): rows in blocks of 256 (the last block holds
// the R < 256 remaining rows) and each row's entries in blocks of BW (32
// values or 8 metadata bytes: 64 features); block (row block, entry block)
// holds its R rows x BW entries row-major and contiguously, blocks ordered by
// row block, then entry block.  Index of entry j of row t:
// Blocked layout of a K-contiguous [N x K] operand: 256-row panels, each cut
// into 64-wide K blocks stored contiguously ([256 x 64] row-major, 32 KB),
// blocks ordered by panel, then K block; nsk = K blocks per panel (K padded
// to 64, N to 256, with zeros).  One K step of a 256-row (or 128-row) tile is
// then one contiguous piece of memory.
__host__ __device__ inline int64_t blocked_index(int64_t n, int64_t k, int64_t nsk) {
  return (((n >> 8) * nsk + (k >> 6)) << 14) + ((n & 255) << 6) + (k & 63);
}

template <int BW>
__device__ __forceinline__ int64_t tiled_index(int64_t t, int64_t j, int64_t tok, int64_t ld) {
  const int64_t tb = t >> 8;
  const int64_t R = tok - (tb << 8) < 256 ? tok - (tb << 8) : 256;
  return (tb << 8) * ld + (j / BW) * R * BW + (t & 255) * BW + (j % BW);
}
// Start of the step at dense contraction index k0 (a multiple of 64) for rows
// from row0 (inside one row block): entry block k0/64, row row0 % 256.
template <int BW>
__device__ __forceinline__ int64_t tiled_step(int64_t row0, int64_t k0, int64_t tok, int64_t ld) {
  const int64_t tb = row0 >> 8;
  const int64_t R = tok - (tb << 8) < 256 ? tok - (tb << 8) : 256;
  return (tb << 8) * ld + (k0 >> 6) * R * BW + (row0 & 255) * BW;
}

template <int BM_, int BN_, int WAVES_M_, int WAVES_N_, int AMODE_, int BMODE_, int EPI_, bool M_FAST_,
          int STAGES_ = 2, bool PIPE_ = true, bool PIN_ = false, int SPK_ = 128, int DEEP_ = 0>
struct GemmCfg {
  // DEEP: separate LDS rings with three stages (prefetched two steps ahead)
  // for one operand, 1 = A or 2 = B, the one streaming from HBM, and two
  // (one step ahead) for the other.  Plain-output epilogues only.
  static constexpr int DEEP = DEEP_;
  // PIPE: double-buffer the MFMA fragments (read sub-step kk+1 during kk's
  // MFMAs); off saves registers.
  static constexpr bool PIPE = PIPE_;
  // PIN: fence the scheduler around each sub-step's MFMAs, so that the reads
  // of the next sub-step are issued ahead of them as written (costs registers).
  static constexpr bool PIN = PIN_;
  static constexpr int BM = BM_, BN = BN_, WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
  static constexpr int NW = WAVES_M_ * WAVES_N_, NT = 64 * NW;
  static constexpr int AMODE = AMODE_, BMODE = BMODE_, EPI = EPI_;
  static constexpr bool M_FAST = M_FAST_;   // consecutive tiles walk M (true) or N (false)
  static constexpr bool SPARSE = AMODE_ == OP_SP;
  // SWAP: the MFMAs take B's fragment as their first operand, so that each
  // lane accumulates runs of consecutive C columns (plain bf16 / fp32 output,
  // written with 16-byte stores).  The 2:4 operand must stay first.
  static constexpr bool SWAP = !SPARSE && (EPI_ == EPI_BF16 || EPI_ == EPI_F32);
  // K-major operands ([K x rows] in memory) are staged K-major in LDS and read
  // with the transposing ds_read_b64_tr_b16.
  static constexpr bool A_KM = AMODE_ == OP_T || AMODE_ == OP_TSP;
  static constexpr bool B_KM = BMODE_ == OP_T;
  // DIRECT: every operand goes global -> LDS by DMA; otherwise (the 2:4
  // K-major operand, expanded in registers) A is register-staged.
  static constexpr bool DIRECT = AMODE_ != OP_TSP;
  static constexpr int STAGES = STAGES_;
  // dense contraction per step: 64, or SPK (64 or 128) for a 2:4 operand
  static constexpr int BK = SPARSE ? SPK_ : 64;
  static_assert(SPK_ == 64 || SPK_ == 128, "2:4 K step");
  static constexpr int KK = SPARSE ? BK / 32 : 4;       // MFMA sub-steps per step
  static constexpr int A_ROWB = SPARSE ? BK : 128;       // bytes per LDS row of A (BK/2 kept or 64 dense values)
  static constexpr int B_ROWB = SPARSE ? 2 * BK : 128;   // bytes per LDS row of B
  static constexpr int M_ROWB = SPARSE ? BK / 8 : 0;     // metadata bytes per row
  static constexpr int A_BYTES = BM * A_ROWB;
  static constexpr int AM_BYTES = BM * M_ROWB;
  static constexpr int B_BYTES = BN * B_ROWB;
  static constexpr int STAGE = A_BYTES + AM_BYTES + B_BYTES;
  static constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  static constexpr int FM = TM / 32, FN = TN / 32;
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile must be a multiple of 32");
  static_assert(DIRECT || STAGES_ == 2, "register staging uses two LDS buffers");
  static_assert(!(A_KM || B_KM) || !SPARSE, "2:4 along K with a K-major partner is not used");
  static_assert(STAGES_ >= 2 && STAGES_ <= 4, "2 to 4 stages");
  // The compressed-activation epilogues stage a BN x BM/2 tile of kept values
  // in one stage buffer and the metadata rows (BM/8 bytes + 4 pad) after the
  // stages.
  static constexpr bool STAGED_EPI = EPI_ == EPI_SPARSIFY || EPI_ == EPI_DH;
  static constexpr int META_PITCH = BM_ / 8 + 4;
  // EPI_DH copies the stored S tile by DMA during the tile's last K step (the
  // uniform two-stage ring only): the metadata rows go in as dword DMAs of 256
  // bytes, META_DMA_PER_WAVE per wave, so their area is rounded up to that.
  static constexpr bool PRE_S = EPI_ == EPI_DH && DEEP_ == 0 && STAGES_ == 2;
  static_assert(EPI_ != EPI_DH || PRE_S, "EPI_DH copies its S tile during the last K step");
  static constexpr int META_DMA_PER_WAVE = (BN_ * META_PITCH / 4 + 64 * NW - 1) / (64 * NW);
  static constexpr int META_BYTES = PRE_S ? META_DMA_PER_WAVE * NW * 256 : (BN_ * META_PITCH + 15) / 16 * 16;
  static constexpr int A_PART = A_BYTES + AM_BYTES;   // one stage of A (and its metadata)
  static constexpr int LDS_BYTES = DEEP_ == 1   ? 3 * A_PART + 2 * B_BYTES
                                   : DEEP_ == 2 ? 2 * A_PART + 3 * B_BYTES
                                                : STAGES_ * STAGE + (STAGED_EPI ? META_BYTES : 0);
  static_assert(DEEP_ == 0 || (STAGES_ == 2 && !STAGED_EPI && DIRECT), "three-stage ring: plain epilogues, direct staging");
  static_assert(!STAGED_EPI || (BM_ == 256 && BN_ * BM_ <= STAGE && DIRECT), "staged epilogue layout");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");
  static_assert(EPI_ != EPI_DH_STE || AMODE_ != OP_TSP, "two operand pairs: direct staging");
  // a blocked B (GemmArgs::b_nsk) needs 128-byte LDS rows of B (64 K per
  // step); only the plain-output products take one, and the other kernels are
  // compiled without the branch
  static constexpr bool B_BLOCKABLE = !B_KM && B_ROWB == 128 && (EPI_ == EPI_BF16 || EPI_ == EPI_F32);
};

// LDS chunk swizzle.  Fragment reads touch 8 consecutive rows at one chunk;
// the transposing stagers write rows 8 apart (rb*8 + j) at one chunk.  XOR-ing
// the chunk with (row ^ row/8) & 7 spreads both patterns over 8 different
// 16-byte bank groups.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row ^ (row >> 3)) & 7); }
// 256-byte rows (the dense operand of a 2:4 product, 128 K per step): 16
// chunks per row; XOR-ing with row % 16 gives the 16 rows that one 16-lane
// group of a fragment read touches 16 different chunk positions.
__device__ __forceinline__ int swz16(int row, int chunk) { return chunk ^ (row & 15); }
// 64-byte rows (kept values of a 2:4 operand, 64 K per step): four rows share
// a 256-byte bank cycle, so the chunk is XOR-ed with (row / 4) % 4 to give 16
// consecutive rows 16 different 16-byte positions.
__device__ __forceinline__ int swz4(int row, int chunk) { return chunk ^ ((row >> 2) & 3); }
template <int ROWB>
__device__ __forceinline__ int swz_row(int row, int chunk) {
  static_assert(ROWB == 64 || ROWB == 128 || ROWB == 256, "row size");
  if constexpr (ROWB == 64)
    return swz4(row, chunk);
  else if constexpr (ROWB == 128)
    return swz(row, chunk);
  else
    return swz16(row, chunk);
}

// Expand 2 groups (4 kept values in 8 bytes + 2 codes in one byte) to 8 dense
// bf16 values packed as a uint4: kept value v0 (v1) of a group lands in slot
// i0 (i1) of its 4 by a 64-bit shift of 16 i0 (16 i1) bits, the other slots 0.
__device__ __forceinline__ uint4 expand2(uint2 kept, uint32_t codes) {
  uint64_t d[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const uint32_t pair = g ? kept.y : kept.x;
    const uint32_t code = (codes >> (4 * g)) & 0xFu;
    const uint32_t s0 = (code & 3u) << 4, s1 = (code >> 2) << 4;
    d[g] = ((uint64_t)(pair & 0xFFFFu) << s0) | ((uint64_t)(pair >> 16) << s1);
  }
  return make_uint4((uint32_t)d[0], (uint32_t)(d[0] >> 32), (uint32_t)d[1], (uint32_t)(d[1] >> 32));
}

// ---- direct global -> LDS staging ------------------------------------------
// Zeros read by lanes whose chunk lies outside the matrix.
static __device__ __attribute__((aligned(16))) uint4 g_dma_zero[1];

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
// One wave-wide LDS DMA: lane i's 16 (or 4) bytes land at LDS address
// lds_wave_base + 16 i (4 i).  The base must be wave-uniform (it goes to M0).
// Issued through inline asm so that the compiler does not guard every later
// LDS access with a full vmcnt(0); the kernel waits with exact counts itself.
// M0 is written here and read only by the DMA that follows; the generated
// code of these kernels uses M0 nowhere else (checked in the ISA).
__device__ __forceinline__ void dma_b128(const void* g, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_wave_base) : "memory", "m0");
}
__device__ __forceinline__ void dma_b32(const void* g, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds_wave_base) : "memory", "m0");
}
// The same DMA addressed as a wave-uniform 64-bit base (SGPRs) plus a 32-bit
// per-lane byte offset: no per-lane 64-bit address arithmetic.  The base is
// uniform by construction; readfirstlane states it to the compiler (and is
// free when it already sits in SGPRs).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t u = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ int64_t uniform_i64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ void dma_b128_s(const void* sbase, uint32_t voff, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(uniform_ptr(sbase)),
               "s"(__builtin_amdgcn_readfirstlane(lds_wave_base))
               : "memory", "m0");
}
__device__ __forceinline__ void dma_b32_s(const void* sbase, uint32_t voff, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(uniform_ptr(sbase)),
               "s"(__builtin_amdgcn_readfirstlane(lds_wave_base))
               : "memory", "m0");
}
// Non-temporal forms (nt: streamed data that is read once and should not
// displace what a workgroup keeps in L2).
__device__ __forceinline__ void dma_b128_nt(const void* g, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(lds_wave_base) : "memory", "m0");
}
__device__ __forceinline__ void dma_b32_nt(const void* g, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off nt" ::"v"(g), "s"(lds_wave_base) : "memory", "m0");
}
__device__ __forceinline__ void dma_b128_nt_s(const void* sbase, uint32_t voff, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" ::"v"(voff), "s"(uniform_ptr(sbase)),
               "s"(__builtin_amdgcn_readfirstlane(lds_wave_base))
               : "memory", "m0");
}
__device__ __forceinline__ void dma_b32_nt_s(const void* sbase, uint32_t voff, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1 nt" ::"v"(voff), "s"(uniform_ptr(sbase)),
               "s"(__builtin_amdgcn_readfirstlane(lds_wave_base))
               : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Workgroup barrier without a memory fence (LDS DMA completion is covered by
// the explicit vmcnt waits; the empty memory clobber keeps the compiler from
// moving LDS reads across it).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// A [ROWS x ROWB] K-contiguous tile (or the kept values of a 2:4 tile) copied
// by DMA: the tile is cut into 1 KB blocks (8 or 4 rows), PER_WAVE blocks per
// wave.  Lane i fills LDS chunk position i of its block; it fetches the
// global chunk that the swizzle maps there.
template <int ROWS, int ROWB, bool KEPT, int NW>
struct DmaTile {
  static constexpr int BLOCKS = ROWS * ROWB / 1024;
  static constexpr int PER_WAVE = BLOCKS / NW;
  static_assert(BLOCKS % NW == 0, "blocks per wave");
  static constexpr int KPC = KEPT ? 16 : 8;    // dense K per 16-byte chunk
  // Issue this wave's loads j in [J0, J1) for the step at k0 into the LDS
  // buffer at byte address lds (wave-uniform).
  // tok > 0 (kept values only): the tiled layout with tok rows.
  template <int J0, int J1>
  __device__ __forceinline__ static void issue(const uint16_t* __restrict__ p, int64_t ld, int64_t row0,
                                               int64_t rows_valid, int64_t k0, int64_t k_valid, uint32_t lds,
                                               int wave, int lane, int64_t tok = 0) {
#pragma unroll
    for (int j = J0; j < J1; ++j) {
      const int blk = wave * PER_WAVE + j;
      const int off = blk * 1024 + lane * 16;
      const int row = off / ROWB, pos = (off % ROWB) / 16;
      const int c = swz_row<ROWB>(row, pos);   // the swizzle is an involution in the chunk index
      const int64_t grow = row0 + row, gk = k0 + (int64_t)c * KPC;
      int64_t idx = grow * ld + (KEPT ? gk / 2 : gk);
      if constexpr (KEPT) {
        if (tok > 0) idx = tiled_index<32>(grow, gk / 2, tok, ld);
      }
      const void* src = (grow < rows_valid && gk < k_valid) ? (const void*)(p + idx) : (const void*)g_dma_zero;
      dma_b128(src, __builtin_amdgcn_readfirstlane(lds + blk * 1024));
    }
  }
  // Unchecked path, for a tile and step that lie inside the matrix: the byte
  // offset of load j's chunk from the tile's first row at the step's first
  // contraction element (constant over the steps), and the issue from a
  // wave-uniform base.
  __device__ __forceinline__ static uint32_t lane_off(int j, int64_t ld, int wave, int lane) {
    const int blk = wave * PER_WAVE + j;
    const int off = blk * 1024 + lane * 16;
    const int row = off / ROWB, pos = (off % ROWB) / 16;
    return (uint32_t)row * (uint32_t)(ld * 2) + (uint32_t)swz_row<ROWB>(row, pos) * 16u;
  }
  __device__ __forceinline__ static const char* step_base(const uint16_t* p, int64_t ld, int64_t row0, int64_t k0) {
    return (const char*)(p + row0 * ld + (KEPT ? k0 / 2 : k0));
  }
  template <int J0, int J1>
  __device__ __forceinline__ static void issue_fast(const char* sbase, const uint32_t* voff, uint32_t lds, int wave) {
#pragma unroll
    for (int j = J0; j < J1; ++j) dma_b128_s(sbase, voff[j], lds + (wave * PER_WAVE + j) * 1024);
  }
};

// Metadata of a 2:4 tile: ROWS rows x MROWB bytes (8 MROWB dense K), dword
// DMA (256 bytes per wave instruction).
template <int ROWS, int MROWB, int NW>
struct DmaMeta {
  static constexpr int BLOCKS = ROWS * MROWB / 256;
  static constexpr int PER_WAVE = BLOCKS / NW;
  static_assert(BLOCKS % NW == 0, "meta blocks per wave");
  // tok > 0: the tiled layout with tok rows.
  template <int J0, int J1>
  __device__ __forceinline__ static void issue(const uint8_t* __restrict__ pm, int64_t ldm, int64_t row0,
                                               int64_t rows_valid, int64_t k0, int64_t k_valid, uint32_t lds,
                                               int wave, int lane, int64_t tok = 0) {
#pragma unroll
    for (int j = J0; j < J1; ++j) {
      const int blk = wave * PER_WAVE + j;
      const int off = blk * 256 + lane * 4;
      const int row = off / MROWB, dw = (off % MROWB) / 4;   // dword dw covers dense K 32 dw .. 32 dw + 31
      const int64_t grow = row0 + row;
      const int64_t idx = tok > 0 ? tiled_index<8>(grow, k0 / 8 + dw * 4, tok, ldm) : grow * ldm + k0 / 8 + dw * 4;
      const void* src = (grow < rows_valid && k0 + 32 * (dw + 1) <= k_valid) ? (const void*)(pm + idx)
                                                                             : (const void*)g_dma_zero;
      dma_b32(src, __builtin_amdgcn_readfirstlane(lds + blk * 256));
    }
  }
  __device__ __forceinline__ static uint32_t lane_off(int j, int64_t ldm, int wave, int lane) {
    const int blk = wave * PER_WAVE + j;
    const int off = blk * 256 + lane * 4;
    return (uint32_t)(off / MROWB) * (uint32_t)ldm + (uint32_t)(off % MROWB);
  }
  __device__ __forceinline__ static const char* step_base(const uint8_t* pm, int64_t ldm, int64_t row0, int64_t k0) {
    return (const char*)(pm + row0 * ldm + k0 / 8);
  }
  template <int J0, int J1>
  __device__ __forceinline__ static void issue_fast(const char* sbase, const uint32_t* voff, uint32_t lds, int wave) {
#pragma unroll
    for (int j = J0; j < J1; ++j) dma_b32_s(sbase, voff[j], lds + (wave * PER_WAVE + j) * 256);
  }
};

// ---- K-major tiles ----------------------------------------------------------
// A K-major operand (stored [K x rows], rows contiguous) is staged as it is:
// LDS row k (one per contraction index of the step, 64 of them) holds the
// tile's ROWS elements, in 32-byte chunks of 16 elements; chunk c of row k
// sits at chunk position c ^ 2 (k & 3).
//
// ds_read_b64_tr_b16 (gfx950, pinned by a probe): within each group of 16
// lanes, lane j reads 4 consecutive 16-bit elements; lane i of the group then
// receives element i % 4 of lane 4q + i/4's read, for q = 0..3.  When lane j
// reads row k0 + j/4 at columns c0 + 4 (j % 4), lane i therefore receives
// column c0 + i of rows k0..k0+3: one MFMA fragment half.  The 32 lanes
// served together touch rows k0..k0+3 at two adjacent logical chunks (c even,
// c + 1); the swizzle spreads these eight 32-byte pieces over eight distinct
// positions, i.e. all 64 banks (each row is a multiple of 256 bytes).
typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int km_swz(int k, int chunk) { return chunk ^ ((k & 3) << 1); }

// Fragment of a v_mfma_f32_32x32x16_bf16 operand from a K-major LDS tile:
// lane l gets columns col0 + l % 32, contraction indices 16 kk + 8 (l / 32) + 0..7.
template <int ROWS>
__device__ __forceinline__ bf16x8 frag_km(const char* base, int kk, int col0, int lane) {
  constexpr int ROWB = ROWS * 2;
  const int grp = lane >> 4, j = lane & 15;
  const int k = kk * 16 + 8 * (grp >> 1) + (j >> 2);
  const int col = col0 + 16 * (grp & 1) + 4 * (j & 3);
  const int c = col >> 4, w = (col & 15) * 2;
  const char* p0 = base + k * ROWB + (km_swz(k, c) << 5) + w;
  const char* p1 = base + (k + 4) * ROWB + (km_swz(k + 4, c) << 5) + w;
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p0);
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p1);
  const s16x4 lo = a, hi = b;
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, v);
}

// A dense K-major tile [64 x ROWS] copied by DMA: 1 KB blocks, PER_WAVE per
// wave; lane i fills the block's 16-byte unit i, i.e. physical unit (i mod
// units per row) of row (block rows + i / units per row), and fetches the
// global 8 elements that the swizzle maps there.
template <int ROWS, int NW>
struct DmaTileKM {
  static constexpr int ROWB = ROWS * 2;
  static constexpr int BLOCKS = 64 * ROWB / 1024;
  static constexpr int PER_WAVE = BLOCKS / NW;
  static_assert(BLOCKS % NW == 0 && ROWB <= 1024, "blocks per wave");
  template <int J0, int J1>
  __device__ __forceinline__ static void issue(const uint16_t* __restrict__ p, int64_t ld, int64_t col0,
                                               int64_t cols_valid, int64_t k0, int64_t k_valid, uint32_t lds,
                                               int wave, int lane) {
#pragma unroll
    for (int j = J0; j < J1; ++j) {
      const int blk = wave * PER_WAVE + j;
      const int off = blk * 1024 + lane * 16;
      const int k = off / ROWB, pu = (off % ROWB) / 16;
      const int col = km_swz(k, pu >> 1) * 16 + (pu & 1) * 8;
      const int64_t gk = k0 + k, gc = col0 + col;
      const void* src = (gk < k_valid && gc < cols_valid) ? (const void*)(p + gk * ld + gc) : (const void*)g_dma_zero;
      dma_b128(src, __builtin_amdgcn_readfirstlane(lds + blk * 1024));
    }
  }
  __device__ __forceinline__ static uint32_t lane_off(int j, int64_t ld, int wave, int lane) {
    const int blk = wave * PER_WAVE + j;
    const int off = blk * 1024 + lane * 16;
    const int k = off / ROWB, pu = (off % ROWB) / 16;
    const int col = km_swz(k, pu >> 1) * 16 + (pu & 1) * 8;
    return (uint32_t)k * (uint32_t)(ld * 2) + (uint32_t)col * 2u;
  }
  __device__ __forceinline__ static const char* step_base(const uint16_t* p, int64_t ld, int64_t col0, int64_t k0) {
    return (const char*)(p + k0 * ld + col0);
  }
  template <int J0, int J1>
  __device__ __forceinline__ static void issue_fast(const char* sbase, const uint32_t* voff, uint32_t lds, int wave) {
#pragma unroll
    for (int j = J0; j < J1; ++j) dma_b128_s(sbase, voff[j], lds + (wave * PER_WAVE + j) * 1024);
  }
};

// A 2:4 K-major tile: rows of kept values [K x cols/2] + metadata [K x cols/8]
// (the compressed activation read along tokens).  Each thread loads the kept
// values (16 bytes) and codes (2 bytes) of 16 consecutive features of one
// contraction row, and after the current step's MFMAs writes them expanded
// (32 bytes) into the K-major LDS tile; no transpose is needed.
template <int ROWS, int NT>
struct StagerKMSP {
  static constexpr int ROWB = ROWS * 2;
  static constexpr int CHUNKS = ROWS / 16;
  static constexpr int NU = 64 * CHUNKS / NT;
  static_assert((64 * CHUNKS) % NT == 0, "units per thread");
  // Unit q (16 features of one contraction row): chunk q % 4 of entry block
  // q / 256 (64 features) at row (q / 4) % 64, so that the 64 lanes of a wave
  // read 16 rows x 64 bytes of one entry block, 1 KB contiguous in the tiled
  // layout.
  __device__ __forceinline__ static int unit_k(int q) { return (q >> 2) & 63; }
  __device__ __forceinline__ static int unit_c(int q) { return (q >> 8) * 4 + (q & 3); }
  uint4 v[NU];
  uint16_t m[NU];
  // The compressed tensor is in the tiled layout with tok rows (tokens =
  // contraction rows here).
  // The step's rows k0 .. k0+63 lie in one block of 256 rows (R of them
  // exist), so every piece is a 32-bit offset from the step's block start.
  __device__ __forceinline__ void load(const uint16_t* __restrict__ pv, int64_t ldv, const uint8_t* __restrict__ pm,
                                       int64_t ldm, int64_t col0, int64_t cols_valid, int64_t k0, int64_t k_valid,
                                       int tid, int64_t tok) {
    const int64_t tb0 = k0 & ~(int64_t)255;
    const int R = (int)(tok - tb0 < 256 ? tok - tb0 : 256);
    const uint16_t* vb = pv + tiled_step<32>(k0, col0, tok, ldv);
    const uint8_t* mb = pm + tiled_step<8>(k0, col0, tok, ldm);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int q = u * NT + tid, k = unit_k(q), c = unit_c(q);
      const int64_t gk = k0 + k, f = col0 + 16 * c;
      v[u] = make_uint4(0u, 0u, 0u, 0u);
      m[u] = 0u;
      if (gk < k_valid && f < cols_valid) {
        v[u] = *(const uint4*)(vb + ((c >> 2) * R * 32 + k * 32 + (c & 3) * 8));
        m[u] = *(const uint16_t*)(mb + ((c >> 2) * R * 8 + k * 8 + (c & 3) * 2));
      }
    }
  }
  // Unchecked path (tile and step inside the matrix, step inside a full block
  // of 256 rows): per-lane byte offsets from the step's block start
  // (tiled_step of its first row and the tile's first column), constant over
  // the steps, and a wave-uniform base per step.  Thread unit (k, c) reads
  // entry block c / 4 at row k, entries 8 (c % 4) .. (values) and 2 (c % 4) ..
  // (metadata bytes).
  __device__ __forceinline__ static void lane_offs(int tid, uint32_t (&ov)[NU], uint32_t (&om)[NU]) {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int q = u * NT + tid, k = unit_k(q), c = unit_c(q);
      ov[u] = (uint32_t)((c >> 2) * 256 * 32 + k * 32 + (c & 3) * 8) * 2u;
      om[u] = (uint32_t)((c >> 2) * 256 * 8 + k * 8 + (c & 3) * 2);
    }
  }
  __device__ __forceinline__ void load_fast(const char* vbase, const char* mbase, const uint32_t (&ov)[NU],
                                            const uint32_t (&om)[NU]) {
    const char* vb = (const char*)uniform_ptr(vbase);
    const char* mb = (const char*)uniform_ptr(mbase);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const u32x4 x = *(const __attribute__((address_space(1))) u32x4*)(vb + ov[u]);
      v[u] = make_uint4(x[0], x[1], x[2], x[3]);
      m[u] = *(const __attribute__((address_space(1))) uint16_t*)(mb + om[u]);
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int q = u * NT + tid, k = unit_k(q), c = unit_c(q);
      char* dst = lds + k * ROWB + (km_swz(k, c) << 5);
      *(uint4*)dst = expand2(make_uint2(v[u].x, v[u].y), m[u] & 0xFFu);
      *(uint4*)(dst + 16) = expand2(make_uint2(v[u].z, v[u].w), m[u] >> 8);
    }
  }
};

// XCD-aware placement: consecutive workgroup ids go to different XCDs (8 on
// MI355X), so remap them so that each XCD receives a contiguous range of
// logical tiles, which then share operand rows in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int pid, int total) {
  constexpr int kXcd = 8;
  const int full = total / kXcd * kXcd;
  if (pid >= full) return pid;
  return (pid % kXcd) * (full / kXcd) + pid / kXcd;
}

// Persistent schedule of the direct-staged kernels: the grid holds at most
// one workgroup per CU, and workgroup b runs tiles first, first + stride, ...
// (< end).  Workgroup ids are dealt to the 8 XCDs round-robin; each XCD gets a
// contiguous share of the tiles, which its workgroups interleave, so the
// tiles in flight on one XCD are neighbours sharing operand rows in its L2.
struct TileRange {
  int first, stride, end;
};
__device__ __forceinline__ TileRange tile_range(int b, int grid, int ntiles) {
  constexpr int kXcd = 8;
  if (grid % kXcd != 0) return {b, grid, ntiles};
  const int x = b % kXcd;
  const int start = (int)((int64_t)x * ntiles / kXcd), end = (int)((int64_t)(x + 1) * ntiles / kXcd);
  return {start + b / kXcd, grid / kXcd, end};
}

template <class Cfg>
__global__ __launch_bounds__(Cfg::NT) void gemm_kernel(const GemmArgs g) {
  constexpr int BM = Cfg::BM, BN = Cfg::BN, BK = Cfg::BK, NT = Cfg::NT, NW = Cfg::NW;
  constexpr int FM = Cfg::FM, FN = Cfg::FN, TM = Cfg::TM, TN = Cfg::TN;
  constexpr bool SPARSE = Cfg::SPARSE;
  constexpr int STAGES = Cfg::STAGES;
  __shared__ __attribute__((aligned(1024))) char smem[Cfg::LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, so derived LDS bases are scalar
  const int wm = wave / Cfg::WAVES_N, wn = wave % Cfg::WAVES_N;
  const int ntiles = g.tiles_m * g.tiles_n;
  // Split-K grids (gridDim.y contraction splits, a multiple of 8): workgroup
  // ids go to the 8 XCDs round-robin in launch order; remap them so that each
  // XCD runs whole splits (every tile of a contraction range), whose tiles
  // read the same rows of both operands at the same time through its L2.
  int bx = blockIdx.x, by = blockIdx.y;
  if (gridDim.y > 1 && gridDim.y % 8 == 0) {
    const int L = blockIdx.x + gridDim.x * blockIdx.y, x = L % 8, j = L / 8;
    by = x * (gridDim.y / 8) + j / gridDim.x;
    bx = j % gridDim.x;
  }
  const int64_t kbeg = (int64_t)by * g.k_split;
  const int64_t kend = kbeg + g.k_split < g.K ? kbeg + g.k_split : g.K;
  const int nsteps = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;
  // EPI_DH_STE: a tile runs its K steps twice, over the two operand pairs
  constexpr bool TWO = Cfg::EPI == EPI_DH_STE;
  const int tsteps = TWO ? 2 * nsteps : nsteps;
  const int lrow = lane & 31, lhalf = lane >> 5;
  // Panel of this workgroup's XCD (m_groups > 1): M tiles [pm_begin, +pm_count),
  // N tiles from pn_begin; tiles are then numbered locally, M fastest.
  const bool panels = Cfg::M_FAST && g.m_groups > 1 && gridDim.x % 8 == 0 && 8 % g.m_groups == 0;
  int pm_begin = 0, pm_count = g.tiles_m, pn_begin = 0, pn_count = g.tiles_n;
  if (panels) {
    const int x = blockIdx.x % 8, per = 8 / g.m_groups, gi = x % g.m_groups, xi = x / g.m_groups;
    pm_begin = gi * g.tiles_m / g.m_groups;
    pm_count = (gi + 1) * g.tiles_m / g.m_groups - pm_begin;
    pn_begin = xi * g.tiles_n / per;
    pn_count = (xi + 1) * g.tiles_n / per - pn_begin;
  }
  auto origin = [&](int tile, int64_t& m0, int64_t& n0) __attribute__((always_inline)) {
    int tm, tn;
    if (panels) {
      tm = pm_begin + tile % pm_count;
      tn = pn_begin + tile / pm_count;
    } else {
      tm = Cfg::M_FAST ? tile % g.tiles_m : tile / g.tiles_n;
      tn = Cfg::M_FAST ? tile / g.tiles_m : tile % g.tiles_n;
    }
    m0 = (int64_t)tm * BM;
    n0 = (int64_t)tn * BN;
  };

  f32x16 acc[FM][FN];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  };
  // EPI_DH_STE: relu(h) of the tile (h = the first pair's product), rounded
  // to bf16 and packed in pairs in the accumulator layout, kept in registers
  // while the second pair accumulates dS^T.
  uint32_t hst[TWO ? FM : 1][TWO ? FN : 1][8];
  auto stash_h = [&]() __attribute__((always_inline)) {
    if constexpr (TWO) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int q = 0; q < 8; ++q) hst[i][j][q] = bf16x2_rne(relu_f32(acc[i][j][2 * q]), relu_f32(acc[i][j][2 * q + 1]));
      zero_acc();
    }
  };

  // MFMAs of one K step on the LDS stage at `base`.  Fragments of sub-step
  // kk+1 are read while sub-step kk's MFMAs run; hook(kk) runs between the
  // reads and the MFMAs of sub-step kk (it issues part of the next stage's
  // loads in the direct path).
  auto compute = [&](const char* lA, const char* lB, auto&& hook) __attribute__((always_inline)) {
    const char* lM = lA + Cfg::A_BYTES;
    if constexpr (!SPARSE) {
      bf16x8 af[2][FM], bfr[2][FN];
      auto read = [&](int kk, int slot) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          if constexpr (Cfg::A_KM) {
            af[slot][i] = frag_km<BM>(lA, kk, wm * TM + i * 32, lane);
          } else {
            const int row = wm * TM + i * 32 + lrow;
            af[slot][i] = *(const bf16x8*)(lA + row * 128 + swz(row, 2 * kk + lhalf) * 16);
          }
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (Cfg::B_KM) {
            bfr[slot][j] = frag_km<BN>(lB, kk, wn * TN + j * 32, lane);
          } else {
            const int row = wn * TN + j * 32 + lrow;
            bfr[slot][j] = *(const bf16x8*)(lB + row * 128 + swz(row, 2 * kk + lhalf) * 16);
          }
        }
      };
      if constexpr (Cfg::PIPE) read(0, 0);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {       // four k16 MFMA steps per 64-wide K step
        const int cur = Cfg::PIPE ? (kk & 1) : 0;
        if constexpr (Cfg::PIPE) {
          if (kk + 1 < 4) read(kk + 1, cur ^ 1);
        } else {
          read(kk, 0);
        }
        hook(kk);
        // keep the reads of sub-step kk+1 ahead of this sub-step's MFMAs (the
        // scheduler would otherwise sink each read next to its consumer)
        if constexpr (Cfg::PIN) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = Cfg::SWAP ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][j], af[cur][i], acc[i][j], 0, 0, 0)
                                  : __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
        if constexpr (Cfg::PIN) __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      constexpr int KK = Cfg::KK;
      uint32_t meta[FM][KK];   // metadata word of sub-step kk (32 dense K) of each row block
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * TM + i * 32 + lrow;
        if constexpr (KK == 4) {
          const uint4 w = *(const uint4*)(lM + row * 16);
          meta[i][0] = w.x; meta[i][1] = w.y; meta[i][2] = w.z; meta[i][3] = w.w;
        } else {
          const uint2 w = *(const uint2*)(lM + row * 8);
          meta[i][0] = w.x; meta[i][1] = w.y;
        }
      }
      bf16x8 af[2][FM];
      bf16x16 bfr[2][FN];
      auto read = [&](int kk, int slot) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < FM; ++i) {
          const int row = wm * TM + i * 32 + lrow;
          af[slot][i] = *(const bf16x8*)(lA + row * Cfg::A_ROWB + swz_row<Cfg::A_ROWB>(row, 2 * kk + lhalf) * 16);
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int row = wn * TN + j * 32 + lrow;
          constexpr int RB = Cfg::B_ROWB;
          const bf16x8 lo = *(const bf16x8*)(lB + row * RB + swz_row<RB>(row, 4 * kk + lhalf) * 16);
          const bf16x8 hi = *(const bf16x8*)(lB + row * RB + swz_row<RB>(row, 4 * kk + 2 + lhalf) * 16);
          bfr[slot][j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
        }
      };
      read(0, 0);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {      // 32-wide smfmac sub-steps
        const int cur = kk & 1;
        if (kk + 1 < KK) read(kk + 1, cur ^ 1);
        hook(kk);
        int idx[FM];
#pragma unroll
        for (int i = 0; i < FM; ++i) idx[i] = (int)(meta[i][kk] >> (16 * lhalf));
        if constexpr (Cfg::PIN) __builtin_amdgcn_sched_barrier(0);   // reads of kk+1 stay ahead of these MFMAs
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_smfmac_f32_32x32x32_bf16(af[cur][i], bfr[cur][j], acc[i][j], idx[i], 0, 0);
        if constexpr (Cfg::PIN) __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  // ---------------------------------------------------------------- epilogues
  // Writes the tile at (m0, n0); `stage` is an LDS stage buffer that no copy
  // is filling (the staged epilogues use it).  EPI_F32 writes a stream-K
  // partial tile to f32_slot when it is set, else the split's partial rows.
  float* f32_slot = nullptr;
  // `pre` runs in the staged epilogues once every wave has finished the
  // main loop's LDS reads (EPI_DH with PRE_S: it issues the next tile's first
  // loads and waits for the S tile copied during the last K step).
  auto epilogue = [&](const int64_t m0, const int64_t n0, char* stage, auto&& pre) __attribute__((always_inline)) {
    if constexpr (Cfg::SWAP) {
      // Accumulator 4b+q of lane l is C[row l%32][col 8b + 4h + q] of its 32x32
      // block (h = l / 32).  N is a multiple of 8, so each 8-column (bf16) or
      // 4-column (fp32) piece is wholly inside or outside the matrix.
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int64_t row = m0 + wm * TM + i * 32 + lrow;
          const int64_t colb = n0 + wn * TN + j * 32;
          if constexpr (Cfg::EPI == EPI_BF16) {
            // pk[b]: columns 8b+4h .. +3 as two bf16 pairs.  One permlane32 swap
            // per dword gives lane half 0 columns 0..15 and half 1 columns 16..31.
            uint32_t pk[4][2];
#pragma unroll
            for (int b = 0; b < 4; ++b)
#pragma unroll
              for (int e = 0; e < 2; ++e)
                pk[b][e] = bf16x2_rne(acc[i][j][4 * b + 2 * e], acc[i][j][4 * b + 2 * e + 1]);
            uint32_t out[2][4];
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
              for (int e = 0; e < 2; ++e) {
                const auto sw = __builtin_amdgcn_permlane32_swap(pk[c][e], pk[c + 2][e], false, false);
                out[c][e] = sw[0];       // half 0: columns 8c + 2e ..; half 1: 16 + 8c + 2e ..
                out[c][2 + e] = sw[1];   // half 0: columns 8c + 4 + 2e ..; half 1: 16 + 8c + 4 + 2e ..
              }
            const int64_t col = colb + 16 * lhalf;
            if (row < g.M) {
              __bf16* dst = (__bf16*)g.C + row * g.ldc + col;
#pragma unroll
              for (int c = 0; c < 2; ++c)
                if (col + 8 * c < g.N) *(uint4*)(dst + 8 * c) = make_uint4(out[c][0], out[c][1], out[c][2], out[c][3]);
            }
          } else if (f32_slot != nullptr) {
            // stream-K partial: the whole tile, tile-local rows and columns
            float* dst = f32_slot + (row - m0) * BN + (colb - n0);
#pragma unroll
            for (int b = 0; b < 4; ++b)
              *(float4*)(dst + 8 * b + 4 * lhalf) =
                  make_float4(acc[i][j][4 * b], acc[i][j][4 * b + 1], acc[i][j][4 * b + 2], acc[i][j][4 * b + 3]);
          } else {
            float* part = (float*)g.C + (int64_t)by * g.M * g.N;
            if (row < g.M) {
#pragma unroll
              for (int b = 0; b < 4; ++b) {
                const int64_t col = colb + 8 * b + 4 * lhalf;
                if (col < g.N)
                  *(float4*)(part + row * g.N + col) =
                      make_float4(acc[i][j][4 * b], acc[i][j][4 * b + 1], acc[i][j][4 * b + 2], acc[i][j][4 * b + 3]);
              }
            }
          }
        }
    } else if constexpr (Cfg::EPI == EPI_F32) {
      // 2:4 products, split-K partial rows (layout as below): 32 lanes store
      // 32 consecutive columns of one row per accumulator.
      float* part = (float*)g.C + (int64_t)by * g.M * g.N;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int64_t col = n0 + wn * TN + j * 32 + lrow;
          const int64_t row = m0 + wm * TM + i * 32 + lhalf * 4;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int dr = (e / 4) * 8 + (e % 4);
            if (row + dr < g.M && col < g.N) part[(row + dr) * g.N + col] = acc[i][j][e];
          }
        }
    } else if constexpr (Cfg::EPI == EPI_BF16) {
      // 2:4 products (the sparse operand stays the MFMA's first): accumulator
      // 4b+q of lane l is C[row 8b + 4h + q][col l%32] of its 32x32 block.
      const bool inside = m0 + BM <= g.M && n0 + BN <= g.N;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int64_t col = n0 + wn * TN + j * 32 + lrow;
          const int64_t row = m0 + wm * TM + i * 32 + lhalf * 4;
          __bf16* base = (__bf16*)g.C + row * g.ldc + col;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int dr = (e / 4) * 8 + (e % 4);
            if (inside || (row + dr < g.M && col < g.N)) base[dr * g.ldc] = (__bf16)acc[i][j][e];
          }
        }
    } else if constexpr (Cfg::EPI == EPI_ACT_DENSE || Cfg::EPI == EPI_DH_DENSE || Cfg::EPI == EPI_DH_STE) {
      // C rows are features f, columns tokens t: accumulators 4b..4b+3 of a
      // lane are features 8b + 4h + 0..3 of token column l % 32.  Lanes l and
      // l+32 exchange halves so that each writes 16 contiguous features
      // (half 0: 0..15, half 1: 16..31 of the 32-row block) of its token row.
      // (EPI_DH_STE: the lane index laundered, so that the store offsets are
      // formed here rather than kept live beside the stashed relu(h).)
      int lr = lrow, lh = lhalf;
      if constexpr (Cfg::EPI == EPI_DH_STE) asm volatile("" : "+v"(lr), "+v"(lh));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int64_t t = n0 + wn * TN + j * 32 + lr;
          const int64_t f32 = m0 + wm * TM + i * 32;
          uint2 mine[4];   // block b: features f32 + 8b + 4h .. +3 as 4 bf16
          if constexpr (Cfg::EPI == EPI_ACT_DENSE) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              uint32_t v[2];
#pragma unroll
              for (int e = 0; e < 2; ++e) {
                // h relu'd and rounded to bf16 (RNE), squared (act_square) and rounded
                const uint32_t r = bf16x2_rne(relu_f32(acc[i][j][4 * b + 2 * e]), relu_f32(acc[i][j][4 * b + 2 * e + 1]));
                if (g.act_square) {
                  const float lo = __builtin_bit_cast(float, r << 16), hi = __builtin_bit_cast(float, r & 0xFFFF0000u);
                  v[e] = bf16x2_rne(lo * lo, hi * hi);
                } else {
                  v[e] = r;
                }
              }
              mine[b] = make_uint2(v[0], v[1]);
            }
          } else if constexpr (Cfg::EPI == EPI_DH_STE) {
            // relu(h) from the stash: accumulator 4b + q of the h product is
            // feature 8b + 4h + q, as for dS
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              uint32_t v[2];
#pragma unroll
              for (int e = 0; e < 2; ++e) {
                const uint32_t rr = hst[i][j][2 * b + e];
                v[e] = bf16x2_rne(acc[i][j][4 * b + 2 * e] * 2.0f * __builtin_bit_cast(float, rr << 16),
                                  acc[i][j][4 * b + 2 * e + 1] * 2.0f * __builtin_bit_cast(float, rr & 0xFFFF0000u));
              }
              mine[b] = make_uint2(v[0], v[1]);
            }
          } else {
            float x[4][4];   // the stored activation of features 8b + 4h + 0..3
            // a subnormal stored s (the raw square root flushes it): bit
            // pattern v in [1, 0x7F], tested as (v - 1) mod 2^16 < 0x7F on the
            // smallest of the lane's values (packed 16-bit integer arithmetic)
            u16x2 vmin = {0xFFFFu, 0xFFFFu};
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              const int64_t f = f32 + 8 * b + 4 * lh;
              uint2 a = make_uint2(0u, 0u);
              if (t < g.N && f < g.f_valid) a = *(const uint2*)(g.act + t * g.ld_act + f);
#pragma unroll
              for (int e = 0; e < 2; ++e) {
                const uint32_t w = e ? a.y : a.x;
                x[b][2 * e] = __builtin_bit_cast(float, w << 16);
                x[b][2 * e + 1] = __builtin_bit_cast(float, w & 0xFFFF0000u);
                vmin = __builtin_elementwise_min(vmin, __builtin_bit_cast(u16x2, w) - (u16x2){1u, 1u});
              }
            }
            const bool tiny = (vmin[0] < vmin[1] ? vmin[0] : vmin[1]) < 0x7Fu;
            if (g.act_square) {   // r = bf16(sqrt(s)) recovers relu(h) exactly
              float rt[4][4];
              if (__builtin_amdgcn_ballot_w64(tiny) == 0) {
#pragma unroll
                for (int b = 0; b < 4; ++b)
#pragma unroll
                  for (int q = 0; q < 4; ++q) rt[b][q] = __builtin_amdgcn_sqrtf(x[b][q]);
              } else {
#pragma unroll
                for (int b = 0; b < 4; ++b)
#pragma unroll
                  for (int q = 0; q < 4; ++q) rt[b][q] = sqrt_for_bf16(x[b][q]);
              }
#pragma unroll
              for (int b = 0; b < 4; ++b)
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                  const uint32_t rr = bf16x2_rne(rt[b][2 * e], rt[b][2 * e + 1]);
                  x[b][2 * e] = __builtin_bit_cast(float, rr << 16);
                  x[b][2 * e + 1] = __builtin_bit_cast(float, rr & 0xFFFF0000u);
                }
            }
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              uint32_t v[2];
#pragma unroll
              for (int e = 0; e < 2; ++e)
                v[e] = bf16x2_rne(acc[i][j][4 * b + 2 * e] * 2.0f * x[b][2 * e],
                                  acc[i][j][4 * b + 2 * e + 1] * 2.0f * x[b][2 * e + 1]);
              mine[b] = make_uint2(v[0], v[1]);
            }
          }
          // Half 0 keeps features 0..15 of the block, half 1 features 16..31:
          // swapping (block 0, block 2) and (block 1, block 3) across the halves
          // leaves each lane two runs of 8 consecutive features.
          uint32_t lo[4], hi[4];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const auto s0 = __builtin_amdgcn_permlane32_swap(e ? mine[0].y : mine[0].x, e ? mine[2].y : mine[2].x,
                                                             false, false);
            const auto s1 = __builtin_amdgcn_permlane32_swap(e ? mine[1].y : mine[1].x, e ? mine[3].y : mine[3].x,
                                                             false, false);
            lo[e] = s0[0];
            lo[2 + e] = s0[1];
            hi[e] = s1[0];
            hi[2 + e] = s1[1];
          }
          const int64_t f = f32 + 16 * lh;
          if (t < g.N) {
            uint16_t* dst = (Cfg::EPI == EPI_ACT_DENSE ? g.act : g.dact) + t * g.ld_act + f;
            if (f + 8 <= g.f_valid) *(uint4*)dst = make_uint4(lo[0], lo[1], lo[2], lo[3]);
            if (f + 16 <= g.f_valid) *(uint4*)(dst + 8) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
          }
        }
    } else {
      static_assert(Cfg::STAGED_EPI, "epilogue mode");
      // C rows are features f, columns tokens t.  Accumulators 4b..4b+3 of a
      // lane are features 8b + 4h + 0..3 of a 32-row block: one whole group of
      // 4 (Algorithm 1).  Lanes l and l+32 hold the even and odd groups of the
      // same 8 features, i.e. the two nibbles of one metadata byte.
      //
      // The tile's compressed rows (one per token: BM/2 kept values and BM/8
      // metadata bytes) are staged in LDS so that global memory sees whole
      // 16-byte (values) and 8-byte (metadata) pieces of each token row.  The
      // values go to the stage buffer of the tile's last K step (free once its
      // MFMAs are done, while the next tile's first loads fill the other one),
      // with 16-byte chunk c of token row t stored at chunk c ^ (t % 16): the
      // lanes of a wave, which touch 32 token rows at one column, then spread
      // over the banks.  Metadata rows (padded by 4 bytes) sit after the stages.
      constexpr int MP = Cfg::META_PITCH;   // bytes per LDS row of metadata (BM/8 + pad)
      char* lv = stage;                     // kept values, one BM-byte row per token (chunk-swizzled)
      char* lm = smem + STAGES * Cfg::STAGE;
      // byte offset of 4-byte word w of token row t's kept values
      auto val_word = [](int t, int w) __attribute__((always_inline)) { return t * BM + ((w >> 2) ^ (t & 15)) * 16 + (w & 3) * 4; };
      const int64_t t_end = g.N - n0;                      // valid tokens in this tile (may exceed BN)
      const int64_t f_end = g.M - m0;                      // valid features (multiple of 64)
      __syncthreads();                                     // main-loop LDS reads are finished

      if constexpr (Cfg::PRE_S) {
        pre();            // the S tile is in LDS (copied during the last K step)
        __syncthreads();
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int tl = wn * TN + j * 32 + lrow;         // token within the tile
          const int fl = wm * TM + i * 32;                // first feature of the 32-row block
          const bool ok = tl < t_end && fl < f_end;
          uint32_t pair[4], codes = 0;
          if constexpr (Cfg::EPI == EPI_SPARSIFY) {
            uint32_t codes = 0;   // code of group b at bits 8b .. 8b+3
#pragma unroll
            for (int b = 0; b < 4; ++b) {
              // h relu'd and rounded to bf16 (RNE; the same bits as rounding
              // first, as the rounding keeps the sign), ranked (ties to the
              // lower index)
              const uint32_t p01 = bf16x2_rne(relu_f32(acc[i][j][4 * b]), relu_f32(acc[i][j][4 * b + 1]));
              const uint32_t p23 = bf16x2_rne(relu_f32(acc[i][j][4 * b + 2]), relu_f32(acc[i][j][4 * b + 3]));
              const Top2 t = top2_keys_hi(p01, p23);
              codes |= top2_code_xor15(t) << (8 * b);
              const float a = __builtin_bit_cast(float, t.first << 2);
              const float c = __builtin_bit_cast(float, t.second << 2);
              pair[b] = bf16x2_rne(a * a, c * c);   // s = relu(h)^2 of the kept pair, index order
            }
            codes ^= 0x0F0F0F0Fu;
            // metadata byte b = code of group 2b (lane half 0) | code of group
            // 2b+1 (half 1) << 4; the swap hands half 0 its partner's codes
            const uint32_t other_codes = __builtin_amdgcn_permlane32_swap(codes, codes, false, false)[1];
            if (ok) {
#pragma unroll
              for (int b = 0; b < 4; ++b)
                *(uint32_t*)(lv + val_word(tl, fl / 4 + 2 * b + lhalf)) = pair[b];
              if (lhalf == 0) *(uint32_t*)(lm + tl * MP + fl / 8) = codes | (other_codes << 4);
            }
          } else {
            // EPI_DH: scale dS at the kept positions of the stored group by
            // 2 relu(h), relu(h) = bf16(sqrt(s)) exactly; result in place.
            if (ok) {
              // group b's code at bits 8b .. 8b+3
              const uint32_t w = *(const uint32_t*)(lm + tl * MP + fl / 8) >> (4 * lhalf);
              uint32_t* loc[4];
              float s[4][2], rt[4][2];
              // a subnormal s (the raw square root flushes it): a positive
              // subnormal bf16 is a bit pattern v in [1, 0x7F], i.e. (v - 1)
              // mod 2^16 < 0x7F; the smallest over the lane's eight values
              // decides (packed 16-bit integer arithmetic)
              u16x2 vmin = {0xFFFFu, 0xFFFFu};
#pragma unroll
              for (int b = 0; b < 4; ++b) {
                loc[b] = (uint32_t*)(lv + val_word(tl, fl / 4 + 2 * b + lhalf));
                const uint32_t sv = *loc[b];
                s[b][0] = __builtin_bit_cast(float, sv << 16);
                s[b][1] = __builtin_bit_cast(float, sv & 0xFFFF0000u);
                vmin = __builtin_elementwise_min(vmin, __builtin_bit_cast(u16x2, sv) - (u16x2){1u, 1u});
              }
              const bool tiny = (vmin[0] < vmin[1] ? vmin[0] : vmin[1]) < 0x7Fu;
              if (__builtin_amdgcn_ballot_w64(tiny) == 0) {
#pragma unroll
                for (int b = 0; b < 4; ++b)
#pragma unroll
                  for (int e = 0; e < 2; ++e) rt[b][e] = __builtin_amdgcn_sqrtf(s[b][e]);
              } else {
#pragma unroll
                for (int b = 0; b < 4; ++b)
#pragma unroll
                  for (int e = 0; e < 2; ++e) rt[b][e] = sqrt_for_bf16(s[b][e]);
              }
#pragma unroll
              for (int b = 0; b < 4; ++b) {
                const uint32_t i0 = __builtin_amdgcn_ubfe(w, 8 * b, 2), i1 = __builtin_amdgcn_ubfe(w, 8 * b + 2, 2);
                float ds[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) ds[q] = acc[i][j][4 * b + q];
                const float d0 = i0 == 0u ? ds[0] : i0 == 1u ? ds[1] : ds[2];
                const float d1 = i1 == 1u ? ds[1] : i1 == 2u ? ds[2] : ds[3];
                const uint32_t rr = bf16x2_rne(rt[b][0], rt[b][1]);   // relu(h), exact
                const float r0 = __builtin_bit_cast(float, rr << 16);
                const float r1 = __builtin_bit_cast(float, rr & 0xFFFF0000u);
                *loc[b] = bf16x2_rne(d0 * 2.0f * r0, d1 * 2.0f * r1);
              }
            }
          }
        }
      __syncthreads();

      // LDS -> global in the tiled layout: the tile's tokens lie in one block
      // of 256 rows (R of them exist) and its features in BM/64 entry blocks,
      // each written as one contiguous run (64 bytes of values, 8 of metadata
      // per token).  Thread q takes 16-byte piece q % 4 of token (q / 4) % BN
      // in entry block q / (4 BN).
      uint16_t* dst = (Cfg::EPI == EPI_SPARSIFY ? g.sv : g.dv) + tiled_step<32>(n0, m0, g.tok, g.ldv);
      const int64_t Rb = g.tok - (n0 & ~(int64_t)255) < 256 ? g.tok - (n0 & ~(int64_t)255) : 256;
      // k2: thread index laundered, so that these offsets are formed here and
      // not kept live across the main loop (measured faster); b3 keeps them
      // (measured faster there, within its registers)
      int td = tid;
      if constexpr (Cfg::EPI == EPI_SPARSIFY) asm volatile("" : "+v"(td));
      // Iteration it covers NT/4 token rows of one entry block: row
      // (it % IPB) NT/4 + td/4, chunk td % 4 (LDS chunk position c ^ (row % 16)
      // = X ^ 4 kb with X fixed per thread), global offset kb R 32 + row 32 +
      // 8 (td % 4) = kb R 32 + (it % IPB) NT/4 32 + 8 td.
      constexpr int RPI = NT / 4, IPB = BN / RPI;
      static_assert(BN % RPI == 0 && BM == 256, "copy-out shape");
      const int t0 = td >> 2, X = (td & 3) ^ (t0 & 15);
#pragma unroll
      for (int it = 0; it < IPB * (BM / 64); ++it) {
        const int kb = it / IPB, rbase = (it % IPB) * RPI, row = rbase + t0;
        if (row < t_end && kb * 64 < f_end) {
          const uint32_t* sp = (const uint32_t*)(lv + row * BM + (X ^ (kb << 2)) * 16);
          // non-temporal: the compressed rows stream out and should not evict
          // the weight panel this XCD keeps in L2
          const u32x4 v = {sp[0], sp[1], sp[2], sp[3]};
          __builtin_nontemporal_store(v, (u32x4*)(dst + kb * Rb * 32 + rbase * 32 + td * 8));
        }
      }
      if constexpr (Cfg::EPI == EPI_SPARSIFY) {
        uint8_t* mdst = g.sm + tiled_step<8>(n0, m0, g.tok, g.ldm);
        constexpr int MCH = BN * (BM / 64);
#pragma unroll
        for (int it = 0; it < (MCH + NT - 1) / NT; ++it) {
          const int q = it * NT + td, kbi = q / BN, row = q % BN;
          if (q < MCH && row < t_end && kbi * 64 < f_end) {
            const uint32_t* sp = (const uint32_t*)(lm + row * MP + kbi * 8);
            const u32x2 v = {sp[0], sp[1]};
            __builtin_nontemporal_store(v, (u32x2*)(mdst + kbi * Rb * 8 + row * 8));
          }
        }
      }
    }
  };

  if constexpr (Cfg::DIRECT) {
    using TA = std::conditional_t<Cfg::A_KM, DmaTileKM<BM, NW>, DmaTile<BM, Cfg::A_ROWB, SPARSE, NW>>;
    using TB = std::conditional_t<Cfg::B_KM, DmaTileKM<BN, NW>, DmaTile<BN, Cfg::B_ROWB, false, NW>>;
    using TMeta = DmaMeta<BM, (SPARSE ? Cfg::M_ROWB : 256), (SPARSE ? NW : 1)>;
    constexpr int LA = TA::PER_WAVE, LB = TB::PER_WAVE, LM = SPARSE ? TMeta::PER_WAVE : 0;
    constexpr int LOADS = LA + LB + LM;   // DMA instructions per wave per step
    const uint32_t smem_lds = lds_u32(smem);
    // Per-lane offsets of the unchecked path, relative to a tile's origin:
    // the same for every tile.
    uint32_t offA[LA], offB[LB], offM[LM > 0 ? LM : 1];
#pragma unroll
    for (int j = 0; j < LA; ++j) offA[j] = TA::lane_off(j, (SPARSE && g.a_tiled) ? 32 : g.lda, wave, lane);
#pragma unroll
    for (int j = 0; j < LB; ++j) offB[j] = TB::lane_off(j, g.ldb, wave, lane);
    if constexpr (SPARSE) {
#pragma unroll
      for (int j = 0; j < LM; ++j) offM[j] = TMeta::lane_off(j, g.a_tiled ? 8 : g.ldam, wave, lane);
    }
    // Steps [0, steps_in) of a tile inside both operands read no element
    // outside them: their loads skip the bounds checks.
    auto steps_in_of = [&](int64_t m0, int64_t n0) __attribute__((always_inline)) {
      int r = 0;
      if (m0 + BM <= g.m_valid && n0 + BN <= g.N) {
        const int64_t k_in = (g.ka_valid < g.kb_valid ? g.ka_valid : g.kb_valid) - kbeg;
        r = k_in <= 0 ? 0 : (int)(k_in / BK < nsteps ? k_in / BK : nsteps);
      }
      return __builtin_amdgcn_readfirstlane(r);
    };
    // Issue this wave's loads of step `step` of the tile at (m0, n0): the A
    // part (with its metadata) at LDS byte offset a_off, the B part at b_off.
    // The checked path (edge tiles, tail steps) passes k0 and the lane index
    // through an empty asm so that its addresses are formed afresh rather
    // than kept in loop-carried registers across the main loop.
    // EPI_DH_STE: steps nsteps .. 2 nsteps - 1 are the K steps of (A2, B2).
    auto issue_a = [&](int64_t m0, int s_in, int step, uint32_t a_off) __attribute__((always_inline)) {
      const bool second = TWO && step >= nsteps;
      if (second) step -= nsteps;
      const uint16_t* pa = second ? g.A2 : g.A;
      const int64_t k0 = kbeg + (int64_t)step * BK;
      const uint32_t base = smem_lds + a_off;
      if (step < s_in) {
        if (SPARSE && g.a_tiled) {
          // tiled 2:4 operand: the step is one contiguous block of rows x 32 values (8 bytes)
          TA::template issue_fast<0, LA>((const char*)(g.A + tiled_step<32>(m0, k0, g.tok, g.lda)), offA, base, wave);
          TMeta::template issue_fast<0, LM>((const char*)(g.Am + tiled_step<8>(m0, k0, g.tok, g.ldam)), offM,
                                            base + Cfg::A_BYTES, wave);
        } else {
          TA::template issue_fast<0, LA>(TA::step_base(pa, g.lda, m0, k0), offA, base, wave);
          if constexpr (SPARSE)
            TMeta::template issue_fast<0, LM>(TMeta::step_base(g.Am, g.ldam, m0, k0), offM, base + Cfg::A_BYTES, wave);
        }
      } else {
        int64_t kc = uniform_i64(k0);
        int lc = lane;
        asm volatile("" : "+s"(kc), "+v"(lc));
        if constexpr (SPARSE) {
          const int64_t tk = g.a_tiled ? g.tok : 0;
          TA::template issue<0, LA>(g.A, g.lda, m0, g.m_valid, kc, g.ka_valid, base, wave, lc, tk);
          TMeta::template issue<0, LM>(g.Am, g.ldam, m0, g.m_valid, kc, g.ka_valid, base + Cfg::A_BYTES, wave, lc, tk);
        } else {
          TA::template issue<0, LA>(pa, g.lda, m0, g.m_valid, kc, g.ka_valid, base, wave, lc);
        }
      }
    };
    auto issue_b = [&](int64_t n0, int s_in, int step, uint32_t b_off) __attribute__((always_inline)) {
      const bool second = TWO && step >= nsteps;
      if (second) step -= nsteps;
      const uint16_t* pb = second ? g.B2 : g.B;
      const int64_t k0 = kbeg + (int64_t)step * BK;
      const uint32_t base = smem_lds + b_off;
      const bool bblk = Cfg::B_BLOCKABLE && g.b_nsk > 0;
      if (step < s_in || bblk) {
        const char* sb = bblk ? (const char*)(pb + blocked_index(n0, k0, g.b_nsk)) : TB::step_base(pb, g.ldb, n0, k0);
        TB::template issue_fast<0, LB>(sb, offB, base, wave);
      } else {
        int64_t kc = uniform_i64(k0);
        int lc = lane;
        asm volatile("" : "+s"(kc), "+v"(lc));
        TB::template issue<0, LB>(pb, g.ldb, n0, g.N, kc, g.kb_valid, base, wave, lc);
      }
    };

    // Persistent schedule: this workgroup runs tiles first, first + stride,
    // ... (< end).  Steps are numbered across its tiles (gs = number of the
    // current tile's step 0); the loads issued ahead run on into the next
    // tile, so its first loads are in flight during this tile's last steps
    // and epilogue.
    const TileRange tr = panels ? TileRange{(int)blockIdx.x / 8, (int)gridDim.x / 8, pm_count * pn_count}
                                : tile_range(bx, gridDim.x, ntiles);
    if (tr.first >= tr.end) return;
    int tile = tr.first;
    int64_t m0, n0;
    origin(tile, m0, n0);
    int s_in = steps_in_of(m0, n0);
    int gs = 0;
    int next = tile + tr.stride;
    bool has_next = next < tr.end;
    int64_t nm0 = 0, nn0 = 0;
    int ns_in = 0;
    auto load_next = [&]() __attribute__((always_inline)) {
      nm0 = 0; nn0 = 0; ns_in = 0;
      if (has_next) {
        origin(next, nm0, nn0);
        ns_in = steps_in_of(nm0, nn0);
      }
    };
    load_next();
    // Issue cursors.  Every operand's source address is linear in the step
    // over a tile's unchecked steps (a prefix of its steps), so each operand
    // keeps the address of the next step it issues, the per-step stride and
    // the number of unchecked steps left.  At a tile's step 0 the general
    // address code sets the cursor up; an unchecked step is then the DMAs plus
    // a pointer add.  Eight waves run their scalar code on the CU's one
    // scalar unit, so the per-step scalar instruction count is what bounds
    // the copy issue.  The two-pair kernel sets its cursors up again at the
    // second pair's step 0.  (The dense-activation epilogues keep the general
    // path: with the cursors they measured no faster.)
    constexpr bool LEAN = Cfg::EPI != EPI_ACT_DENSE && Cfg::EPI != EPI_DH_DENSE;
    // A 2:4 operand's metadata advances by 1/8 of its kept values' stride
    // (tiled: 8 R against 64 R bytes; rows: BK/8 against BK bytes).  A stride
    // is at most BK rows of a pitch the entry points bound by 65536 elements
    // (about 8 MB), so 32 bits hold it.
    const char* ca_p = nullptr;   // A (kept values for a 2:4 operand)
    const char* ca_m = nullptr;   // its metadata
    uint32_t ca_st = 0;
    int ca_n = 0;
    const char* cb_p = nullptr;
    uint32_t cb_st = 0;
    int cb_n = 0;
    auto a_src = [&](int64_t tm0, int64_t k0, bool second, const char*& pv, const char*& pm) __attribute__((always_inline)) {
      if (SPARSE && g.a_tiled) {
        pv = (const char*)(g.A + tiled_step<32>(tm0, k0, g.tok, g.lda));
        pm = (const char*)(g.Am + tiled_step<8>(tm0, k0, g.tok, g.ldam));
      } else {
        pv = TA::step_base(TWO && second ? g.A2 : g.A, g.lda, tm0, k0);
        if constexpr (SPARSE) pm = TMeta::step_base(g.Am, g.ldam, tm0, k0);
      }
    };
    auto b_src = [&](int64_t tn0, int64_t k0, bool second) __attribute__((always_inline)) {
      const bool bblk = Cfg::B_BLOCKABLE && g.b_nsk > 0;
      return bblk ? (const char*)(g.B + blocked_index(tn0, k0, g.b_nsk))
                  : TB::step_base(TWO && second ? g.B2 : g.B, g.ldb, tn0, k0);
    };
    auto setup_a = [&](int64_t tm0, int tin, bool second) __attribute__((always_inline)) {
      const char *v0 = nullptr, *m0p = nullptr, *v1 = nullptr, *m1p = nullptr;
      a_src(tm0, kbeg, second, v0, m0p);
      a_src(tm0, kbeg + BK, second, v1, m1p);
      (void)m1p;
      ca_p = (const char*)uniform_ptr(v0);
      ca_st = __builtin_amdgcn_readfirstlane((uint32_t)(v1 - v0));
      if constexpr (SPARSE) ca_m = (const char*)uniform_ptr(m0p);
      ca_n = tin;
    };
    auto setup_b = [&](int64_t tn0, int tin, bool second) __attribute__((always_inline)) {
      const char* p0 = b_src(tn0, kbeg, second);
      cb_p = (const char*)uniform_ptr(p0);
      cb_st = __builtin_amdgcn_readfirstlane((uint32_t)(b_src(tn0, kbeg + BK, second) - p0));
      cb_n = (Cfg::B_BLOCKABLE && g.b_nsk > 0) ? nsteps : tin;
    };
    // Lookahead step x (relative to the current tile's step 0) lies in this
    // tile (x < tsteps) or in the next one; issue its A / B part if it exists.
    // A cursor is set up at step 0 of each operand pair of a tile.
    auto pair_start = [&](int x) __attribute__((always_inline)) {
      const int xs = x < tsteps ? x : x - tsteps;
      return xs == 0 || (TWO && xs == nsteps);
    };
    auto ahead_a = [&](int x, uint32_t a_off) __attribute__((always_inline)) {
      const bool here = x < tsteps;
      if (!(here || (has_next && x - tsteps < tsteps))) return;
      if constexpr (LEAN) {
        if (pair_start(x)) setup_a(here ? m0 : nm0, here ? s_in : ns_in, (here ? x : x - tsteps) >= nsteps);
        if (ca_n > 0) {
          const uint32_t base = smem_lds + a_off;
          TA::template issue_fast<0, LA>(ca_p, offA, base, wave);
          if constexpr (SPARSE) {
            TMeta::template issue_fast<0, LM>(ca_m, offM, base + Cfg::A_BYTES, wave);
            ca_m += ca_st >> 3;
          }
          ca_p += ca_st;
          --ca_n;
          return;
        }
      }
      issue_a(here ? m0 : nm0, here ? s_in : ns_in, here ? x : x - tsteps, a_off);
    };
    auto ahead_b = [&](int x, uint32_t b_off) __attribute__((always_inline)) {
      const bool here = x < tsteps;
      if (!(here || (has_next && x - tsteps < tsteps))) return;
      if constexpr (LEAN) {
        if (pair_start(x)) setup_b(here ? n0 : nn0, here ? s_in : ns_in, (here ? x : x - tsteps) >= nsteps);
        if (cb_n > 0) {
          TB::template issue_fast<0, LB>(cb_p, offB, smem_lds + b_off, wave);
          cb_p += cb_st;
          --cb_n;
          return;
        }
      }
      issue_b(here ? n0 : nn0, here ? s_in : ns_in, here ? x : x - tsteps, b_off);
    };
    auto exists = [&](int x) __attribute__((always_inline)) { return x < tsteps || (has_next && x - tsteps < tsteps); };
    // Steady-state issue from the cursors: the caller guarantees an unchecked
    // step of the current tile (so the counts are positive).
    auto fast_a = [&](uint32_t a_off) __attribute__((always_inline)) {
      const uint32_t base = smem_lds + a_off;
      TA::template issue_fast<0, LA>(ca_p, offA, base, wave);
      if constexpr (SPARSE) {
        TMeta::template issue_fast<0, LM>(ca_m, offM, base + Cfg::A_BYTES, wave);
        ca_m += ca_st >> 3;
      }
      ca_p += ca_st;
      --ca_n;
    };
    auto fast_b = [&](uint32_t b_off) __attribute__((always_inline)) {
      TB::template issue_fast<0, LB>(cb_p, offB, smem_lds + b_off, wave);
      cb_p += cb_st;
      --cb_n;
    };

    if constexpr (Cfg::DEEP != 0) {
      // The deep operand's stage of global step q is q % 3, the other's q % 2;
      // A's ring comes first.  Step s issues the shallow operand's step s+1,
      // then the deep one's step s+2.
      constexpr bool DA = Cfg::DEEP == 1;
      constexpr int LOADS_DEEP = DA ? LA + LM : LB;
      constexpr int NA = DA ? 3 : 2;
      auto a_off = [](int q) { return (uint32_t)((q % NA) * Cfg::A_PART); };
      auto b_off = [](int q) { return (uint32_t)(NA * Cfg::A_PART + (q % (DA ? 2 : 3)) * Cfg::B_BYTES); };
      // x: step relative to the current tile's step 0; q = gs + x
      auto ahead_deep = [&](int x, int q) __attribute__((always_inline)) {
        if constexpr (DA) ahead_a(x, a_off(q)); else ahead_b(x, b_off(q));
      };
      auto ahead_shallow = [&](int x, int q) __attribute__((always_inline)) {
        if constexpr (DA) ahead_b(x, b_off(q)); else ahead_a(x, a_off(q));
      };
      ahead_deep(0, 0);
      ahead_shallow(0, 0);
      ahead_deep(1, 1);
      for (;;) {
        zero_acc();
        for (int s = 0; s < tsteps; ++s) {
          if constexpr (LEAN) {
            // Steady state: steps 1 .. s_in - 3 issue unchecked steps s+1 and
            // s+2 of this tile from the cursors; ring positions advance
            // without a modulo.
            if (s == 1 || (TWO && s == nsteps + 1)) {
              // (two-pair kernel: each pair's run separately, so that the
              // cursor set-up at the second pair's step 0 and stash_h at the
              // first pair's last step stay in the general body)
              const int s_end = (TWO && s > nsteps ? nsteps : 0) + s_in - 2;
              int r3 = (gs + s) % 3, r2 = (gs + s) & 1;   // (gs + s) mod 3, mod 2
              for (; s < s_end; ++s) {
                wait_vmcnt<LOADS_DEEP>();
                lds_barrier();
                const int r3n2 = r3 == 0 ? 2 : r3 - 1;   // (gs + s + 2) mod 3
                const int a_r = DA ? r3 : r2, b_r = DA ? r2 : r3;   // stages of step s
                // the shallow operand's step s+1 before this step's MFMAs (it
                // is needed next step), the deep one's step s+2 after them
                if constexpr (DA) fast_b(NA * Cfg::A_PART + (r2 ^ 1) * Cfg::B_BYTES);
                else fast_a((r2 ^ 1) * Cfg::A_PART);
                compute(smem + a_r * Cfg::A_PART, smem + NA * Cfg::A_PART + b_r * Cfg::B_BYTES, [](int) {});
                if constexpr (DA) fast_a(r3n2 * Cfg::A_PART);
                else fast_b(NA * Cfg::A_PART + r3n2 * Cfg::B_BYTES);
                r3 = r3 == 2 ? 0 : r3 + 1;
                r2 ^= 1;
              }
              if (s >= tsteps) break;
            }
          }
          // Step s needs both operands' step s; the loads issued after the
          // shallow operand's step s are the deep one's step s+1 (issued with
          // it at step s-1).  At a tile's first step the previous epilogue's
          // stores are outstanding too: wait for all.
          if (s > 0 && exists(s + 1))
            wait_vmcnt<LOADS_DEEP>();
          else
            wait_vmcnt<0>();
          lds_barrier();   // every wave's loads of step s landed; step s-1's reads are done
          ahead_shallow(s + 1, gs + s + 1);
          ahead_deep(s + 2, gs + s + 2);
          compute(smem + a_off(gs + s), smem + b_off(gs + s), [](int) {});
          if (TWO && s == nsteps - 1) stash_h();
        }
        epilogue(m0, n0, smem, [] {});
        if (!has_next) break;
        gs += tsteps;
        tile = next;
        m0 = nm0;
        n0 = nn0;
        s_in = ns_in;
        next = tile + tr.stride;
        has_next = next < tr.end;
        load_next();
      }
    } else {
      // Stage (gs + s) % STAGES holds step s, A part then B part; step s
      // issues the loads STAGES - 1 steps ahead.
      auto st_off = [](int q) { return (uint32_t)((q % STAGES) * Cfg::STAGE); };
      // PRE_S: the stored S rows of the tile at (m0, n0) -> LDS by DMA, values
      // to the stage buffer at byte offset `off` (token row t's 16-byte chunk c
      // at chunk position c ^ (t % 16), the layout the epilogue reads) and
      // metadata rows to the area after the stages (pitch META_PITCH bytes).
      // Lanes whose piece lies outside the matrix (or in a row's pad dword)
      // copy the zero block.
      auto issue_s_tile = [&](int64_t tm0, int64_t tn0, uint32_t off) __attribute__((always_inline)) {
        if constexpr (Cfg::PRE_S) {
          const int64_t t_end = g.N - tn0, f_end = g.M - tm0;
          constexpr int VPW = BN * BM / 1024 / NW;    // 1 KB value blocks per wave
          static_assert((BN * BM / 1024) % NW == 0, "value blocks per wave");
          constexpr int MPD = Cfg::META_PITCH / 4;    // dwords per metadata row (the last is pad)
          constexpr int MPW = Cfg::META_DMA_PER_WAVE;
          const uint32_t lm_off = STAGES * Cfg::STAGE;
          // The stored S is tiled and the tile's tokens lie in one block of
          // 256 rows (R of them exist): value chunk c of token row t is
          // entries 8 (c % 4) .. of entry block c / 4, metadata dword w is
          // bytes 4 (w % 2) .. of entry block w / 2, at 32-bit offsets from
          // wave-uniform bases.  Pieces outside the matrix (rows >= t_end,
          // features >= f_end, a row's pad dword) re-read a valid piece of
          // the tile instead: the epilogue never reads those LDS positions.
          const int64_t Rb = g.tok - (tn0 & ~(int64_t)255) < 256 ? g.tok - (tn0 & ~(int64_t)255) : 256;
          const char* vbase = (const char*)(g.sv + tiled_step<32>(tn0, tm0, g.tok, g.ldv));
          const char* mbase = (const char*)(g.sm + tiled_step<8>(tn0, tm0, g.tok, g.ldm));
          const int t_last = (int)(t_end < BN ? t_end : BN) - 1;
          const int c_lim = (int)(f_end < BM ? f_end : BM) / 16;     // valid value chunks per row
          // lane index laundered so that the offsets are formed here rather
          // than hoisted out of the main loop into live registers
          int ln = lane;
          asm volatile("" : "+v"(ln));
#pragma unroll
          for (int j = 0; j < VPW; ++j) {
            const int blk = wave * VPW + j;
            const int b = blk * 1024 + ln * 16;
            int row = b / BM, c = ((b % BM) / 16) ^ (row & 15);
            row = row < t_last ? row : t_last;
            c = c < c_lim ? c : 0;
            const uint32_t o = (uint32_t)((c >> 2) * (int)Rb * 32 + row * 32 + (c & 3) * 8) * 2u;
            dma_b128_nt_s(vbase, o, smem_lds + off + blk * 1024);
          }
#pragma unroll
          for (int j = 0; j < MPW; ++j) {
            const int blk = wave * MPW + j;
            const int q = blk * 64 + ln;
            int row = q / MPD, w = q % MPD;
            row = row < t_last ? row : t_last;
            w = (w < MPD - 1 && 32 * w < f_end) ? w : 0;
            dma_b32_nt_s(mbase, (uint32_t)((w >> 1) * (int)Rb * 8 + row * 8 + (w & 1) * 4), smem_lds + lm_off + blk * 256);
          }
        }
      };
#pragma unroll
      for (int p = 0; p < STAGES - 1; ++p) {
        ahead_a(p, st_off(p));
        ahead_b(p, st_off(p) + Cfg::A_PART);
      }
      static_assert(!TWO || !Cfg::PRE_S, "two operand pairs with a plain epilogue");
      for (;;) {
        zero_acc();
        for (int s = 0; s < tsteps; ++s) {
          if constexpr (LEAN) {
            // Steady state: steps 1 .. s_in - STAGES + 1 issue unchecked
            // steps of this tile from the cursors (the later steps already
            // issued all exist, so the wait count is fixed); ring positions
            // advance without a modulo.
            if (s == 1 || (TWO && s == nsteps + 1)) {
              constexpr int W = STAGES >= 4 ? 2 * LOADS : STAGES == 3 ? LOADS : 0;
              const int s_end = (TWO && s > nsteps ? nsteps : 0) + s_in - (STAGES - 1);   // per operand pair
              int rc = (gs + s) % STAGES;   // stage of step s
              for (; s < s_end; ++s) {
                wait_vmcnt<W>();
                lds_barrier();
                const int ri = rc == 0 ? STAGES - 1 : rc - 1;   // stage of step s + STAGES - 1
                const char* st = smem + rc * Cfg::STAGE;
                if constexpr (STAGES == 2) {
                  fast_a(ri * Cfg::STAGE);
                  fast_b(ri * Cfg::STAGE + Cfg::A_PART);
                }
                compute(st, st + Cfg::A_PART, [](int) {});
                if constexpr (STAGES > 2) {
                  // copies of step s + STAGES - 1 after this step's MFMAs: its
                  // stage was last read in step s - 1 (before the barrier), and
                  // it has a whole step to land
                  fast_a(ri * Cfg::STAGE);
                  fast_b(ri * Cfg::STAGE + Cfg::A_PART);
                }
                rc = rc == STAGES - 1 ? 0 : rc + 1;
              }
              if (s >= tsteps) break;
            }
          }
          // wait for this wave's loads of step s.  The loads of the up to
          // STAGES - 2 later steps already issued (after those of s: memory
          // operations complete in issue order) may stay in flight.  At a
          // tile's first step the previous epilogue's stores are outstanding
          // too: wait for all.
          int ahead = 0;
          if (s > 0) {
#pragma unroll
            for (int j = 1; j <= STAGES - 2; ++j) ahead += exists(s + j) ? 1 : 0;
          }
          if (STAGES >= 4 && ahead >= 2)
            wait_vmcnt<2 * LOADS>();
          else if (STAGES >= 3 && ahead >= 1)
            wait_vmcnt<LOADS>();
          else
            wait_vmcnt<0>();
          lds_barrier();   // every wave's loads of step s landed; step s-1's reads are done
          const int la = s + STAGES - 1;
          if (Cfg::PRE_S && la == nsteps) {
            // last step: the free buffer takes this tile's S rows instead of
            // the next tile's first step
            issue_s_tile(m0, n0, st_off(gs + la));
          } else {
            ahead_a(la, st_off(gs + la));
            ahead_b(la, st_off(gs + la) + Cfg::A_PART);
          }
          const char* st = smem + st_off(gs + s);
          compute(st, st + Cfg::A_PART, [](int) {});
          if (TWO && s == nsteps - 1) stash_h();
        }
        if constexpr (Cfg::PRE_S) {
          // the next tile's first step goes to the buffer the last step read
          // (every wave is past those reads when `pre` runs); this tile's S
          // rows, issued before it, have landed once at most its LOADS remain
          const uint32_t q0 = st_off(gs + nsteps - 1);
          epilogue(m0, n0, smem + st_off(gs + nsteps), [&] {
            ahead_a(nsteps, q0);
            ahead_b(nsteps, q0 + Cfg::A_PART);
            if (has_next)
              wait_vmcnt<LOADS>();
            else
              wait_vmcnt<0>();
          });
        } else {
          const int last = tsteps > 0 ? (gs + tsteps - 1) % STAGES : 0;
          epilogue(m0, n0, smem + last * Cfg::STAGE, [] {});
        }
        if (!has_next) break;
        gs += Cfg::PRE_S ? nsteps - 1 : tsteps;
        tile = next;
        m0 = nm0;
        n0 = nn0;
        s_in = ns_in;
        next = tile + tr.stride;
        has_next = next < tr.end;
        load_next();
      }
    }
  } else {
    // A: the 2:4 K-major operand, expanded in registers; B: DMA.  The next
    // step's A loads and B DMA are issued before the current step's MFMAs; A
    // is written to LDS after them; one barrier per step.
    using TB = std::conditional_t<Cfg::B_KM, DmaTileKM<BN, NW>, DmaTile<BN, Cfg::B_ROWB, false, NW>>;
    const uint32_t smem_lds = lds_u32(smem);
    uint32_t offB[TB::PER_WAVE];
#pragma unroll
    for (int j = 0; j < TB::PER_WAVE; ++j) offB[j] = TB::lane_off(j, g.ldb, wave, lane);

    // Accumulate steps [0, ns) of the K range starting at kb of the tile at (m0, n0).
    auto run_tile = [&](int64_t m0, int64_t n0, int64_t kb, int ns) __attribute__((always_inline)) {
      zero_acc();
      StagerKMSP<BM, NT> sa;
      int b_steps_in = 0;   // steps whose B loads need no bounds checks
      if (n0 + BN <= g.N) {
        const int64_t k_in = g.kb_valid - kb;
        b_steps_in = k_in <= 0 ? 0 : (int)(k_in / BK < ns ? k_in / BK : ns);
      }
      b_steps_in = __builtin_amdgcn_readfirstlane(b_steps_in);
      int a_steps_in = 0;   // steps whose A loads need no bounds checks (and lie in full row blocks)
      if (m0 + BM <= g.m_valid) {
        const int64_t k_full = g.ka_valid < (g.tok & ~(int64_t)255) ? g.ka_valid : (g.tok & ~(int64_t)255);
        const int64_t k_in = k_full - kb;
        a_steps_in = k_in <= 0 ? 0 : (int)(k_in / BK < ns ? k_in / BK : ns);
      }
      a_steps_in = __builtin_amdgcn_readfirstlane(a_steps_in);
      // Copy cursors (the scalar code of eight waves shares one scalar unit,
      // so the unchecked steps avoid the general address arithmetic).  In
      // the tiled layout a step's 64 token rows of kept values (metadata) lie
      // 4096 (512) bytes after the previous step's inside a 256-row block; at
      // a block boundary the next block's rows follow 512 lda - 3 * 4096
      // (256 ldam - 3 * 512) bytes on (full blocks: R = 256).  B advances BK
      // rows (K-major) or BK elements.
      static_assert(BK == 64, "64 token rows per step");
      const char* cv = (const char*)uniform_ptr(g.A + tiled_step<32>(kb, m0, g.tok, g.lda));
      const char* cm = (const char*)uniform_ptr(g.Am + tiled_step<8>(kb, m0, g.tok, g.ldam));
      const int64_t jv = uniform_i64(512 * g.lda - 3 * 4096), jm = uniform_i64(256 * g.ldam - 3 * 512);
      uint32_t tpos = __builtin_amdgcn_readfirstlane((uint32_t)(kb & 255));   // token row in its block of the next load
      const char* cb = (const char*)uniform_ptr(TB::step_base(g.B, g.ldb, n0, kb));
      const uint32_t sb = __builtin_amdgcn_readfirstlane((uint32_t)(TB::step_base(g.B, g.ldb, n0, kb + BK) - TB::step_base(g.B, g.ldb, n0, kb)));
      auto load_a = [&](int step) __attribute__((always_inline)) {
        const int64_t k0 = kb + (int64_t)step * BK;
        if (step < a_steps_in) {
          // per-lane offsets formed here from a laundered thread index (cheaper
          // than keeping them in registers across the main loop)
          uint32_t aov[StagerKMSP<BM, NT>::NU], aom[StagerKMSP<BM, NT>::NU];
          int tc = tid;
          asm volatile("" : "+v"(tc));
          StagerKMSP<BM, NT>::lane_offs(tc, aov, aom);
          sa.load_fast(cv, cm, aov, aom);
          tpos = (tpos + 64) & 255;
          const bool cross = tpos == 0;
          cv += cross ? jv : 4096;
          cm += cross ? jm : 512;
        } else {
          int64_t kc = uniform_i64(k0);   // addresses formed afresh (see the direct path)
          int tc = tid;
          asm volatile("" : "+s"(kc), "+v"(tc));
          sa.load(g.A, g.lda, g.Am, g.ldam, m0, g.m_valid, kc, g.ka_valid, tc, g.tok);
        }
      };
      auto issue_b = [&](int step) __attribute__((always_inline)) {
        const int64_t k0 = kb + (int64_t)step * BK;
        const uint32_t base = smem_lds + (uint32_t)((step & 1) * Cfg::STAGE) + Cfg::A_BYTES;
        if (step < b_steps_in) {
          TB::template issue_fast<0, TB::PER_WAVE>(cb, offB, base, wave);
          cb += sb;
        } else
          TB::template issue<0, TB::PER_WAVE>(g.B, g.ldb, n0, g.N, k0, g.kb_valid, base, wave, lane);
      };
      if (ns > 0) {
        load_a(0);
        issue_b(0);
        sa.store(smem, tid);
        wait_vmcnt<0>();
        __syncthreads();
      }
      for (int s = 0; s < ns; ++s) {
        const int buf = s & 1;
        const bool more = s + 1 < ns;
        if (more) {
          load_a(s + 1);
          issue_b(s + 1);
        }
        // The expanded A of step s+1 is written to the other buffer (last
        // read in step s-1, before the previous barrier) ahead of this step's
        // last MFMA sub-step, so that its VALU work overlaps the MFMAs still
        // in flight.  (Measured: 5 % faster than after the step; earlier
        // sub-steps wait longer for A's loads or spill.)
        compute(smem + buf * Cfg::STAGE, smem + buf * Cfg::STAGE + Cfg::A_PART, [&](int kk) {
          if (kk == 3 && more) sa.store(smem + (buf ^ 1) * Cfg::STAGE, tid);
        });
        wait_vmcnt<0>();   // B's DMA of step s+1 has landed
        __syncthreads();   // A's LDS writes and B's DMA of step s+1 are complete
      }
    };
    int64_t m0, n0;
    if (g.stream_steps > 0) {
      // Stream-K: this workgroup's share [beg, end) of the tiles x S steps,
      // one partial tile per tile it touches.
      const int64_t S = g.stream_steps, I = (int64_t)ntiles * S;
      const int64_t beg = (int64_t)blockIdx.x * I / gridDim.x, end = (int64_t)(blockIdx.x + 1) * I / gridDim.x;
      const int64_t t_first = beg / S;
      for (int64_t it = beg; it < end;) {
        const int t = (int)(it / S);
        const int64_t k_first = it - (int64_t)t * S;
        const int64_t k_last = end - (int64_t)t * S < S ? end - (int64_t)t * S : S;
        origin(t, m0, n0);
        run_tile(m0, n0, k_first * BK, (int)(k_last - k_first));
        f32_slot = (float*)g.C + ((int64_t)blockIdx.x * g.stream_segs + (t - t_first)) * (BM * BN);
        epilogue(m0, n0, smem, [] {});
        it = (int64_t)t * S + k_last;
      }
    } else {
      origin(xcd_remap(bx, ntiles), m0, n0);
      run_tile(m0, n0, kbeg, nsteps);
      epilogue(m0, n0, smem, [] {});
    }
  }
}

}  // namespace elas
