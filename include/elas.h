/*
 * elas.h -- C ABI of the MI355X (gfx950) implementation of the ELAS low-rank
 * FFN with 2:4 activation sparsity (ELAS, arXiv 2605.03667).
 *
 * The block (Fig. 1 caption; Eq. 1-3, Algorithm 1), tokens as rows:
 *
 *     P = x U_up                x [T,d], U_up [d,r]          (Eq. 1 factors)
 *     H = P V_up                V_up [r,d_ff]
 *     s = max(0,H)^2            Eq. 2
 *     S = mask_top2(s) * s      Algorithm 1 / Eq. 3, groups of 4 along d_ff
 *     Z = S U_down              U_down [d_ff,r]  (2:4 sparse x dense GEMM)
 *     Y = Z V_down              V_down [r,d]
 *
 * With W = A B of Eq. 1 acting on row vectors, U = B^T and V = A^T.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * - bf16 tensors are passed as uint16_t bit patterns; float32 as float.
 * - Every tensor pointer is a DEVICE pointer owned by the caller.  The library
 *   never allocates, frees or keeps device memory (workspace is the caller's).
 * - Dense tensors are row-major and contiguous.  Every pointer must be 16-byte
 *   aligned.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *   work is enqueued on it asynchronously; the calls do not synchronise
 *   (except in the debug mode, elas_debug_sync below).
 * - Arguments are validated on the host before anything is enqueued.  On an
 *   error nothing is launched, outputs are untouched, the return value is the
 *   error code and elas_last_error() (thread-local) describes it.  A failed
 *   kernel launch returns ELAS_ERR_DEVICE; faults inside kernels surface at the
 *   caller's next synchronisation, as for any HIP work.
 * - Calls on one stream are ordered; calls that share output or workspace
 *   buffers must not run concurrently on different streams.
 *
 * Compressed 2:4 layout ("sparse rows")
 * -------------------------------------
 * A matrix Z [M x N] whose every group of 4 consecutive row entries (features
 * 4j..4j+3) keeps exactly 2 entries (Algorithm 1) is stored as
 *   vals [M x ldv] bf16 : group j's kept values at vals[i][2j], vals[i][2j+1],
 *                         in ascending feature order;
 *   meta [M x ldm] bytes: group j's code  i0 | (i1 << 2)  (i0 < i1 are the
 *                         kept positions inside the group) in byte j/2, low
 *                         nibble for even j, high nibble for odd j.
 * Row pitches: ldv = 32 * ceil(N/64) values and ldm = 8 * ceil(N/64) bytes
 * (rows padded to a multiple of 64 features so every row is 16-byte aligned).
 * Padding groups (j >= N/4) hold values 0 and code 0x4 (positions 0 and 1), so
 * a padded row is itself a valid 2:4 row whose extra entries are zero.
 * Per kept value this is 2 bytes plus 2 bits: 0.5625 of dense bf16, the ratio
 * of the paper's Table 2 (Sec. 4.2.2).
 *
 * Tiled compressed layout (the FFN's saved S)
 * -------------------------------------------
 * elas_lowrank_ffn_fwd stores the compressed S in the same buffers
 * (M x ldv values, M x ldm bytes, M = T) with the same row contents, but
 * tiled so that the 2:4 products read whole contiguous blocks: rows are cut
 * into blocks of 256 (the last block holds the R = M - 256 b remaining rows,
 * otherwise R = 256), and within a row block each row's entries into blocks
 * of BW = 32 values (ldv) or BW = 8 metadata bytes (ldm), i.e. 64 features.
 * Entry block c of row block b holds its R rows x BW entries row-major and
 * contiguously; blocks follow one another by row block, then entry block.
 * Entry j of row i (values: ld = ldv, BW = 32; metadata: ld = ldm, BW = 8) is
 *   element  (i / 256) * 256 * ld + (j / BW) * R * BW + (i % 256) * BW + j % BW.
 * elas_sparsify_24 and elas_spmm_24 use the row layout above.
 */
#ifndef ELAS_H
#define ELAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes -------------------------------------------------------- */
#define ELAS_OK              0
#define ELAS_ERR_NULL        1  /* a required pointer is NULL                      */
#define ELAS_ERR_SHAPE       2  /* a size is out of range or not a required multiple */
#define ELAS_ERR_ALIGN       3  /* a pointer is not 16-byte aligned                */
#define ELAS_ERR_WORKSPACE   4  /* workspace missing or smaller than required      */
#define ELAS_ERR_FLAGS       5  /* unknown or unsupported flag bits                */
#define ELAS_ERR_DEVICE      6  /* a HIP call or kernel launch failed              */

/* ---- flags ---------------------------------------------------------------- */
/* elas_sparsify_24: what the top-2 selection ranks (Algorithm 1). */
#define ELAS_SPARSIFY_RELU2  0u /* s = max(0,h)^2 is ranked and stored (ELAS's activation) */
#define ELAS_SPARSIFY_RAW    1u /* h itself is ranked by |h| and stored unchanged          */

/* elas_lowrank_ffn_fwd / _bwd: activation mode (both calls must agree). */
#define ELAS_MODE_SPARSE24   0u /* the ReLU^2 output is pruned to 2:4 and stored compressed    */
#define ELAS_MODE_DENSE      2u /* dense activations, no selection (the paper's dense warm-up,
                                   Sec. 3.4 and Algorithm 2; also the dense comparison run)   */
/* elas_lowrank_ffn_bwd only: gradient through the 2:4 selection. */
#define ELAS_BWD_STE         4u /* straight-through estimator of Eq. 4: the selection is the
                                   identity in the backward, dH = dS * 2 relu(h) everywhere
                                   (relu(h) recomputed from P and V_up); default is the
                                   masked derivative dH = dS * mask * 2 relu(h)               */

/* elas_lowrank_ffn_fwd only: orientation of the four factors. */
#define ELAS_FACTORS_AB      8u /* the factors are given as the A and B of Eq. 1 (W = A B, the
                                   orientation a linear layer stores): U_up^T [r,d],
                                   V_up^T [d_ff,r], U_down^T [r,d_ff], V_down^T [d,r].  This is
                                   the kernels' operand layout, so nothing is re-laid out (for
                                   inference with pre-arranged weights); results are identical */

/* elas_lowrank_ffn_fwd only, sparse mode: launch shape.  Without either flag the forward is
   the four-kernel sequence (on MI355X faster than the fused launch at every supported shape
   but one).  Both compute the same block (Eq. 1-3, Algorithm 1) and write the same outputs in
   the same layouts; their fp32 sums run in a different order, so results can differ in the
   last bits (and a group whose ranking ties within that difference can keep another pair).
   Both flags together, or ELAS_FWD_FUSED with ELAS_MODE_DENSE: ELAS_ERR_FLAGS. */
#define ELAS_FWD_FUSED      16u /* one launch per call: each workgroup computes P, S, Z and Y
                                   for its block of tokens, with P and a d_ff chunk of S in LDS
                                   and Z accumulated on chip (the fully fused forward).  Needs
                                   d a multiple of 64 up to 1024 and r = 128 or 256, else
                                   ELAS_ERR_SHAPE                                              */
#define ELAS_FWD_UNFUSED    32u /* the four-kernel sequence (k1 .. k4)                         */

/* elas_spmm_24: layout of the dense operand B. */
#define ELAS_B_KN            0  /* B is [K x N] row-major                         */
#define ELAS_B_NK            1  /* B is [N x K] row-major (B^T stored)            */

/* Human-readable name of a status code (static string). */
const char* elas_status_string(int status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* elas_last_error(void);

/* Row pitches of the compressed layout for a row of N features:
 * values per row (ldv) and metadata bytes per row (ldm).  N must be > 0. */
int64_t elas_vals_ld(int64_t N);
int64_t elas_meta_ld(int64_t N);

/*
 * elas_sparsify_24 -- Algorithm 1 (Sec. 3.3.1) with Eq. 2 in front of it.
 *
 * h     [M x N] bf16, device, read only.
 * vals  [M x elas_vals_ld(N)] bf16, device, written (compressed layout above).
 * meta  [M x elas_meta_ld(N)] bytes, device, written.
 * flags ELAS_SPARSIFY_RELU2: key and value are s = max(0,h)^2 computed in fp32
 *       (h*h is exact in fp32 for 2^-63 <= |h| < 2^64), ranked exactly as the
 *       real numbers s, ties to the lower index; kept values are s rounded to
 *       bf16, nearest-even.  relu(NaN) = 0.
 *       ELAS_SPARSIFY_RAW: key |h|, kept values are h's bits unchanged.
 * Requires M >= 0, N > 0, N % 8 == 0.  M == 0 is a no-op (pointers are then
 * not inspected and may be NULL).
 */
int elas_sparsify_24(const uint16_t* h, int64_t M, int64_t N, uint32_t flags,
                     uint16_t* vals, uint8_t* meta, void* stream);

/*
 * elas_spmm_24 -- C = A B with A 2:4-sparse along K (the paper's sparse x
 * dense product of the down projection, Fig. 1 caption and Sec. 4.2.2).
 *
 * a_vals, a_meta  A [M x K] in the compressed layout (pitches for N := K).
 * b               B, bf16, [K x N] (b_layout ELAS_B_KN) or [N x K] (ELAS_B_NK).
 * c               C [M x N] bf16, written; products accumulate in fp32 and are
 *                 rounded to bf16 (nearest-even) once.
 * workspace       device scratch of at least elas_spmm_24_workspace_bytes()
 *                 bytes (may be NULL when that is 0).
 * Requires M >= 0, K > 0, K % 8 == 0, N > 0, N % 8 == 0, K and N at most 65536.
 * M == 0 is a no-op (pointers are then not inspected and may be NULL).
 */
size_t elas_spmm_24_workspace_bytes(int64_t M, int64_t K, int64_t N, int b_layout);
int elas_spmm_24(const uint16_t* a_vals, const uint8_t* a_meta, int64_t M, int64_t K,
                 const uint16_t* b, int64_t N, int b_layout, uint16_t* c,
                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * elas_lowrank_ffn_fwd -- forward of the block above.
 *
 * Inputs (bf16, device, read only): x [T,d], U_up [d,r], V_up [r,d_ff],
 *   U_down [d_ff,r], V_down [r,d].
 * Outputs (bf16, device, written):
 *   y      [T,d]
 *   P      [T,r]   saved for the backward (P = x U_up, rounded to bf16)
 *   s_vals sparse mode: T x elas_vals_ld(d_ff) values, compressed S (kept s in
 *          bf16) in the tiled layout above
 *          dense mode:  [T x d_ff] dense S = relu(H)^2 in bf16, row-major
 *   s_meta sparse mode: T x elas_meta_ld(d_ff) bytes, its 2-bit indices, tiled;
 *          dense mode: not used (may be NULL)
 *   Z      [T,r]   saved for the backward
 * Rounding points: P, H (before ReLU^2), the kept s, Z and y are rounded to
 * bf16 (nearest-even); every product accumulates in fp32.  The 2:4 selection
 * ranks max(0, bf16(H))^2 exactly, ties to the lower index.
 * flags: ELAS_MODE_SPARSE24 (0) or ELAS_MODE_DENSE, optionally | ELAS_FACTORS_AB
 *   (the four factor pointers then hold the transposed matrices listed there).
 * workspace >= elas_lowrank_ffn_fwd_workspace_bytes(T, d, d_ff, r, flags).  The
 * size depends on T and is not monotonic in it (small token counts add fp32
 * split-K partials), so query it for every T a buffer is reused for.
 * Requires T >= 0, d, d_ff, r > 0, multiples of 8 and at most 65536.  T == 0 is
 * a no-op (pointers are then not inspected and may be NULL).
 */
size_t elas_lowrank_ffn_fwd_workspace_bytes(int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags);
int elas_lowrank_ffn_fwd(const uint16_t* x, const uint16_t* U_up, const uint16_t* V_up,
                         const uint16_t* U_down, const uint16_t* V_down,
                         int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags,
                         uint16_t* y, uint16_t* P, uint16_t* s_vals, uint8_t* s_meta,
                         uint16_t* Z, void* workspace, size_t workspace_bytes, void* stream);

/*
 * elas_lowrank_ffn_fwd_noalloc -- for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): elas_lowrank_ffn_fwd with the same arguments, flags,
 * outputs and results (bit for bit), but without a workspace argument.  Its
 * workspace is a static device array of ELAS_NOALLOC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends; the call
 * itself allocates nothing (no hipMalloc, no allocating library routine).
 * The first call on a device looks the array's address up there.
 * Errors: as elas_lowrank_ffn_fwd, plus ELAS_ERR_WORKSPACE when the shape
 * needs more workspace than the array holds
 * (elas_lowrank_ffn_fwd_workspace_bytes > ELAS_NOALLOC_SCRATCH_BYTES; at the
 * largest model shape, d = 2048, d_ff = 5464, r = 512, it needs about 31 MB
 * at any token count), and ELAS_ERR_DEVICE if the address lookup fails.
 * Each call overwrites every part of the array it reads (nothing needs to
 * start at zero).  All calls on one device share the array: calls that
 * overlap in time on one device (different streams or threads) race and must
 * be ordered by the caller.
 */
#define ELAS_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
size_t elas_noalloc_scratch_bytes(void);
int elas_lowrank_ffn_fwd_noalloc(const uint16_t* x, const uint16_t* U_up, const uint16_t* V_up,
                                 const uint16_t* U_down, const uint16_t* V_down,
                                 int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags,
                                 uint16_t* y, uint16_t* P, uint16_t* s_vals, uint8_t* s_meta,
                                 uint16_t* Z, void* stream);

/*
 * elas_lowrank_ffn_bwd -- backward of the block (Sec. 3.3.2, Sec. 3.4).
 *
 * dy [T,d] bf16 is dL/dY; x, U_up, V_up, U_down, V_down as in the forward;
 * P, s_vals, s_meta, Z are the forward's saved outputs (read only; s_meta
 * unused in dense mode).
 * Outputs: dx [T,d] bf16 (written); dU_up [d,r], dV_up [r,d_ff],
 *   dU_down [d_ff,r], dV_down [r,d] fp32 (overwritten, not accumulated).
 * Gradient through the activation:
 *   default (sparse mode): dH = dS * mask * 2 relu(h) with the stored mask,
 *     the derivative of the sparsified forward; relu(h) is recovered exactly
 *     from the stored bf16 s.  The full-width activation is never read:
 *     dU_down = S^T dZ and dV_up = P^T dH use the compressed form.
 *   ELAS_BWD_STE (after a sparse forward): Eq. 4, dH = dS * 2 relu(h) at every
 *     position; relu(h) = relu(bf16(P V_up)) is recomputed tile by tile inside
 *     the dH kernel (no d_ff-wide activation is stored).
 *   ELAS_MODE_DENSE (after a dense forward): dH = dS * 2 relu(h), dense.
 * Rounding points: dZ, dH, dP and dx are rounded to bf16.
 * flags: 0, ELAS_BWD_STE or ELAS_MODE_DENSE (the forward's mode).
 * workspace >= elas_lowrank_ffn_bwd_workspace_bytes(T, d, d_ff, r, flags).
 * Same size rules as the forward; T == 0 writes zero weight gradients (only
 * the four gradient pointers and the workspace are then inspected).
 */
size_t elas_lowrank_ffn_bwd_workspace_bytes(int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags);
int elas_lowrank_ffn_bwd(const uint16_t* dy, const uint16_t* x, const uint16_t* U_up,
                         const uint16_t* V_up, const uint16_t* U_down, const uint16_t* V_down,
                         int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags,
                         const uint16_t* P, const uint16_t* s_vals, const uint8_t* s_meta,
                         const uint16_t* Z,
                         uint16_t* dx, float* dU_up, float* dV_up, float* dU_down, float* dV_down,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * elas_fullrank_ffn_fwd -- forward of the full-rank ReLU^2 FFN, the block the
 * paper's FFN speed-up table compares ELAS against (Table 3, Sec. 4.2.3).
 * The weights are the full matrices W of Eq. 1 (acting on column vectors, as
 * a linear layer stores them); with tokens as rows:
 *
 *     H = x W_up^T,   S = max(0,H)^2,   Y = S W_down^T
 *
 * Inputs (bf16, device, read only): x [T,d], W_up [d_ff,d], W_down [d,d_ff].
 * Outputs (bf16, device, written): y [T,d] and S [T,d_ff], the dense
 *   activation (what a training step would keep for its backward).
 * Rounding points: H (before ReLU^2), S and y are rounded to bf16
 * (nearest-even); both products accumulate in fp32.  No workspace.
 * Requires T >= 0, d, d_ff > 0, multiples of 8 and at most 65536.  T == 0 is a
 * no-op (pointers are then not inspected and may be NULL).
 */
int elas_fullrank_ffn_fwd(const uint16_t* x, const uint16_t* W_up, const uint16_t* W_down,
                          int64_t T, int64_t d, int64_t d_ff, uint16_t* y, uint16_t* S, void* stream);

/*
 * elas_meta_to_canonical / elas_vals_to_canonical -- read back the compressed
 * S that elas_lowrank_ffn_fwd saves (tiled layout above; the storage of the
 * kept values plus index information of Sec. 4.2.2) in the canonical form:
 * row i's N/8 metadata bytes (resp. N/2 kept values) contiguous, no padding,
 * group j's code in byte j/2 as in the row layout.
 * HOST memory on both sides (copy the device buffers to the host first):
 *   meta_tiled [M x elas_meta_ld(N)] bytes -> meta_canonical [M x N/8] bytes;
 *   vals_tiled [M x elas_vals_ld(N)] bf16  -> vals_canonical [M x N/2] bf16.
 * Requires M >= 0, N > 0, N % 8 == 0, N <= 65536; M == 0 is a no-op.  NULL
 * buffers give ELAS_ERR_NULL.  Synchronous; no device work.
 */
int elas_meta_to_canonical(const uint8_t* meta_tiled, int64_t M, int64_t N, uint8_t* meta_canonical);
int elas_vals_to_canonical(const uint16_t* vals_tiled, int64_t M, int64_t N, uint16_t* vals_canonical);

/*
 * Debug mode (ELAS_DEBUG_SYNC).  When on, every kernel an entry point
 * launches is followed by a synchronisation of the caller's stream, and a
 * failure is returned by that entry point as ELAS_ERR_DEVICE naming the
 * kernel (elas_last_error), instead of surfacing at the caller's next
 * synchronisation.  For debugging only: it serialises host and device and
 * must not be used while the stream is being captured into a graph.
 * The initial state is on when the environment variable ELAS_DEBUG_SYNC is
 * set to anything but "0" at load time.  elas_debug_sync(1 / 0) switches it
 * on / off, elas_debug_sync(-1) leaves it; each returns the previous state.
 */
int elas_debug_sync(int enable);

/*
 * Per-kernel timing (diagnostics for benchmarks; not thread-safe).
 *
 * elas_timing_enable(1) clears earlier records and starts recording: every
 * kernel the entry points launch is then bracketed by two hipEvents recorded
 * on the caller's stream.  elas_timing_enable(0) stops recording.
 * elas_timing_collect() waits for the recorded events and aggregates them per
 * kernel tag; it returns the number of tags (or -ELAS_ERR_DEVICE).
 * elas_timing_entry(i, ...) returns tag i's name (NUL-terminated, truncated to
 * name_cap), its number of launches and their summed duration in ms.
 * elas_timing_only(tag) restricts recording to the launches of one kernel tag
 * (the string is copied), so that a timed region carries only that kernel's
 * events; NULL or "" restores recording of every launch.  Always ELAS_OK.
 */
int elas_timing_enable(int enable);
int elas_timing_only(const char* tag);
int elas_timing_collect(void);
int elas_timing_entry(int i, char* name, int name_cap, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* ELAS_H */
