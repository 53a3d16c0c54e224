// Launch sequences of the ELAS low-rank 2:4 FFN on one GPU: forward (ELAS
// Fig. 1 caption; Eq. 1-3, Algorithm 1), backward (Sec. 3.3.2, Sec. 3.4) and
// the standalone 2:4 sparse x dense product.  Everything runs on the caller's
// stream in the caller's workspace; nothing here allocates.
#include <algorithm>
#include <atomic>

#include "gemm.h"
#include "internal.h"

namespace elas {

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Carves consecutive aligned regions out of the caller's workspace.
struct Carver {
  char* p;
  size_t used = 0;
  template <class T>
  T* take(size_t count) {
    T* r = p ? (T*)(p + used) : nullptr;
    used += align_up(count * sizeof(T));
    return r;
  }
};

// ---- small kernels -----------------------------------------------------------

// Transposing job: out[j][i] = in[i][j] for i < rows, j < cols; 0 elsewhere
// in [out_rows x out_cols].  Copying job (transpose = 0): out[i][j] = in[i][j],
// 0 elsewhere.  The output is row-major with pitch ldo, or blocked
// (blocked_index) when nsk > 0.
struct TransposeJob {
  const uint16_t* in;
  uint16_t* out;
  int64_t rows, cols, ldi, out_rows, out_cols, ldo;
  int tiles_x;      // 64-wide tiles along out_cols
  int tile_begin;   // first flat tile index of this job
  int transpose;
  int64_t nsk;
};
__device__ __forceinline__ int64_t job_pos(const TransposeJob& jb, int64_t row, int64_t col) {
  return jb.nsk > 0 ? blocked_index(row, col, jb.nsk) : row * jb.ldo + col;
}
// Up to four transposes in one launch (the weight factors of one call): the
// flat tile index selects the job, so small factors share the launch.
constexpr int kMaxTransposeJobs = 4;
struct TransposeBatch {
  TransposeJob job[kMaxTransposeJobs];
  int n;
};

__global__ __launch_bounds__(256) void transpose_pad_kernel(TransposeBatch tb) {
  // 64 x 64 tile, moved in 16-byte pieces (8 bf16): thread t reads row
  // i0 + t/8 (+32) at columns j0 + 8 (t%8), and writes output row j0 + t/8
  // (+32) at columns i0 + 8 (t%8).  cols, ldi, out_cols and ldo are
  // multiples of 8 (model dimensions), so a piece is wholly inside or outside.
  // The LDS rows are padded to 72 elements so that the column reads of the
  // write phase fall in distinct banks.
  __shared__ __attribute__((aligned(16))) uint16_t tile[64][72];
  int q = 0;
#pragma unroll
  for (int k = 1; k < kMaxTransposeJobs; ++k)
    if (k < tb.n && (int)blockIdx.x >= tb.job[k].tile_begin) q = k;
  const TransposeJob& jb = tb.job[q];
  const int t = (int)blockIdx.x - jb.tile_begin;
  const int r = threadIdx.x / 8, c = threadIdx.x % 8;
  if (!jb.transpose) {   // (uniform over the workgroup: one job per tile)
    const int64_t r0 = (int64_t)(t / jb.tiles_x) * 64, c0 = (int64_t)(t % jb.tiles_x) * 64;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t i = r0 + r + 32 * h, j = c0 + 8 * c;
      if (i < jb.out_rows && j < jb.out_cols) {
        uint4 v = make_uint4(0u, 0u, 0u, 0u);
        if (i < jb.rows && j < jb.cols) v = *(const uint4*)(jb.in + i * jb.ldi + j);
        *(uint4*)(jb.out + job_pos(jb, i, j)) = v;
      }
    }
    return;
  }
  const int64_t i0 = (int64_t)(t % jb.tiles_x) * 64, j0 = (int64_t)(t / jb.tiles_x) * 64;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int a = r + 32 * h;
    const int64_t i = i0 + a, j = j0 + 8 * c;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (i < jb.rows && j < jb.cols) v = *(const uint4*)(jb.in + i * jb.ldi + j);
    *(uint4*)&tile[a][8 * c] = v;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int a = r + 32 * h;                       // output row j0 + a = input column
    const int64_t jj = j0 + a, ii = i0 + 8 * c;
    if (jj < jb.out_rows && ii < jb.out_cols) {
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) w[k] = (uint32_t)tile[8 * c + 2 * k][a] | ((uint32_t)tile[8 * c + 2 * k + 1][a] << 16);
      *(uint4*)(jb.out + job_pos(jb, jj, ii)) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// Collects transposes and launches them together.
struct Transposes {
  TransposeBatch tb{};
  int tiles = 0;
  void add(const uint16_t* in, int64_t rows, int64_t cols, int64_t ldi, uint16_t* out, int64_t out_rows,
           int64_t out_cols, int64_t ldo, int transpose = 1, int64_t nsk = 0) {
    TransposeJob& j = tb.job[tb.n++];
    j = TransposeJob{in, out, rows, cols, ldi, out_rows, out_cols, ldo, (int)cdiv(out_cols, 64), tiles, transpose, nsk};
    tiles += j.tiles_x * (int)cdiv(out_rows, 64);
  }
  hipError_t launch(hipStream_t st) {
    if (tiles == 0) return hipSuccess;
    TimedLaunch tl("weight_transpose", st);
    hipLaunchKernelGGL(transpose_pad_kernel, dim3((unsigned)tiles), dim3(256), 0, st, tb);
    return hipGetLastError();
  }
};

hipError_t transpose_pad(const uint16_t* in, int64_t rows, int64_t cols, int64_t ldi, uint16_t* out,
                         int64_t out_rows, int64_t out_cols, int64_t ldo, hipStream_t st) {
  Transposes t;
  t.add(in, rows, cols, ldi, out, out_rows, out_cols, ldo);
  return t.launch(st);
}

// Writes a 64 x 64 (m, n) tile of sums held as acc[i] = row m0 + ty + 16 i,
// float4 columns n0 + 4 tx: to out[m][n], or to out[n][m] when transposing
// (through LDS, so that consecutive threads store consecutive m).  N and a
// non-transposed ldo are multiples of 4 (the model dimensions are multiples
// of 8).
__device__ __forceinline__ void reduce_store(const float4 (&acc)[4], int64_t m0, int64_t n0, int tx, int ty,
                                             int64_t N, int64_t rows_out, int transpose, float* __restrict__ out,
                                             int64_t ldo, float (*tile)[65]) {
  const int64_t n = n0 + 4 * tx;
  if (!transpose) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t m = m0 + ty + 16 * i;
      if (m < rows_out && n < N) *(float4*)(out + m * ldo + n) = acc[i];
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    tile[4 * tx + 0][ty + 16 * i] = acc[i].x;
    tile[4 * tx + 1][ty + 16 * i] = acc[i].y;
    tile[4 * tx + 2][ty + 16 * i] = acc[i].z;
    tile[4 * tx + 3][ty + 16 * i] = acc[i].w;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < 64 * 64; q += 256) {
    const int r = q / 64, c = q % 64;
    const int64_t on = n0 + r, om = m0 + c;
    if (on < N && om < rows_out) out[on * ldo + om] = tile[r][c];
  }
}

// out[m][n] (or out[n][m]) = sum over the splits k, in order (so the result
// is deterministic), of part[k][m][n], for rows m < rows_out; one 64 x 64
// (m, n) tile per block.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int splits, int64_t M,
                                                           int64_t N, int64_t rows_out, int transpose,
                                                           float* __restrict__ out, int64_t ldo) {
  __shared__ float tile[64][65];
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int64_t n = n0 + 4 * tx;
  float4 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  // Splits are read four at a time (16 loads in flight per thread) and added
  // in split order, so the result does not depend on the grouping.
  int k = 0;
  for (; k + 4 <= splits; k += 4) {
    float4 v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float* pk = part + (int64_t)(k + u) * M * N;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + ty + 16 * i;
        v[u][i] = (m < rows_out && n < N) ? *(const float4*)(pk + m * N + n) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[i].x += v[u][i].x; acc[i].y += v[u][i].y; acc[i].z += v[u][i].z; acc[i].w += v[u][i].w;
      }
  }
  for (; k < splits; ++k) {
    const float* pk = part + (int64_t)k * M * N;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t m = m0 + ty + 16 * i;
      if (m < rows_out && n < N) {
        const float4 v = *(const float4*)(pk + m * N + n);
        acc[i].x += v.x; acc[i].y += v.y; acc[i].z += v.z; acc[i].w += v.w;
      }
    }
  }
  reduce_store(acc, m0, n0, tx, ty, N, rows_out, transpose, out, ldo, tile);
}

// bf16 result of a split-K product with a bf16 output: out[m][n] =
// bf16(sum over the splits k, in order, of part[k][m][n]); one 4-column piece
// per thread (N and ldo are multiples of 8).
__global__ __launch_bounds__(256) void splitk_reduce_bf16_kernel(const float* __restrict__ part, int splits, int64_t M,
                                                                int64_t N, uint16_t* __restrict__ out, int64_t ldo) {
  const int64_t pieces = N / 4;
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= M * pieces) return;
  const int64_t m = q / pieces, n = (q % pieces) * 4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int k = 0; k < splits; ++k) {
    const float4 v = *(const float4*)(part + ((int64_t)k * M + m) * N + n);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  *(uint2*)(out + m * ldo + n) = make_uint2(bf16x2_rne(acc.x, acc.y), bf16x2_rne(acc.z, acc.w));
}

// The stream-K counterpart: workgroup w of `wgs` owns iterations
// [w I / wgs, (w+1) I / wgs) of the I = ntiles x S (tile, K step) space and
// wrote the partial of the j-th tile it touched to part + (w segs + j) 256^2
// (256 x 256 row-major).  The sums run over the workgroups in order, i.e. in
// K order, so the result is deterministic.
__global__ __launch_bounds__(256) void streamk_reduce_kernel(const float* __restrict__ part, int wgs, int segs,
                                                            int64_t S, int tiles_n, int64_t ntiles, int64_t N,
                                                            int64_t rows_out, int transpose, float* __restrict__ out,
                                                            int64_t ldo) {
  __shared__ float tile[64][65];
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  const int64_t t = (m0 / 256) * tiles_n + n0 / 256;
  const int lm = (int)(m0 % 256), ln = (int)(n0 % 256) + 4 * tx;
  const int64_t I = ntiles * S, tb = t * S, te = tb + S;
  auto beg_of = [&](int64_t w) { return w * I / wgs; };
  int64_t w = tb * wgs / I;   // the workgroup whose range holds iteration tb
  while (w > 0 && beg_of(w) > tb) --w;
  while (beg_of(w + 1) <= tb) ++w;
  float4 acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  // The workgroups [w, w_end) that touch tile t, read four at a time (16
  // loads in flight per thread) and added in workgroup order.
  int64_t w_end = w;
  while (w_end < wgs && beg_of(w_end) < te) ++w_end;
  for (; w < w_end; w += 4) {
    float4 v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t wu = w + u;
      const int64_t b = beg_of(wu), e = beg_of(wu + 1);
      const bool has = wu < w_end && e > b;
      const float* slot = part + ((int64_t)wu * segs + (t - b / S)) * 65536;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        v[u][i] = has ? *(const float4*)(slot + (int64_t)(lm + ty + 16 * i) * 256 + ln) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[i].x += v[u][i].x; acc[i].y += v[u][i].y; acc[i].z += v[u][i].z; acc[i].w += v[u][i].w;
      }
  }
  reduce_store(acc, m0, n0, tx, ty, N, rows_out, transpose, out, ldo, tile);
}

__global__ __launch_bounds__(256) void fill_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n) p[e] = 0.f;
}

hipError_t fill_zero(float* p, int64_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  TimedLaunch tl("fill_zero", st);
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

// ---- GEMM configurations -----------------------------------------------------
// Tile shapes picked by measurement on MI355X at the 1B FFN shapes: eight
// waves (two per SIMD) hide LDS and global latency better than four larger
// wave tiles.
// Dense products with both operands K-contiguous: 256 x BN tiles, 4 x 2 waves.
template <int BN, int EPI, bool M_FAST, int DEEP = 0>
using CfgNT = GemmCfg<256, BN, 4, 2, OP_K, OP_K, EPI, M_FAST, 2, true, false, 128, DEEP>;
// Plain bf16 outputs (A = the token-major activation streaming from HBM, B =
// a weight factor resident in L2): A gets three LDS stages, B two.
using CfgNT3 = CfgNT<256, EPI_BF16, false, 1>;
// 2:4 sparse A (smfmac) times K-contiguous B: 256 x 256 tiles, 4 x 2 waves
// (64 x 128 per wave), 64 dense K per step in three LDS stages (150 KB).  The
// full-width N tile halves the re-reads of the compressed operand, which
// streams from HBM, and the third stage covers more of its latency.
// (Measured: 22% faster than 256 x 128 tiles with 128-K steps in two stages.)
using CfgSP = GemmCfg<256, 256, 4, 2, OP_SP, OP_K, EPI_BF16, false, 3, true, false, 64>;
// Contraction over tokens (K = T): both operands stored [T x rows].
// Both operands are K-major: the dense ones go to LDS by DMA, the 2:4 one is
// expanded in registers; fragments are read with the transposing LDS read.
// K = T weight-gradient products (both operands token-major and streaming;
// a three-stage ring for one of them measured no gain).
template <int AMODE>
using CfgTT = GemmCfg<256, 256, 4, 2, AMODE, OP_T, EPI_F32, false>;

// Compute units of the current device (cached per device id).
// (Relaxed atomics: concurrent first calls store the same value.)
int device_cus() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <class Cfg>
hipError_t launch(const char* tag, GemmArgs g, int splits, hipStream_t st) {
  if (g.b_nsk > 0 && (!Cfg::B_BLOCKABLE || g.ldb != 64)) return hipErrorInvalidValue;
  g.tiles_m = (int)cdiv(g.M, Cfg::BM);
  g.tiles_n = (int)cdiv(g.N, Cfg::BN);
  if (splits <= 1) {
    splits = 1;
    g.k_split = cdiv(g.K, Cfg::BK) * Cfg::BK;
  }
  // Direct-staged kernels are persistent: one workgroup per CU at most, each
  // looping over its tiles.
  const int tiles = g.tiles_m * g.tiles_n;
  const int cus = device_cus();
  const int wgs = Cfg::DIRECT && tiles > cus ? cus : tiles;
  const dim3 grid((unsigned)wgs, (unsigned)splits);
  TimedLaunch tl(tag, st);
  hipLaunchKernelGGL(gemm_kernel<Cfg>, grid, dim3(Cfg::NT), 0, st, g);
  return hipGetLastError();
}

// Small problems: when 256-wide tiles would leave more than a quarter of the
// CUs without a tile, 128 x 128 tiles (4 waves of 64 x 64) give four times as
// many (twice as many for the staged 2:4 epilogues, which need 256 features).
using CfgSPs = GemmCfg<128, 128, 2, 2, OP_SP, OP_K, EPI_BF16, false, 3, true, false, 64>;

bool few_tiles(int64_t M, int64_t N, int bm, int bn) { return cdiv(M, bm) * cdiv(N, bn) * 4 < 3LL * device_cus(); }

// Split-K of a bf16-output product with few 128 x 128 tiles and a long K:
// enough splits to cover the CUs once, each at least 8 K steps of bk; the fp32
// partials [splits x M x N] are then summed in split order and rounded once.
struct SmallSplit {
  int splits;
  int64_t k_split;
};
SmallSplit plan_small_split(int64_t M, int64_t N, int64_t K, int bk) {
  const int64_t tiles = cdiv(M, 128) * cdiv(N, 128), cus = device_cus();
  const int64_t steps = cdiv(K, bk);
  if (tiles == 0 || tiles * 2 > cus || steps < 16) return {1, K};   // (no rows: nothing to split)
  int64_t s = cus / tiles;
  if (s > steps / 8) s = steps / 8;
  if (s < 2) return {1, K};
  const int64_t k_split = cdiv(cdiv(K, s), bk) * bk;
  return {(int)cdiv(K, k_split), k_split};
}
size_t small_split_bytes(int64_t M, int64_t N, int64_t K, int bk) {
  const SmallSplit p = plan_small_split(M, N, K, bk);
  return p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
}
template <int EPI, bool M_FAST>
using CfgNTs = GemmCfg<128, 128, 2, 2, OP_K, OP_K, EPI, M_FAST>;
using CfgSPsf = GemmCfg<128, 128, 2, 2, OP_SP, OP_K, EPI_F32, false, 3, true, false, 64>;

hipError_t reduce_bf16(const float* part, int splits, int64_t M, int64_t N, uint16_t* out, int64_t ldo,
                       hipStream_t st) {
  TimedLaunch tl("splitk_reduce_bf16", st);
  hipLaunchKernelGGL(splitk_reduce_bf16_kernel, dim3((unsigned)cdiv(M * (N / 4), 256)), dim3(256), 0, st, part, splits,
                     M, N, out, ldo);
  return hipGetLastError();
}

// 2:4 A times K-contiguous B, bf16 out (`part`: split-K partials, may be null).
hipError_t launch_sp(const char* tag, GemmArgs g, hipStream_t st, float* part = nullptr) {
  if (few_tiles(g.M, g.N, 256, 256)) {
    const SmallSplit p = part ? plan_small_split(g.M, g.N, g.K, CfgSPsf::BK) : SmallSplit{1, g.K};
    if (p.splits > 1) {
      uint16_t* out = (uint16_t*)g.C;
      const int64_t ldo = g.ldc;
      g.C = part;
      g.ldc = g.N;
      g.k_split = p.k_split;
      hipError_t e = launch<CfgSPsf>(tag, g, p.splits, st);
      if (e != hipSuccess) return e;
      return reduce_bf16(part, p.splits, g.M, g.N, out, ldo, st);
    }
    return launch<CfgSPs>(tag, g, 1, st);
  }
  return launch<CfgSP>(tag, g, 1, st);
}
// Epilogues that select and compress 2:4 groups (features along M).
// With more than 3 MB of A rows (the d_ff-wide weight factor: 5.6 MB at 1B,
// beyond an XCD's 4 MB L2) and an even number of 256-row tiles, two panels.
template <int EPI>
hipError_t launch_staged(const char* tag, GemmArgs g, hipStream_t st) {
  if (few_tiles(g.M, g.N, 256, 256)) return launch<CfgNT<128, EPI, true>>(tag, g, 1, st);
  const int64_t tiles_m = cdiv(g.M, 256);
  if (tiles_m % 2 == 0 && tiles_m * 256 * g.K * 2 > (int64_t(3) << 20)) g.m_groups = 2;
  return launch<CfgNT<256, EPI, true>>(tag, g, 1, st);
}
// Epilogues that write or read the dense activation (features along M).
template <int EPI>
hipError_t launch_act(const char* tag, const GemmArgs& g, hipStream_t st) {
  if (few_tiles(g.M, g.N, 256, 256)) return launch<CfgNTs<EPI, true>>(tag, g, 1, st);
  return launch<CfgNT<256, EPI, true, 2>>(tag, g, 1, st);
}

// Dense product C[M x N] = A[M x K] * Bt[N x K]^T in bf16 (`part`: split-K
// partials for small problems, may be null).
// b_nsk > 0: Bt is blocked (blocked_index, b_nsk K blocks per panel; ldb is
// then ignored).
hipError_t gemm_nt_bf16(const char* tag, const uint16_t* A, int64_t lda, const uint16_t* Bt, int64_t ldb, uint16_t* C, int64_t ldc,
                        int64_t M, int64_t N, int64_t K, hipStream_t st, float* part = nullptr, int64_t b_nsk = 0) {
  GemmArgs g{};
  g.A = A; g.lda = lda; g.B = Bt; g.ldb = b_nsk > 0 ? 64 : ldb; g.b_nsk = b_nsk; g.C = C; g.ldc = ldc;
  g.M = M; g.N = N; g.K = K; g.m_valid = M; g.ka_valid = K; g.kb_valid = K;
  if (few_tiles(M, N, 256, N <= 128 ? 128 : 256)) {
    const SmallSplit p = part ? plan_small_split(M, N, K, 64) : SmallSplit{1, K};
    if (p.splits > 1) {
      g.C = part;
      g.ldc = N;
      g.k_split = p.k_split;
      const hipError_t e = launch<CfgNTs<EPI_F32, false>>(tag, g, p.splits, st);
      if (e != hipSuccess) return e;
      return reduce_bf16(part, p.splits, M, N, C, ldc, st);
    }
    return launch<CfgNTs<EPI_BF16, false>>(tag, g, 1, st);
  }
  if (N <= 128) return launch<CfgNT<128, EPI_BF16, false>>(tag, g, 1, st);
  return launch<CfgNT3>(tag, g, 1, st);
}

// Work split of a K = T product.  Split-K: enough workgroups to cover the 256
// CUs once, each split at least 8 K steps long (more splits fill the CUs more
// evenly but cost more partial-sum traffic than they save at the 1B shapes);
// below 16 steps (T < 1024) and for outputs under 2^20 elements, splits may be
// 2 steps long, since there the latency of a few long workgroups dominates
// (measured: the 60M backward at 512 tokens 134 -> 93 us; the same rule was
// slower at 2048 tokens and above, and for the 1B shape's larger outputs).
// When that leaves more than a tenth of the CUs idle, the register-staged
// (2:4) products use stream-K instead: 256 workgroups with equal shares of
// the tiles x K steps, each at least 8 steps.
constexpr int kStreamWgs = 256;
// Products that even split fill at most half the CUs with 256 x 256 tiles
// (short K at small token counts) use 128 x 128 tiles and split-K only.
struct SplitPlan {
  int splits;
  int64_t k_split;
  int64_t stream_steps;   // > 0: stream-K with this many K steps per tile
  int segs;               // stream-K partial tiles per workgroup
  bool small;             // 128 x 128 tiles
};
SplitPlan plan_tiles(int64_t M, int64_t N, int64_t K, int tb) {
  const int64_t tiles = cdiv(M, tb) * cdiv(N, tb);
  const int64_t steps = cdiv(K, 64);
  const int64_t min_steps = steps < 16 && M * N < (1 << 20) ? 2 : 8;
  int64_t s = 256 / tiles;
  if (s < 1) s = 1;
  if (s > steps / min_steps) s = steps / min_steps > 0 ? steps / min_steps : 1;
  const int64_t k_split = cdiv(cdiv(K, s), 64) * 64;
  return {(int)cdiv(K, k_split), k_split, 0, 0, tb == 128};
}
SplitPlan plan_splits(int64_t M, int64_t N, int64_t K, bool allow_stream) {
  if (K <= 0) return {0, 0, 0, 0, false};
  const SplitPlan big = plan_tiles(M, N, K, 256);
  const int64_t tiles = cdiv(M, 256) * cdiv(N, 256), steps = cdiv(K, 64);
  if (tiles * big.splits * 2 <= kStreamWgs) {
    const SplitPlan sm = plan_tiles(M, N, K, 128);
    if (cdiv(M, 128) * cdiv(N, 128) * sm.splits > 2 * tiles * big.splits) return sm;
  }
  if (allow_stream && tiles * big.splits * 10 < 9LL * kStreamWgs && tiles * steps >= 8LL * kStreamWgs) {
    const int64_t longest = cdiv(tiles * steps, kStreamWgs);
    return {1, K, steps, (int)((longest - 1) / steps + 2), false};
  }
  return big;
}
size_t partial_bytes(int64_t M, int64_t N, int64_t K, bool allow_stream) {
  const SplitPlan p = plan_splits(M, N, K, allow_stream);
  if (p.stream_steps > 0) return (size_t)kStreamWgs * p.segs * 256 * 256 * sizeof(float);
  return (size_t)p.splits * M * N * sizeof(float);
}

// C = A^T B summed over K = T rows, reduced into out (optionally transposed),
// keeping rows m < rows_out.  A is [K x M] dense (OP_T) or 2:4 compressed
// along M (OP_TSP); B is [K x N] dense.
template <int AMODE>
using CfgTTs = GemmCfg<128, 128, 2, 2, AMODE, OP_T, EPI_F32, false>;

template <int AMODE>
hipError_t gemm_tt_f32(const char* tag, const uint16_t* A, int64_t lda, const uint8_t* Am, int64_t ldam, const uint16_t* B,
                       int64_t ldb, int64_t M, int64_t N, int64_t K, float* part, float* out, int64_t rows_out,
                       bool transpose, int64_t ldo, hipStream_t st) {
  if (K == 0) return hipSuccess;
  using Cfg = CfgTT<AMODE>;
  const SplitPlan p = plan_splits(M, N, K, AMODE == OP_TSP);
  GemmArgs g{};
  g.A = A; g.lda = lda; g.Am = Am; g.ldam = ldam; g.B = B; g.ldb = ldb;
  g.M = M; g.N = N; g.K = K; g.m_valid = M; g.ka_valid = K; g.kb_valid = K;
  g.k_split = p.k_split; g.C = part; g.ldc = N;
  if (AMODE == OP_TSP) g.tok = K;   // the compressed operand is tiled over its K (token) rows
  const dim3 rgrid((unsigned)cdiv(N, 64), (unsigned)cdiv(rows_out, 64));
  if (p.stream_steps > 0) {
    static_assert(Cfg::BM == 256 && Cfg::BN == 256, "stream-K partial tiles are 256 x 256");
    g.stream_steps = p.stream_steps;
    g.stream_segs = p.segs;
    g.tiles_m = (int)cdiv(M, Cfg::BM);
    g.tiles_n = (int)cdiv(N, Cfg::BN);
    {
      TimedLaunch tl(tag, st);
      hipLaunchKernelGGL(gemm_kernel<Cfg>, dim3(kStreamWgs), dim3(Cfg::NT), 0, st, g);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    TimedLaunch tl("splitk_reduce", st);
    hipLaunchKernelGGL(streamk_reduce_kernel, rgrid, dim3(256), 0, st, part, kStreamWgs, p.segs, p.stream_steps,
                       g.tiles_n, (int64_t)g.tiles_m * g.tiles_n, N, rows_out, transpose ? 1 : 0, out, ldo);
    return hipGetLastError();
  }
  hipError_t e = p.small ? launch<CfgTTs<AMODE>>(tag, g, p.splits, st) : launch<Cfg>(tag, g, p.splits, st);
  if (e != hipSuccess) return e;
  TimedLaunch tl("splitk_reduce", st);
  hipLaunchKernelGGL(splitk_reduce_kernel, rgrid, dim3(256), 0, st, part, p.splits, M, N, rows_out,
                     transpose ? 1 : 0, out, ldo);
  return hipGetLastError();
}

struct FwdWs {
  uint16_t *U_upT, *V_upT, *U_downT, *V_downT;
  float* part;   // split-K partials of the long-K products at small token counts
  size_t bytes;
};
// (ab: the caller passes the factors already K-contiguous; no copies)
FwdWs fwd_ws(char* p, int64_t T, int64_t d, int64_t F, int64_t r, bool ab) {
  const int64_t Fp = pad64(F);
  Carver c{p};
  FwdWs w{};
  if (!ab) {
    w.U_upT = c.take<uint16_t>(r * d);
    w.V_upT = c.take<uint16_t>(Fp * r);
    w.U_downT = c.take<uint16_t>(r * Fp);
    w.V_downT = c.take<uint16_t>(d * r);
  }
  size_t pb = small_split_bytes(T, r, d, 64);                 // k1
  pb = std::max(pb, small_split_bytes(T, r, Fp, 64));          // k3 (2:4 or dense)
  pb = std::max(pb, small_split_bytes(T, d, r, 64));           // k4
  w.part = pb ? c.take<float>(pb / sizeof(float)) : nullptr;
  w.bytes = c.used;
  return w;
}

struct BwdWs {
  uint16_t *dZ, *dH, *dP, *V_upT;
  uint16_t *V_upB, *V_downB;   // V_up [r x F] and V_down [r x d] blocked (the B operands of b5, b1)
  float* part;
  size_t bytes;
};
// dH is compressed [T x ldv] in the sparse backward and dense [T x F] in the
// dense and straight-through ones; the straight-through backward also holds
// V_up^T (relu(h) is recomputed tile by tile inside the dH kernel).
BwdWs bwd_ws(char* p, int64_t T, int64_t d, int64_t F, int64_t r, bool dense, bool ste) {
  const int64_t Fp = pad64(F);
  Carver c{p};
  BwdWs w{};
  w.dZ = c.take<uint16_t>(T * r);
  w.dH = c.take<uint16_t>(T * ((dense || ste) ? F : vals_ld(F)));
  w.dP = c.take<uint16_t>(T * r);
  if (ste) w.V_upT = c.take<uint16_t>(Fp * r);
  w.V_upB = c.take<uint16_t>(pad256(r) * Fp);
  w.V_downB = c.take<uint16_t>(pad256(r) * pad64(d));
  // split-K partials of the products over tokens (d_ff-wide ones have Fp rows
  // when read compressed, F rows when dense)
  size_t pb = partial_bytes(r, d, T, false);
  const size_t p2 = partial_bytes(Fp, r, T, true), p3 = partial_bytes(d, r, T, false), p4 = partial_bytes(F, r, T, false);
  if (p2 > pb) pb = p2;
  if (p3 > pb) pb = p3;
  if (p4 > pb) pb = p4;
  // split-K of the long-K bf16 products at small token counts (b1, b5, b8)
  pb = std::max(pb, small_split_bytes(T, r, d, 64));
  pb = std::max(pb, small_split_bytes(T, r, Fp, 64));
  pb = std::max(pb, small_split_bytes(T, d, r, 64));
  w.part = c.take<float>(pb / sizeof(float));
  w.bytes = c.used;
  return w;
}

#define ELAS_TRY(...)                        \
  do {                                       \
    hipError_t e_ = (__VA_ARGS__);           \
    if (e_ != hipSuccess) return e_;         \
  } while (0)

}  // namespace

size_t spmm_workspace_bytes(int64_t K, int64_t N, int b_layout) {
  return b_layout == 0 ? align_up((size_t)K * N * sizeof(uint16_t)) : 0;
}

size_t fwd_workspace_bytes(int64_t T, int64_t d, int64_t F, int64_t r, bool dense, bool ab) {
  (void)dense;
  return fwd_ws(nullptr, T, d, F, r, ab).bytes;
}

size_t bwd_workspace_bytes(int64_t T, int64_t d, int64_t F, int64_t r, bool dense, bool ste) {
  return bwd_ws(nullptr, T, d, F, r, dense, ste).bytes;
}

hipError_t run_spmm24(const uint16_t* a_vals, const uint8_t* a_meta, int64_t M, int64_t K, const uint16_t* b,
                      int64_t N, bool b_is_nk, uint16_t* c, void* ws, hipStream_t st) {
  if (M == 0) return hipSuccess;
  const uint16_t* bt = b;
  int64_t ldb = K;
  if (!b_is_nk) {   // B [K x N] -> B^T [N x K] in the workspace
    uint16_t* t = (uint16_t*)ws;
    ELAS_TRY(transpose_pad(b, K, N, N, t, N, K, K, st));
    bt = t;
  }
  GemmArgs g{};
  g.A = a_vals; g.lda = vals_ld(K); g.Am = a_meta; g.ldam = meta_ld(K);
  g.B = bt; g.ldb = ldb;
  g.M = M; g.N = N; g.K = pad64(K); g.m_valid = M; g.ka_valid = pad64(K); g.kb_valid = K;
  g.C = c; g.ldc = N;
  return launch_sp("spmm24", g, st);
}

hipError_t run_fwd(const FfnArgs& a, hipStream_t st) {
  const int64_t T = a.T, d = a.d, F = a.F, r = a.r, Fp = pad64(F);
  const FwdWs w = fwd_ws((char*)a.ws, T, d, F, r, a.ab);
  // Weight factors K-contiguous for the MFMA operands: laid out here, or
  // given so (ELAS_FACTORS_AB: unpadded d_ff, whose missing rows / columns
  // the loads read as zero, exactly like the zero padding of the copies).
  const uint16_t *U_upT = a.U_up, *V_upT = a.V_up, *U_downT = a.U_down, *V_downT = a.V_down;
  int64_t F_rows = F, ld_ud = F;   // rows of V_up^T, pitch (= K extent) of U_down^T
  if (!a.ab) {
    Transposes tr;
    tr.add(a.U_up, d, r, r, w.U_upT, r, d, d);          // [r x d]
    tr.add(a.V_up, r, F, F, w.V_upT, Fp, r, r);         // [Fp x r], zero rows >= F
    tr.add(a.U_down, F, r, r, w.U_downT, r, Fp, Fp);    // [r x Fp], zero cols >= F
    tr.add(a.V_down, r, d, d, w.V_downT, d, r, r);      // [d x r]
    ELAS_TRY(tr.launch(st));
    U_upT = w.U_upT; V_upT = w.V_upT; U_downT = w.U_downT; V_downT = w.V_downT;
    F_rows = Fp;
    ld_ud = Fp;
  }
  // The one-launch forward only on request: measured slower than the four
  // kernels below at every supported shape but one.
  if (!a.dense && a.fused == 1)
    return run_fused_fwd(a.x, U_upT, V_upT, U_downT, V_downT, T, d, F, r, F_rows, ld_ud, a.y, a.P, a.s_vals,
                         a.s_meta, a.Z, st);
  // P = x U_up
  ELAS_TRY(gemm_nt_bf16("k1_up_gemm", a.x, d, U_upT, d, a.P, r, T, r, d, st, w.part));
  if (!a.dense) {
    // H^T = V_up^T P^T with ReLU^2 + 2:4 selection + compression in the epilogue
    GemmArgs g{};
    g.A = V_upT; g.lda = r; g.B = a.P; g.ldb = r;
    g.M = Fp; g.N = T; g.K = r; g.m_valid = F_rows; g.ka_valid = r; g.kb_valid = r;
    g.sv = a.s_vals; g.sm = a.s_meta; g.ldv = vals_ld(F); g.ldm = meta_ld(F); g.tok = T;   // S written tiled
    ELAS_TRY(launch_staged<EPI_SPARSIFY>("k2_up_relu2_sparsify", g, st));
    // Z = S U_down on the 2:4 operand
    GemmArgs z{};
    z.A = a.s_vals; z.lda = vals_ld(F); z.Am = a.s_meta; z.ldam = meta_ld(F); z.a_tiled = 1; z.tok = T;
    z.B = U_downT; z.ldb = ld_ud;
    z.M = T; z.N = r; z.K = Fp; z.m_valid = T; z.ka_valid = Fp; z.kb_valid = ld_ud;
    z.C = a.Z; z.ldc = r;
    ELAS_TRY(launch_sp("k3_spmm_down", z, st, w.part));
  } else {
    // dense activations: S = relu(H)^2 written [T x F], then a dense product
    GemmArgs g{};
    g.A = V_upT; g.lda = r; g.B = a.P; g.ldb = r;
    g.M = Fp; g.N = T; g.K = r; g.m_valid = F_rows; g.ka_valid = r; g.kb_valid = r;
    g.act = a.s_vals; g.ld_act = F; g.f_valid = F; g.act_square = 1;
    ELAS_TRY(launch_act<EPI_ACT_DENSE>("k2_up_relu2_dense", g, st));
    ELAS_TRY(gemm_nt_bf16("k3_down_gemm_dense", a.s_vals, F, U_downT, ld_ud, a.Z, r, T, r, F, st, w.part));
  }
  // Y = Z V_down
  ELAS_TRY(gemm_nt_bf16("k4_down_gemm", a.Z, r, V_downT, r, a.y, d, T, d, r, st, w.part));
  return hipSuccess;
}

// Full-rank ReLU^2 FFN forward (the comparison of Table 3, Sec. 4.2.3).  The
// weights come in the orientation of Eq. 1 (W_up [F x d], W_down [d x F]),
// which is already the K-contiguous operand layout, so nothing is re-laid out:
// S = relu(x W_up^T)^2 through the fused dense-activation epilogue of the
// dense-mode up projection, then Y = S W_down^T.
hipError_t run_fullrank_fwd(const uint16_t* x, const uint16_t* W_up, const uint16_t* W_down, int64_t T,
                            int64_t d, int64_t F, uint16_t* y, uint16_t* S, hipStream_t st) {
  // S^T = relu(W_up x^T)^2, written token-major [T x F]
  GemmArgs g{};
  g.A = W_up; g.lda = d; g.B = x; g.ldb = d;
  g.M = F; g.N = T; g.K = d; g.m_valid = F; g.ka_valid = d; g.kb_valid = d;
  g.act = S; g.ld_act = F; g.f_valid = F; g.act_square = 1;
  ELAS_TRY(launch_act<EPI_ACT_DENSE>("fr_up_relu2", g, st));
  // Y = S W_down^T
  ELAS_TRY(gemm_nt_bf16("fr_down_gemm", S, F, W_down, F, y, d, T, d, F, st));
  return hipSuccess;
}

hipError_t run_bwd(const FfnArgs& a, hipStream_t st) {
  const int64_t T = a.T, d = a.d, F = a.F, r = a.r, Fp = pad64(F);
  const int64_t ldv = vals_ld(F), ldm = meta_ld(F);
  if (T == 0) {
    ELAS_TRY(fill_zero(a.dU_up, d * r, st));
    ELAS_TRY(fill_zero(a.dV_up, r * F, st));
    ELAS_TRY(fill_zero(a.dU_down, F * r, st));
    ELAS_TRY(fill_zero(a.dV_down, r * d, st));
    return hipSuccess;
  }
  const BwdWs w = bwd_ws((char*)a.ws, T, d, F, r, a.dense, a.ste);
  // V_up and V_down are the K-contiguous B operands of dP and dZ as they are,
  // but the row pitch of V_up (d_ff elements) need not be a multiple of 64
  // bytes, so that each 128-byte row piece of a K step would straddle two
  // cache lines.  Both are copied blocked (one contiguous 32 KB block per
  // tile K step: measured 7 % faster for dP at 1B), and V_up^T for the
  // straight-through backward, in one launch.
  const int64_t nsk_vu = Fp / 64, nsk_vd = pad64(d) / 64;
  {
    Transposes tr;
    tr.add(a.V_up, r, F, F, w.V_upB, pad256(r), Fp, 0, 0, nsk_vu);
    tr.add(a.V_down, r, d, d, w.V_downB, pad256(r), pad64(d), 0, 0, nsk_vd);
    if (a.ste) tr.add(a.V_up, r, F, F, w.V_upT, Fp, r, r);      // [Fp x r], zero rows >= F
    ELAS_TRY(tr.launch(st));
  }
  // dZ = dY V_down^T
  ELAS_TRY(gemm_nt_bf16("b1_dZ", a.dy, d, w.V_downB, d, w.dZ, r, T, r, d, st, w.part, nsk_vd));
  // dV_down = Z^T dY
  ELAS_TRY(gemm_tt_f32<OP_T>("b2_dV_down", a.Z, r, nullptr, 0, a.dy, d, r, d, T, w.part, a.dV_down, r, false, d, st));
  if (!a.dense && !a.ste) {
    // dH = (dZ U_down^T) * mask * 2 relu(H), computed as dS^T = U_down dZ^T
    GemmArgs g{};
    g.A = a.U_down; g.lda = r; g.B = w.dZ; g.ldb = r;
    g.M = Fp; g.N = T; g.K = r; g.m_valid = F; g.ka_valid = r; g.kb_valid = r;
    g.sv = a.s_vals; g.sm = a.s_meta; g.ldv = ldv; g.ldm = ldm; g.dv = w.dH; g.tok = T;   // S read, dH written, tiled
    ELAS_TRY(launch_staged<EPI_DH>("b3_dH_masked", g, st));
    // dU_down = S^T dZ from the compressed S
    ELAS_TRY(gemm_tt_f32<OP_TSP>("b4_dU_down", a.s_vals, ldv, a.s_meta, ldm, w.dZ, r, Fp, r, T, w.part, a.dU_down, F,
                                 false, r, st));
    // dP = dH V_up^T on the 2:4 operand (V_up blocked)
    GemmArgs p{};
    p.A = w.dH; p.lda = ldv; p.Am = a.s_meta; p.ldam = ldm; p.a_tiled = 1; p.tok = T;
    p.B = w.V_upB; p.ldb = 64; p.b_nsk = nsk_vu;
    p.M = T; p.N = r; p.K = Fp; p.m_valid = T; p.ka_valid = Fp; p.kb_valid = F;
    p.C = w.dP; p.ldc = r;
    ELAS_TRY(launch_sp("b5_spmm_dP", p, st, w.part));
    // dV_up = P^T dH, computed as dV_up^T = dH^T P and written transposed
    ELAS_TRY(gemm_tt_f32<OP_TSP>("b6_dV_up", w.dH, ldv, a.s_meta, ldm, a.P_in, r, Fp, r, T, w.part, a.dV_up, F, true, F,
                                 st));
  } else {
    // dense dH [T x F] = dS * 2 r at every position: r = bf16(sqrt(s)) from the
    // dense S (dense mode), or relu(h) recomputed from P and V_up (straight-
    // through estimator of Eq. 4 after a sparse forward)
    GemmArgs g{};
    g.A = a.U_down; g.lda = r; g.B = w.dZ; g.ldb = r;
    g.M = Fp; g.N = T; g.K = r; g.m_valid = F; g.ka_valid = r; g.kb_valid = r;
    g.ld_act = F; g.f_valid = F; g.dact = w.dH;
    if (a.ste) {
      // one kernel per tile: h^T = V_up^T P^T over the first r contraction
      // steps (V_up^T rows >= F read as zero), relu(h) kept in registers, then
      // dS^T = U_down dZ^T over the next r
      g.A = w.V_upT; g.B = a.P_in; g.A2 = a.U_down; g.B2 = w.dZ;
      ELAS_TRY(launch_act<EPI_DH_STE>("b3_dH_ste", g, st));
    } else {
      g.act = const_cast<uint16_t*>(a.s_vals); g.act_square = 1;
      ELAS_TRY(launch_act<EPI_DH_DENSE>("b3_dH_dense", g, st));
    }
    if (a.dense) {
      // dU_down = S^T dZ with the dense S
      ELAS_TRY(gemm_tt_f32<OP_T>("b4_dU_down_dense", a.s_vals, F, nullptr, 0, w.dZ, r, F, r, T, w.part, a.dU_down, F,
                                 false, r, st));
    } else {
      ELAS_TRY(gemm_tt_f32<OP_TSP>("b4_dU_down", a.s_vals, ldv, a.s_meta, ldm, w.dZ, r, Fp, r, T, w.part, a.dU_down,
                                   F, false, r, st));
    }
    // dP = dH V_up^T (dense)
    ELAS_TRY(gemm_nt_bf16("b5_dP_dense", w.dH, F, w.V_upB, F, w.dP, r, T, r, F, st, w.part, nsk_vu));
    // dV_up^T = dH^T P (dense), written transposed
    ELAS_TRY(gemm_tt_f32<OP_T>("b6_dV_up_dense", w.dH, F, nullptr, 0, a.P_in, r, F, r, T, w.part, a.dV_up, F, true,
                               F, st));
  }
  // dU_up = x^T dP
  ELAS_TRY(gemm_tt_f32<OP_T>("b7_dU_up", a.x, d, nullptr, 0, w.dP, r, d, r, T, w.part, a.dU_up, d, false, r, st));
  // dx = dP U_up^T   (U_up [d x r] is already K-contiguous)
  ELAS_TRY(gemm_nt_bf16("b8_dx", w.dP, r, a.U_up, r, a.dx, d, T, d, r, st, w.part));
  return hipSuccess;
}

}  // namespace elas
