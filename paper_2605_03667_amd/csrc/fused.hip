// Fused forward of the ELAS low-rank FFN for compact factor shapes: one launch
// computes P = x U_up, the 2:4-pruned S = top2(relu(P V_up)^2), Z = S U_down
// and Y = Z V_down (Eq. 1-3, Algorithm 1; the block of the Fig. 1 caption) for
// a block of tokens per workgroup.  P and the current d_ff chunk of S stay in
// LDS, Z accumulates in registers across d_ff, and only the saved activations
// (P, the compressed S, Z) and Y are written.  The weight factors are read
// K-contiguous (the operand layout of the four-kernel path) and served from L2.
//
// Every product is computed as C^T = W * Act^T on v_mfma_f32_32x32x16_bf16:
// A is a factor (rows = output features, K contiguous, from global memory), B
// the activation block (rows = tokens, K contiguous, from LDS; x in phase 1
// comes from global memory too).  Accumulator e of lane l then holds feature
// 8(e/4) + 4(l/32) + e%4 of a 32-feature block for token l%32, so each lane
// owns whole groups of 4 consecutive features: the 2:4 selection needs no data
// exchange, and the outputs leave as 8-byte pieces of 4 consecutive features.
#include "gemm.h"
#include "internal.h"

namespace elas {

namespace {

struct FusedArgs {
  const uint16_t* x;         // [T x d]
  const uint16_t* U_upT;     // [r x d]
  const uint16_t* V_upT;     // [F_rows x r]; rows >= F_rows read as 0
  const uint16_t* U_downT;   // [r x ld_ud]; columns >= F_cols read as 0
  const uint16_t* V_downT;   // [d x r]
  uint16_t* P;               // [T x r]
  uint16_t* sv;              // kept values of S, tiled (tok = T), pitch ldv
  uint8_t* sm;               // metadata of S, tiled, pitch ldm
  uint16_t* Z;               // [T x r]
  uint16_t* y;               // [T x d]
  int64_t T, ldv, ldm, ld_ud;
  int d, r, Fp, F_rows, F_cols;
};

constexpr int kFusedThreads = 256;   // 4 waves, one per SIMD
constexpr int kChunk = 128;          // d_ff features per chunk (32 per wave)
constexpr int kMaxR = 256;

__device__ __forceinline__ bf16x8 as_frag(uint4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ uint4 load16(const uint16_t* p, bool ok) {
  return ok ? *(const uint4*)p : make_uint4(0u, 0u, 0u, 0u);
}
__device__ __forceinline__ f32x16 mfma(uint4 a, uint4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_frag(a), as_frag(b), c, 0, 0, 0);
}
__device__ __forceinline__ void zero16(f32x16& a) {
#pragma unroll
  for (int e = 0; e < 16; ++e) a[e] = 0.f;
}

// TB token blocks of 32 per workgroup; NR = r / 128 (32-wide output blocks of
// the r-wide products per wave).
template <int TB, int NR>
__global__ __launch_bounds__(kFusedThreads) void fused_fwd_kernel(const FusedArgs a) {
  constexpr int BT = 32 * TB;
  constexpr int R = 128 * NR;               // r
  constexpr int PP = 2 * R + 16;            // bytes per LDS row of P / Z (16-byte skew per row)
  constexpr int SP = 2 * kChunk + 16;       // bytes per LDS row of an expanded S chunk
  constexpr int RK = R / 16;                // k16 steps over r
  __shared__ __attribute__((aligned(16))) char ps[BT * PP];          // P, later Z
  __shared__ __attribute__((aligned(16))) char ss[2][BT * SP];       // S chunks (double buffer)

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 31, lh = lane >> 5;
  const int64_t t0 = (int64_t)blockIdx.x * BT;
  const int64_t T = a.T;
  const int d = a.d;

  // ---- phase 1: P^T = U_up^T x^T (K = d), output blocks wave + 4 i ------------
  {
    f32x16 acc[NR][TB];
#pragma unroll
    for (int i = 0; i < NR; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j) zero16(acc[i][j]);
    uint4 fa[2][NR][4], fb[2][TB][4];
    auto load = [&](int kc, uint4 (&la)[NR][4], uint4 (&lb)[TB][4]) __attribute__((always_inline)) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const int k = kc * 64 + ks * 16 + 8 * lh;
#pragma unroll
        for (int i = 0; i < NR; ++i) la[i][ks] = *(const uint4*)(a.U_upT + (int64_t)((wave + 4 * i) * 32 + lr) * d + k);
#pragma unroll
        for (int j = 0; j < TB; ++j) {
          const int64_t t = t0 + 32 * j + lr;
          lb[j][ks] = load16(a.x + t * d + k, t < T);
        }
      }
    };
    auto compute = [&](uint4 (&la)[NR][4], uint4 (&lb)[TB][4]) __attribute__((always_inline)) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int i = 0; i < NR; ++i)
#pragma unroll
          for (int j = 0; j < TB; ++j) acc[i][j] = mfma(la[i][ks], lb[j][ks], acc[i][j]);
    };
    const int nk = d / 64;   // chunks of 64 along d, loaded one chunk ahead
    load(0, fa[0], fb[0]);
    for (int kc = 0; kc < nk; kc += 2) {
      if (kc + 1 < nk) load(kc + 1, fa[1], fb[1]);
      compute(fa[0], fb[0]);
      if (kc + 1 < nk) {
        if (kc + 2 < nk) load(kc + 2, fa[0], fb[0]);
        compute(fa[1], fb[1]);
      }
    }
    // P rounded to bf16: to the saved P and to LDS (phase 2's B operand)
#pragma unroll
    for (int i = 0; i < NR; ++i)
#pragma unroll
      for (int j = 0; j < TB; ++j)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int n = (wave + 4 * i) * 32 + 8 * b + 4 * lh, tl = 32 * j + lr;
          const uint2 v = make_uint2(bf16x2_rne(acc[i][j][4 * b], acc[i][j][4 * b + 1]),
                                     bf16x2_rne(acc[i][j][4 * b + 2], acc[i][j][4 * b + 3]));
          *(uint2*)(ps + tl * PP + 2 * n) = v;
          if (t0 + tl < T) *(uint2*)(a.P + (t0 + tl) * R + n) = v;
        }
  }
  __syncthreads();

  // ---- phases 2 + 3 over d_ff chunks of 128 features -------------------------
  // Phase 2: H^T of features c*128 + 32 wave .. +31 (K = r), ReLU^2, top-2 of
  // each group of 4, compressed to the saved S and expanded into LDS.
  // Phase 3: Z^T += U_down^T[:, chunk] S_chunk^T (K = 128), output blocks
  // wave + 4 i.  A chunk's A operands are loaded one phase ahead.
  f32x16 accz[NR][TB];
#pragma unroll
  for (int i = 0; i < NR; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j) zero16(accz[i][j]);
  uint4 f2[RK], f3[NR][8];
  auto load2 = [&](int c) __attribute__((always_inline)) {
    const int f = c * kChunk + 32 * wave + lr;
#pragma unroll
    for (int ks = 0; ks < RK; ++ks) f2[ks] = load16(a.V_upT + (int64_t)f * R + ks * 16 + 8 * lh, f < a.F_rows);
  };
  auto load3 = [&](int c) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const int f = c * kChunk + ks * 16 + 8 * lh;
#pragma unroll
      for (int i = 0; i < NR; ++i)
        f3[i][ks] = load16(a.U_downT + (int64_t)((wave + 4 * i) * 32 + lr) * a.ld_ud + f, f < a.F_cols);
    }
  };
  const int nchunks = (a.Fp + kChunk - 1) / kChunk;
  load2(0);
  load3(0);
  for (int c = 0; c < nchunks; ++c) {
    char* sbuf = ss[c & 1];
    f32x16 acch[TB];
#pragma unroll
    for (int j = 0; j < TB; ++j) zero16(acch[j]);
#pragma unroll
    for (int ks = 0; ks < RK; ++ks)
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const uint4 bv = *(const uint4*)(ps + (32 * j + lr) * PP + 32 * ks + 16 * lh);
        acch[j] = mfma(f2[ks], bv, acch[j]);
      }
    if (c + 1 < nchunks) load2(c + 1);
    const int f0 = c * kChunk + 32 * wave;   // first feature of this wave's block
#pragma unroll
    for (int j = 0; j < TB; ++j) {
      const int tl = 32 * j + lr;
      const int64_t t = t0 + tl;
      uint32_t codes = 0;   // code of group b at bits 8b .. 8b+3
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        // h = bf16(H) relu'd (rounding keeps the sign), ranked with ties to
        // the lower index; kept s = bf16(relu(h)^2) in index order
        const uint32_t p01 = bf16x2_rne(relu_f32(acch[j][4 * b]), relu_f32(acch[j][4 * b + 1]));
        const uint32_t p23 = bf16x2_rne(relu_f32(acch[j][4 * b + 2]), relu_f32(acch[j][4 * b + 3]));
        const Top2 k = top2_keys_hi(p01, p23);
        const uint32_t code = top2_code_xor15(k) ^ 0xFu;   // i0 | i1 << 2
        codes |= code << (8 * b);
        const float v0 = __builtin_bit_cast(float, k.first << 2);
        const float v1 = __builtin_bit_cast(float, k.second << 2);
        const uint32_t pair = bf16x2_rne(v0 * v0, v1 * v1);
        // expanded group (kept values at slots i0, i1, zeros elsewhere) for phase 3
        const uint64_t e = ((uint64_t)(pair & 0xFFFFu) << (16 * (code & 3u))) |
                           ((uint64_t)(pair >> 16) << (16 * (code >> 2)));
        *(uint2*)(sbuf + tl * SP + 2 * (32 * wave + 8 * b + 4 * lh)) = make_uint2((uint32_t)e, (uint32_t)(e >> 32));
        if (t < T && f0 < a.Fp) {
          const int g = (f0 + 8 * b + 4 * lh) / 4;   // group index along d_ff
          *(uint32_t*)(a.sv + tiled_index<32>(t, 2 * g, T, a.ldv)) = pair;
        }
      }
      // metadata byte f/8 = code of the even group (lane half 0) | code of the
      // odd group (half 1) << 4; the swap hands half 0 its partner's codes
      const uint32_t other = __builtin_amdgcn_permlane32_swap(codes, codes, false, false)[1];
      if (lh == 0 && t < T && f0 < a.Fp) *(uint32_t*)(a.sm + tiled_index<8>(t, f0 / 8, T, a.ldm)) = codes | (other << 4);
    }
    __syncthreads();   // the S chunk is complete; the other buffer is free (see below)
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const uint4 bv = *(const uint4*)(sbuf + (32 * j + lr) * SP + 32 * ks + 16 * lh);
#pragma unroll
        for (int i = 0; i < NR; ++i) accz[i][j] = mfma(f3[i][ks], bv, accz[i][j]);
      }
    if (c + 1 < nchunks) load3(c + 1);
    // Chunk c + 2 rewrites this buffer only after the barrier of chunk c + 1,
    // which every wave reaches after finishing these reads.
  }

  // ---- phase 4: Z rounded to bf16 (saved, and to LDS), Y^T = V_down^T Z^T ----
  // (P's LDS rows are free: every wave passed the last chunk's barrier after
  // its last phase-2 read.)
#pragma unroll
  for (int i = 0; i < NR; ++i)
#pragma unroll
    for (int j = 0; j < TB; ++j)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int n = (wave + 4 * i) * 32 + 8 * b + 4 * lh, tl = 32 * j + lr;
        const uint2 v = make_uint2(bf16x2_rne(accz[i][j][4 * b], accz[i][j][4 * b + 1]),
                                   bf16x2_rne(accz[i][j][4 * b + 2], accz[i][j][4 * b + 3]));
        *(uint2*)(ps + tl * PP + 2 * n) = v;
        if (t0 + tl < T) *(uint2*)(a.Z + (t0 + tl) * R + n) = v;
      }
  __syncthreads();
  {
    uint4 f4[2][RK];
    auto load4 = [&](int nb, uint4 (&l)[RK]) __attribute__((always_inline)) {
#pragma unroll
      for (int ks = 0; ks < RK; ++ks) l[ks] = *(const uint4*)(a.V_downT + (int64_t)(nb * 32 + lr) * R + ks * 16 + 8 * lh);
    };
    auto block = [&](int nb, uint4 (&l)[RK]) __attribute__((always_inline)) {
      f32x16 acc[TB];
#pragma unroll
      for (int j = 0; j < TB; ++j) zero16(acc[j]);
#pragma unroll
      for (int ks = 0; ks < RK; ++ks)
#pragma unroll
        for (int j = 0; j < TB; ++j) {
          const uint4 bv = *(const uint4*)(ps + (32 * j + lr) * PP + 32 * ks + 16 * lh);
          acc[j] = mfma(l[ks], bv, acc[j]);
        }
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        const int64_t t = t0 + 32 * j + lr;
        if (t < T) {
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int n = nb * 32 + 8 * b + 4 * lh;
            *(uint2*)(a.y + t * d + n) = make_uint2(bf16x2_rne(acc[j][4 * b], acc[j][4 * b + 1]),
                                                    bf16x2_rne(acc[j][4 * b + 2], acc[j][4 * b + 3]));
          }
        }
      }
    };
    // this wave's output blocks are wave, wave + 4, ...; the next one's A
    // operands load while the current one computes
    const int nblk = d / 32;
    if (wave < nblk) load4(wave, f4[0]);
    for (int nb = wave; nb < nblk; nb += 8) {
      if (nb + 4 < nblk) load4(nb + 4, f4[1]);
      block(nb, f4[0]);
      if (nb + 4 < nblk) {
        if (nb + 8 < nblk) load4(nb + 8, f4[0]);
        block(nb + 4, f4[1]);
      }
    }
  }
}

template <int TB, int NR>
hipError_t launch_fused(const FusedArgs& a, hipStream_t st) {
  const unsigned blocks = (unsigned)((a.T + 32 * TB - 1) / (32 * TB));
  TimedLaunch tl("f3_fused_fwd", st);
  hipLaunchKernelGGL((fused_fwd_kernel<TB, NR>), dim3(blocks), dim3(kFusedThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace

bool fused_fwd_supported(int64_t d, int64_t r) {
  return d % 64 == 0 && d <= 1024 && r % 128 == 0 && r <= kMaxR;
}

hipError_t run_fused_fwd(const uint16_t* x, const uint16_t* U_upT, const uint16_t* V_upT, const uint16_t* U_downT,
                         const uint16_t* V_downT, int64_t T, int64_t d, int64_t F, int64_t r, int64_t F_rows,
                         int64_t ld_ud, uint16_t* y, uint16_t* P, uint16_t* s_vals, uint8_t* s_meta, uint16_t* Z,
                         hipStream_t st) {
  if (T == 0) return hipSuccess;
  if (!fused_fwd_supported(d, r)) return hipErrorInvalidValue;
  FusedArgs a{};
  a.x = x; a.U_upT = U_upT; a.V_upT = V_upT; a.U_downT = U_downT; a.V_downT = V_downT;
  a.P = P; a.sv = s_vals; a.sm = s_meta; a.Z = Z; a.y = y;
  a.T = T; a.ldv = vals_ld(F); a.ldm = meta_ld(F); a.ld_ud = ld_ud;
  a.d = (int)d; a.r = (int)r; a.Fp = (int)pad64(F); a.F_rows = (int)F_rows; a.F_cols = (int)ld_ud;
  // Two token blocks per workgroup once one-block workgroups would cover the
  // CUs twice over: each factor read from L2 then serves 64 tokens.
  const bool two = T > 2 * 256 * 32;
  if (r == 128) return two ? launch_fused<2, 1>(a, st) : launch_fused<1, 1>(a, st);
  return two ? launch_fused<2, 2>(a, st) : launch_fused<1, 2>(a, st);
}

}  // namespace elas
