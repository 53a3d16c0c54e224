// Standalone 2:4 activation sparsification (ELAS, Sec. 3.3.1, Algorithm 1,
// with Eq. 2's ReLU^2 in front).  HBM-bound streaming kernel: one thread per
// 16 features of a row (4 groups) reads 32 bytes and writes 16 bytes of kept
// values plus 2 bytes of metadata.  Consecutive threads take consecutive
// 16-feature chunks of a row, so a wave reads 2 KB of one row contiguously.
#include "device.h"
#include "internal.h"

namespace elas {

template <bool RAW>
__global__ __launch_bounds__(256) void sparsify24_kernel(const uint16_t* __restrict__ h, int64_t row0, uint32_t rows,
                                                         int64_t N, uint32_t chunks, uint16_t* __restrict__ vals,
                                                         uint8_t* __restrict__ meta, int64_t ldv, int64_t ldm) {
  // rows * chunks < 2^31 (the host cuts larger inputs into slabs), so the
  // thread -> (row, chunk) split uses 32-bit arithmetic.
  const uint32_t t = blockIdx.x * 256u + threadIdx.x;
  if (t >= rows * chunks) return;
  const uint32_t rl = t / chunks;
  const uint32_t c = t - rl * chunks;
  const int64_t row = row0 + rl;
  const int64_t f0 = (int64_t)c * 16;
  const uint16_t* src = h + row * N + f0;
  u32x4 lo = {0u, 0u, 0u, 0u}, hi = {0u, 0u, 0u, 0u};
  // N % 8 == 0, so each 8-feature half is entirely inside or entirely past
  // the row; halves past it read as zeros (all-zero groups keep positions 0,1
  // with value 0, which is the padding content).
  if (f0 + 8 <= N) lo = __builtin_nontemporal_load((const u32x4*)src);
  if (f0 + 16 <= N) hi = __builtin_nontemporal_load((const u32x4*)(src + 8));
  const uint32_t w[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  uint32_t out[4];
  uint32_t code16 = 0u;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    uint32_t code, pair;
    if constexpr (RAW) {
      // rank |h| (sign bit cleared); keep the signed values
      const Top2 k = top2_keys(w[2 * g] & 0x7FFF7FFFu, w[2 * g + 1] & 0x7FFF7FFFu);
      code = top2_code_of(k);
      pair = pick_pair(code, w[2 * g] & 0xFFFFu, w[2 * g] >> 16, w[2 * g + 1] & 0xFFFFu, w[2 * g + 1] >> 16);
    } else {
      // relu (NaN -> 0), rank by value with ties to the lower index, keep
      // relu(h)^2 rounded to bf16
      const Top2 k = top2_keys(relu_bits2(w[2 * g]), relu_bits2(w[2 * g + 1]));
      code = top2_code_of(k);
      const float a = __builtin_bit_cast(float, k.first << 16), b = __builtin_bit_cast(float, k.second << 16);
      pair = bf16x2_rne(a * a, b * b);
    }
    out[g] = pair;
    code16 |= code << (4 * g);
  }
  uint4 o = {out[0], out[1], out[2], out[3]};
  *(uint4*)(vals + row * ldv + (int64_t)c * 8) = o;
  *(uint16_t*)(meta + row * ldm + (int64_t)c * 2) = (uint16_t)code16;
}

hipError_t launch_sparsify24(const uint16_t* h, int64_t M, int64_t N, bool raw, uint16_t* vals,
                             uint8_t* meta, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int64_t ldv = vals_ld(N), ldm = meta_ld(N);
  const int64_t chunks = ldv / 8;             // 16 features per thread, padding included
  const int64_t slab = ((int64_t(1) << 31) - 1) / chunks;   // rows per launch: rows * chunks < 2^31
  TimedLaunch tl("sparsify24", stream);
  for (int64_t r0 = 0; r0 < M; r0 += slab) {
    const int64_t rows = M - r0 < slab ? M - r0 : slab;
    const dim3 grid((unsigned)((rows * chunks + 255) / 256)), block(256);
    if (raw)
      hipLaunchKernelGGL(sparsify24_kernel<true>, grid, block, 0, stream, h, r0, (uint32_t)rows, N, (uint32_t)chunks,
                         vals, meta, ldv, ldm);
    else
      hipLaunchKernelGGL(sparsify24_kernel<false>, grid, block, 0, stream, h, r0, (uint32_t)rows, N,
                         (uint32_t)chunks, vals, meta, ldv, ldm);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace elas
