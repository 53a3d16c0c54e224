// Standalone 2:4 activation sparsification (ELAS, Sec. 3.3.1, Algorithm 1,
// with Eq. 2's ReLU^2 in front).  HBM-bound streaming kernel: one thread per
// 16 features of a row (4 groups) reads 32 bytes and writes 16 bytes of kept
// values plus 2 bytes of metadata.  Consecutive threads take consecutive
// 16-feature chunks of a row, so a wave reads 2 KB of one row contiguously.
#include "device.h"
#include "internal.h"

namespace elas {

template <bool RAW>
__global__ __launch_bounds__(256) void sparsify24_kernel(const uint16_t* __restrict__ h, int64_t M,
                                                         int64_t N, int64_t chunks, uint16_t* __restrict__ vals,
                                                         uint8_t* __restrict__ meta, int64_t ldv,
                                                         int64_t ldm) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= M * chunks) return;
  const int64_t row = t / chunks;
  const int64_t c = t - row * chunks;
  const int64_t f0 = c * 16;
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
    const uint32_t e0 = w[2 * g] & 0xFFFFu, e1 = w[2 * g] >> 16;
    const uint32_t e2 = w[2 * g + 1] & 0xFFFFu, e3 = w[2 * g + 1] >> 16;
    uint32_t code, pair;
    if constexpr (RAW) {
      code = top2_code(e0 & 0x7FFFu, e1 & 0x7FFFu, e2 & 0x7FFFu, e3 & 0x7FFFu);
      pair = pick_pair(code, e0, e1, e2, e3);
    } else {
      const uint32_t r0 = relu_bits(e0), r1 = relu_bits(e1), r2 = relu_bits(e2), r3 = relu_bits(e3);
      code = top2_code(r0, r1, r2, r3);
      const uint32_t kept = pick_pair(code, r0, r1, r2, r3);
      const float a = bf16_to_f32(kept & 0xFFFFu), b = bf16_to_f32(kept >> 16);
      pair = f32_to_bf16_rne(a * a) | (f32_to_bf16_rne(b * b) << 16);
    }
    out[g] = pair;
    code16 |= code << (4 * g);
  }
  uint4 o = {out[0], out[1], out[2], out[3]};
  *(uint4*)(vals + row * ldv + c * 8) = o;
  *(uint16_t*)(meta + row * ldm + c * 2) = (uint16_t)code16;
}

hipError_t launch_sparsify24(const uint16_t* h, int64_t M, int64_t N, bool raw, uint16_t* vals,
                             uint8_t* meta, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int64_t ldv = vals_ld(N), ldm = meta_ld(N);
  const int64_t chunks = ldv / 8;             // 16 features per thread, padding included
  const int64_t threads = M * chunks;
  const dim3 grid((unsigned)((threads + 255) / 256)), block(256);
  TimedLaunch tl("sparsify24", stream);
  if (raw)
    hipLaunchKernelGGL(sparsify24_kernel<true>, grid, block, 0, stream, h, M, N, chunks, vals, meta, ldv, ldm);
  else
    hipLaunchKernelGGL(sparsify24_kernel<false>, grid, block, 0, stream, h, M, N, chunks, vals, meta, ldv, ldm);
  return hipGetLastError();
}

}  // namespace elas
