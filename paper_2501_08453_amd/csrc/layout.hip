// Transposed token tiles (layout described in common.hpp): a memory-bound
// reformatting pass that lets the attention kernels fetch every operand whose
// contraction runs over tokens (V^T in the forward; Q^T, dO^T and K^T in the
// backward) with plain 16-byte LDS reads instead of transposing reads.
#include "common.hpp"

namespace vcja {
namespace {

template <int D>
__global__ __launch_bounds__(256) void token_tiles_kernel(const __bf16* __restrict__ x, __bf16* __restrict__ xt,
                                                          int H, int N, int ntile) {
  constexpr int CPR = D / 8;       // 16-byte chunks per token row
  constexpr int RS = D + 8;        // LDS row stride (elements)
  constexpr int OCH = kTileRow / 8;  // 16-byte chunks per output row (9)
  __shared__ __attribute__((aligned(16))) __bf16 buf[kTileTok * RS];
  const int tile = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const size_t tok = (size_t)H * D;
  const __bf16* src = x + (size_t)b * N * tok + (size_t)h * D;
  for (int c = threadIdx.x; c < kTileTok * CPR; c += 256) {
    const int t = c / CPR, col = (c % CPR) * 8;
    const int n = tile * kTileTok + t;
    bf16x8 v = zero_bf16x8();
    if (n < N) v = *(const bf16x8*)(src + (size_t)n * tok + col);
    *(bf16x8*)&buf[t * RS + col] = v;
  }
  __syncthreads();
  __bf16* dst = xt + (((size_t)b * H + h) * ntile + tile) * tile_elems(D);
  for (int c = threadIdx.x; c < D * OCH; c += 256) {
    const int d = c / OCH, pc = c % OCH;
    bf16x8 v = zero_bf16x8();
    if (pc < kTileTok / 8) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = buf[tok_pos(pc * 8 + i) * RS + d];  // tok_pos is an involution
    }
    *(bf16x8*)(dst + (size_t)d * kTileRow + pc * 8) = v;
  }
}

}  // namespace

hipError_t launch_token_tiles(const __bf16* x, __bf16* xt, int B, int H, int N, int head_dim, hipStream_t s) {
  const int ntile = (N + kTileTok - 1) / kTileTok;
  dim3 grid(ntile, H, B);
  if (head_dim == 128)
    hipLaunchKernelGGL(token_tiles_kernel<128>, grid, dim3(256), 0, s, x, xt, H, N, ntile);
  else
    hipLaunchKernelGGL(token_tiles_kernel<64>, grid, dim3(256), 0, s, x, xt, H, N, ntile);
  return hipGetLastError();
}

}  // namespace vcja
