// Weight layout conversion run once at model load: row-major bf16 W [N][K]
// into the fragment-tiled storage every bf16 projection kernel reads
// (wt_chunk in common.h).  Reads are coalesced along k; the padding rows of
// the last 16-row block are written as zeros.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace axon {

__global__ void __launch_bounds__(256) tile_weight_kernel(const bf16* __restrict__ src, bf16* __restrict__ dst,
                                                          int64_t N, int K) {
  const int cpr = K / 8;
  const int64_t total = (N + 15) / 16 * 16 * cpr;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += (int64_t)gridDim.x * 256) {
    const int64_t n = q / cpr;
    const int c = (int)(q % cpr);
    bf16x8 v = {};
    if (n < N) v = *(const bf16x8*)(src + n * K + (int64_t)c * 8);
    *(bf16x8*)(dst + wt_chunk(n, c, K)) = v;
  }
}

// dst[r][k0 .. k0+7] = src[k0 .. k0+7][perm[r]]: consecutive threads take
// consecutive rows r, so each of the 8 source reads is coalesced along n
__global__ void __launch_bounds__(256) transpose_rows_kernel(const bf16* __restrict__ src, bf16* __restrict__ dst,
                                                             int K, int N, const int32_t* __restrict__ perm) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  const int k0 = blockIdx.y * 8;
  if (r >= N) return;
  const int c = perm ? perm[r] : r;
  bf16x8 v;
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] = src[(int64_t)(k0 + j) * N + c];
  *(bf16x8*)(dst + (int64_t)r * K + k0) = v;
}

void launch_transpose_rows(const bf16* src, bf16* dst, int K, int N, const int32_t* perm, hipStream_t s) {
  if (K <= 0 || N <= 0) return;
  transpose_rows_kernel<<<dim3((N + 255) / 256, K / 8), 256, 0, s>>>(src, dst, K, N, perm);
}

void launch_tile_weight(const bf16* src, bf16* dst, int64_t N, int K, hipStream_t s) {
  const int64_t total = (N + 15) / 16 * 16 * (K / 8);
  const int64_t grid = std::min<int64_t>((total + 255) / 256, 16384);
  if (grid > 0) tile_weight_kernel<<<(unsigned)grid, 256, 0, s>>>(src, dst, N, K);
}

}  // namespace axon
