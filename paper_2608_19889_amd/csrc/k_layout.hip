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

void launch_tile_weight(const bf16* src, bf16* dst, int64_t N, int K, hipStream_t s) {
  const int64_t total = (N + 15) / 16 * 16 * (K / 8);
  const int64_t grid = std::min<int64_t>((total + 255) / 256, 16384);
  if (grid > 0) tile_weight_kernel<<<(unsigned)grid, 256, 0, s>>>(src, dst, N, K);
}

}  // namespace axon
