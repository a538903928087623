// Row kernels of the GPT-2 family (the complete GPT-2 definition of the
// Technical Supplement): token + learned-position embedding with the first
// LayerNorm, and LayerNorm with gain and bias.  One workgroup of 256 threads
// per row; a thread keeps its (up to 8) groups of 4 features in registers, so
// the mean, the variance around it and the output come from one read of the
// row.  HBM/latency bound.
#include "common.h"
#include "kernels.h"

namespace axon {

constexpr int LN_MAXV = 8;  // rows of up to 8 * 1024 features

// h = (v - mean) / sqrt(var + eps) * g + beta for the thread's feature
// groups; mean and the (biased) variance over the D features of the row
AXON_DEV void ln_store(const f32x4 (&v)[LN_MAXV], int D, float eps, const bf16* __restrict__ g,
                       const bf16* __restrict__ beta, bf16* __restrict__ hr, float* red) {
  const int t4 = threadIdx.x * 4;
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < LN_MAXV; ++j)
    if (t4 + j * 1024 < D) sum += (v[j][0] + v[j][1]) + (v[j][2] + v[j][3]);
  const float mean = block_sum(sum, red) / (float)D;
  float sq = 0.f;
#pragma unroll
  for (int j = 0; j < LN_MAXV; ++j)
    if (t4 + j * 1024 < D) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float d = v[j][c] - mean;
        sq += d * d;
      }
    }
  const float rstd = rsqrtf(block_sum(sq, red) / (float)D + eps);
#pragma unroll
  for (int j = 0; j < LN_MAXV; ++j) {
    const int i = t4 + j * 1024;
    if (i < D) {
      const bf16x4 gv = *(const bf16x4*)(g + i), bv = *(const bf16x4*)(beta + i);
      bf16x4 o;
#pragma unroll
      for (int c = 0; c < 4; ++c) o[c] = (bf16)((v[j][c] - mean) * rstd * (float)gv[c] + (float)bv[c]);
      *(bf16x4*)(hr + i) = o;
    }
  }
}

__global__ void __launch_bounds__(256) embed_pos_ln_kernel(const int32_t* __restrict__ tok,
                                                           const bf16* __restrict__ wte,
                                                           const bf16* __restrict__ wpe,
                                                           const bf16* __restrict__ g, const bf16* __restrict__ beta,
                                                           float* __restrict__ x, bf16* __restrict__ h, int D, int V,
                                                           int P, float eps, const int32_t* __restrict__ cu, int nseq,
                                                           const int32_t* __restrict__ ent_base,
                                                           const int32_t* __restrict__ len) {
  __shared__ float red[16];
  const int t = blockIdx.x;
  int pos;
  if (len) {
    pos = len[t];
  } else {
    const int e = seq_of_token(cu, nseq, t);
    pos = (ent_base ? ent_base[e] : 0) + t - cu[e];
  }
  pos = min(max(pos, 0), P - 1);           // validated on the host; never read out of the table
  const int id = min(max(tok[t], 0), V - 1);  // ids outside [0, V) are clamped, never dereferenced
  f32x4 v[LN_MAXV];
#pragma unroll
  for (int j = 0; j < LN_MAXV; ++j) {
    const int i = threadIdx.x * 4 + j * 1024;
    if (i < D) {
      const bf16x4 a = *(const bf16x4*)(wte + wt_chunk(id, i >> 3, D) + (i & 7));  // fragment-tiled table
      const bf16x4 b = *(const bf16x4*)(wpe + (int64_t)pos * D + i);
#pragma unroll
      for (int c = 0; c < 4; ++c) v[j][c] = (float)a[c] + (float)b[c];
      *(f32x4*)(x + (int64_t)t * D + i) = v[j];
    }
  }
  ln_store(v, D, eps, g, beta, h + (int64_t)t * D, red);
}

__global__ void __launch_bounds__(256) layernorm_kernel(const float* __restrict__ x, const bf16* __restrict__ g,
                                                        const bf16* __restrict__ beta, bf16* __restrict__ h, int D,
                                                        float eps, const int32_t* __restrict__ cu_last) {
  __shared__ float red[16];
  const int i_out = blockIdx.x;
  const int r = cu_last ? cu_last[i_out + 1] - 1 : i_out;
  f32x4 v[LN_MAXV];
#pragma unroll
  for (int j = 0; j < LN_MAXV; ++j) {
    const int i = threadIdx.x * 4 + j * 1024;
    if (i < D) v[j] = *(const f32x4*)(x + (int64_t)r * D + i);
  }
  ln_store(v, D, eps, g, beta, h + (int64_t)i_out * D, red);
}

void launch_embed_pos_ln(const int32_t* tok, const bf16* wte, const bf16* wpe, const bf16* g, const bf16* beta,
                         float* x, bf16* h, int T, int D, int V, int P, float eps, const int32_t* cu, int nseq,
                         const int32_t* ent_base, const int32_t* len, hipStream_t s) {
  if (T <= 0) return;
  embed_pos_ln_kernel<<<T, 256, 0, s>>>(tok, wte, wpe, g, beta, x, h, D, V, P, eps, cu, nseq, ent_base, len);
}

void launch_layernorm(const float* x, const bf16* g, const bf16* beta, bf16* h, int rows, int D, float eps,
                      const int32_t* cu_last, hipStream_t s) {
  if (rows <= 0) return;
  layernorm_kernel<<<rows, 256, 0, s>>>(x, g, beta, h, D, eps, cu_last);
}

}  // namespace axon
