// Row kernels: embedding gather + RMSNorm, residual reduction + RMSNorm,
// greedy argmax, slot-length bookkeeping.  All are HBM/latency bound; rows are
// read with 16-byte vector accesses, one workgroup per row.
#include "common.h"
#include "kernels.h"

namespace axon {

// 4 consecutive elements of a T row as floats
AXON_DEV f32x4 load4(const float* p) { return *(const f32x4*)p; }
AXON_DEV f32x4 load4(const bf16* p) {
  bf16x4 v = *(const bf16x4*)p;
  return f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}
AXON_DEV void store4(float* p, f32x4 v) { *(f32x4*)p = v; }
AXON_DEV void store4(bf16* p, f32x4 v) {
  *(bf16x4*)p = bf16x4{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
}

// element i of embedding row id: bf16 tables are fragment-tiled (they double
// as the tied output head), float tables are row-major
AXON_DEV const float* emb_at(const float* e, int id, int i, int D) { return e + (int64_t)id * D + i; }
AXON_DEV const bf16* emb_at(const bf16* e, int id, int i, int D) { return e + wt_chunk(id, i >> 3, D) + (i & 7); }

// x[r,:] = E[tok[r],:] (as float); h[r,:] = x * rsqrt(mean(x^2) + eps) * g
template <typename T>
__global__ void __launch_bounds__(256) embed_rmsnorm_kernel(const int32_t* __restrict__ tok,
                                                            const T* __restrict__ emb,
                                                            const T* __restrict__ g,
                                                            float* __restrict__ x, T* __restrict__ h,
                                                            int D, int V, float eps, int h_pair) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  const int id = min(max(tok[r], 0), V - 1);  // ids outside [0, V) are clamped, never dereferenced
  float* xr = x + (int64_t)r * D;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < D; i += blockDim.x * 4) {
    f32x4 v = load4(emb_at(emb, id, i, D));
    store4(xr + i, v);
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  ss = block_sum(ss, red);
  const float inv = rsqrtf(ss / (float)D + eps);
  for (int i = threadIdx.x * 4; i < D; i += blockDim.x * 4) {
    f32x4 v = load4(emb_at(emb, id, i, D)), gv = load4(g + i);
    store4(h + (h_pair ? xp_off(r, i, D) : (int64_t)r * D + i),
           f32x4{v[0] * inv * gv[0], v[1] * inv * gv[1], v[2] * inv * gv[2], v[3] * inv * gv[3]});
  }
}

// Optionally x[r,:] += sum_s parts[s][r,:] (split-K partial products of the
// projection that feeds the residual), then h[i,:] = rmsnorm(x[r,:]) * g with
// r = i, or r = cu[i+1]-1 (last position of sequence i) when ``cu_last`` is set;
// h rows in the row-pair layout when h_pair is set (both kernels).
template <typename T>
__global__ void __launch_bounds__(256) resid_rmsnorm_kernel(float* __restrict__ x,
                                                            const float* __restrict__ parts,
                                                            int nparts, int64_t part_stride,
                                                            const T* __restrict__ g, T* __restrict__ h,
                                                            int D, float eps,
                                                            const int32_t* __restrict__ cu_last, int h_pair) {
  __shared__ float red[16];
  const int i_out = blockIdx.x;
  const int r = cu_last ? cu_last[i_out + 1] - 1 : i_out;
  float* xr = x + (int64_t)r * D;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < D; i += blockDim.x * 4) {
    f32x4 v = load4(xr + i);
    if (nparts > 0) {
      for (int s = 0; s < nparts; ++s) {
        f32x4 p = load4(parts + s * part_stride + (int64_t)r * D + i);
        v[0] += p[0]; v[1] += p[1]; v[2] += p[2]; v[3] += p[3];
      }
      store4(xr + i, v);
    }
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  ss = block_sum(ss, red);
  const float inv = rsqrtf(ss / (float)D + eps);
  for (int i = threadIdx.x * 4; i < D; i += blockDim.x * 4) {
    f32x4 v = load4(xr + i), gv = load4(g + i);
    store4(h + (h_pair ? xp_off(i_out, i, D) : (int64_t)i_out * D + i),
           f32x4{v[0] * inv * gv[0], v[1] * inv * gv[1], v[2] * inv * gv[2], v[3] * inv * gv[3]});
  }
}

// next[r] = argmax_v logits[r, v] (lowest index among equal maxima); when
// ``len`` is set, len[r] += 1 (the decode step has appended one position).
// The row read is cu_last[i+1]-1 when ``cu_last`` is set (last position of
// sequence i in a packed all-positions logits matrix), else i.
__global__ void __launch_bounds__(1024) argmax_kernel(const float* __restrict__ logits, int V,
                                                      int32_t* __restrict__ next,
                                                      int32_t* __restrict__ len,
                                                      const int32_t* __restrict__ cu_last) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const int i_out = blockIdx.x;
  const int r = cu_last ? cu_last[i_out + 1] - 1 : i_out;
  const float* row = logits + (int64_t)r * V;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < V; i += blockDim.x) {
    float v = row[i];
    if (v > best) { best = v; bi = i; }  // ascending scan: first maximum per thread
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    float ov = __shfl_xor(best, m, 64);
    int oi = __shfl_xor(bi, m, 64);
    if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) { sv[w] = best; si[w] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < (int)(blockDim.x >> 6); ++k)
      if (sv[k] > best || (sv[k] == best && si[k] < bi)) { best = sv[k]; bi = si[k]; }
    next[i_out] = bi == 0x7fffffff ? 0 : bi;
    if (len) len[i_out] += 1;
  }
}

__global__ void set_lengths_kernel(const int32_t* __restrict__ cu, int32_t* __restrict__ len, int n) {
  int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < n) len[b] = cu[b + 1] - cu[b];
}

__global__ void set_step_lengths_kernel(const int32_t* __restrict__ cu, const int32_t* __restrict__ ent_slot,
                                        const int32_t* __restrict__ ent_base, int32_t* __restrict__ len, int n) {
  int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) len[ent_slot[e]] = ent_base[e] + cu[e + 1] - cu[e];
}

// ---------------------------------------------------------------- launchers

template <typename T>
void launch_embed_rmsnorm(const int32_t* tok, const T* emb, const T* g, float* x, T* h, int rows, int D, int V,
                          float eps, hipStream_t s, bool h_pair) {
  if (rows <= 0) return;
  embed_rmsnorm_kernel<T><<<rows, 256, 0, s>>>(tok, emb, g, x, h, D, V, eps, h_pair ? 1 : 0);
}

template <typename T>
void launch_resid_rmsnorm(float* x, const float* parts, int nparts, int64_t part_stride, const T* g, T* h,
                          int rows, int D, float eps, const int32_t* cu_last, hipStream_t s, bool h_pair) {
  if (rows <= 0) return;
  resid_rmsnorm_kernel<T><<<rows, 256, 0, s>>>(x, parts, nparts, part_stride, g, h, D, eps, cu_last, h_pair ? 1 : 0);
}

void launch_argmax(const float* logits, int rows, int V, int32_t* next, int32_t* len, hipStream_t s) {
  if (rows <= 0) return;
  argmax_kernel<<<rows, 1024, 0, s>>>(logits, V, next, len, nullptr);
}

void launch_argmax_rows(const float* logits, int nseq, int V, int32_t* next, const int32_t* cu, hipStream_t s) {
  if (nseq <= 0) return;
  argmax_kernel<<<nseq, 1024, 0, s>>>(logits, V, next, nullptr, cu);
}

void launch_set_lengths(const int32_t* cu, int32_t* len, int n, hipStream_t s) {
  if (n <= 0) return;
  set_lengths_kernel<<<(n + 255) / 256, 256, 0, s>>>(cu, len, n);
}

void launch_set_step_lengths(const int32_t* cu, const int32_t* ent_slot, const int32_t* ent_base, int32_t* len,
                             int n, hipStream_t s) {
  if (n <= 0) return;
  set_step_lengths_kernel<<<(n + 255) / 256, 256, 0, s>>>(cu, ent_slot, ent_base, len, n);
}

template void launch_embed_rmsnorm<float>(const int32_t*, const float*, const float*, float*, float*, int, int,
                                          int, float, hipStream_t, bool);
template void launch_embed_rmsnorm<bf16>(const int32_t*, const bf16*, const bf16*, float*, bf16*, int, int, int,
                                         float, hipStream_t, bool);
template void launch_resid_rmsnorm<float>(float*, const float*, int, int64_t, const float*, float*, int, int,
                                          float, const int32_t*, hipStream_t, bool);
template void launch_resid_rmsnorm<bf16>(float*, const float*, int, int64_t, const bf16*, bf16*, int, int,
                                         float, const int32_t*, hipStream_t, bool);

}  // namespace axon
