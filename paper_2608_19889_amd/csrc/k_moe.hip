// Mixture-of-experts routing around the grouped expert GEMMs.
//
// The MoE built-in's softmax top-k router (Built-In Libraries, "Activations
// and specialized modules"), the "stacked experts" form that replaces a loop
// over experts (Compiler, Phase 2 graph rewriting): every token's k choices
// become rows of one grouped GEMM, ordered by expert and, within an expert,
// by (token, choice), so the result does not depend on scheduling.
//   route:   probabilities = softmax over the experts of the router logits;
//            the top_k by probability (ties to the lowest expert index) with
//            their probabilities as weights (divided by their sum when
//            normalized)
//   plan:    per-expert row counts, row and 256-row tile offsets, and for each
//            grouped row its token (the GEMM's gather) and for each choice its
//            grouped row
//   combine: x[t] += sum over the token's choices j (in order) of
//            w[t][j] * y[grouped row of (t, j)]
#include "common.h"
#include "kernels.h"

namespace axon {

constexpr int MOE_MAX_E = 256, MOE_MAX_K = 8;

// one wavefront per token; lane l holds experts l, l + 64, l + 128, l + 192
__global__ void __launch_bounds__(256) moe_route_kernel(const float* __restrict__ logits, int ldl, int T, int E,
                                                        int k, int norm, int32_t* __restrict__ topi,
                                                        float* __restrict__ topw) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // whole wavefronts; no barrier follows
  float p[MOE_MAX_E / 64];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < MOE_MAX_E / 64; ++j) {
    const int e = lane + 64 * j;
    p[j] = e < E ? logits[(int64_t)t * ldl + e] : -INFINITY;
    mx = fmaxf(mx, p[j]);
  }
  mx = wave_max(mx);
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < MOE_MAX_E / 64; ++j) {
    p[j] = lane + 64 * j < E ? __expf(p[j] - mx) : 0.f;
    sum += p[j];
  }
  sum = wave_sum(sum);
  const float inv = 1.f / sum;
#pragma unroll
  for (int j = 0; j < MOE_MAX_E / 64; ++j) p[j] = lane + 64 * j < E ? p[j] * inv : -1.f;  // -1: never chosen
  float wsel[MOE_MAX_K];
  int isel[MOE_MAX_K];
  float wsum = 0.f;
  for (int c = 0; c < k; ++c) {
    // the largest remaining probability, lowest expert index on ties
    float bv = -2.f;
    int bi = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < MOE_MAX_E / 64; ++j)
      if (p[j] > bv) { bv = p[j]; bi = lane + 64 * j; }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = __shfl_xor(bv, m, 64);
      const int oi = __shfl_xor(bi, m, 64);
      if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
    }
    wsel[c] = bv;
    isel[c] = bi;
    wsum += bv;
#pragma unroll
    for (int j = 0; j < MOE_MAX_E / 64; ++j)
      if (lane + 64 * j == bi) p[j] = -1.f;
  }
  if (lane == 0) {
    const float sc = norm ? 1.f / wsum : 1.f;
    for (int c = 0; c < k; ++c) {
      topi[(int64_t)t * k + c] = isel[c];
      topw[(int64_t)t * k + c] = wsel[c] * sc;
    }
  }
}

// rows of expert blockIdx.x among the n choices
__global__ void __launch_bounds__(256) moe_count_kernel(const int32_t* __restrict__ topi, int n,
                                                        int32_t* __restrict__ cnt) {
  __shared__ int part[4];
  const int e = blockIdx.x;
  int c = 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) c += topi[i] == e;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) c += __shfl_xor(c, m, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) cnt[e] = part[0] + part[1] + part[2] + part[3];
}

// off[e] = rows before expert e, toff[e] = 256-row tiles before expert e (E + 1 entries each)
__global__ void moe_scan_kernel(const int32_t* __restrict__ cnt, int E, int32_t* __restrict__ off,
                                int32_t* __restrict__ toff) {
  if (threadIdx.x != 0) return;
  int r = 0, tl = 0;
  for (int e = 0; e < E; ++e) {
    off[e] = r;
    toff[e] = tl;
    r += cnt[e];
    tl += (cnt[e] + 255) / 256;
  }
  off[E] = r;
  toff[E] = tl;
}

// Expert blockIdx.x's rows in choice order: the i-th choice (i = t*k + j)
// with topi[i] == e becomes grouped row off[e] + (number of earlier such
// choices); xrow[row] = its token, inv[i] = row.
__global__ void __launch_bounds__(256) moe_scatter_kernel(const int32_t* __restrict__ topi, int n, int k,
                                                          const int32_t* __restrict__ off,
                                                          int32_t* __restrict__ xrow, int32_t* __restrict__ inv) {
  __shared__ int wcount[4];
  const int e = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int base = off[e];
  for (int i0 = 0; i0 < n; i0 += 256) {
    const int i = i0 + threadIdx.x;
    const bool hit = i < n && topi[i] == e;
    const uint64_t bal = __ballot(hit);
    if (lane == 0) wcount[wave] = __popcll(bal);
    __syncthreads();
    int before = 0;
    for (int w = 0; w < wave; ++w) before += wcount[w];
    const int total = wcount[0] + wcount[1] + wcount[2] + wcount[3];
    if (hit) {
      const int row = base + before + __popcll(bal & ((1ull << lane) - 1));
      xrow[row] = i / k;
      inv[i] = row;
    }
    base += total;
    __syncthreads();  // wcount is rewritten by the next chunk
  }
}

// x[t][:] += sum_j w[t][j] * y[inv[t*k + j]][:], 4 features per thread and
// 1024 per workgroup.  With xg: also xg[t] = bf16(x[t] * g) and the sum of
// squares of the workgroup's 1024 new x values in ss_out[blockIdx.x * T + t]
// (the next layer's normalization, applied by the projection that reads xg).
__global__ void __launch_bounds__(256) moe_combine_kernel(float* __restrict__ x, const float* __restrict__ y,
                                                          const int32_t* __restrict__ inv,
                                                          const float* __restrict__ w, int D, int k,
                                                          const bf16* __restrict__ g, bf16* __restrict__ xg,
                                                          float* __restrict__ ss_out) {
  __shared__ float red[16];
  const int t = blockIdx.y;
  const int n = (blockIdx.x * 256 + threadIdx.x) * 4;
  float sq = 0.f;
  if (n < D) {
    f32x4 acc = *(const f32x4*)(x + (int64_t)t * D + n);
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const float wj = w[(int64_t)t * k + j];
      const f32x4 v = *(const f32x4*)(y + (int64_t)inv[(int64_t)t * k + j] * D + n);
      s[0] += wj * v[0];
      s[1] += wj * v[1];
      s[2] += wj * v[2];
      s[3] += wj * v[3];
    }
    acc += s;
    *(f32x4*)(x + (int64_t)t * D + n) = acc;
    if (xg) {
      bf16x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        o[j] = (bf16)(acc[j] * (float)g[n + j]);
        sq += acc[j] * acc[j];
      }
      *(bf16x4*)(xg + (int64_t)t * D + n) = o;
    }
  }
  if (xg) {  // grid-uniform: every thread of the workgroup reaches the barrier
    sq = block_sum(sq, red);
    if (threadIdx.x == 0) ss_out[(int64_t)blockIdx.x * gridDim.y + t] = sq;
  }
}

// out[row] = h[xrow[row]] (bf16 rows of D, 8 elements per thread)
__global__ void __launch_bounds__(256) moe_gather_kernel(const bf16* __restrict__ h, const int32_t* __restrict__ xrow,
                                                         int D, bf16* __restrict__ out) {
  const int row = blockIdx.y;
  const int i = (blockIdx.x * 256 + threadIdx.x) * 8;
  if (i >= D) return;
  *(bf16x8*)(out + (int64_t)row * D + i) = *(const bf16x8*)(h + (int64_t)xrow[row] * D + i);
}

void launch_moe_gather(const bf16* h, const int32_t* xrow, int rows, int D, bf16* out, hipStream_t s) {
  if (rows <= 0) return;
  moe_gather_kernel<<<dim3((D / 8 + 255) / 256, rows), 256, 0, s>>>(h, xrow, D, out);
}

void launch_moe_route(const float* logits, int ldl, int T, int E, int k, int norm, int32_t* topi, float* topw,
                      hipStream_t s) {
  if (T <= 0) return;
  moe_route_kernel<<<(T + 3) / 4, 256, 0, s>>>(logits, ldl, T, E, k, norm, topi, topw);
}

void launch_moe_plan(const int32_t* topi, int T, int E, int k, int32_t* cnt, int32_t* off, int32_t* toff,
                     int32_t* xrow, int32_t* inv, hipStream_t s) {
  const int n = T * k;
  moe_count_kernel<<<E, 256, 0, s>>>(topi, n, cnt);
  moe_scan_kernel<<<1, 64, 0, s>>>(cnt, E, off, toff);
  moe_scatter_kernel<<<E, 256, 0, s>>>(topi, n, k, off, xrow, inv);
}

void launch_moe_combine(float* x, const float* y, const int32_t* inv, const float* w, int T, int D, int k,
                        hipStream_t s, const bf16* g, bf16* xg, float* ss_out) {
  if (T <= 0) return;
  moe_combine_kernel<<<dim3(moe_combine_blocks(D), T), 256, 0, s>>>(x, y, inv, w, D, k, g, xg, ss_out);
}

}  // namespace axon
