// Backward pass of the Llama-family decoder (training): the loss, the
// reverse of each forward step that is not a projection, and the layout
// helpers that let the projection gradients run on the prefill GEMM.
//
// Every projection Y = X W^T (X [T][K], W [N][K]) has two gradients, both run
// by gemm_bf16 (out[r][c] = sum_k A[r][k] B[c][k], B fragment-tiled):
//   dX = dY W       : A = dY [T][N],   B = W^T tiled [K][N]  (contraction N)
//   dW = dY^T X     : A = dY^T [N][Tp], B = X^T tiled [K][Tp] (contraction Tp,
//                     the token count padded to 32 with zero columns)
// so the weights get a transposed tiled copy once, and the activations and
// their gradients are transposed per use (transpose_pad_kernel).
//
// Attention backward recomputes the probabilities from the forward pass's
// per-(query, head) log2-sum-exp: P = 2^(s sc - lse) with sc = log2(e) /
// sqrt(hd); dP = dO V^T; dS = P (dP - D) with D = rowsum(dO O); dQ = dS K /
// sqrt(hd); dK = dS^T Q / sqrt(hd); dV = P^T dO, all on the matrix cores.
// One wavefront per 32-query block and head accumulates dQ over the keys; one
// per 32-key block and query head accumulates that head's share of dK and dV
// over the later queries, and the shares of a group's heads are summed in
// order.  No atomics, so every gradient but the embedding's is
// deterministic.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace axon {

constexpr float LOG2E = 1.4426950408889634f;

AXON_DEV float block_max(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float m = -INFINITY;
  for (int i = 0; i < nw; ++i) m = fmaxf(m, red[i]);
  return m;
}

// ---------------------------------------------------------------- the loss

// Row t of logits [T][ldl]: lse = log sum_v exp(logit_v) over v < V; a target
// in [0, V) counts (rowloss = lse - logit_target, valid = 1), any other value
// does not (0, 0).
__global__ void __launch_bounds__(256) ce_rows_kernel(const float* __restrict__ logits, int ldl, int V,
                                                      const int32_t* __restrict__ targets,
                                                      float* __restrict__ rowloss, float* __restrict__ valid,
                                                      float* __restrict__ lse_out) {
  __shared__ float red[16];
  const int t = blockIdx.x;
  const float* row = logits + (int64_t)t * ldl;
  float mx = -INFINITY;
  for (int v = threadIdx.x; v < V; v += 256) mx = fmaxf(mx, row[v]);
  mx = block_max(mx, red);
  float sum = 0.f;
  for (int v = threadIdx.x; v < V; v += 256) sum += __expf(row[v] - mx);
  sum = block_sum(sum, red);
  if (threadIdx.x == 0) {
    const float lse = mx + __logf(sum);
    const int tg = targets[t];
    const bool ok = tg >= 0 && tg < V;
    rowloss[t] = ok ? lse - row[tg] : 0.f;
    valid[t] = ok ? 1.f : 0.f;
    lse_out[t] = lse;
  }
}

// loss = sum(rowloss) / N over the N counted rows (0 when none); scal[0] = 1/N
// (0 when none).  One workgroup, fixed summation order.
__global__ void __launch_bounds__(256) ce_reduce_kernel(const float* __restrict__ rowloss,
                                                        const float* __restrict__ valid, int T,
                                                        float* __restrict__ loss, float* __restrict__ scal) {
  __shared__ float red[16];
  float s = 0.f, n = 0.f;
  for (int t = threadIdx.x; t < T; t += 256) {
    s += rowloss[t];
    n += valid[t];
  }
  s = block_sum(s, red);
  n = block_sum(n, red);
  if (threadIdx.x == 0) {
    loss[0] = n > 0.f ? s / n : 0.f;
    scal[0] = n > 0.f ? 1.f / n : 0.f;
  }
}

// dlogits[t][v] = (softmax_v - [v == target]) / N for counted rows, else 0;
// columns V .. ldl-1 are zero.  4 columns per thread (ldl % 4 == 0).
__global__ void __launch_bounds__(256) ce_grad_kernel(const float* __restrict__ logits, int ldl, int V,
                                                      const int32_t* __restrict__ targets,
                                                      const float* __restrict__ valid,
                                                      const float* __restrict__ lse, const float* __restrict__ scal,
                                                      bf16* __restrict__ dlog) {
  const int t = blockIdx.y;
  const int v0 = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (v0 >= ldl) return;
  const bool ok = valid[t] > 0.f;
  const float l = lse[t], inv = scal[0];
  const int tg = targets[t];
  bf16x4 o;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = v0 + j;
    float g = 0.f;
    if (ok && v < V) g = (__expf(logits[(int64_t)t * ldl + v] - l) - (v == tg ? 1.f : 0.f)) * inv;
    o[j] = (bf16)g;
  }
  *(bf16x4*)(dlog + (int64_t)t * ldl + v0) = o;
}

// ---------------------------------------------------------------- layouts

// Element offset of (row c, column col) of a [C][dld] matrix stored in the
// A-operand fragments of the attention backward's Q^T / dO^T / K^T products
// (C and dld multiples of 32): fragment (c / 32, col / 32, kk) is 1 KB of 64
// lanes x 8 values, lane hl * 32 + c % 32 holding the block's columns kk * 16 +
// kap(hl, j), j = 0..7, kap(hl, j) = (j / 4) * 8 + 4 hl + j % 4 (the order of
// the dS / P operand it multiplies), so a wavefront's fragment is one
// contiguous read.
AXON_DEV int64_t frag_off(int64_t c, int64_t col, int64_t dld) {
  const int q = (int)(col & 31), kk = q >> 4, r16 = q & 15;
  const int hl = (r16 >> 2) & 1, j = (r16 >> 3) * 4 + (r16 & 3);
  return ((((c >> 5) * (dld >> 5) + (col >> 5)) * 2 + kk) * 64 + hl * 32 + (c & 31)) * 8 + j;
}

// dst[c][col(t)] = src[t][c] through a 64 x 64 LDS tile, both sides
// coalesced: rows t < T are read (rows T .. Tmax-1 give zeros), col(t) = t,
// or with cu: e * SP + (t - cu[e]) for t's sequence e (t < T only).  C % 4
// == 0, ld % 4 == 0.  frag: dst in the fragment order of frag_off.
__global__ void __launch_bounds__(256) transpose_tile_kernel(const bf16* __restrict__ src, int64_t ld, int T, int Tmax,
                                                             int C, bf16* __restrict__ dst, int64_t dld,
                                                             const int32_t* __restrict__ cu, int nseq, int SP,
                                                             bool frag = false) {
  __shared__ bf16 tile[64][66];
  const int t0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int t = t0 + ty + 16 * r, c = c0 + tx * 4;
    bf16x4 v = {(bf16)0.f, (bf16)0.f, (bf16)0.f, (bf16)0.f};
    if (t < T && c < C) v = *(const bf16x4*)(src + (int64_t)t * ld + c);
#pragma unroll
    for (int j = 0; j < 4; ++j) tile[ty + 16 * r][tx * 4 + j] = v[j];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int c = c0 + ty + 16 * r;
    if (c >= C) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = t0 + tx * 4 + j;
      if (t >= (cu ? T : Tmax)) continue;
      int64_t col = t;
      if (cu) {
        const int e = seq_of_token(cu, nseq, t);
        col = (int64_t)e * SP + (t - cu[e]);
      }
      dst[frag ? frag_off(c, col, dld) : (int64_t)c * dld + col] = tile[tx * 4 + j][ty + 16 * r];
    }
  }
}

// dst[k][n] = W[n][k] from the fragment-tiled W [N][K]; dst rows are Np
// apart (the caller zeroes columns N .. Np-1)
__global__ void __launch_bounds__(256) untile_transpose_kernel(const bf16* __restrict__ W, int64_t N, int K,
                                                               bf16* __restrict__ dst, int64_t Np) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (n, k-chunk)
  const int kc = K / 8;
  if (q >= N * kc) return;
  const int64_t n = q / kc;
  const int c = (int)(q % kc);
  const bf16x8 v = *(const bf16x8*)(W + wt_chunk(n, c, K));
#pragma unroll
  for (int j = 0; j < 8; ++j) dst[(int64_t)(c * 8 + j) * Np + n] = v[j];
}

__global__ void __launch_bounds__(256) to_bf16_kernel(const float* __restrict__ src, bf16* __restrict__ dst,
                                                      int64_t n4) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  const f32x4 v = *(const f32x4*)(src + i * 4);
  *(bf16x4*)(dst + i * 4) = bf16x4{(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
}

// ---------------------------------------------------------------- norms, MLP

// RMSNorm y = x r g, r = rsqrt(mean(x^2) + eps): dx (= or +=) r g dy - x r^3
// mean(g dy x); dgrow = dy x r (summed over rows by the column sum)
__global__ void __launch_bounds__(256) rmsnorm_bwd_kernel(const float* __restrict__ x, const bf16* __restrict__ g,
                                                          const float* __restrict__ dy, int ldy, int D, float eps,
                                                          float* __restrict__ dx, int accumulate,
                                                          float* __restrict__ dgrow) {
  __shared__ float red[16];
  const int t = blockIdx.x;
  const float* xr = x + (int64_t)t * D;
  const float* dyr = dy + (int64_t)t * ldy;
  float ss = 0.f, sgd = 0.f;
  for (int i = threadIdx.x; i < D; i += 256) {
    const float xv = xr[i];
    ss += xv * xv;
    sgd += (float)g[i] * dyr[i] * xv;
  }
  ss = block_sum(ss, red);
  sgd = block_sum(sgd, red);
  const float r = rsqrtf(ss / (float)D + eps);
  const float c = r * r * r * sgd / (float)D;
  float* dxr = dx + (int64_t)t * D;
  for (int i = threadIdx.x; i < D; i += 256) {
    const float xv = xr[i], d = dyr[i];
    const float v = r * (float)g[i] * d - xv * c;
    dxr[i] = accumulate ? dxr[i] + v : v;
    dgrow[(int64_t)t * D + i] = d * xv * r;
  }
}

// gate/up pre-activations gu [T][2I] in the interleaved row order (16 gate
// rows, then the 16 matching up rows); da [T][I]: dgu = (da u silu'(g),
// da silu(g)) in the same order, silu'(g) = s (1 + g (1 - s)), s = sigmoid(g)
__global__ void __launch_bounds__(256) swiglu_bwd_kernel(const float* __restrict__ gu, const float* __restrict__ da,
                                                         bf16* __restrict__ dgu, int T, int I) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)T * I) return;
  const int t = (int)(idx / I), f = (int)(idx % I);
  const int64_t rg = (int64_t)t * 2 * I + (f / 16) * 32 + (f % 16);
  const float g = gu[rg], u = gu[rg + 16], d = da[idx];
  const float s = 1.f / (1.f + __expf(-g));
  dgu[rg] = (bf16)(d * u * s * (1.f + g * (1.f - s)));
  dgu[rg + 16] = (bf16)(d * g * s);
}

// column sums of src [T][C] (rows ld apart) in two deterministic passes:
// part[chunk][c] over rows chunk*rpc .., then dst[c] = sum over chunks
__global__ void __launch_bounds__(256) colsum_part_kernel(const float* __restrict__ src, int64_t ld, int T, int C,
                                                          int rpc, float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  const int t0 = blockIdx.y * rpc, t1 = min(T, t0 + rpc);
  float s = 0.f;
  for (int t = t0; t < t1; ++t) s += src[(int64_t)t * ld + c];
  part[(int64_t)blockIdx.y * C + c] = s;
}
__global__ void __launch_bounds__(256) colsum_final_kernel(const float* __restrict__ part, int nchunks, int C,
                                                           float* __restrict__ dst) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  float s = 0.f;
  for (int i = 0; i < nchunks; ++i) s += part[(int64_t)i * C + c];
  dst[c] = s;
}

// ---------------------------------------------------------------- attention

// D[t][h] = sum_d dO[t][h][d] O[t][h][d]; D and the forward's log2-sum-exp
// are also copied into the packed per-head rows lsep / dsump [H][W] (column
// e*SP + position), where the 4 consecutive queries a lane of the dK / dV
// kernel needs are one 16-byte load
__global__ void __launch_bounds__(256) attn_bwd_d_kernel(const bf16* __restrict__ dob, const bf16* __restrict__ o,
                                                         int TH, int hd, float* __restrict__ dsum,
                                                         const float* __restrict__ lse, const int32_t* __restrict__ cu,
                                                         int nseq, int H, int SP, int64_t W,
                                                         float* __restrict__ lsep, float* __restrict__ dsump) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= TH) return;
  const bf16* a = dob + (int64_t)i * hd;
  const bf16* b = o + (int64_t)i * hd;
  float s = 0.f;
  for (int d = 0; d < hd; d += 8) {
    const bf16x8 x = *(const bf16x8*)(a + d), y = *(const bf16x8*)(b + d);
#pragma unroll
    for (int j = 0; j < 8; ++j) s += (float)x[j] * (float)y[j];
  }
  dsum[i] = s;
  const int t = i / H, h = i % H;
  const int e = seq_of_token(cu, nseq, t);
  const int64_t col = (int64_t)h * W + (int64_t)e * SP + (t - cu[e]);
  lsep[col] = lse[i];
  dsump[col] = s;
}

// ---- MFMA attention backward.  v_mfma_f32_32x32x16_bf16 with lane L, half
// hl = L / 32, column c = L % 32: A operand = row c, k = 8 hl .. 8 hl + 7;
// B operand = column c, the same k; accumulator element i = row (i/4)*8 +
// 4 hl + i%4, column c.  The accumulator of a 32 x 32 block therefore holds,
// per lane, 16 rows of one column: taken 8 at a time (k-steps kk = 0, 1) it
// is directly a B operand whose k slot (hl, j) stands for row kk*16 +
// kap(hl, j), kap(hl, j) = (j/4)*8 + 4 hl + j%4, and the A operand of that
// product reads its rows in the same order: two runs of 4 consecutive
// positions, which the transposed copies (positions contiguous) serve as two
// 8-byte reads.
//
// Packed copies, per sequence e at columns / rows e*SP + position (SP = the
// longest sequence rounded up to 32, plus 32 positions of finite padding, so
// a block's reads past its sequence end stay inside the sequence's range;
// W = the packed width), every one stored in MFMA fragment order so that a
// wavefront's operand fragment is one contiguous 1 KB read:
//   kr, vr  K and V rows (row_frag_off: fragment = 32 positions x 16 dims)
//   qt, dot, kt  Q^T, dO^T [H*hd][W], K^T [KV*hd][W] (frag_off)

// Element offset of dimension d of packed row col of kv head g in kr / vr:
// fragment (g, col / 32, d / 16) holds lane (d % 16) / 8 * 32 + col % 32,
// values d % 8 (the A / B operand lane order of a 32-row x 16-k fragment)
AXON_DEV int64_t row_frag_off(int64_t g, int64_t col, int d, int hd, int64_t W) {
  return (((g * (W >> 5) + (col >> 5)) * (hd >> 4) + (d >> 4)) * 64 + ((d & 15) >> 3) * 32 + (col & 31)) * 8 + (d & 7);
}

// the layer's K / V rows from the cache into kr / vr (row e*SP + position)
// and K^T into kt.  Workgroup = 16 positions p0 .. p0+15 of one sequence
// (p0 % 16 == 0, blockIdx.x counts the sequences' 16-position blocks in
// order) x one kv head: the cache's K block (positions x 8-dim chunks) and
// V^T block (dims x 16 positions) are staged in LDS, then every output leaves
// in 16-byte stores: 8 dims of one position (kr, vr) or 8 positions of one
// dim (kt, in the kap order of its fragment).  Positions past the sequence
// end are written as zeros, which is what the zero-filled padding holds.
template <int HD>
__global__ void __launch_bounds__(256) attn_bwd_pack_kernel(KVView kv, const int32_t* __restrict__ cu, int nseq,
                                                            int SP, int64_t W, bf16* __restrict__ kr,
                                                            bf16* __restrict__ vr, bf16* __restrict__ kt) {
  __shared__ bf16 ks[16][HD + 8];  // K rows (padded: the kt gather reads a column)
  __shared__ bf16 vs[HD][16 + 8];  // V^T rows
  const int h = blockIdx.y, tid = threadIdx.x;
  int e = 0, blk = blockIdx.x;
  for (; e < nseq - 1; ++e) {
    const int nb = (cu[e + 1] - cu[e] + 15) / 16;
    if (blk < nb) break;
    blk -= nb;
  }
  const int p0 = blk * 16, len = cu[e + 1] - cu[e];
  const bf16 zero = (bf16)0.f;
  // K: thread -> (position, 8-dim chunk); V^T: thread -> (dim, 8 positions)
  for (int i = tid; i < 16 * (HD / 8); i += 256) {
    const int pp = i / (HD / 8), d0 = (i % (HD / 8)) * 8, p = p0 + pp;
    bf16x8 v = {zero, zero, zero, zero, zero, zero, zero, zero};
    if (p < len) v = *(const bf16x8*)((const bf16*)kv.k + k_el(kv, e, h, p, d0));
    *(bf16x8*)&ks[pp][d0] = v;
  }
  for (int i = tid; i < HD * 2; i += 256) {
    const int d = i / 2, half = i % 2;
    // the block's V^T row of dim d holds positions p0 .. p0+15 contiguously
    const bf16x8 v = *(const bf16x8*)((const bf16*)kv.v + v_el(kv, e, h, min(p0, len - 1) & ~15, d) + half * 8);
#pragma unroll
    for (int j = 0; j < 8; ++j) vs[d][half * 8 + j] = p0 + half * 8 + j < len ? v[j] : zero;
  }
  __syncthreads();
  const int64_t col0 = (int64_t)e * SP + p0;
  for (int i = tid; i < 16 * (HD / 8); i += 256) {
    const int pp = i / (HD / 8), d0 = (i % (HD / 8)) * 8;
    bf16x8 vv;
#pragma unroll
    for (int j = 0; j < 8; ++j) vv[j] = vs[d0 + j][pp];
    *(bf16x8*)(kr + row_frag_off(h, col0 + pp, d0, HD, W)) = *(const bf16x8*)&ks[pp][d0];
    *(bf16x8*)(vr + row_frag_off(h, col0 + pp, d0, HD, W)) = vv;
  }
  // kt: dim d, half hl of the 16 positions (kap(hl, j) = (j/4)*8 + 4 hl + j%4)
  for (int i = tid; i < HD * 2; i += 256) {
    const int d = i / 2, hl = i % 2;
    bf16x8 v;
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = ks[(j / 4) * 8 + hl * 4 + j % 4][d];
    *(bf16x8*)(kt + frag_off((int64_t)h * HD + d, col0 + hl * 4, W)) = v;
  }
}

AXON_DEV int kap(int hl, int j) { return (j >> 2) * 8 + hl * 4 + (j & 3); }

// the 32-position block blockIdx.x of the sequences in order: (sequence, first position)
AXON_DEV void locate_block(const int32_t* __restrict__ cu, int nseq, int& e, int& p0) {
  int blk = blockIdx.x;
  for (e = 0; e < nseq - 1; ++e) {
    const int nb = (cu[e + 1] - cu[e] + 31) / 32;
    if (blk < nb) break;
    blk -= nb;
  }
  p0 = blk * 32;
}

// dQ of 32 queries (one head): over the key blocks up to the last query,
// S^T = K Q^T and dP^T = V dO^T (k = head dim), then dQ^T += K^T dS^T (k =
// the block's 32 keys).  One wavefront per workgroup; no LDS.
template <int HD>
__global__ void __launch_bounds__(64) attn_bwd_dq_kernel(const bf16* __restrict__ q, const bf16* __restrict__ dob,
                                                         const bf16* __restrict__ kr, const bf16* __restrict__ vr,
                                                         const bf16* __restrict__ kt, const float* __restrict__ lse,
                                                         const float* __restrict__ dsum,
                                                         const int32_t* __restrict__ cu, int nseq, int H, int KVh,
                                                         int SP, int64_t W, float* __restrict__ dq) {
  int e, q0;
  locate_block(cu, nseq, e, q0);
  const int h = blockIdx.y, kvh = h / (H / KVh);
  const int tok0 = cu[e], S = cu[e + 1] - tok0;
  const int lane = threadIdx.x, hl = lane >> 5, c = lane & 31;
  const int myq = q0 + c;
  const int64_t tq = tok0 + min(myq, S - 1);  // columns past the sequence read its last query (not stored)
  bf16x8 qf[HD / 16], df[HD / 16];
#pragma unroll
  for (int s = 0; s < HD / 16; ++s) {
    qf[s] = *(const bf16x8*)(q + (tq * H + h) * HD + s * 16 + hl * 8);
    df[s] = *(const bf16x8*)(dob + (tq * H + h) * HD + s * 16 + hl * 8);
  }
  const float sc = LOG2E / sqrtf((float)HD);
  const float l2 = lse[tq * H + h], Dq = dsum[tq * H + h];
  f32x16 acc[HD / 32];
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) acc[b] = f32x16{};
  const int kend = min(S, q0 + 32);
  for (int kb0 = 0; kb0 < kend; kb0 += 32) {
    f32x16 st = {}, dpt = {};
    const int64_t kfr = ((int64_t)kvh * (W >> 5) + (((int64_t)e * SP + kb0) >> 5)) * (HD / 16) * 512 + lane * 8;
#pragma unroll
    for (int s = 0; s < HD / 16; ++s) {
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(kr + kfr + s * 512), qf[s], st, 0, 0, 0);
      dpt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(vr + kfr + s * 512), df[s], dpt, 0, 0, 0);
    }
    // dS as a bf16 pair hi + lo: a row of dS sums to zero, so dQ = dS K
    // cancels, and rounding dS to one bf16 would leave an error of 2^-9 of
    // the row's absolute sum times the keys' common part
    bf16x8 dsh[2], dsl[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = kb0 + (i >> 2) * 8 + hl * 4 + (i & 3);
      const float p = (key <= myq && myq < S) ? exp2f(st[i] * sc - l2) : 0.f;
      const float ds = p * (dpt[i] - Dq);
      const bf16 hi = (bf16)ds;
      dsh[i >> 3][i & 7] = hi;
      dsl[i >> 3][i & 7] = (bf16)(ds - (float)hi);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int b = 0; b < HD / 32; ++b) {
        const bf16x8 a =
            *(const bf16x8*)(kt + frag_off((int64_t)kvh * HD + b * 32 + c, (int64_t)e * SP + kb0 + kk * 16, W) +
                             hl * 256);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, dsh[kk], acc[b], 0, 0, 0);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, dsl[kk], acc[b], 0, 0, 0);
      }
  }
  if (myq >= S) return;
  const float rs = 1.f / sqrtf((float)HD);
  float* out = dq + ((int64_t)(tok0 + myq) * H + h) * HD;
#pragma unroll
  for (int b = 0; b < HD / 32; ++b)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d = b * 32 + g * 8 + hl * 4;
      *(f32x4*)(out + d) = f32x4{acc[b][g * 4] * rs, acc[b][g * 4 + 1] * rs, acc[b][g * 4 + 2] * rs,
                                 acc[b][g * 4 + 3] * rs};
    }
}

// dK and dV of 32 keys from one query head h = blockIdx.y (kv head h / group):
// over the query blocks from the key block on, S = Q K^T and dP = dO V^T (k =
// head dim), then dV^T += dO^T P and dK^T += Q^T dS (k = the block's 32
// queries).  Writes the head's share into dk / dv [T][H][hd] (the heads of a
// group are summed by attn_bwd_group_sum_kernel; with one head per group they
// are the result).
template <int HD>
__global__ void __launch_bounds__(64) attn_bwd_dkv_kernel(const bf16* __restrict__ q, const bf16* __restrict__ dob,
                                                          const bf16* __restrict__ kr, const bf16* __restrict__ vr,
                                                          const bf16* __restrict__ qt, const bf16* __restrict__ dot,
                                                          const float* __restrict__ lsep,
                                                          const float* __restrict__ dsump,
                                                          const int32_t* __restrict__ cu, int nseq, int H, int KVh,
                                                          int SP, int64_t W, float* __restrict__ dk,
                                                          float* __restrict__ dv) {
  int e, kb0;
  locate_block(cu, nseq, e, kb0);
  const int h = blockIdx.y, kvh = h / (H / KVh);
  const int tok0 = cu[e], S = cu[e + 1] - tok0;
  const int lane = threadIdx.x, hl = lane >> 5, c = lane & 31;
  const int mykey = kb0 + c;
  bf16x8 kf[HD / 16], vf[HD / 16];
  // this lane's key mykey (padded rows past the sequence), fragments of 16 dims
  const int64_t kfr = ((int64_t)kvh * (W >> 5) + (((int64_t)e * SP + kb0) >> 5)) * (HD / 16) * 512 + lane * 8;
#pragma unroll
  for (int s = 0; s < HD / 16; ++s) {
    kf[s] = *(const bf16x8*)(kr + kfr + s * 512);
    vf[s] = *(const bf16x8*)(vr + kfr + s * 512);
  }
  const float sc = LOG2E / sqrtf((float)HD);
  f32x16 akk[HD / 32], avv[HD / 32];
#pragma unroll
  for (int b = 0; b < HD / 32; ++b) {
    akk[b] = f32x16{};
    avv[b] = f32x16{};
  }
  {
    for (int qb0 = kb0; qb0 < S; qb0 += 32) {
      const int64_t tq = tok0 + min(qb0 + c, S - 1);  // rows past the sequence read its last query
      f32x16 sq = {}, dpq = {};
#pragma unroll
      for (int s = 0; s < HD / 16; ++s) {
        sq = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(q + (tq * H + h) * HD + s * 16 + hl * 8), kf[s],
                                                     sq, 0, 0, 0);
        dpq = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(const bf16x8*)(dob + (tq * H + h) * HD + s * 16 + hl * 8),
                                                      vf[s], dpq, 0, 0, 0);
      }
      // the statistics of queries qb0 + g*8 + hl*4 .. +3 (packed rows; past
      // the sequence end they are whatever the padding holds, and unused)
      const int64_t srow = (int64_t)h * W + (int64_t)e * SP + qb0 + hl * 4;
      f32x4 lq[4], dq4[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        lq[g] = *(const f32x4*)(lsep + srow + g * 8);
        dq4[g] = *(const f32x4*)(dsump + srow + g * 8);
      }
      // P in bf16; dS as a bf16 pair hi + lo (dK = dS^T Q sums a row of dS,
      // which sums to zero, against the queries: see the dQ kernel)
      bf16x8 pb[2], dsh[2], dsl[2];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int qi = qb0 + (i >> 2) * 8 + hl * 4 + (i & 3);
        const bool ok = qi < S && mykey <= qi;
        const float p = ok ? exp2f(sq[i] * sc - lq[i >> 2][i & 3]) : 0.f;
        pb[i >> 3][i & 7] = (bf16)p;
        const float ds = ok ? p * (dpq[i] - dq4[i >> 2][i & 3]) : 0.f;
        const bf16 hi = (bf16)ds;
        dsh[i >> 3][i & 7] = hi;
        dsl[i >> 3][i & 7] = (bf16)(ds - (float)hi);
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int b = 0; b < HD / 32; ++b) {
          const int64_t off = frag_off((int64_t)h * HD + b * 32 + c, (int64_t)e * SP + qb0 + kk * 16, W) + hl * 256;
          const bf16x8 ao = *(const bf16x8*)(dot + off);
          const bf16x8 aq = *(const bf16x8*)(qt + off);
          avv[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ao, pb[kk], avv[b], 0, 0, 0);
          akk[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq, dsh[kk], akk[b], 0, 0, 0);
          akk[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq, dsl[kk], akk[b], 0, 0, 0);
        }
    }
  }
  if (mykey >= S) return;
  const float rs = 1.f / sqrtf((float)HD);
  const int64_t orow = ((int64_t)(tok0 + mykey) * H + h) * HD;
#pragma unroll
  for (int b = 0; b < HD / 32; ++b)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int d = b * 32 + g * 8 + hl * 4;
      *(f32x4*)(dk + orow + d) = f32x4{akk[b][g * 4] * rs, akk[b][g * 4 + 1] * rs, akk[b][g * 4 + 2] * rs,
                                       akk[b][g * 4 + 3] * rs};
      *(f32x4*)(dv + orow + d) = f32x4{avv[b][g * 4], avv[b][g * 4 + 1], avv[b][g * 4 + 2], avv[b][g * 4 + 3]};
    }
}

// dk[t][kvh] = sum over the group's heads (in order) of dkh[t][head], same for v
__global__ void __launch_bounds__(256) attn_bwd_group_sum_kernel(const float* __restrict__ dkh,
                                                                 const float* __restrict__ dvh, int64_t n, int group,
                                                                 int hd, float* __restrict__ dk,
                                                                 float* __restrict__ dv) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // over T * KV * hd
  if (i >= n) return;
  const int64_t row = i / hd, d = i % hd;  // row = t * KV + kvh
  const int64_t base = row * group * hd + d;
  float a = 0.f, b = 0.f;
  for (int g = 0; g < group; ++g) {
    a += dkh[base + (int64_t)g * hd];
    b += dvh[base + (int64_t)g * hd];
  }
  dk[i] = a;
  dv[i] = b;
}

// Gradients at the rotated q / k and at v back through RoPE (the transpose of
// a rotation rotates by the opposite angle) into the fused QKV layout: dqkv
// [T][nq] bf16 in the projection's row order (within a head, groups of 8 =
// 4 first halves and their partners), dqkv_f [T][nq] float in the original
// order (for the bias gradient; may be null).  One thread per (token, head,
// pair i < hd/2).
__global__ void __launch_bounds__(256) rope_bwd_kernel(const float* __restrict__ dq, const float* __restrict__ dk,
                                                       const float* __restrict__ dv, const float* __restrict__ cos_t,
                                                       const float* __restrict__ sin_t,
                                                       const int32_t* __restrict__ cu, int nseq, int T, int H,
                                                       int KVh, int hd, bf16* __restrict__ dqkv,
                                                       float* __restrict__ dqkv_f) {
  const int half = hd / 2, NH = H + 2 * KVh;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)T * NH * half) return;
  const int i = (int)(idx % half);
  const int hh = (int)((idx / half) % NH);
  const int t = (int)(idx / ((int64_t)half * NH));
  const float* src = hh < H ? dq + ((int64_t)t * H + hh) * hd
                            : (hh < H + KVh ? dk + ((int64_t)t * KVh + hh - H) * hd
                                            : dv + ((int64_t)t * KVh + hh - H - KVh) * hd);
  float y1 = src[i], y2 = src[i + half];
  if (hh < H + KVh) {
    const int pos = t - cu[seq_of_token(cu, nseq, t)];
    const float c = cos_t[(int64_t)pos * half + i], s = sin_t[(int64_t)pos * half + i];
    const float x1 = y1 * c + y2 * s, x2 = y2 * c - y1 * s;
    y1 = x1;
    y2 = x2;
  }
  const int64_t nq = (int64_t)NH * hd;
  const int r1 = 8 * (i / 4) + (i % 4);  // row of element i in the grouped order; its partner is 4 later
  dqkv[(int64_t)t * nq + hh * hd + r1] = (bf16)y1;
  dqkv[(int64_t)t * nq + hh * hd + r1 + 4] = (bf16)y2;
  if (dqkv_f) {
    dqkv_f[(int64_t)t * nq + hh * hd + i] = y1;
    dqkv_f[(int64_t)t * nq + hh * hd + i + half] = y2;
  }
}

// Rows of a projection gradient [R][D] in the kernel layout, back to the
// weight map's tensors: mode 0 (fused QKV, heads q then k then v, grouped rows)
// into dst0 / dst1 / dst2 = q / k / v; mode 1 (gate/up interleaved in blocks
// of 16) into dst0 / dst1 = gate / up.  4 columns per thread.
__global__ void __launch_bounds__(256) scatter_rows_kernel(const float* __restrict__ src, int D, int mode, int hd,
                                                           int H, int KVh, float* __restrict__ dst0,
                                                           float* __restrict__ dst1, float* __restrict__ dst2) {
  const int r = blockIdx.x;
  const int c = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (c >= D) return;
  float* dst;
  if (mode == 0) {
    const int hh = r / hd, rr = r % hd, g = rr / 8, j = rr % 8;
    const int L = hh * hd + (j < 4 ? 4 * g + j : hd / 2 + 4 * g + j - 4);
    dst = hh < H ? dst0 + (int64_t)L * D
                 : (hh < H + KVh ? dst1 + (int64_t)(L - H * hd) * D : dst2 + (int64_t)(L - (H + KVh) * hd) * D);
  } else {
    const int b = r / 32, j = r % 32;
    dst = j < 16 ? dst0 + (int64_t)(b * 16 + j) * D : dst1 + (int64_t)(b * 16 + j - 16) * D;
  }
  *(f32x4*)(dst + c) = *(const f32x4*)(src + (int64_t)r * D + c);
}

// dE[tok[t]] += dx[t] (tokens repeat, hence atomic additions)
__global__ void __launch_bounds__(256) embed_bwd_kernel(const int32_t* __restrict__ tok, const float* __restrict__ dx,
                                                        int D, int V, float* __restrict__ dE) {
  const int t = blockIdx.x;
  const int id = min(max(tok[t], 0), V - 1);
  for (int d = threadIdx.x; d < D; d += 256) atomicAdd(dE + (int64_t)id * D + d, dx[(int64_t)t * D + d]);
}

// ---------------------------------------------------------------- launchers

void launch_ce_loss(const float* logits, int ldl, int V, const int32_t* targets, int T, float* rowloss, float* valid,
                    float* lse, float* loss, float* scal, bf16* dlog, hipStream_t s) {
  ce_rows_kernel<<<T, 256, 0, s>>>(logits, ldl, V, targets, rowloss, valid, lse);
  ce_reduce_kernel<<<1, 256, 0, s>>>(rowloss, valid, T, loss, scal);
  ce_grad_kernel<<<dim3((ldl / 4 + 255) / 256, T), 256, 0, s>>>(logits, ldl, V, targets, valid, lse, scal, dlog);
}

void launch_transpose_pad(const bf16* src, int ld, int T, int C, bf16* dst, int Tp, hipStream_t s) {
  if (C <= 0 || Tp <= 0) return;
  transpose_tile_kernel<<<dim3((Tp + 63) / 64, (C + 63) / 64), 256, 0, s>>>(src, ld, T, Tp, C, dst, Tp, nullptr, 0, 0);
}

void launch_untile_transpose(const bf16* W, int64_t N, int K, bf16* dst, int64_t Np, hipStream_t s) {
  const int64_t n = N * (K / 8);
  if (n > 0) untile_transpose_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(W, N, K, dst, Np);
}

void launch_to_bf16(const float* src, bf16* dst, int64_t n, hipStream_t s) {
  const int64_t n4 = n / 4;
  if (n4 > 0) to_bf16_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, s>>>(src, dst, n4);
}

void launch_rmsnorm_bwd(const float* x, const bf16* g, const float* dy, int ldy, int T, int D, float eps, float* dx,
                        int accumulate, float* dgrow, hipStream_t s) {
  if (T > 0) rmsnorm_bwd_kernel<<<T, 256, 0, s>>>(x, g, dy, ldy, D, eps, dx, accumulate, dgrow);
}

void launch_swiglu_bwd(const float* gu, const float* da, bf16* dgu, int T, int I, hipStream_t s) {
  const int64_t n = (int64_t)T * I;
  if (n > 0) swiglu_bwd_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(gu, da, dgu, T, I);
}

int colsum_chunks(int T) { return std::max(1, std::min(256, (T + 63) / 64)); }

void launch_colsum(const float* src, int64_t ld, int T, int C, float* part, float* dst, hipStream_t s) {
  if (T <= 0 || C <= 0) return;
  const int nch = colsum_chunks(T), rpc = (T + nch - 1) / nch;
  colsum_part_kernel<<<dim3((C + 255) / 256, nch), 256, 0, s>>>(src, ld, T, C, rpc, part);
  colsum_final_kernel<<<(C + 255) / 256, 256, 0, s>>>(part, nch, C, dst);
}

bool attn_bwd_layout_ok(int H, int KVh, int hd, int SP, int64_t W) {
  // frag_off / row_frag_off cut rows, columns and packed positions into
  // 32-wide fragments and head dimensions into 16-wide k-steps
  return H > 0 && KVh > 0 && H % KVh == 0 && (hd == 64 || hd == 128) && SP > 0 && SP % 32 == 0 && W % 32 == 0 &&
         ((int64_t)H * hd) % 32 == 0 && ((int64_t)KVh * hd) % 32 == 0;
}

bool launch_attn_bwd(const bf16* q, KVView kv, const bf16* o, const bf16* dob, const float* lse, float* dsum,
                     float* statp, const int32_t* cu, const int32_t* h_cu, int nseq, int T, int H, int SP, int64_t W,
                     bf16* kr, bf16* vr, bf16* kt, bf16* qt, bf16* dot, float* dq, float* dkh, float* dvh, float* dk,
                     float* dv, hipStream_t s) {
  if (!attn_bwd_layout_ok(H, kv.kv_heads, kv.hd, SP, W)) return false;
  if (T <= 0) return true;
  const int KVh = kv.kv_heads, hd = kv.hd, group = H / KVh;
  float* lsep = statp;
  float* dsump = statp + (int64_t)H * W;
  attn_bwd_d_kernel<<<(T * H + 255) / 256, 256, 0, s>>>(dob, o, T * H, hd, dsum, lse, cu, nseq, H, SP, W, lsep, dsump);
  int blocks16 = 0;
  for (int e = 0; e < nseq; ++e) blocks16 += (h_cu[e + 1] - h_cu[e] + 15) / 16;
  if (hd == 64) attn_bwd_pack_kernel<64><<<dim3(blocks16, KVh), 256, 0, s>>>(kv, cu, nseq, SP, W, kr, vr, kt);
  else attn_bwd_pack_kernel<128><<<dim3(blocks16, KVh), 256, 0, s>>>(kv, cu, nseq, SP, W, kr, vr, kt);
  transpose_tile_kernel<<<dim3((T + 63) / 64, (H * hd + 63) / 64), 256, 0, s>>>(q, (int64_t)H * hd, T, T, H * hd, qt,
                                                                                 W, cu, nseq, SP, true);
  transpose_tile_kernel<<<dim3((T + 63) / 64, (H * hd + 63) / 64), 256, 0, s>>>(dob, (int64_t)H * hd, T, T, H * hd,
                                                                                 dot, W, cu, nseq, SP, true);
  int blocks = 0;
  for (int e = 0; e < nseq; ++e) blocks += (h_cu[e + 1] - h_cu[e] + 31) / 32;
  float* dkt = group > 1 ? dkh : dk;  // per-head shares, summed below when a group has several heads
  float* dvt = group > 1 ? dvh : dv;
  if (hd == 64) {
    attn_bwd_dq_kernel<64><<<dim3(blocks, H), 64, 0, s>>>(q, dob, kr, vr, kt, lse, dsum, cu, nseq, H, KVh, SP, W, dq);
    attn_bwd_dkv_kernel<64><<<dim3(blocks, H), 64, 0, s>>>(q, dob, kr, vr, qt, dot, lsep, dsump, cu, nseq, H, KVh, SP,
                                                           W, dkt, dvt);
  } else {
    attn_bwd_dq_kernel<128><<<dim3(blocks, H), 64, 0, s>>>(q, dob, kr, vr, kt, lse, dsum, cu, nseq, H, KVh, SP, W, dq);
    attn_bwd_dkv_kernel<128><<<dim3(blocks, H), 64, 0, s>>>(q, dob, kr, vr, qt, dot, lsep, dsump, cu, nseq, H, KVh, SP,
                                                            W, dkt, dvt);
  }
  if (group > 1) {
    const int64_t n = (int64_t)T * KVh * hd;
    attn_bwd_group_sum_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(dkh, dvh, n, group, hd, dk, dv);
  }
  return true;
}

void launch_rope_bwd(const float* dq, const float* dk, const float* dv, const float* cos_t, const float* sin_t,
                     const int32_t* cu, int nseq, int T, int H, int KVh, int hd, bf16* dqkv, float* dqkv_f,
                     hipStream_t s) {
  const int64_t n = (int64_t)T * (H + 2 * KVh) * (hd / 2);
  if (n > 0)
    rope_bwd_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(dq, dk, dv, cos_t, sin_t, cu, nseq, T, H, KVh, hd,
                                                                dqkv, dqkv_f);
}

void launch_scatter_rows(const float* src, int R, int D, int mode, int hd, int H, int KVh, float* dst0, float* dst1,
                         float* dst2, hipStream_t s) {
  if (R > 0) scatter_rows_kernel<<<dim3(R, (D / 4 + 255) / 256), 256, 0, s>>>(src, D, mode, hd, H, KVh, dst0, dst1, dst2);
}

void launch_embed_bwd(const int32_t* tok, const float* dx, int T, int D, int V, float* dE, hipStream_t s) {
  if (T > 0) embed_bwd_kernel<<<T, 256, 0, s>>>(tok, dx, D, V, dE);
}

}  // namespace axon
