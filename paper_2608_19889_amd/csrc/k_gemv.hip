// Few-token projections for the decode step (M <= 64 tokens), fused with
// their neighbours.  HBM-bound on the weight stream.
//
// A workgroup owns 16*RB output features of W [N][K] and the whole K range;
// its KS wavefronts split K into contiguous chunks, run
// v_mfma_f32_16x16x32_bf16 with W as the A operand (16 rows per block) and the
// tokens as the B operand (16 columns per block, NB blocks), and reduce their
// partial tiles through LDS in a fixed order (deterministic, no split-K
// partials in HBM).
//
// Normalized operand (NORM): RMSNorm(x) g enters as bf16(x[t][k] * g[k]),
// written by the producer of x together with per-workgroup partial sums of
// squares of x; the accumulator is scaled by inv[t] = rsqrt(sum of squares /
// K + eps) in the epilogue.  This replaces a separate normalization kernel.
//
// Epilogues:
//   GV_HEAD  logits (optional) + per-workgroup (max, first index) per token
//   GV_RESID x[t][n] += acc (+ bias[n]); writes bf16(x * g_next) for the
//            next normalized projection and per-workgroup sums of squares of
//            the new x (unless xg_out is null: GPT-2's LayerNorm is a kernel)
//   GV_GELU  a[t][n] = bf16(gelu_tanh(acc + bias[n])) (GPT-2 MLP)
//   GV_SILU  rows come in blocks of 16 gate rows + the 16 matching up rows:
//            a[t][f] = bf16(silu(gate) * up)
//   GV_ROPE  rows of the fused QKV projection are permuted so that an 8-row
//            group holds 4 rotation-pair first halves and their partners:
//            bias + rotary embedding at position len[t], then q -> q_out,
//            k -> K pages, v -> transposed V pages.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace axon {

AXON_DEV float silu_g(float z) { return z / (1.f + __expf(-z)); }

constexpr int GV_U = 4;  // k-steps of 32 per pipeline stage

// v(0) + v(1) + ... + v(n - 1) in that order, 8 independent (LDS) reads per
// round instead of a chain of dependent ones
template <typename V>
AXON_DEV float ordered_sum(int n, const V& v) {
  float s = 0.f;
  for (int j0 = 0; j0 < n; j0 += 8) {
    float r[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = v(min(j0 + q, n - 1));
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (j0 + q < n) s += r[q];
  }
  return s;
}

// Epilogue operands that do not depend on the projection's result, loaded by
// the fused kernel before its weight stream (one epilogue item per thread).
// bf16 values are kept as their raw bits and every field is pinned (an empty
// asm that "modifies" it) after the stream: otherwise the compiler converts
// or combines a value next to its load and waits for that load before the
// stream starts.
struct GvPre {
  float x;         // residual: x[t][n]
  uint32_t g;      // residual: bits of the next gain at n
  int pos;         // rope: the token's position
  uint32_t b1, b2; // rope: bits of the pair's biases
};
AXON_DEV float bf16_bits(uint32_t b) { return __uint_as_float(b << 16); }
AXON_DEV void pin(float& v) { asm volatile("" : "+v"(v)); }
AXON_DEV void pin(uint32_t& v) { asm volatile("" : "+v"(v)); }
AXON_DEV void pin(int& v) { asm volatile("" : "+v"(v)); }

// The epilogues of a tile of ROWS output features x COLS token columns
// starting at feature n0; total(row, col) is the finished (normalized) dot
// product.  wg / nwg index the per-tile partials (sums of squares, argmax).
// aux: LDS of at least max(ROWS, 16) x (COLS + 1) floats.
// PRE: ``pre`` holds the operands of item ``tid`` (the tile has at most one
// item per thread).
template <int ROWS, int COLS, int NT, int EPI, bool PRE = false, typename Total>
AXON_DEV void gv_epilogue(const GemvArgs& a, int n0, int tid, float* aux, int wg, int nwg, const Total& total,
                          const GvPre& pre = GvPre{}) {
  const int M = a.M, lane = tid & 63, wave = tid >> 6;
  auto s_aux = [&](int row, int col) -> float& { return aux[row * (COLS + 1) + col]; };
  if constexpr (EPI == GV_RESID) {
    // features fastest: each token's outputs are contiguous in memory
    // with a bias (GPT-2) the next normalization is a separate LayerNorm: no
    // xg / sums of squares (xg_out and ss_out null)
    for (int it = tid; it < ROWS * M; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      float sq = 0.f;
      if (n < a.N) {
        float* p = a.out_f32 + (int64_t)col * a.ldo + n;
        float v = (PRE ? pre.x : *p) + total(row, col);
        if (a.bias) v += (float)a.bias[n];
        *p = v;
        sq = v * v;
        if (a.xg_out)
          a.xg_out[a.out_tiled ? xt_off(col, n) : (int64_t)col * a.ldo + n] =
              (bf16)(v * (PRE ? bf16_bits(pre.g) : (float)a.gain_next[n]));
      }
      s_aux(row, col) = sq;
    }
    __syncthreads();
    if (tid < M && a.ss_out)
      a.ss_out[(int64_t)wg * M + tid] = ordered_sum(ROWS, [&](int row) { return s_aux(row, tid); });
  } else if constexpr (EPI == GV_SILU) {
    // each 32-row block: rows 0..15 gate, 16..31 the matching up rows
    for (int it = tid; it < (ROWS / 2) * M; it += NT) {
      const int fl = it % (ROWS / 2), col = it / (ROWS / 2);
      const int blk = fl / 16, f = fl % 16;
      if (n0 + blk * 32 >= a.N) continue;  // N is a multiple of 32 (16 gate + 16 up rows)
      const float g = total(blk * 32 + f, col), u = total(blk * 32 + 16 + f, col);
      const int fo = n0 / 2 + fl;
      a.out_t[a.out_tiled ? xt_off(col, fo) : (int64_t)col * a.ldo + fo] = (bf16)(silu_g(g) * u);
    }
  } else if constexpr (EPI == GV_GELU) {
    for (int it = tid; it < ROWS * M; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      if (n < a.N) a.out_t[(int64_t)col * a.ldo + n] = (bf16)gelu_tanh_f(total(row, col) + (float)a.bias[n]);
    }
  } else if constexpr (EPI == GV_ROPE) {
    // an 8-row group of a head = first halves i = 4g..4g+3 and their partners
    const int hd = a.kv.hd, half = hd / 2;
    const int head = n0 / hd, g0 = (n0 % hd) / 8;
    const int KVh = a.kv.kv_heads;
    for (int it = tid; it < (ROWS / 2) * M; it += NT) {
      const int pr = it % (ROWS / 2), t = it / (ROWS / 2);
      const int gl = pr / 4, i4 = pr % 4;
      const int i = (g0 + gl) * 4 + i4;  // rotation pair (i, i + hd/2) of this head
      float x1 = total(gl * 8 + i4, t), x2 = total(gl * 8 + 4 + i4, t);
      if (a.bias) {
        x1 += PRE ? bf16_bits(pre.b1) : (float)a.bias[head * hd + i];
        x2 += PRE ? bf16_bits(pre.b2) : (float)a.bias[head * hd + half + i];
      }
      const int pos = PRE ? pre.pos : a.len[t];
      const int sl = a.slot ? a.slot[t] : t;
      if (head < a.H + KVh) {
        const float cs = a.cos_t[(int64_t)pos * half + i], sn = a.sin_t[(int64_t)pos * half + i];
        const float y1 = x1 * cs - x2 * sn, y2 = x2 * cs + x1 * sn;
        if (head < a.H) {
          bf16* dst = a.q_out + ((int64_t)t * a.H + head) * hd;
          dst[i] = (bf16)y1;
          dst[i + half] = (bf16)y2;
        } else {
          bf16* kc = (bf16*)a.kv.k;
          kc[k_el(a.kv, sl, head - a.H, pos, i)] = (bf16)y1;
          kc[k_el(a.kv, sl, head - a.H, pos, i + half)] = (bf16)y2;
        }
      } else {
        const int kvh = head - a.H - KVh;
        bf16* vc = (bf16*)a.kv.v;
        vc[v_el(a.kv, sl, kvh, pos, i)] = (bf16)x1;
        vc[v_el(a.kv, sl, kvh, pos, i + half)] = (bf16)x2;
      }
    }
  } else if constexpr (EPI == GV_F32) {
    for (int it = tid; it < ROWS * M; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      if (n < a.N) a.out_f32[(int64_t)col * a.ldo + n] = total(row, col);
    }
  } else {  // GV_HEAD
    for (int it = tid; it < ROWS * M; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      float v = -INFINITY;
      if (n < a.N) {
        v = total(row, col);
        if (a.out_f32) a.out_f32[(int64_t)col * a.ldo + n] = v;
      }
      s_aux(row, col) = v;
    }
    __syncthreads();
    // per token, the largest logit of the tile and its lowest index (a
    // wavefront per token)
    for (int t = wave; t < M; t += NT / 64) {
      float best = -INFINITY;
      int bi = 0x7fffffff;
      for (int row = lane; row < ROWS; row += 64) {
        const float v = s_aux(row, t);
        if (v > best) { best = v; bi = n0 + row; }
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const float ov = __shfl_xor(best, m, 64);
        const int oi = __shfl_xor(bi, m, 64);
        if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
      }
      if (lane == 0) {
        a.am_val[(int64_t)t * nwg + wg] = best;
        a.am_idx[(int64_t)t * nwg + wg] = bi;
      }
    }
  }
}

// XT: the token operand is in tile order (xt_off; one token block)
template <int ROWS, int KS, int NB, bool NORM, int EPI, int U = GV_U, bool XT = false>
__global__ void __launch_bounds__(KS * 64) gemv_fused_kernel(GemvArgs a) {
  static_assert(!XT || NB == 1, "the tile order holds one block of 16 tokens");
  constexpr int RB = ROWS < 16 ? 1 : ROWS / 16;  // 16-row MFMA blocks (an 8-row tile leaves 8 rows idle)
  constexpr int COLS = NB * 16;
  constexpr int NT = KS * 64;
  __shared__ float red[KS][RB * 16][COLS + 1];
  __shared__ float s_ss[NT];
  __shared__ float s_inv[64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = blockIdx.x * ROWS;
  const int K = a.K, M = a.M;
  // K range of the workgroup (split K: split blockIdx.y of gridDim.y, each a
  // multiple of 32), divided among the KS wavefronts in whole stages
  const int klen = EPI == GV_PART ? ((K + gridDim.y - 1) / gridDim.y + 31) / 32 * 32 : K;
  const int kbase = EPI == GV_PART ? min(K, (int)blockIdx.y * klen) : 0;
  const int kloc = min(K - kbase, klen);
  const int kc = ((kloc + KS - 1) / KS + 32 * U - 1) / (32 * U) * (32 * U);
  const int k0 = kbase + min(kloc, wave * kc), k1 = kbase + min(kloc, wave * kc + kc);
  const int r16 = lane & 15;

  // Every load below is unconditional (a load under a lane condition makes
  // the compiler wait for all outstanding loads where the branches join).
  // W is fragment-tiled: the A fragment of row block r at k (a multiple of
  // 32) is this lane's 16-byte chunk of the 1 KB tile (row block, k / 32).
  // Rows past N read row N-1 and token columns past M read token M-1: those
  // MFMA rows / columns only reach outputs that are never stored.  In an
  // 8-row workgroup lanes 8..15 repeat rows 0..7 (same addresses, no extra
  // traffic).
  const bf16* wrow[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int n = n0 + r * 16 + (ROWS >= 16 ? r16 : (r16 & 7));
    wrow[r] = a.W + wt_chunk(min(n, a.N - 1), lane >> 4, K);
  }
  auto woff = [](int k) -> int64_t { return (int64_t)(k >> 5) * 512; };
  // token fragments: lane (r16, lane / 16) reads 16 bytes of token r16
  // (tokens past M-1 read token M-1: no bytes beyond the tokens' own), from
  // row r16 (row-major) or, in tile order, from the k-step's 1 KB at 16 k
  // (xt_off)
  const bf16* xrow[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c)
    xrow[c] = XT ? a.X + ((lane >> 4) * 16 + min(r16, M - 1)) * 8
                 : a.X + (int64_t)min(c * 16 + r16, M - 1) * K + (lane >> 4) * 8;
  auto xoff = [](int k) -> int64_t { return XT ? (int64_t)k * 16 : (int64_t)k; };

  // sums of squares of the normalized rows: the first SSR partials of this
  // thread are loaded into registers now (index clamped, excluded in the sum)
  // and consumed after the stream
  // (tokens x slices threads; no more slices than the partials need, which
  // keeps the per-token sum over slices short)
  constexpr int SSR = 16;
  float ss_reg[SSR];
  const int ss_slices = NORM ? min(NT / M, max(1, (a.ss_n + SSR - 1) / SSR)) : 1;
  const int ss_t = tid % M, ss_sl = tid / M;
  if constexpr (NORM) {
    // only the wavefronts holding slices load (a wave-uniform branch)
    if (wave * 64 < ss_slices * M) {
#pragma unroll
      for (int i = 0; i < SSR; ++i) {
        const int j = min(ss_sl + i * ss_slices, a.ss_n - 1);
        ss_reg[i] = a.ss_in[(int64_t)j * M + ss_t];
      }
    } else {
#pragma unroll
      for (int i = 0; i < SSR; ++i) ss_reg[i] = 0.f;
    }
  }

  f32x4 acc[RB][NB];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c) acc[r][c] = f32x4{};

  // software-pipelined stream over the full stages of [k0, k1): stage s+1 is
  // loaded while stage s feeds the MFMAs; the rest (k1 - k0 is a multiple of
  // 32) in single k-steps
  bf16x8 wa[U][RB], xb[U][NB];
  auto load_stage = [&](int k) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int r = 0; r < RB; ++r) wa[u][r] = *(const bf16x8*)(wrow[r] + woff(k + u * 32));
#pragma unroll
      for (int c = 0; c < NB; ++c) xb[u][c] = *(const bf16x8*)(xrow[c] + xoff(k + u * 32));
    }
  };
  auto mfma_stage = [&](const bf16x8 (&wv)[U][RB], const bf16x8 (&xv)[U][NB]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int c = 0; c < NB; ++c)
          acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wv[u][r], xv[u][c], acc[r][c], 0, 0, 0);
  };
  // epilogue operands (one item per thread), loaded behind the first stage
  constexpr bool PRE = (EPI == GV_RESID && ROWS * COLS <= NT) || (EPI == GV_ROPE && (ROWS / 2) * COLS <= NT);
  GvPre pre{};
  auto prefetch = [&] {
    if constexpr (PRE && EPI == GV_RESID) {
      const int it = min(tid, ROWS * M - 1);
      const int n = min(n0 + it % ROWS, a.N - 1), col = it / ROWS;
      pre.x = a.out_f32[(int64_t)col * a.ldo + n];
      pre.g = a.gain_next ? *(const unsigned short*)(a.gain_next + n) : 0u;
    } else if constexpr (PRE && EPI == GV_ROPE) {
      const int it = min(tid, (ROWS / 2) * M - 1);
      const int pr = it % (ROWS / 2), t = it / (ROWS / 2);
      const int hd = a.kv.hd, half = hd / 2, head = n0 / hd;
      const int i = ((n0 % hd) / 8 + pr / 4) * 4 + pr % 4;
      pre.pos = a.len[t];
      // no bias: read the weights instead (any valid address; not used)
      const bf16* bp = a.bias ? a.bias : a.W;
      pre.b1 = *(const unsigned short*)(bp + head * hd + i);
      pre.b2 = *(const unsigned short*)(bp + head * hd + half + i);
    }
  };
  auto pin_pre = [&] {
    if constexpr (PRE && EPI == GV_RESID) {
      pin(pre.x);
      pin(pre.g);
    } else if constexpr (PRE && EPI == GV_ROPE) {
      pin(pre.pos);
      pin(pre.b1);
      pin(pre.b2);
    }
  };
  const int nst = (k1 - k0) / (32 * U);
  if (nst > 0) load_stage(k0);
  prefetch();
  if (nst > 0) {
    for (int st = 1; st < nst; ++st) {
      bf16x8 ca[U][RB], cb[U][NB];
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int r = 0; r < RB; ++r) ca[u][r] = wa[u][r];
#pragma unroll
        for (int c = 0; c < NB; ++c) cb[u][c] = xb[u][c];
      }
      load_stage(k0 + st * 32 * U);
      mfma_stage(ca, cb);
    }
    mfma_stage(wa, xb);
  }
  for (int k = k0 + nst * 32 * U; k < k1; k += 32) {
    bf16x8 w1[RB], x1[NB];
#pragma unroll
    for (int r = 0; r < RB; ++r) w1[r] = *(const bf16x8*)(wrow[r] + woff(k));
#pragma unroll
    for (int c = 0; c < NB; ++c) x1[c] = *(const bf16x8*)(xrow[c] + xoff(k));
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int c = 0; c < NB; ++c) acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w1[r], x1[c], acc[r][c], 0, 0, 0);
  }

  // the prefetched values are used from here on (see GvPre)
  pin_pre();
  if constexpr (NORM) {
#pragma unroll
    for (int i = 0; i < SSR; ++i) pin(ss_reg[i]);
  }
  // ---- cross-wavefront reduction: acc[r][c][i] = C[n0 + r*16 + (lane/16)*4 + i][c*16 + lane%16]
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][r * 16 + (lane >> 4) * 4 + i][c * 16 + r16] = acc[r][c][i];
  if constexpr (NORM) {
    float ss_part = 0.f;
    // selects, not branches: a lane-divergent branch per term costs more
    // than the adds
    const bool ss_own = ss_sl < ss_slices;
#pragma unroll
    for (int i = 0; i < SSR; ++i) ss_part += ss_own && ss_sl + i * ss_slices < a.ss_n ? ss_reg[i] : 0.f;
    // partials beyond the prefetched ones: 16 independent loads per round
    // (a load-add loop would wait for every load in turn)
    if (ss_sl < ss_slices) {
      for (int j0 = ss_sl + SSR * ss_slices; j0 < a.ss_n; j0 += SSR * ss_slices) {
        float v[SSR];
#pragma unroll
        for (int i = 0; i < SSR; ++i) v[i] = a.ss_in[(int64_t)min(j0 + i * ss_slices, a.ss_n - 1) * M + ss_t];
#pragma unroll
        for (int i = 0; i < SSR; ++i)
          if (j0 + i * ss_slices < a.ss_n) ss_part += v[i];
      }
    }
    s_ss[tid] = ss_part;
  }
  __syncthreads();
  if constexpr (NORM) {
    if (tid < M) {
      const float tot = ordered_sum(ss_slices, [&](int sl) { return s_ss[sl * M + tid]; });
      s_inv[tid] = rsqrtf(tot / (float)K + a.eps);
    }
    __syncthreads();
  }
  auto total = [&](int row, int col) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < KS; ++w) s += red[w][row][col];
    if constexpr (NORM) s *= s_inv[col];
    return s;
  };

  if constexpr (EPI == GV_PART) {
    // raw tile sums of this K split: part[split][col][n0 + row]
    for (int it = tid; it < ROWS * COLS; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      if (col < M && n < a.N) a.part[((int64_t)blockIdx.y * M + col) * a.N + n] = total(row, col);
    }
  } else {
    // the residual and head epilogues overwrite element (row, col) of their
    // scratch only after the same thread has read total(row, col): the first
    // wavefront's tile serves as that scratch
    gv_epilogue<ROWS, COLS, NT, EPI, PRE>(a, n0, tid, &red[0][0][0], blockIdx.x, gridDim.x, total, pre);
  }
}

// Projections of 17..64 tokens: the 4 wavefronts of a workgroup split the
// output rows (16 * RB each) over the workgroup's whole K range and share the
// token operand, which is staged through LDS in B-fragment lane order (a
// wavefront reads 1 KB per fragment with consecutive 16-byte lanes, no bank
// conflicts), double-buffered with one barrier per stage of U k-steps.  There
// is no cross-wavefront reduction, so registers and LDS stay small enough for
// several workgroups per CU (the weight stream needs many bytes in flight).
// Same operands, K splitting (EPI == GV_PART) and epilogues as
// gemv_fused_kernel.
// GROUPED (mixture-of-experts decode, GemvArgs::g_*): expert e = blockIdx.y
// owns rows g_off[e] .. g_off[e+1]-1 (a workgroup with none leaves at once)
// and multiplies W + e * g_wstride; its token column c reads X row
// g_xrow[g_off[e] + c] (row g_off[e] + c without g_xrow) and writes output
// row g_off[e] + c.
template <int RB, int NB, bool NORM, int EPI, int U, bool GROUPED = false>
__global__ void __launch_bounds__(256) gemv_wide_kernel(GemvArgs a) {
  constexpr int NT = 256, ROWS = 64 * RB, COLS = NB * 16;
  constexpr int XCH = U * NB * 64;  // 16-byte token chunks per stage
  static_assert(XCH % NT == 0, "stage must split evenly over the threads");
  constexpr int XPT = XCH / NT;
  constexpr int XS_FLOATS = 2 * XCH * 4, TOT_FLOATS = ROWS * (COLS + 1);
  // token stages while streaming, then the finished tile for the epilogue
  __shared__ float smem[XS_FLOATS > TOT_FLOATS ? XS_FLOATS : TOT_FLOATS];
  __shared__ float s_ss[NT];
  __shared__ float s_inv[64];
  bf16x8* xs = (bf16x8*)smem;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n0 = blockIdx.x * ROWS;
  const int K = a.K;
  int M = a.M, r0 = 0;
  if constexpr (GROUPED) {
    r0 = a.g_off[blockIdx.y];
    M = a.g_off[blockIdx.y + 1] - r0;
    if (M == 0) return;  // no token chose this expert: leave before any barrier
    a.W += (int64_t)blockIdx.y * a.g_wstride;
  }
  const int klen = EPI == GV_PART ? ((K + gridDim.y - 1) / gridDim.y + 31) / 32 * 32 : K;
  const int kb = EPI == GV_PART ? min(K, (int)blockIdx.y * klen) : 0;
  const int nsteps = (min(K, kb + klen) - kb) / 32;  // k-steps of 32 (K is a multiple of 32)
  const int nst = (nsteps + U - 1) / U;               // stages; the last may be partial
  const int r16 = lane & 15;

  // weights: this wavefront's row blocks (rows past N read row N-1, never stored)
  const bf16* wrow[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int n = n0 + (wave * RB + r) * 16 + r16;
    wrow[r] = a.W + wt_chunk(min(n, a.N - 1), lane >> 4, K);
  }
  // token chunks this thread stages: chunk q = (u * NB + c) * 64 + l holds
  // lane l's B fragment of token block c at k-step u (token columns past M
  // read token M-1)
  const bf16* xsrc[XPT];
  int xu[XPT];
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int q = tid + i * NT, l = q & 63, c = (q >> 6) % NB;
    xu[i] = (q >> 6) / NB;
    int64_t xr = min(c * 16 + (l & 15), M - 1);
    if constexpr (GROUPED) xr = a.g_xrow ? a.g_xrow[r0 + xr] : r0 + xr;
    xsrc[i] = a.X + xr * K + (l >> 4) * 8;
  }
  auto kstep = [&](int j) { return kb + min(j, nsteps - 1) * 32; };  // clamped: every load is unconditional

  constexpr int SSR = 16;
  float ss_reg[SSR];
  const int ss_slices = NORM ? min(NT / M, max(1, (a.ss_n + SSR - 1) / SSR)) : 1;
  const int ss_t = tid % M, ss_sl = tid / M;
  if constexpr (NORM) {
    if (wave * 64 < ss_slices * M) {
#pragma unroll
      for (int i = 0; i < SSR; ++i) {
        const int j = min(ss_sl + i * ss_slices, a.ss_n - 1);
        ss_reg[i] = a.ss_in[(int64_t)j * M + ss_t];
      }
    } else {
#pragma unroll
      for (int i = 0; i < SSR; ++i) ss_reg[i] = 0.f;
    }
  }

  f32x4 acc[RB][NB];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c) acc[r][c] = f32x4{};

  bf16x8 xr[XPT];
  bf16x8 wA[U][RB], wB[U][RB];
  auto load_x = [&](int st) {
#pragma unroll
    for (int i = 0; i < XPT; ++i) xr[i] = *(const bf16x8*)(xsrc[i] + kstep(st * U + xu[i]));
  };
  auto store_x = [&](int buf) {
#pragma unroll
    for (int i = 0; i < XPT; ++i) xs[buf * XCH + tid + i * NT] = xr[i];
  };
  auto load_w = [&](bf16x8 (&w)[U][RB], int st) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int r = 0; r < RB; ++r) w[u][r] = *(const bf16x8*)(wrow[r] + (int64_t)(kstep(st * U + u) >> 5) * 512);
  };
  auto compute = [&](const bf16x8 (&w)[U][RB], int st) {
    const bf16x8* xb = xs + (st & 1) * XCH + lane;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (st * U + u < nsteps) {  // workgroup-uniform: the last stage may be partial
        bf16x8 xv[NB];
#pragma unroll
        for (int c = 0; c < NB; ++c) xv[c] = xb[(u * NB + c) * 64];
#pragma unroll
        for (int r = 0; r < RB; ++r)
#pragma unroll
          for (int c = 0; c < NB; ++c)
            acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[u][r], xv[c], acc[r][c], 0, 0, 0);
      }
    }
  };
  // stage st: barrier (its tokens landed for every wavefront; the other
  // buffer is no longer read), MFMAs, stage the tokens of st + 1, issue the
  // loads of st + 2 into the weight registers just consumed
  auto stage = [&](bf16x8 (&w)[U][RB], int st) {
    __syncthreads();
    compute(w, st);
    if (st + 1 < nst) store_x((st + 1) & 1);
    if (st + 2 < nst) {
      load_x(st + 2);
      load_w(w, st + 2);
    }
  };
  if (nst > 0) {
    load_x(0);
    load_w(wA, 0);
    store_x(0);
    if (nst > 1) {
      load_x(1);
      load_w(wB, 1);
    }
    for (int st = 0; st < nst; st += 2) {
      stage(wA, st);
      if (st + 1 < nst) stage(wB, st + 1);
    }
  }

  // the prefetched sums of squares are used from here on (see GvPre)
  if constexpr (NORM) {
#pragma unroll
    for (int i = 0; i < SSR; ++i) pin(ss_reg[i]);
  }
  // finished tile -> LDS (over the token stages): tot[row][col]
  __syncthreads();
  float* tot = smem;
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        tot[((wave * RB + r) * 16 + (lane >> 4) * 4 + i) * (COLS + 1) + c * 16 + r16] = acc[r][c][i];
  if constexpr (NORM) {
    float ss_part = 0.f;
    // selects, not branches: a lane-divergent branch per term costs more
    // than the adds
    const bool ss_own = ss_sl < ss_slices;
#pragma unroll
    for (int i = 0; i < SSR; ++i) ss_part += ss_own && ss_sl + i * ss_slices < a.ss_n ? ss_reg[i] : 0.f;
    if (ss_sl < ss_slices) {
      for (int j0 = ss_sl + SSR * ss_slices; j0 < a.ss_n; j0 += SSR * ss_slices) {
        float v[SSR];
#pragma unroll
        for (int i = 0; i < SSR; ++i) v[i] = a.ss_in[(int64_t)min(j0 + i * ss_slices, a.ss_n - 1) * M + ss_t];
#pragma unroll
        for (int i = 0; i < SSR; ++i)
          if (j0 + i * ss_slices < a.ss_n) ss_part += v[i];
      }
    }
    s_ss[tid] = ss_part;
  }
  __syncthreads();
  if constexpr (NORM) {
    if (tid < M) {
      const float tot = ordered_sum(ss_slices, [&](int sl) { return s_ss[sl * M + tid]; });
      s_inv[tid] = rsqrtf(tot / (float)K + a.eps);
    }
    __syncthreads();
  }
  auto total = [&](int row, int col) {
    float s = tot[row * (COLS + 1) + col];
    if constexpr (NORM) s *= s_inv[col];
    return s;
  };
  if constexpr (EPI == GV_PART) {
    // partial sums of this K split (already scaled by the token's RMSNorm
    // factor when NORM): part[split][col][n0 + row]
    for (int it = tid; it < ROWS * M; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      if (n < a.N) a.part[((int64_t)blockIdx.y * M + col) * a.N + n] = total(row, col);
    }
  } else if constexpr (EPI == GV_F32) {
    for (int it = tid; it < ROWS * M; it += NT) {
      const int row = it % ROWS, col = it / ROWS, n = n0 + row;
      if (n < a.N) a.out_f32[(int64_t)(r0 + col) * a.ldo + n] = total(row, col);
    }
  } else {
    // the residual and head epilogues overwrite element (row, col) of their
    // scratch only after the same thread has read total(row, col): the tile
    // itself serves as that scratch
    if constexpr (GROUPED) {
      a.M = M;
      a.out_t += (int64_t)r0 * a.ldo;
    }
    gv_epilogue<ROWS, COLS, NT, EPI>(a, n0, tid, tot, blockIdx.x, gridDim.x, total);
  }
}

// Epilogue of a split-K projection: total = the K splits' partial sums in
// split order (deterministic; a normalized projection's partials already
// carry the token's RMSNorm factor), then the projection's epilogue on tiles
// of EROWS features.
template <int EROWS, int NB, int EPI>
__global__ void __launch_bounds__(256) gemv_split_epilogue_kernel(GemvArgs a, int nsplit) {
  constexpr int COLS = NB * 16, NT = 256;
  static_assert(EROWS >= 16, "the tile doubles as the epilogue scratch");
  // the tile's totals; the residual and head epilogues overwrite element
  // (row, col) only after the same thread has read it, so it is also their
  // scratch
  __shared__ float s_tot[EROWS * (COLS + 1)];
  const int tid = threadIdx.x, M = a.M;
  const int n0 = blockIdx.x * EROWS;
  // staged rows-fastest (the partials are [split][token][n]: coalesced), the
  // splits in order; 4 splits' loads in flight per round
  constexpr int IT = (EROWS * COLS + NT - 1) / NT;
  const int items = EROWS * M;
  float sum[IT];
#pragma unroll
  for (int j = 0; j < IT; ++j) sum[j] = 0.f;
  for (int sp0 = 0; sp0 < nsplit; sp0 += 4) {
    float v[IT][4];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int it = min(tid + j * NT, items - 1);
      const int n = min(n0 + it % EROWS, a.N - 1), c = it / EROWS;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[j][q] = a.part[((int64_t)min(sp0 + q, nsplit - 1) * M + c) * a.N + n];
    }
#pragma unroll
    for (int j = 0; j < IT; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (sp0 + q < nsplit) sum[j] += v[j][q];
  }
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    const int it = tid + j * NT;
    if (it < items) s_tot[(it % EROWS) * (COLS + 1) + it / EROWS] = sum[j];
  }
  __syncthreads();
  auto total = [&](int row, int col) { return s_tot[row * (COLS + 1) + col]; };
  gv_epilogue<EROWS, COLS, NT, EPI>(a, n0, tid, s_tot, blockIdx.x, gridDim.x, total);
}

// Residual epilogue of a split-K projection by token rows: workgroup
// (chunk, t) owns features [1024 chunk, 1024 chunk + 1024) of token t, 4 per
// thread: x[t][n] += the splits' partials (split order), xg = bf16(x *
// g_next), and one sum of squares of the new x per (chunk, token).  Few
// partials per token keep the next normalized projection's prologue short.
// N must be a multiple of 4 (float4 / 4 x bf16 accesses).
__global__ void __launch_bounds__(256) gemv_split_resid_kernel(GemvArgs a, int nsplit) {
  const int t = blockIdx.y, tid = threadIdx.x, M = a.M;
  const int n = min(blockIdx.x * GV_RESID_ROWS + tid * 4, a.N - 4);  // clamped: loads are unconditional
  const bool own = blockIdx.x * GV_RESID_ROWS + tid * 4 < a.N;
  float4 s = {0.f, 0.f, 0.f, 0.f};
  for (int sp0 = 0; sp0 < nsplit; sp0 += 4) {
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = *(const float4*)(a.part + ((int64_t)min(sp0 + q, nsplit - 1) * M + t) * a.N + n);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (sp0 + q < nsplit) {
        s.x += v[q].x; s.y += v[q].y; s.z += v[q].z; s.w += v[q].w;
      }
  }
  float* xp = a.out_f32 + (int64_t)t * a.ldo + n;
  const float4 x0 = *(const float4*)xp;
  float4 x = {x0.x + s.x, x0.y + s.y, x0.z + s.z, x0.w + s.w};
  if (a.bias) {
    const bf16x4 bb = *(const bf16x4*)(a.bias + n);
    x.x += (float)bb[0]; x.y += (float)bb[1]; x.z += (float)bb[2]; x.w += (float)bb[3];
  }
  float sq = 0.f;
  if (own) {
    *(float4*)xp = x;
    if (a.xg_out) {
      const bf16x4 g = *(const bf16x4*)(a.gain_next + n);
      bf16x4 o;
      o[0] = (bf16)(x.x * (float)g[0]);
      o[1] = (bf16)(x.y * (float)g[1]);
      o[2] = (bf16)(x.z * (float)g[2]);
      o[3] = (bf16)(x.w * (float)g[3]);
      *(bf16x4*)(a.xg_out + (int64_t)t * a.ldo + n) = o;
    }
    sq = x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) sq += __shfl_xor(sq, m, 64);
  __shared__ float s_w[4];
  if ((tid & 63) == 0) s_w[tid >> 6] = sq;
  __syncthreads();
  if (tid == 0 && a.ss_out) a.ss_out[(int64_t)blockIdx.x * M + t] = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
}

// next[t] = index of the largest partial maximum (lowest index on ties);
// len[t] += 1 when ``len`` is set.
__global__ void __launch_bounds__(1024) argmax_final_kernel(const float* __restrict__ val,
                                                            const int32_t* __restrict__ idx, int nparts,
                                                            int32_t* __restrict__ next, int32_t* __restrict__ len) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const int t = blockIdx.x;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  // 4 independent partial loads per thread and round (a compare-as-you-load
  // loop waits for every load in turn); the order of the candidates does
  // not matter: the largest value wins, ties go to the lowest index
  const float* vr = val + (int64_t)t * nparts;
  const int32_t* ir = idx + (int64_t)t * nparts;
  for (int j0 = threadIdx.x; j0 < nparts; j0 += 4 * 1024) {
    float v[4];
    int i[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = min(j0 + u * 1024, nparts - 1);
      v[u] = vr[j];
      i[u] = ir[j];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (v[u] > best || (v[u] == best && i[u] < bi)) { best = v[u]; bi = i[u]; }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(best, m, 64);
    const int oi = __shfl_xor(bi, m, 64);
    if (ov > best || (ov == best && oi < bi)) { best = ov; bi = oi; }
  }
  if ((threadIdx.x & 63) == 0) { sv[threadIdx.x >> 6] = best; si[threadIdx.x >> 6] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 16; ++w)
      if (sv[w] > best || (sv[w] == best && si[w] < bi)) { best = sv[w]; bi = si[w]; }
    next[t] = bi == 0x7fffffff ? 0 : bi;
    if (len) len[t] += 1;
  }
}

// x[t] = E[tok[t]] as float, xg[t] = bf16(x[t] * g), ss_out[t] = sum of
// squares of the row (a single partial for the first projection's normalization)
__global__ void __launch_bounds__(256) embed_ss_kernel(const int32_t* __restrict__ tok, const bf16* __restrict__ emb,
                                                       const bf16* __restrict__ g, float* __restrict__ x,
                                                       bf16* __restrict__ xg, float* __restrict__ ss_out, int D,
                                                       int V, bool xg_tiled) {
  __shared__ float red[16];
  const int t = blockIdx.x;
  const int id = min(max(tok[t], 0), V - 1);
  float* xr = x + (int64_t)t * D;
  float ss = 0.f;
  for (int i = threadIdx.x * 8; i < D; i += blockDim.x * 8) {
    const bf16x8 v = *(const bf16x8*)(emb + wt_chunk(id, i >> 3, D));  // fragment-tiled table
    f32x4 lo, hi;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lo[j] = (float)v[j];
      hi[j] = (float)v[j + 4];
      ss += lo[j] * lo[j] + hi[j] * hi[j];
    }
    *(f32x4*)(xr + i) = lo;
    *(f32x4*)(xr + i + 4) = hi;
    const bf16x8 gv = *(const bf16x8*)(g + i);
    bf16x8 o;
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = (bf16)((float)v[j] * (float)gv[j]);
    *(bf16x8*)(xg + (xg_tiled ? xt_off(t, i) : (int64_t)t * D + i)) = o;  // i % 8 == 0: 16 contiguous bytes
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) ss_out[t] = ss;
}

// ---------------------------------------------------------------- launchers

// Workgroup shape per epilogue and token count: ROWS output features, KS
// wavefronts splitting K, U k-steps of 32 per pipeline stage.  Chosen by
// timing every candidate on weights streamed from HBM (not from the 256 MB
// last-level cache): narrow projections need enough row blocks to occupy all
// 256 CUs (one CU streams only ~25 GB/s); more token columns favour more rows
// per workgroup (each token fragment is reused across them) and a shallower
// pipeline (register pressure).
GvShape gemv_shape(int N, int K, int M, int epi) {
  N = std::max(N, 1);
  const int nb = (M + 15) / 16;
  if (epi == GV_F32) {
    // float rows (a router's tens of logits): K split over up to 32
    // workgroups per 64-row block, since one CU alone streams slowly
    const int blocks = (N + 63) / 64;
    const int ksplit = std::max(1, std::min(K / 64, (32 + blocks - 1) / blocks));
    return {64, 4, nb == 2 ? 2 : 4, ksplit, 16, 1};
  }
  if ((epi == GV_SILU || epi == GV_GELU) && nb >= 2 && (N + 63) / 64 < 256) {
    // narrow gate/up (shared experts) or GELU up projection: K split towards
    // ~512 workgroups; 32-row SiLU epilogue tiles hold 16 gate rows and their
    // 16 up rows
    const int blocks = (N + 63) / 64;
    const int ksplit = std::max(2, std::min(12, (512 + blocks / 2) / blocks));
    return {64, 4, nb == 2 ? 2 : 4, ksplit, epi == GV_SILU ? 32 : 16, 1};
  }
  if (nb == 1) {
    // from timing every (rows, wavefronts, k-steps) candidate on weights
    // streamed from HBM, 1B- and 7B-shaped layers at 8 and 16 tokens (token
    // operands in tile order)
    if (epi == GV_SILU) return {32, 8, 4, 1, 0};
    if (epi == GV_GELU) return {32, 4, 4, 1, 0};
    if (epi == GV_HEAD) return {32, 8, 4, 1, 0};
    // QKV + RoPE: with a long K, 32-row tiles halve the token-operand reads
    // per weight byte (10.7 against 14.4 us on the 7B shape)
    if (epi == GV_ROPE) return K >= 3072 ? GvShape{32, 8, 4, 1, 0} : GvShape{16, 16, 4, 1, 0};
    if (N / 16 < 192) return K >= 2048 ? GvShape{8, 8, 8, 1, 0} : GvShape{8, 16, 2, 1, 0};
    return {16, 8, 4, 1, 0};
  }
  // 17..64 tokens: the row-splitting kernel (gemv_wide_kernel), whose token
  // fragments are reused by 4 or 8 row blocks per workgroup.  3 token blocks
  // need 4 k-steps per stage (the stage is split evenly over 256 threads).
  // Shapes and split counts from timing the candidates on weights streamed
  // from HBM (7B- and 32B-shaped layers at 32 and 64 tokens).
  if (epi == GV_RESID || epi == GV_ROPE) {
    // narrow projections: K split over workgroups, then a second kernel sums
    // the splits and runs the epilogue (the residual one by token rows of
    // 1024 features, the others on 16-row tiles).  Long K: 128-row tiles
    // towards ~252 workgroups; short K: 64-row tiles towards ~504 (33..64
    // tokens) or ~1008 (17..32 tokens) workgroups, which keeps enough weight
    // bytes in flight per CU
    const int erows = epi == GV_RESID && N % 4 == 0 ? GV_RESID_ROWS : 16;
    const int rb = K >= 8192 ? 2 : 1;
    const int blocks = (N + 64 * rb - 1) / (64 * rb);
    const int target = rb == 2 ? 252 : nb >= 3 ? 504 : 1008;
    const int ksplit = std::max(2, std::min(12, (target + blocks / 2) / blocks));
    return {64 * rb, 4, rb == 2 || nb >= 3 ? 4 : 2, ksplit, erows, 1};
  }
  if (epi == GV_SILU || epi == GV_GELU) {
    if (nb == 2) return {128, 4, 2, 1, 0, 1};
    return {64, 4, nb == 3 ? 4 : 2, 1, 0, 1};
  }
  return {128, 4, nb == 4 ? 2 : 4, 1, 0, 1};  // head
}

int gemv_rows(int N, int K, int M, int epi) {
  const GvShape sh = gemv_shape(N, K, M, epi);
  return sh.ksplit > 1 ? sh.erows : sh.rows;
}

int64_t gemv_workspace_floats(int N, int K, int M, int epi) {
  const GvShape sh = gemv_shape(N, K, M, epi);
  return sh.ksplit > 1 ? (int64_t)sh.ksplit * M * N : 0;
}

template <int ROWS, int KS, int U, int NB, bool NORM, int EPI>
static bool gv(const GemvArgs& a, hipStream_t s) {
  if constexpr (NB == 1) {
    if (a.x_tiled) {
      klaunch(gemv_fused_kernel<ROWS, KS, NB, NORM, EPI, U, true>, dim3((a.N + ROWS - 1) / ROWS), dim3(KS * 64), 0, s,
              a);
      return true;
    }
  }
  klaunch(gemv_fused_kernel<ROWS, KS, NB, NORM, EPI, U>, dim3((a.N + ROWS - 1) / ROWS), dim3(KS * 64), 0, s, a);
  return true;
}

template <int RB, int U, int NB, bool NORM, int EPI>
static bool gvw(const GemvArgs& a, hipStream_t s) {
  klaunch(gemv_wide_kernel<RB, NB, NORM, EPI, U>, dim3((a.N + 64 * RB - 1) / (64 * RB)), dim3(256), 0, s, a);
  return true;
}

// every unsplit shape gemv_shape can return, per (epilogue, normalization,
// token blocks)
template <int EPI, bool NORM>
static bool gv_dispatch(const GemvArgs& a, const GvShape& sh, int nb, hipStream_t s) {
#define AXON_GV(R, KS_, U_, NB_) \
  if (!sh.wide && sh.rows == R && sh.ks == KS_ && sh.u == U_ && nb == NB_) return gv<R, KS_, U_, NB_, NORM, EPI>(a, s);
#define AXON_GVW(R, U_, NB_) \
  if (sh.wide && sh.rows == R && sh.u == U_ && nb == NB_) return gvw<R / 64, U_, NB_, NORM, EPI>(a, s);
  if constexpr (EPI == GV_SILU || EPI == GV_GELU) {
    AXON_GV(32, 4, 4, 1) AXON_GV(32, 8, 4, 1) AXON_GVW(128, 2, 2) AXON_GVW(64, 4, 3) AXON_GVW(64, 2, 4)
  } else if constexpr (EPI == GV_HEAD) {
    AXON_GV(32, 8, 4, 1) AXON_GVW(128, 4, 2) AXON_GVW(128, 4, 3) AXON_GVW(128, 2, 4)
  } else {
    AXON_GV(8, 16, 2, 1) AXON_GV(8, 8, 8, 1) AXON_GV(16, 8, 4, 1) AXON_GV(16, 16, 4, 1) AXON_GV(32, 8, 4, 1)
  }
#undef AXON_GVW
#undef AXON_GV
  return false;
}

// split K: partial sums (grid N/rows x ksplit, normalized when NORM) then the
// epilogue kernel; a timed launch starts its events with the first kernel
// and stops with the second
template <int RB, int U, int NB, bool NORM, int EPI>
static bool gv_split(const GemvArgs& a, const GvShape& sh, hipStream_t s) {
  auto k1 = gemv_wide_kernel<RB, NB, NORM, GV_PART, U>;
  const bool rows = EPI == GV_RESID && sh.erows == GV_RESID_ROWS;
  constexpr int ER = EPI == GV_SILU ? 32 : 16;  // the SiLU epilogue pairs 16 gate and 16 up rows
  if (!rows && sh.erows != ER) return false;
  auto k2 = rows ? gemv_split_resid_kernel : gemv_split_epilogue_kernel<ER, NB, EPI>;
  const dim3 g1((a.N + 64 * RB - 1) / (64 * RB), sh.ksplit);
  const dim3 g2 = rows ? dim3((a.N + GV_RESID_ROWS - 1) / GV_RESID_ROWS, a.M) : dim3((a.N + ER - 1) / ER);
  const TimingSlot t = g_timing_slot;
  g_timing_slot = TimingSlot{};
  if (t.start) {
    hipExtLaunchKernelGGL(k1, g1, dim3(256), 0, s, t.start, nullptr, 0, a);
    hipExtLaunchKernelGGL(k2, g2, dim3(256), 0, s, nullptr, t.stop, 0, a, sh.ksplit);
  } else {
    k1<<<g1, 256, 0, s>>>(a);
    k2<<<g2, 256, 0, s>>>(a, sh.ksplit);
  }
  return true;
}

template <int EPI, bool NORM>
static bool gv_split_nb(const GemvArgs& a, const GvShape& sh, int nb, hipStream_t s) {
  if (!sh.wide || !a.part) return false;
#define AXON_GVS(R, U_, NB_) \
  if (sh.rows == R && sh.u == U_ && nb == NB_) return gv_split<R / 64, U_, NB_, NORM, EPI>(a, sh, s);
  if constexpr (EPI == GV_F32) {
    AXON_GVS(64, 4, 1) AXON_GVS(64, 2, 2) AXON_GVS(64, 4, 3) AXON_GVS(64, 4, 4)
  } else if constexpr (EPI == GV_SILU || EPI == GV_GELU) {
    AXON_GVS(64, 2, 2) AXON_GVS(64, 4, 3) AXON_GVS(64, 4, 4)
  } else {
    AXON_GVS(64, 2, 2) AXON_GVS(64, 4, 3) AXON_GVS(64, 4, 4)
    AXON_GVS(128, 4, 2) AXON_GVS(128, 4, 3) AXON_GVS(128, 4, 4)
  }
#undef AXON_GVS
  return false;
}

bool launch_gemv_fused(const GemvArgs& a, int epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return true;
  if (a.M > 64) return false;
  const GvShape sh = gemv_shape(a.N, a.K, a.M, epi);
  const int nb = (a.M + 15) / 16;
  const bool norm = a.ss_in != nullptr;
  // the tile order serves the unsplit one-block kernel only
  if ((a.x_tiled || a.out_tiled) && (a.M > XT_ROWS || sh.wide || sh.ksplit > 1 || epi == GV_F32)) return false;
  if (a.out_tiled && epi != GV_RESID && epi != GV_SILU) return false;
  if (sh.ksplit > 1) {
    if (epi == GV_RESID) return !norm && gv_split_nb<GV_RESID, false>(a, sh, nb, s);
    if (epi == GV_ROPE) return norm ? gv_split_nb<GV_ROPE, true>(a, sh, nb, s) : gv_split_nb<GV_ROPE, false>(a, sh, nb, s);
    if (epi == GV_SILU) return norm && gv_split_nb<GV_SILU, true>(a, sh, nb, s);
    if (epi == GV_GELU) return !norm && a.bias && gv_split_nb<GV_GELU, false>(a, sh, nb, s);
    if (epi == GV_F32) return !norm && gv_split_nb<GV_F32, false>(a, sh, nb, s);
    return false;
  }
  switch (epi) {
    case GV_SILU: return norm && gv_dispatch<GV_SILU, true>(a, sh, nb, s);
    case GV_ROPE: return norm ? gv_dispatch<GV_ROPE, true>(a, sh, nb, s) : gv_dispatch<GV_ROPE, false>(a, sh, nb, s);
    case GV_GELU: return !norm && a.bias && gv_dispatch<GV_GELU, false>(a, sh, nb, s);
    case GV_RESID: return !norm && gv_dispatch<GV_RESID, false>(a, sh, nb, s);
    case GV_HEAD: return norm ? gv_dispatch<GV_HEAD, true>(a, sh, nb, s) : gv_dispatch<GV_HEAD, false>(a, sh, nb, s);
    case GV_F32:  // float rows out (router logits): 64-row workgroups
      if (norm) return false;
      if (nb == 1) return gvw<1, 4, 1, false, GV_F32>(a, s);
      if (nb == 2) return gvw<1, 2, 2, false, GV_F32>(a, s);
      if (nb == 3) return gvw<1, 4, 3, false, GV_F32>(a, s);
      return gvw<1, 2, 4, false, GV_F32>(a, s);
    default: return false;
  }
}

template <int NB, int EPI>
static void grouped_launch(const GemvArgs& a, int n_experts, hipStream_t s) {
  // 64-row workgroups, 4 k-steps per stage (measured on the DeepSeek-MoE-16B
  // shape at 32 tokens: 5.48 TB/s; 2 k-steps 5.38, 128-row workgroups 5.32)
  constexpr int U = 4;
  klaunch(gemv_wide_kernel<1, NB, false, EPI, U, true>, dim3((a.N + 63) / 64, n_experts), dim3(256), 0, s, a);
}

bool launch_gemv_grouped(const GemvArgs& a, int epi, int n_experts, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0 || n_experts <= 0) return true;
  if (a.M > 64 || (epi != GV_SILU && epi != GV_F32)) return false;
  const int nb = (a.M + 15) / 16;
  if (epi == GV_SILU) {
    if (nb == 1) grouped_launch<1, GV_SILU>(a, n_experts, s);
    else if (nb == 2) grouped_launch<2, GV_SILU>(a, n_experts, s);
    else if (nb == 3) grouped_launch<3, GV_SILU>(a, n_experts, s);
    else grouped_launch<4, GV_SILU>(a, n_experts, s);
  } else {
    if (nb == 1) grouped_launch<1, GV_F32>(a, n_experts, s);
    else if (nb == 2) grouped_launch<2, GV_F32>(a, n_experts, s);
    else if (nb == 3) grouped_launch<3, GV_F32>(a, n_experts, s);
    else grouped_launch<4, GV_F32>(a, n_experts, s);
  }
  return true;
}

void launch_argmax_final(const float* val, const int32_t* idx, int nparts, int M, int32_t* next, int32_t* len,
                         hipStream_t s) {
  if (M <= 0) return;
  argmax_final_kernel<<<M, 1024, 0, s>>>(val, idx, nparts, next, len);
}

void launch_embed_ss(const int32_t* tok, const bf16* emb, const bf16* g, float* x, bf16* xg, float* ss_out, int M,
                     int D, int V, hipStream_t s, bool xg_tiled) {
  if (M <= 0) return;
  embed_ss_kernel<<<M, 256, 0, s>>>(tok, emb, g, x, xg, ss_out, D, V, xg_tiled);
}

}  // namespace axon
