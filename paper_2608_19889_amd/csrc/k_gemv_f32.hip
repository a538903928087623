// Few-token projections of the float32 models (float weights, up to 16
// tokens): the float32 counterpart of the fused decode projections of
// k_gemv.hip, so that a float32 decode step is 5 kernels per layer instead of
// separate projection, normalization, rotation and SiLU kernels.
//
// A workgroup owns 8 output rows; each of its 4 wavefronts computes two of
// them for every token, lanes along K (16-byte loads of the row-major weight
// rows and of the token rows), with compensated (Kahan) float32 sums per lane
// and a butterfly sum across the wavefront, so the error does not grow with
// K.  The two rows of a wavefront are chosen by the epilogue:
//   GV_ROPE  rotation pair: an 8-row group of the permuted QKV rows holds 4
//            first halves and their partners, wavefront w takes rows w and
//            w + 4 of the group
//   GV_SILU  gate row f and its up row f + 16 (gate/up interleaved in blocks
//            of 16 rows), wavefront w of workgroup g: f = 16 (g / 4) + 4 (g % 4) + w
//   GV_RESID, GV_HEAD  rows 2w and 2w + 1 of the tile
// Normalized operand (NORM): X holds x * g and the sums are scaled by
// rsqrt(sum of squares / K + eps) of the token, from the per-workgroup
// partial sums of squares the producer of x wrote.
#include "common.h"
#include "kernels.h"

namespace axon {

AXON_DEV float silu_f32(float z) { return z / (1.f + expf(-z)); }

// row r of the workgroup's tile (0..7) -> matrix row
template <int EPI>
AXON_DEV int f32_tile_row(int wg, int r) {
  const int w = r >> 1, second = r & 1;
  if constexpr (EPI == GV_ROPE) return 8 * wg + w + 4 * second;
  else if constexpr (EPI == GV_SILU) return 32 * (wg >> 2) + 4 * (wg & 3) + w + 16 * second;
  else return 8 * wg + r;
}

template <int MT, bool NORM, int EPI>
__global__ void __launch_bounds__(256) gemv_f32_fused_kernel(GemvF32Args a) {
  constexpr int UK = MT >= 8 ? 1 : MT >= 4 ? 2 : 4;  // 16-byte chunks per lane in flight per operand row
  __shared__ float s_tot[8][MT];
  __shared__ float s_aux[8][MT];
  __shared__ float s_ss[256];
  __shared__ float s_inv[MT];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wg = blockIdx.x, M = a.M, K = a.K;
  const int n0 = f32_tile_row<EPI>(wg, 2 * w), n1 = f32_tile_row<EPI>(wg, 2 * w + 1);
  const float* w0 = a.W + (int64_t)min(n0, a.N - 1) * K;
  const float* w1 = a.W + (int64_t)min(n1, a.N - 1) * K;

  // partial sums of squares of the normalized rows: thread (slice, token)
  // adds partials slice, slice + nsl, ... (loaded ahead of the stream)
  const int nsl = NORM ? max(1, min(256 / M, a.ss_n)) : 1;
  const int ss_t = tid % M, ss_s = tid / M;
  float ss_part = 0.f;
  if constexpr (NORM) {
    if (ss_s < nsl)
      for (int j = ss_s; j < a.ss_n; j += nsl) ss_part += a.ss_in[(int64_t)j * M + ss_t];
  }

  float acc0[MT], cmp0[MT], acc1[MT], cmp1[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc0[t] = cmp0[t] = acc1[t] = cmp1[t] = 0.f;
  // s + w x with the rounding error of the sum carried in c (the true sum is s - c)
  auto kahan = [](float& s, float& c, float wv, float x) {
    const float y = fmaf(wv, x, -c);
    const float u = s + y;
    c = (u - s) - y;
    s = u;
  };
  for (int kb = lane * 4; kb < K; kb += 256 * UK) {
    f32x4 wv0[UK], wv1[UK], xv[UK][MT];
#pragma unroll
    for (int u = 0; u < UK; ++u) {
      const int k = min(kb + u * 256, K - 4);  // past K: any valid chunk, zeroed at use
      wv0[u] = *(const f32x4*)(w0 + k);
      wv1[u] = *(const f32x4*)(w1 + k);
#pragma unroll
      for (int t = 0; t < MT; ++t) xv[u][t] = *(const f32x4*)(a.X + (int64_t)min(t, M - 1) * K + k);
    }
#pragma unroll
    for (int u = 0; u < UK; ++u) {
      const bool ok = kb + u * 256 < K;
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float x = ok ? xv[u][t][j] : 0.f;
          kahan(acc0[t], cmp0[t], wv0[u][j], x);
          kahan(acc1[t], cmp1[t], wv1[u][j], x);
        }
    }
  }
  // wavefront sums (every lane gets them); lane 0 files them
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const float v0 = wave_sum(acc0[t] - cmp0[t]), v1 = wave_sum(acc1[t] - cmp1[t]);
    if (lane == 0) {
      s_tot[2 * w][t] = v0;
      s_tot[2 * w + 1][t] = v1;
    }
  }
  if constexpr (NORM) s_ss[tid] = ss_part;
  __syncthreads();
  if constexpr (NORM) {
    if (tid < M) {
      float tot = 0.f;
      for (int sl = 0; sl < nsl; ++sl) tot += s_ss[sl * M + tid];
      s_inv[tid] = rsqrtf(tot / (float)K + a.eps);
    }
    __syncthreads();
  }
  auto total = [&](int r, int t) { return NORM ? s_tot[r][t] * s_inv[t] : s_tot[r][t]; };

  if constexpr (EPI == GV_RESID) {
    // x[t][n] += total; xg = x * g_next; one sum of squares per (workgroup, token)
    if (tid < 8 * M) {
      const int r = tid % 8, t = tid / 8, n = 8 * wg + r;
      float sq = 0.f;
      if (n < a.N) {
        float* p = a.out + (int64_t)t * a.ldo + n;
        const float v = *p + total(r, t);
        *p = v;
        sq = v * v;
        if (a.xg_out) a.xg_out[(int64_t)t * a.ldo + n] = v * a.gain_next[n];
      }
      s_aux[r][t] = sq;
    }
    __syncthreads();
    if (tid < M && a.ss_out) {
      float s = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) s += s_aux[r][tid];
      a.ss_out[(int64_t)wg * M + tid] = s;
    }
  } else if constexpr (EPI == GV_SILU) {
    if (tid < 4 * M) {
      const int j = tid % 4, t = tid / 4;
      const int f = 16 * (wg >> 2) + 4 * (wg & 3) + j;  // gate row 32 (wg / 4) + 4 (wg % 4) + j
      if (2 * f < a.N) a.out[(int64_t)t * a.ldo + f] = silu_f32(total(2 * j, t)) * total(2 * j + 1, t);
    }
  } else if constexpr (EPI == GV_ROPE) {
    if (tid < 4 * M) {
      const int j = tid % 4, t = tid / 4;
      const int hd = a.kv.hd, half = hd / 2, KVh = a.kv.kv_heads;
      const int nf = 8 * wg + j;  // first-half row; its partner is nf + 4
      const int head = nf / hd, i = ((nf % hd) / 8) * 4 + j;
      float x1 = total(2 * j, t), x2 = total(2 * j + 1, t);
      if (a.bias) {
        x1 += a.bias[head * hd + i];
        x2 += a.bias[head * hd + half + i];
      }
      const int pos = a.len[t];
      const int sl = a.slot ? a.slot[t] : t;
      if (head < a.H + KVh) {
        const float cs = a.cos_t[(int64_t)pos * half + i], sn = a.sin_t[(int64_t)pos * half + i];
        const float y1 = x1 * cs - x2 * sn, y2 = x2 * cs + x1 * sn;
        if (head < a.H) {
          float* dst = a.q_out + ((int64_t)t * a.H + head) * hd;
          dst[i] = y1;
          dst[i + half] = y2;
        } else {
          float* kc = (float*)a.kv.k;
          kc[k_el(a.kv, sl, head - a.H, pos, i)] = y1;
          kc[k_el(a.kv, sl, head - a.H, pos, i + half)] = y2;
        }
      } else {
        float* vc = (float*)a.kv.v;
        vc[v_el(a.kv, sl, head - a.H - KVh, pos, i)] = x1;
        vc[v_el(a.kv, sl, head - a.H - KVh, pos, i + half)] = x2;
      }
    }
  } else {  // GV_HEAD: logits and, per token, the tile's largest logit and its lowest index
    if (tid < 8 * M) {
      const int r = tid % 8, t = tid / 8, n = 8 * wg + r;
      float v = -INFINITY;
      if (n < a.N) {
        v = total(r, t);
        if (a.out) a.out[(int64_t)t * a.ldo + n] = v;
      }
      s_aux[r][t] = v;
    }
    __syncthreads();
    if (tid < M) {
      float best = -INFINITY;
      int bi = 0x7fffffff;
      for (int r = 0; r < 8; ++r)
        if (s_aux[r][tid] > best) {
          best = s_aux[r][tid];
          bi = 8 * wg + r;
        }
      a.am_val[(int64_t)tid * gridDim.x + wg] = best;
      a.am_idx[(int64_t)tid * gridDim.x + wg] = bi;
    }
  }
}

// ============================================================================
// Short-context decode: attention fused into the O projection.  Every
// workgroup first computes the attention output of all tokens and heads
// itself, into LDS (a wavefront per (token, kv head) item: the item's query
// heads scored against 64 keys at a time, online softmax per head, P V with
// lane d owning output dimension d), then runs the residual O projection on it
// as gemv_f32_fused_kernel<., false, GV_RESID> does.  This repeats the
// attention in every workgroup, which is cheap only while contexts and the
// model are small (the launcher's caller checks); it saves the attention
// kernel and one memory round trip per layer.  The first weight stage of the
// projection is loaded before the attention, behind its loads.
// ============================================================================
constexpr int AO_MAXG = 8;
constexpr float AO_LOG2E = 1.4426950408889634f;

template <int MT, int HD>
__global__ void __launch_bounds__(256) attn_o_f32_kernel(GemvF32Args a, const float* __restrict__ q, KVView kv) {
  constexpr int UK = MT >= 8 ? 1 : MT >= 4 ? 2 : 4;
  constexpr int DL = HD / 64;
  extern __shared__ float xo[];  // [M][H * HD]: the attention output, the projection's operand
  __shared__ float qs[4][AO_MAXG][HD];
  __shared__ f32x4 ps[4][AO_MAXG][16];
  __shared__ float sm[4][AO_MAXG], sl[4][AO_MAXG], sa[4][AO_MAXG];
  __shared__ float so[4][AO_MAXG][HD];
  __shared__ float s_tot[8][MT];
  __shared__ float s_aux[8][MT];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wg = blockIdx.x, M = a.M, K = a.K, H = a.H;
  const int n0 = 8 * wg + 2 * w, n1 = n0 + 1;
  const float* w0 = a.W + (int64_t)min(n0, a.N - 1) * K;
  const float* w1 = a.W + (int64_t)min(n1, a.N - 1) * K;
  // first weight stage (k chunks lane*4 + 256 u)
  f32x4 wv0[UK], wv1[UK];
#pragma unroll
  for (int u = 0; u < UK; ++u) {
    const int k = min(lane * 4 + u * 256, K - 4);
    wv0[u] = *(const f32x4*)(w0 + k);
    wv1[u] = *(const f32x4*)(w1 + k);
  }

  // ---- attention: item (t, kvh) = (it / KVh, it % KVh), wavefront it % 4
  const int KVh = kv.kv_heads, G = H / KVh;
  const float sc = AO_LOG2E / sqrtf((float)HD);
  const float* kb = (const float*)kv.k;
  const float* vb = (const float*)kv.v;
  for (int it = w; it < M * KVh; it += 4) {
    const int t = it / KVh, kvh = it % KVh;
    const int pos = a.len[t], slot = a.slot ? a.slot[t] : t;
    const int lo = kv.window ? max(0, pos - kv.window + 1) : 0;
    for (int i = lane; i < G * HD; i += 64) {
      qs[w][i / HD][i % HD] = q[((int64_t)t * H + kvh * G) * HD + i];
      so[w][i / HD][i % HD] = 0.f;
    }
    if (lane < G) {
      sm[w][lane] = -INFINITY;
      sl[w][lane] = 0.f;
    }
    for (int j0 = lo & ~63; j0 <= pos; j0 += 64) {
      const int j = j0 + lane;
      const bool valid = j >= lo && j <= pos;
      f32x4 kr[HD / 4];
      const float* kp = kb + k_el(kv, slot, kvh, min(max(j, lo), pos), 0);
#pragma unroll
      for (int d = 0; d < HD / 4; ++d) kr[d] = *(const f32x4*)(kp + (d >> 1) * 128 + (d & 1) * 4);
      f32x4 vr[DL][16];
#pragma unroll
      for (int i = 0; i < DL; ++i)
#pragma unroll
        for (int blk = 0; blk < 4; ++blk) {
          const float* vp = vb + v_el(kv, slot, kvh, min(j0 + blk * 16, pos & ~15), lane + 64 * i);
#pragma unroll
          for (int c = 0; c < 4; ++c) vr[i][blk * 4 + c] = *(const f32x4*)(vp + c * 4);
        }
      for (int h = 0; h < G; ++h) {
        float dot = 0.f;
#pragma unroll
        for (int d = 0; d < HD / 4; ++d) {
          dot = fmaf(qs[w][h][4 * d], kr[d][0], dot);
          dot = fmaf(qs[w][h][4 * d + 1], kr[d][1], dot);
          dot = fmaf(qs[w][h][4 * d + 2], kr[d][2], dot);
          dot = fmaf(qs[w][h][4 * d + 3], kr[d][3], dot);
        }
        const float s = valid ? dot * sc : -INFINITY;
        const float m_old = sm[w][h];
        const float m_new = fmaxf(m_old, wave_max(s));  // finite: the chunk holds a key in [lo, pos]
        const float alpha = exp2f(m_old - m_new);
        const float p = valid ? exp2f(s - m_new) : 0.f;
        const float lsum = wave_sum(p);
        ((float*)ps[w][h])[lane] = p;
        if (lane == 0) {
          sl[w][h] = sl[w][h] * alpha + lsum;
          sm[w][h] = m_new;
          sa[w][h] = alpha;
        }
      }
#pragma unroll
      for (int i = 0; i < DL; ++i)
        for (int h = 0; h < G; ++h) {
          float acc = so[w][h][lane + 64 * i] * sa[w][h];
#pragma unroll
          for (int c = 0; c < 16; ++c) {
            const f32x4 pv = ps[w][h][c];
            acc = fmaf(pv[0], vr[i][c][0], acc);
            acc = fmaf(pv[1], vr[i][c][1], acc);
            acc = fmaf(pv[2], vr[i][c][2], acc);
            acc = fmaf(pv[3], vr[i][c][3], acc);
          }
          so[w][h][lane + 64 * i] = acc;
        }
    }
    for (int i = lane; i < G * HD; i += 64)
      xo[t * K + (kvh * G + i / HD) * HD + i % HD] = so[w][i / HD][i % HD] / sl[w][i / HD];
  }
  __syncthreads();

  // ---- residual O projection over the LDS operand
  float acc0[MT], cmp0[MT], acc1[MT], cmp1[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc0[t] = cmp0[t] = acc1[t] = cmp1[t] = 0.f;
  for (int kb0 = lane * 4; kb0 < K; kb0 += 256 * UK) {
    if (kb0 != lane * 4) {
#pragma unroll
      for (int u = 0; u < UK; ++u) {
        const int k = min(kb0 + u * 256, K - 4);
        wv0[u] = *(const f32x4*)(w0 + k);
        wv1[u] = *(const f32x4*)(w1 + k);
      }
    }
#pragma unroll
    for (int u = 0; u < UK; ++u) {
      const int k = kb0 + u * 256;
      if (k >= K) break;
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const f32x4 x = *(const f32x4*)(xo + min(t, M - 1) * K + k);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float y = fmaf(wv0[u][j], x[j], -cmp0[t]);
          float s = acc0[t] + y;
          cmp0[t] = (s - acc0[t]) - y;
          acc0[t] = s;
          y = fmaf(wv1[u][j], x[j], -cmp1[t]);
          s = acc1[t] + y;
          cmp1[t] = (s - acc1[t]) - y;
          acc1[t] = s;
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const float v0 = wave_sum(acc0[t] - cmp0[t]), v1 = wave_sum(acc1[t] - cmp1[t]);
    if (lane == 0) {
      s_tot[2 * w][t] = v0;
      s_tot[2 * w + 1][t] = v1;
    }
  }
  __syncthreads();
  if (tid < 8 * M) {
    const int r = tid % 8, t = tid / 8, n = 8 * wg + r;
    float sq = 0.f;
    if (n < a.N) {
      float* p = a.out + (int64_t)t * a.ldo + n;
      const float v = *p + s_tot[r][t];
      *p = v;
      sq = v * v;
      if (a.xg_out) a.xg_out[(int64_t)t * a.ldo + n] = v * a.gain_next[n];
    }
    s_aux[r][t] = sq;
  }
  __syncthreads();
  if (tid < M && a.ss_out) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) s += s_aux[r][tid];
    a.ss_out[(int64_t)wg * M + tid] = s;
  }
}

bool attn_o_f32_fits(int M, int H, int KVh, int hd, int max_ctx) {
  return M >= 1 && M <= 4 && (hd == 64 || hd == 128) && H % KVh == 0 && H / KVh <= AO_MAXG &&
         (int64_t)M * H * hd * 4 <= 16384 && max_ctx <= 128;
}

template <int MT, int HD>
static void ao_launch(const GemvF32Args& a, const float* q, KVView kv, hipStream_t s) {
  const size_t lds = (size_t)a.M * a.K * sizeof(float);
  klaunch(attn_o_f32_kernel<MT, HD>, dim3((a.N + 7) / 8), dim3(256), (uint32_t)lds, s, a, q, kv);
}

bool launch_attn_o_f32(const GemvF32Args& a, const float* q, KVView kv, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return true;
  if (a.ss_in || a.K != a.H * kv.hd || a.K % 4 != 0) return false;
  if (!attn_o_f32_fits(a.M, a.H, kv.kv_heads, kv.hd, 0)) return false;
  if (kv.hd == 64) {
    if (a.M == 1) ao_launch<1, 64>(a, q, kv, s);
    else if (a.M <= 2) ao_launch<2, 64>(a, q, kv, s);
    else ao_launch<4, 64>(a, q, kv, s);
  } else {
    if (a.M == 1) ao_launch<1, 128>(a, q, kv, s);
    else if (a.M <= 2) ao_launch<2, 128>(a, q, kv, s);
    else ao_launch<4, 128>(a, q, kv, s);
  }
  return true;
}

// x[t] = E[tok[t]], xg[t] = x[t] * g, ss_out[t] = sum of squares of the row
// (the first projection's single partial)
__global__ void __launch_bounds__(256) embed_ss_f32_kernel(const int32_t* __restrict__ tok,
                                                           const float* __restrict__ emb, const float* __restrict__ g,
                                                           float* __restrict__ x, float* __restrict__ xg,
                                                           float* __restrict__ ss_out, int D, int V, int M) {
  __shared__ float red[16];
  const int t = blockIdx.x;
  const int id = min(max(tok[t], 0), V - 1);
  const float* e = emb + (int64_t)id * D;
  float sq = 0.f;
  for (int k = threadIdx.x; k < D; k += 256) {
    const float v = e[k];
    x[(int64_t)t * D + k] = v;
    xg[(int64_t)t * D + k] = v * g[k];
    sq += v * v;
  }
  sq = block_sum(sq, red);
  if (threadIdx.x == 0) ss_out[t] = sq;  // partial 0 of token t ([1][M])
}

template <int MT, bool NORM, int EPI>
static void f32_launch(const GemvF32Args& a, hipStream_t s) {
  const int nwg = EPI == GV_SILU ? (a.N + 31) / 32 * 4 : (a.N + 7) / 8;
  klaunch(gemv_f32_fused_kernel<MT, NORM, EPI>, dim3(nwg), dim3(256), 0, s, a);
}

template <int MT>
static bool f32_dispatch(const GemvF32Args& a, int epi, hipStream_t s) {
  const bool norm = a.ss_in != nullptr;
  switch (epi) {
    case GV_ROPE:
      if (!norm) return false;
      f32_launch<MT, true, GV_ROPE>(a, s);
      return true;
    case GV_SILU:
      if (!norm) return false;
      f32_launch<MT, true, GV_SILU>(a, s);
      return true;
    case GV_RESID:
      if (norm) return false;
      f32_launch<MT, false, GV_RESID>(a, s);
      return true;
    case GV_HEAD:
      if (!norm) return false;
      f32_launch<MT, true, GV_HEAD>(a, s);
      return true;
    default:
      return false;
  }
}

bool launch_gemv_f32_fused(const GemvF32Args& a, int epi, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return true;
  if (a.M > GEMV_F32_MAX_M || a.K % 4 != 0) return false;
  if (epi == GV_SILU && a.N % 32 != 0) return false;
  if (epi == GV_ROPE && (a.N % 8 != 0 || a.kv.hd % 8 != 0)) return false;
  if (a.M == 1) return f32_dispatch<1>(a, epi, s);
  if (a.M <= 2) return f32_dispatch<2>(a, epi, s);
  if (a.M <= 4) return f32_dispatch<4>(a, epi, s);
  if (a.M <= 8) return f32_dispatch<8>(a, epi, s);
  return f32_dispatch<16>(a, epi, s);
}

int gemv_f32_parts(int N, int epi) { return epi == GV_SILU ? (N + 31) / 32 * 4 : (N + 7) / 8; }

void launch_embed_ss_f32(const int32_t* tok, const float* emb, const float* g, float* x, float* xg, float* ss_out,
                         int M, int D, int V, hipStream_t s) {
  if (M <= 0) return;
  embed_ss_f32_kernel<<<M, 256, 0, s>>>(tok, emb, g, x, xg, ss_out, D, V, M);
}

}  // namespace axon
