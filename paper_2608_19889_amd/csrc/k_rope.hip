// Bias + rotary position embedding + KV-cache write.
//
// The projection output row of a token holds H query heads, then KV key
// heads, then KV value heads (head_dim each); within a head the columns come
// in groups of 8 = 4 first-half elements i and their rotation partners
// i + hd/2 (qkv_col below), the row order the fused decode projection needs.  Queries and keys are rotated by
// their absolute position with rotate-half pairing (element i with i + hd/2,
// angle pos * theta^(-2i/hd), cos/sin read from a float table built in double
// precision on the host); queries go to q_out [T][H][hd], keys to the K pages,
// values (unrotated) to the transposed V pages.
#include "common.h"
#include "kernels.h"

namespace axon {

constexpr int ROPE_TT = 16;  // tokens per workgroup

AXON_DEV void token_slot_pos(int t, int nseq, const int32_t* __restrict__ cu, const int32_t* __restrict__ len,
                             const int32_t* __restrict__ ent_slot, const int32_t* __restrict__ ent_base, int& slot,
                             int& pos) {
  if (len) {
    slot = t;
    pos = len[t];
  } else {
    const int e = seq_of_token(cu, nseq, t);
    slot = ent_slot ? ent_slot[e] : e;
    pos = (ent_base ? ent_base[e] : 0) + t - cu[e];
  }
}

// column of element j of head h in the permuted projection output
template <int HD>
AXON_DEV int qkv_col(int h, int j) {
  constexpr int HALF = HD / 2;
  const int jj = j < HALF ? j : j - HALF;
  return h * HD + (jj / 4) * 8 + (j < HALF ? 0 : 4) + jj % 4;
}

template <typename T, int HD>
__global__ void __launch_bounds__(256) rope_kv_kernel(const float* __restrict__ parts, int nparts, int64_t pstride,
                                                      const T* __restrict__ bias, const float* __restrict__ cos_t,
                                                      const float* __restrict__ sin_t, T* __restrict__ q_out,
                                                      KVView kv, int T_tokens, int nseq,
                                                      const int32_t* __restrict__ cu,
                                                      const int32_t* __restrict__ len, int H,
                                                      const int32_t* __restrict__ ent_slot,
                                                      const int32_t* __restrict__ ent_base) {
  __shared__ float vt[ROPE_TT][HD + 1];
  const int KVh = kv.kv_heads;
  const int nqkv = (H + 2 * KVh) * HD;
  const int t0 = blockIdx.x * ROPE_TT;
  const int head = blockIdx.y;
  const int off = head * HD;
  // element j of this head for token t (bias indexed in the original order)
  auto val = [&](int t, int j) {
    const float* p = parts + (int64_t)t * nqkv + qkv_col<HD>(head, j);
    float v = 0.f;
    for (int s = 0; s < nparts; ++s) v += p[s * pstride];
    if (bias) v += to_f32(bias[off + j]);
    return v;
  };
  if (head < H + KVh) {
    constexpr int HALF = HD / 2;
    for (int idx = threadIdx.x; idx < ROPE_TT * HALF; idx += blockDim.x) {
      const int t = t0 + idx / HALF, i = idx % HALF;
      if (t >= T_tokens) continue;
      int slot, pos;
      token_slot_pos(t, nseq, cu, len, ent_slot, ent_base, slot, pos);
      const float x1 = val(t, i), x2 = val(t, i + HALF);
      const float c = cos_t[(int64_t)pos * HALF + i], s = sin_t[(int64_t)pos * HALF + i];
      const float y1 = x1 * c - x2 * s, y2 = x2 * c + x1 * s;
      if (head < H) {
        T* dst = q_out + ((int64_t)t * H + head) * HD;
        dst[i] = from_f32<T>(y1);
        dst[i + HALF] = from_f32<T>(y2);
      } else {
        T* kc = (T*)kv.k;
        kc[k_el(kv, slot, head - H, pos, i)] = from_f32<T>(y1);
        kc[k_el(kv, slot, head - H, pos, i + HALF)] = from_f32<T>(y2);
      }
    }
  } else {
    const int kvh = head - H - KVh;
    for (int idx = threadIdx.x; idx < ROPE_TT * HD; idx += blockDim.x) {
      const int tt = idx / HD, d = idx % HD;
      if (t0 + tt < T_tokens) vt[tt][d] = val(t0 + tt, d);
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < ROPE_TT * HD; idx += blockDim.x) {
      const int d = idx / ROPE_TT, tt = idx % ROPE_TT;
      const int t = t0 + tt;
      if (t >= T_tokens) continue;
      int slot, pos;
      token_slot_pos(t, nseq, cu, len, ent_slot, ent_base, slot, pos);
      ((T*)kv.v)[v_el(kv, slot, kvh, pos, d)] = from_f32<T>(vt[tt][d]);
    }
  }
}

template <typename T>
void launch_rope_kv(const float* parts, int nparts, int64_t part_stride, const T* bias, const float* cos_t,
                    const float* sin_t, T* q_out, KVView kv, int T_tokens, int nseq, const int32_t* cu,
                    const int32_t* len, int H, hipStream_t s, const int32_t* ent_slot, const int32_t* ent_base) {
  if (T_tokens <= 0) return;
  dim3 grid((T_tokens + ROPE_TT - 1) / ROPE_TT, H + 2 * kv.kv_heads);
  if (kv.hd == 64)
    rope_kv_kernel<T, 64><<<grid, 256, 0, s>>>(parts, nparts, part_stride, bias, cos_t, sin_t, q_out, kv,
                                               T_tokens, nseq, cu, len, H, ent_slot, ent_base);
  else
    rope_kv_kernel<T, 128><<<grid, 256, 0, s>>>(parts, nparts, part_stride, bias, cos_t, sin_t, q_out, kv,
                                                T_tokens, nseq, cu, len, H, ent_slot, ent_base);
}

template void launch_rope_kv<float>(const float*, int, int64_t, const float*, const float*, const float*, float*,
                                    KVView, int, int, const int32_t*, const int32_t*, int, hipStream_t,
                                    const int32_t*, const int32_t*);
template void launch_rope_kv<bf16>(const float*, int, int64_t, const bf16*, const float*, const float*, bf16*,
                                   KVView, int, int, const int32_t*, const int32_t*, int, hipStream_t,
                                   const int32_t*, const int32_t*);

}  // namespace axon
