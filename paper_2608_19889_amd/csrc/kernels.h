// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on the
// given stream and returns immediately; shapes are validated by the caller.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace axon {

// Epilogues of the projection GEMMs (out[t][n] = sum_k X[t][k] * W[n][k]).
enum Epi : int {
  EPI_F32 = 0,    // out_f32[t * ldo + n] = acc
  EPI_RESID = 1,  // out_f32[t * ldo + n] += acc   (residual stream, float)
  EPI_SILU = 2,   // W rows interleaved in blocks of 16 gate rows then 16 up rows;
                  // out_t[t * ldo + f] = silu(gate_f) * up_f
  EPI_PART = 3    // out_f32[split * part_stride + t * ldo + n] = acc (split-K partial)
};

struct EpiArgs {
  float* out_f32;
  void* out_t;
  int ldo;
  int64_t part_stride;
};

// ---- row kernels (k_norm.hip)
template <typename T>
void launch_embed_rmsnorm(const int32_t* tok, const T* emb, const T* g, float* x, T* h, int rows, int D, int V,
                          float eps, hipStream_t s);
template <typename T>
void launch_resid_rmsnorm(float* x, const float* parts, int nparts, int64_t part_stride, const T* g, T* h,
                          int rows, int D, float eps, const int32_t* cu_last, hipStream_t s);
void launch_argmax(const float* logits, int rows, int V, int32_t* next, int32_t* len, hipStream_t s);
// argmax of row cu[i+1]-1 for each sequence i
void launch_argmax_rows(const float* logits, int nseq, int V, int32_t* next, const int32_t* cu, hipStream_t s);
void launch_set_lengths(const int32_t* cu, int32_t* len, int n, hipStream_t s);

// ---- projections (k_gemm.hip)
// Many-token GEMM (prefill): bf16 MFMA tiles.  Requires K % 64 == 0, N % 32 == 0.
void launch_gemm_bf16(const bf16* W, const bf16* X, int N, int M, int K, int epi, const EpiArgs& ep,
                      hipStream_t s);
// Few-token GEMM (decode, M <= 64): streams W once.  Returns the number of
// K splits used (> 1 means EPI_PART partials were written to ep.out_f32 with
// stride ep.part_stride, and the caller's reduction applies the epilogue).
int plan_gemv_splits(int N, int M, int K);
void launch_gemv_bf16(const bf16* W, const bf16* X, int N, int M, int K, int splits, int epi,
                      const EpiArgs& ep, hipStream_t s);
// float32 check-mode GEMM (any M): EPI_F32 / EPI_RESID / EPI_PART(split 0 only).
void launch_gemm_f32(const float* W, const float* X, int N, int M, int K, int epi, const EpiArgs& ep,
                     hipStream_t s);
// a[t][f] = silu(sum_s gate) * sum_s up over split-K partials of the
// interleaved gate/up projection ([nparts][M][2I] floats).
template <typename T>
void launch_silu_reduce(const float* parts, int nparts, int64_t part_stride, T* a, int M, int I,
                        hipStream_t s);
// out[t][n] = sum_s parts[s][t][n]
void launch_sum_reduce(const float* parts, int nparts, int64_t part_stride, float* out, int M, int N,
                       hipStream_t s);

// ---- bias + rotary + KV-cache write (k_rope.hip)
// qkv rows are sum_s parts[s][t][:] (+ bias): q heads, then k heads, then v heads.
// Token t belongs to sequence seq(t) at position pos(t): prefill uses cu
// (positions restart at 0 per sequence), decode (len != nullptr) uses slot t at
// position len[t].
template <typename T>
void launch_rope_kv(const float* parts, int nparts, int64_t part_stride, const T* bias, const float* cos_t,
                    const float* sin_t, T* q_out, KVView kv, int T_tokens, int nseq, const int32_t* cu,
                    const int32_t* len, int H, hipStream_t s);

// ---- attention (k_attn.hip)
// Causal prefill attention over the cache; o [T][H*hd].
template <typename T>
void launch_attn_prefill(const T* q, KVView kv, T* o, int T_tokens, int nseq, const int32_t* cu,
                         const int32_t* h_cu, int H, hipStream_t s);
// Decode attention: one query per slot at position len[b] (after the step's
// key/value were written), context len[b] + 1; split over key chunks.
int plan_decode_chunks(int max_ctx);
template <typename T>
void launch_attn_decode(const T* q, KVView kv, T* o, float* part, int B, int H, const int32_t* len,
                        int max_ctx, hipStream_t s);

}  // namespace axon
