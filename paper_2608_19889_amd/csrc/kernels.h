// Host-side launchers of the gfx950 kernels.  Every launcher enqueues on the
// given stream and returns immediately; shapes are validated by the caller.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace axon {

// Measurement hook: when the runtime arms this slot, the next kernel launched
// through klaunch() carries the two events in its own dispatch
// (hipExtLaunchKernelGGL), so their elapsed time is that kernel's execution.
struct TimingSlot {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local TimingSlot g_timing_slot;

template <typename Kern, typename... Args>
void klaunch(Kern kern, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  if (g_timing_slot.start) {
    const TimingSlot t = g_timing_slot;
    g_timing_slot = TimingSlot{};
    hipExtLaunchKernelGGL(kern, grid, block, shmem, s, t.start, t.stop, 0, args...);
  } else {
    kern<<<grid, block, shmem, s>>>(args...);
  }
}

// Epilogues of the projection GEMMs (out[t][n] = sum_k X[t][k] * W[n][k]).
enum Epi : int {
  EPI_F32 = 0,    // out_f32[t * ldo + n] = acc
  EPI_RESID = 1,  // out_f32[t * ldo + n] += acc   (residual stream, float)
  EPI_SILU = 2,   // W rows interleaved in blocks of 16 gate rows then 16 up rows;
                  // out_t[t * ldo + f] = silu(gate_f) * up_f
  EPI_PART = 3,   // (reserved)
  EPI_ROPE = 4,   // bf16 fused QKV projection (rows in the rotation-pair order of
                  // the decode projections): bias + rotary embedding, then q ->
                  // q_out, k -> K pages, v -> transposed V pages
  EPI_GELU = 5    // out_t[t * ldo + n] = gelu_tanh(acc + bias[n])  (GPT-2 MLP, bf16)
};
// EPI_F32 / EPI_RESID add EpiArgs::bias[n] to acc when it is set.

struct EpiArgs {
  float* out_f32;
  void* out_t;
  int ldo;
  int64_t part_stride;
  // EPI_ROPE.  Token t is at position t - cu[seq] of sequence seq (prefill,
  // len == nullptr) or at position len[t] of slot t (decode).
  const bf16* bias;  // [(H+2KV)hd] in the original head order, or null
  const float* cos_t;
  const float* sin_t;
  bf16* q_out;       // [T][H][hd]
  KVView kv;
  const int32_t* cu;
  int nseq;
  const int32_t* len;
  int H;
  // prefill entry e (tokens cu[e] .. cu[e+1]-1): cache slot ent_slot[e] and
  // position of its first token ent_base[e]; null: slot e, position 0
  const int32_t* ent_slot;
  const int32_t* ent_base;
  // grouped GEMM (mixture of experts): expert e multiplies its matrix W + e *
  // g_wstride with rows g_off[e] .. g_off[e+1]-1 of the grouped operand; row a
  // of it is X row g_xrow[a] (a when null), output row a.  g_toff[e] = sum of
  // ceil(rows / 256) over the experts before e.
  const int32_t* g_off;
  const int32_t* g_toff;
  const int32_t* g_xrow;
  int64_t g_wstride;
  int g_E;
  // row-pair layout (xp_off) of the token operand X, and of the bf16 output
  // out_t of the SiLU epilogue; 0: row-major
  int xpair;
  int opair;
};

// ---- GPT-2 rows (k_layernorm.hip).  Token t is at position len[t] (decode)
// or, with len null, ent_base[e] + t - cu[e] of its entry e (0-based when
// ent_base is null).
// x[t] = wte[tok[t]] + wpe[pos] (float; wte fragment-tiled, wpe row-major
// [P][D]); h[t] = LayerNorm(x[t]) * g + beta (bf16)
void launch_embed_pos_ln(const int32_t* tok, const bf16* wte, const bf16* wpe, const bf16* g, const bf16* beta,
                         float* x, bf16* h, int T, int D, int V, int P, float eps, const int32_t* cu, int nseq,
                         const int32_t* ent_base, const int32_t* len, hipStream_t s);
// h[i] = LayerNorm(x[r]) * g + beta with r = i, or r = cu_last[i+1]-1 (the
// last position of sequence i) when cu_last is set
void launch_layernorm(const float* x, const bf16* g, const bf16* beta, bf16* h, int rows, int D, float eps,
                      const int32_t* cu_last, hipStream_t s);
// dst[r][k] = src[k][perm ? perm[r] : r] (bf16): a [K][N] matrix stored
// [in][out] transposed to [N][K], rows optionally permuted
void launch_transpose_rows(const bf16* src, bf16* dst, int K, int N, const int32_t* perm, hipStream_t s);

// ---- backward pass (k_train.hip)
// loss over logits [T][ldl] (V real columns, ldl % 4 == 0) and targets
// (counted when in [0, V)): loss[0] = mean cross-entropy, dlog [T][ldl] bf16 =
// its gradient (zero padding); rowloss / valid / lse [T] and scal [1] scratch
void launch_ce_loss(const float* logits, int ldl, int V, const int32_t* targets, int T, float* rowloss, float* valid,
                    float* lse, float* loss, float* scal, bf16* dlog, hipStream_t s);
// dst [C][Tp] = src [T][C]^T (rows ld apart), zero columns T .. Tp-1 (Tp % 8 == 0)
void launch_transpose_pad(const bf16* src, int ld, int T, int C, bf16* dst, int Tp, hipStream_t s);
// dst [K][Np] (row-major) = W^T for the fragment-tiled W [N][K]
void launch_untile_transpose(const bf16* W, int64_t N, int K, bf16* dst, int64_t Np, hipStream_t s);
void launch_to_bf16(const float* src, bf16* dst, int64_t n, hipStream_t s);  // n % 4 == 0
// RMSNorm backward: dx (accumulate ? += : =) and per-row gain terms dgrow [T][D]
void launch_rmsnorm_bwd(const float* x, const bf16* g, const float* dy, int ldy, int T, int D, float eps, float* dx,
                        int accumulate, float* dgrow, hipStream_t s);
void launch_swiglu_bwd(const float* gu, const float* da, bf16* dgu, int T, int I, hipStream_t s);
// dst[c] = sum_t src[t][c], deterministic; part holds colsum_chunks(T) * C floats
int colsum_chunks(int T);
void launch_colsum(const float* src, int64_t ld, int T, int C, float* part, float* dst, hipStream_t s);
// attention backward over nseq fresh sequences in slots 0.. (contiguous cache):
// dq [T][H][hd], dk / dv [T][KV][hd] (float), from q / o / dO [T][H][hd] bf16,
// the forward's log2-sum-exp lse [T][H]; dsum [T][H] scratch.  Packed copies
// (scratch, finite at allocation): kr / vr [nseq*SP][KV][hd], kt [KV*hd][W],
// qt / dot [H*hd][W], W >= nseq*SP, SP >= the longest sequence rounded up to
// 32, plus 32
// dkh / dvh [T][H][hd] scratch (the per-head shares of dk / dv)
// false (nothing launched) unless the packed fragment layouts fit the shape:
// attn_bwd_layout_ok(H, kv heads, head_dim, SP, W)
bool attn_bwd_layout_ok(int H, int KVh, int hd, int SP, int64_t W);
bool launch_attn_bwd(const bf16* q, KVView kv, const bf16* o, const bf16* dob, const float* lse, float* dsum,
                     float* statp /* [2][H][W] */, const int32_t* cu, const int32_t* h_cu, int nseq, int T, int H,
                     int SP, int64_t W,
                     bf16* kr, bf16* vr, bf16* kt, bf16* qt, bf16* dot, float* dq, float* dkh, float* dvh, float* dk,
                     float* dv, hipStream_t s);
// back through RoPE into the fused QKV row order (bf16) and the original order
// (float, may be null)
void launch_rope_bwd(const float* dq, const float* dk, const float* dv, const float* cos_t, const float* sin_t,
                     const int32_t* cu, int nseq, int T, int H, int KVh, int hd, bf16* dqkv, float* dqkv_f,
                     hipStream_t s);
// projection gradient rows back to the weight map's tensors (mode 0: QKV into
// q / k / v; mode 1: gate/up into gate / up)
void launch_scatter_rows(const float* src, int R, int D, int mode, int hd, int H, int KVh, float* dst0, float* dst1,
                         float* dst2, hipStream_t s);
void launch_embed_bwd(const int32_t* tok, const float* dx, int T, int D, int V, float* dE, hipStream_t s);

// ---- weight layout (k_layout.hip): fragment-tiled copy of row-major bf16
// W [N][K] (K % 32 == 0) into dst of round_up(N, 16) * K elements
void launch_tile_weight(const bf16* src, bf16* dst, int64_t N, int K, hipStream_t s);

// ---- row kernels (k_norm.hip); a bf16 embedding table is fragment-tiled.
// h_pair: h in the row-pair layout (xp_off; D % 32 == 0), else row-major.
template <typename T>
void launch_embed_rmsnorm(const int32_t* tok, const T* emb, const T* g, float* x, T* h, int rows, int D, int V,
                          float eps, hipStream_t s, bool h_pair = false);
template <typename T>
void launch_resid_rmsnorm(float* x, const float* parts, int nparts, int64_t part_stride, const T* g, T* h,
                          int rows, int D, float eps, const int32_t* cu_last, hipStream_t s, bool h_pair = false);
void launch_argmax(const float* logits, int rows, int V, int32_t* next, int32_t* len, hipStream_t s);
// argmax of row cu[i+1]-1 for each sequence i
void launch_argmax_rows(const float* logits, int nseq, int V, int32_t* next, const int32_t* cu, hipStream_t s);
void launch_set_lengths(const int32_t* cu, int32_t* len, int n, hipStream_t s);
// len[ent_slot[e]] = ent_base[e] + cu[e+1] - cu[e] for the n entries of a step
void launch_set_step_lengths(const int32_t* cu, const int32_t* ent_slot, const int32_t* ent_base, int32_t* len,
                             int n, hipStream_t s);

// ---- projections (k_gemm.hip)
// Many-token GEMM (prefill): bf16 MFMA tiles.  Requires K % 64 == 0, N % 32 == 0
// (EPI_ROPE: the head dimension a multiple of 32).  ep.xpair: X in the row-pair
// layout (xp_off); ep.opair: the SiLU epilogue's output in that layout.
void launch_gemm_bf16(const bf16* W, const bf16* X, int N, int M, int K, int epi, const EpiArgs& ep,
                      hipStream_t s);
// Grouped GEMM of the experts (ep.g_*): rows of all experts together at most
// max_rows; launches enough 256 x 256 tiles for any split of them over the
// experts (surplus workgroups exit at once).  EPI_F32 or EPI_SILU.
void launch_gemm_bf16_grouped(const bf16* W, const bf16* X, int N, int K, int max_rows, int epi, const EpiArgs& ep,
                              hipStream_t s);
// split K over gridDim.y = ksplit workgroup rows: float32 partials
// part[s * part_stride + m * N + n] (the 256 x 256 kernel; ksplit divides K /
// 32).  gemm_ksplit: the split worth taking for an output of few 256-tiles
// (1: none).
void launch_gemm_bf16_split(const bf16* W, const bf16* X, int N, int M, int K, int ksplit, float* part,
                            int64_t part_stride, hipStream_t s, bool xpair = false);
int gemm_ksplit(int N, int M, int K);
// out[i] (accumulate ? += : =) sum of parts[s * stride + i] over s in order (n % 4 == 0)
void launch_sum_parts(float* out, const float* parts, int nparts, int64_t stride, int64_t n, int accumulate,
                      hipStream_t s);
// float32 check-mode GEMM (any M): EPI_F32 / EPI_RESID / EPI_PART(split 0 only).
void launch_gemm_f32(const float* W, const float* X, int N, int M, int K, int epi, const EpiArgs& ep,
                     hipStream_t s);
// a[t][f] = silu(sum_s gate) * sum_s up over split-K partials of the
// interleaved gate/up projection ([nparts][M][2I] floats).
template <typename T>
void launch_silu_reduce(const float* parts, int nparts, int64_t part_stride, T* a, int M, int I,
                        hipStream_t s);
// ---- fused decode projections (k_gemv.hip)
enum GvEpi : int { GV_HEAD = 0, GV_RESID = 1, GV_SILU = 2, GV_ROPE = 3, GV_PART = 4 /* internal: split-K partials */,
                   GV_F32 = 5 /* grouped experts: float rows out_f32[row][n] */,
                   GV_GELU = 6 /* out_t[t][n] = bf16(gelu_tanh(acc + bias[n])) */ };

struct GemvArgs {
  const bf16* W;  // [N][K]
  int N, K, M;
  // B operand X [M][K] bf16.  Normalized operand (ss_in != nullptr): X holds
  // bf16(x * g) and the result is scaled by rsqrt(sum of squares / K + eps)
  const bf16* X;
  const float* ss_in;  // [ss_n][M] partial sums of squares of the rows of x
  int ss_n;
  float eps;
  // epilogue outputs
  float* out_f32;  // GV_HEAD logits [M][ldo] (may be null) / GV_RESID x [M][ldo]
  int ldo;
  bf16* out_t;     // GV_SILU a [M][ldo]
  float* ss_out;   // GV_RESID: [N / gemv_rows][M], or null
  bf16* xg_out;    // GV_RESID: bf16(x * gain_next) [M][ldo], or null (then ss_out too)
  const bf16* gain_next;
  float* am_val;   // GV_HEAD: [M][N / gemv_rows] partial maxima
  int32_t* am_idx;
  // GV_ROPE: [(H+2KV)hd] in the original (unpermuted) order; GV_RESID /
  // GV_GELU: [N] added to acc; or null
  const bf16* bias;
  const float* cos_t;
  const float* sin_t;
  bf16* q_out;  // [M][H][hd]
  KVView kv;
  const int32_t* len;   // token t is at position len[t] ...
  const int32_t* slot;  // ... of cache slot slot[t] (t when null)
  int H;
  // split K (projections of 17..64 tokens): workspace of ksplit * M * N floats
  // (gemv_workspace_floats), owned by the caller
  float* part;
  // grouped experts (launch_gemv_grouped): expert e multiplies W + e *
  // g_wstride with its rows g_off[e] .. g_off[e+1]-1; row r reads X row
  // g_xrow[r] (row r when g_xrow is NULL) and writes output row r (M is an
  // upper bound of any expert's rows)
  const int32_t* g_off;
  const int32_t* g_xrow;
  int64_t g_wstride;
  // tile order (xt_off) of the token operands, up to 16 tokens, unsplit
  // fused projections only: x_tiled -- X is stored in it; out_tiled -- the
  // epilogue writes xg_out (GV_RESID) or out_t (GV_SILU) in it
  int x_tiled;
  int out_tiled;
};
constexpr int GEMV_MAX_M = 64;      // token columns one fused projection handles
constexpr int GV_RESID_ROWS = 1024;  // features per workgroup of the split-K residual epilogue
struct GvShape {
  int rows, ks, u;  // output rows per workgroup, wavefronts splitting K, k-steps of 32 per stage
  int ksplit;       // workgroups splitting K (1: fused epilogue; else partials + an epilogue kernel)
  int erows;        // rows per workgroup of the epilogue kernel (ksplit > 1)
  int wide = 0;     // 1: gemv_wide_kernel (4 wavefronts splitting the rows, ks unused)
};
// floats of GemvArgs::part a launch of this shape needs (0 when unsplit)
int64_t gemv_workspace_floats(int N, int K, int M, int epi);
GvShape gemv_shape(int N, int K, int M, int epi);
int gemv_rows(int N, int K, int M, int epi);  // output rows per workgroup (ss partial count = N / rows)
// false (nothing launched) when M > GEMV_MAX_M or the normalization does not
// match the epilogue (GV_SILU and GV_ROPE need ss_in, GV_RESID must not have it)
bool launch_gemv_fused(const GemvArgs& a, int epi, hipStream_t s);
void launch_argmax_final(const float* val, const int32_t* idx, int nparts, int M, int32_t* next, int32_t* len,
                         hipStream_t s);
// Few-token grouped expert projections (mixture-of-experts decode): a
// workgroup per (64-row block, expert), the expert's rows (at most a.M <= 64)
// gathered through g_xrow; GV_SILU (out_t rows, interleaved gate/up W) or
// GV_F32 (out_f32 rows).  false when a.M > 64.
bool launch_gemv_grouped(const GemvArgs& a, int epi, int n_experts, hipStream_t s);
// xg_tiled: xg in the tile order of the few-token projections (M <= 16)
void launch_embed_ss(const int32_t* tok, const bf16* emb, const bf16* g, float* x, bf16* xg, float* ss_out, int M,
                     int D, int V, hipStream_t s, bool xg_tiled = false);

// ---- float32 few-token projections (k_gemv_f32.hip): float weights [N][K]
// row-major (QKV rows in the rotation-pair order, gate/up interleaved in
// blocks of 16 rows), up to GEMV_F32_MAX_M tokens, the epilogues of
// GV_ROPE / GV_SILU (normalized operand), GV_RESID, GV_HEAD (normalized)
struct GemvF32Args {
  const float* W;
  int N, K, M;
  const float* X;       // [M][K]: x * g (normalized operand) or the plain operand
  const float* ss_in;   // [ss_n][M] partial sums of squares of x, or null
  int ss_n;
  float eps;
  float* out;           // GV_RESID x [M][ldo] (+=) / GV_SILU a [M][ldo] / GV_HEAD logits [M][ldo] or null
  int ldo;
  float* xg_out;        // GV_RESID: x * gain_next [M][ldo], or null
  const float* gain_next;
  float* ss_out;        // GV_RESID: [gemv_f32_parts(N)][M]
  float* am_val;        // GV_HEAD: [M][gemv_f32_parts(N)] per-workgroup maxima
  int32_t* am_idx;
  const float* bias;    // GV_ROPE: [(H+2KV)hd] in the original head order, or null
  const float* cos_t;
  const float* sin_t;
  float* q_out;         // [M][H][hd]
  KVView kv;
  const int32_t* len;   // token t at position len[t] of slot slot[t] (t when null)
  const int32_t* slot;
  int H;
};
constexpr int GEMV_F32_MAX_M = 16;
// false (nothing launched) for more than GEMV_F32_MAX_M tokens or a shape or
// normalization the epilogue does not take
bool launch_gemv_f32_fused(const GemvF32Args& a, int epi, hipStream_t s);
int gemv_f32_parts(int N, int epi);  // workgroups of a launch (partials per token)
// Short-context decode (attention recomputed by every workgroup of the O
// projection): whether a step of M tokens with contexts up to max_ctx keys
// qualifies, and the fused attention + residual O projection (a: the
// GV_RESID projection with K = H * hd; q [M][H][hd]; token t at position
// a.len[t] of slot a.slot[t]).  false (nothing launched) outside those limits.
bool attn_o_f32_fits(int M, int H, int KVh, int hd, int max_ctx);
bool launch_attn_o_f32(const GemvF32Args& a, const float* q, KVView kv, hipStream_t s);
void launch_embed_ss_f32(const int32_t* tok, const float* emb, const float* g, float* x, float* xg, float* ss_out,
                         int M, int D, int V, hipStream_t s);

// ---- bias + rotary + KV-cache write (k_rope.hip)
// qkv rows are sum_s parts[s][t][:] (+ bias): q heads, then k heads, then v heads.
// Token t belongs to entry e(t) of cu: prefill puts it in slot ent_slot[e] at
// position ent_base[e] + t - cu[e] (slot e, position t - cu[e] when the arrays
// are null); decode (len != nullptr) uses slot t at position len[t].
template <typename T>
void launch_rope_kv(const float* parts, int nparts, int64_t part_stride, const T* bias, const float* cos_t,
                    const float* sin_t, T* q_out, KVView kv, int T_tokens, int nseq, const int32_t* cu,
                    const int32_t* len, int H, hipStream_t s, const int32_t* ent_slot = nullptr,
                    const int32_t* ent_base = nullptr);

// ---- attention (k_attn.hip)
// Causal prefill attention over the cache; o [T][H*hd] (bf16 with o_pair: in
// the row-pair layout, xp_off with K = H*hd).  The workgroups cover
// the nseq entries listed in ents (device) / h_ents (host copy), or entries
// 0..nseq-1 when both are null; entry e's tokens cu[e] .. cu[e+1]-1 are at
// positions ent_base[e] + 0, 1, ... of slot ent_slot[e] and attend to every
// earlier key of that slot (null arrays: slot e from position 0).
template <typename T>
void launch_attn_prefill(const T* q, KVView kv, T* o, int T_tokens, int nseq, const int32_t* cu,
                         const int32_t* h_cu, int H, hipStream_t s, const int32_t* ents = nullptr,
                         const int32_t* h_ents = nullptr, const int32_t* ent_slot = nullptr,
                         const int32_t* ent_base = nullptr, float* lse = nullptr, bool o_pair = false);
// Decode attention: one query per slot at position len[b] (after the step's
// key/value were written), context len[b] + 1; keys split over
// plan_decode_splits() workgroups per (slot, kv head).  ``part`` holds
// B * H * splits * (hd + 2) floats; the last split of a (slot, kv head)
// merges them.
int plan_decode_splits(int B, int kv_heads, int max_ctx);
// Item b reads query row rows[b] and writes output row rows[b] (b when null),
// in cache slot slots[b] (b when null), at position len[b]; bf16 only for the
// indirection (the float32 path reaches such items through launch_attn_prefill).
// p[0 .. n) = 0, as a kernel (graph-capture safe)
void launch_zero_i32(int32_t* p, int n, hipStream_t s);
// cnt: int32 [B][kv heads], zero before the launch and left zero after it
// (split arrival counters).  o_tiled (bf16, B <= 16, no rows): o [B][H hd]
// in the tile order of the few-token projections (xt_off).
template <typename T>
void launch_attn_decode(const T* q, KVView kv, T* o, float* part, int32_t* cnt, int B, int H, const int32_t* len,
                        int max_ctx, hipStream_t s, const int32_t* rows = nullptr,
                        const int32_t* slots = nullptr, bool o_tiled = false);

// ---- mixture of experts (k_moe.hip)
// topi / topw [T][k]: the top_k experts of each token (E <= 256, k <= 8) from
// float logits [T][ldl], and their softmax probabilities (over all E),
// divided by their sum when norm
void launch_moe_route(const float* logits, int ldl, int T, int E, int k, int norm, int32_t* topi, float* topw,
                      hipStream_t s);
// grouped-GEMM plan of the T*k choices: cnt [E], off / toff [E+1] (rows and
// 256-row tiles before each expert), xrow [T*k] (token of each grouped row),
// inv [T*k] (grouped row of choice t*k + j)
void launch_moe_plan(const int32_t* topi, int T, int E, int k, int32_t* cnt, int32_t* off, int32_t* toff,
                     int32_t* xrow, int32_t* inv, hipStream_t s);
// out[r] = h[xrow[r]] for r < rows (bf16 rows of D, D % 8 == 0)
void launch_moe_gather(const bf16* h, const int32_t* xrow, int rows, int D, bf16* out, hipStream_t s);
// x[t] += sum_j w[t][j] * y[inv[t*k+j]] (float rows of D, D % 4 == 0).  With
// xg: also xg = bf16(x * g) and per-token sums of squares of the new x in
// moe_combine_blocks(D) partials, ss_out[part * T + t].
inline int moe_combine_blocks(int D) { return (D / 4 + 255) / 256; }
void launch_moe_combine(float* x, const float* y, const int32_t* inv, const float* w, int T, int D, int k,
                        hipStream_t s, const bf16* g = nullptr, bf16* xg = nullptr, float* ss_out = nullptr);

}  // namespace axon
