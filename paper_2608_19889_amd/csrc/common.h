// Shared device-side types and helpers for the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

#define AXON_DEV __device__ __forceinline__

AXON_DEV float to_f32(float v) { return v; }
AXON_DEV float to_f32(bf16 v) { return (float)v; }
template <typename T> AXON_DEV T from_f32(float v);
template <> AXON_DEV float from_f32<float>(float v) { return v; }
template <> AXON_DEV bf16 from_f32<bf16>(float v) { return (bf16)v; }  // round to nearest even

// GELU, tanh form (GPT-2's gelu_new): 0.5 z (1 + tanh(u)), u = sqrt(2/pi) (z +
// 0.044715 z^3), with tanh(u) = 1 - 2 / (e^{2u} + 1) (an overflowing e^{2u}
// gives 1, an underflowing one -1).
AXON_DEV float gelu_tanh_f(float z) {
  const float u = 0.7978845608028654f * (z + 0.044715f * z * z * z);
  return 0.5f * z * (2.f - 2.f / (__expf(2.f * u) + 1.f));
}

// The value that lane l ^ 32 (l ^ 16) of the wavefront holds, by the gfx950
// permlane swaps: a register exchange between half-wavefronts (16-lane rows),
// no LDS round trip as with ds_bpermute.  A swap of v with itself leaves
// lane l the pair (its own value, the partner's) in half order.
AXON_DEV float lane_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}
AXON_DEV float lane_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float((threadIdx.x & 16) ? r[0] : r[1]);
}

// DPP lane moves within 16-lane rows: CTRL 0xB1 / 0x4E = quad_perm
// [1,0,3,2] / [2,3,0,1] (lane l ^ 1, l ^ 2), 0x141 = row_half_mirror (lane j
// of an 8-lane half <- 7 - j), 0x140 = row_mirror (lane j of a row <- 15 - j).
template <int CTRL>
AXON_DEV float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
// Sum / maximum over the 64 lanes of a wavefront, every lane the same
// result: a butterfly of register moves (no LDS round trip).  After the l ^ 1
// and l ^ 2 steps a value is uniform over its 4-lane group, so the half-row
// mirror adds the other group of its 8 lanes (as l ^ 4 would) and, the value
// then uniform over 8 lanes, the row mirror the other half of its row (as
// l ^ 8 would); both operands of every add are the same pair in either lane.
AXON_DEV float wave_sum(float v) {
  v += dpp_move<0xB1>(v);
  v += dpp_move<0x4E>(v);
  v += dpp_move<0x141>(v);
  v += dpp_move<0x140>(v);
  v += lane_xor16(v);
  v += lane_xor32(v);
  return v;
}
AXON_DEV float wave_max(float v) {
  v = fmaxf(v, dpp_move<0xB1>(v));
  v = fmaxf(v, dpp_move<0x4E>(v));
  v = fmaxf(v, dpp_move<0x141>(v));
  v = fmaxf(v, dpp_move<0x140>(v));
  v = fmaxf(v, lane_xor16(v));
  v = fmaxf(v, lane_xor32(v));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); every thread gets the result.
AXON_DEV float block_sum(float v, float* red /* >= 16 floats of shared memory */) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}

// Sequence index of packed token t given prefix sums cu[0..nseq] (cu[0] = 0).
AXON_DEV int seq_of_token(const int32_t* __restrict__ cu, int nseq, int t) {
  int lo = 0, hi = nseq - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// KV-cache addressing.  One layout serves the contiguous and the paged cache:
// a "page" holds ``ps`` consecutive positions of one sequence for every kv head.
//   K  page: [KV][ps][hd]      (row per position, head_dim contiguous)
//   V^T page: [KV][hd][ps]     (row per head-dim index, positions contiguous)
// Contiguous cache: page = slot, ps = per-slot capacity.  Paged cache: page =
// block_table[slot * bt_stride + pos / ps].
struct KVView {
  void* k;            // this layer's K pages
  void* v;            // this layer's V^T pages
  const int32_t* bt;  // block table or nullptr (contiguous)
  int bt_stride;
  int ps;             // positions per page
  int kv_heads;
  int hd;
  int window = 0;     // sliding window W: a query at position p sees keys (p - W, p]; 0 = all
};

AXON_DEV int64_t kv_page(const KVView& c, int slot, int pos) {
  return c.bt ? (int64_t)c.bt[(int64_t)slot * c.bt_stride + pos / c.ps] : (int64_t)slot;
}
// Within a page, each kv head owns a slab of ps x hd elements, cut into
// blocks of 16 positions (16 hd contiguous elements each; ps is a multiple of
// 16).  K block: [hd / 8][16 positions][8 dims]: the 8-dim chunk of a
// position is 16 contiguous bytes and a chunk's 16 positions 256 bytes, so
// the 16-position x 32-dim MFMA fragment of a key block is one contiguous
// 1 KB read in lane order.  V block: [hd][16 positions], V^T of the block:
// 4 consecutive positions of a dimension are 8 contiguous bytes, 16 dims x 16
// positions one contiguous 512-byte read.
AXON_DEV int64_t kv_block(const KVView& c, int slot, int kvh, int pos) {  // first element of pos's block
  return ((kv_page(c, slot, pos) * c.kv_heads + kvh) * c.ps + (pos % c.ps & ~15)) * (int64_t)c.hd;
}
// element offset of K[pos][d] for (slot, kv head)
AXON_DEV int64_t k_el(const KVView& c, int slot, int kvh, int pos, int d) {
  return kv_block(c, slot, kvh, pos) + (d >> 3) * 128 + (pos & 15) * 8 + (d & 7);
}
// element offset of V[pos][d] for (slot, kv head)
AXON_DEV int64_t v_el(const KVView& c, int slot, int kvh, int pos, int d) {
  return kv_block(c, slot, kvh, pos) + d * 16 + (pos & 15);
}

// Fragment-tiled storage of a bf16 weight matrix W [N][K] (K % 32 == 0).  Rows
// come in blocks of 16 (the last block zero-padded); each block is cut along k
// into 16 x 32 tiles of 1 KB, stored one after another, and a tile holds its
// 64 16-byte chunks in the lane order of a v_mfma 16x16x32 A operand: chunk
// (r, s) = row r of the block, k values 8s..8s+7 of the tile, at position
// r + 16 s.  A wavefront's fragment load is one contiguous 1 KB read, and a
// row block is one contiguous stream along k.
// Token operand of the few-token projections in tile order: element (t, k)
// of a [16][K] bf16 operand (t < 16, K a multiple of 32) sits where the B
// fragment of v_mfma_f32_16x16x32_bf16 for k-step k / 32 wants it, so a
// wavefront's fragment is one contiguous 1 KB read (lane L = 16 ((k / 8) % 4)
// + t holds k values 8 (L / 16) .. +7 of token t).  Rows t >= the token count
// are neither written nor read (their lanes read token count - 1).
AXON_DEV int64_t xt_off(int t, int64_t k) { return (k >> 5) * 512 + ((((k >> 3) & 3) << 4) + t) * 8 + (k & 7); }
constexpr int XT_ROWS = 16;  // tokens of the tile order (one B fragment column block)

// Row-pair layout of a bf16 token operand [T][K] (K a multiple of 32) of the
// prefill GEMMs: rows 2p and 2p+1 are stored together in slices of 32 k values,
// row 2p's slice then row 2p+1's, so that the two 64-byte pieces a 32-deep
// k-tile takes from the pair fill one 128-byte line (row-major rows left every
// such piece half a line, and the GEMM's tile loads ran 15-20% slower).  A
// buffer of an odd row count holds one row more.
AXON_DEV int64_t xp_off(int64_t t, int64_t k, int K) {
  return ((t >> 1) * (K >> 5) + (k >> 5)) * 64 + (t & 1) * 32 + (k & 31);
}

// Element offset of W[n][8c .. 8c+7] (c = k-chunk index, k = 8c):
AXON_DEV int64_t wt_chunk(int64_t n, int c, int K) {
  return (((n >> 4) * (K >> 5) + (c >> 2)) * 64 + (n & 15) + 16 * (c & 3)) * 8;
}
