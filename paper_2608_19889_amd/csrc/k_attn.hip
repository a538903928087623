// Causal grouped-query attention over the KV cache.
//
// softmax(q k^T / sqrt(hd)) v per query head, keys 0..pos of the query's own
// sequence, kv head = query head / (H / KV).  Softmax runs online in base 2
// with float statistics.
//
// Both bf16 kernels compute S^T = K Q^T (keys as MFMA rows, queries as
// columns), so that a lane owns one query column: the row maximum and sum of a
// query are then in-lane reductions plus one or two cross-lane exchanges, and
// the probabilities already sit in the lane layout of the B operand of the
// following O^T = V^T P^T product (the k index of that product is permuted to
// match, and V^T is read with the same permutation from the transposed V pages).
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace axon {

constexpr float LOG2E = 1.4426950408889634f;

// Page of position ``pos`` of ``slot`` for a wave-uniform (slot, pos), the
// cache kind fixed at compile time (no branch on bt): read through the
// constant address space, so that it is a scalar load whose wait does not
// hold up the wavefront's outstanding vector loads.  The page table is not
// written while a kernel runs.
template <bool PAGED>
AXON_DEV int64_t kv_page_of(const KVView& c, int slot, int pos) {
  if constexpr (!PAGED) {
    return slot;
  } else {
    typedef const __attribute__((address_space(4))) int32_t* cptr;
    const cptr bt = (cptr)(uintptr_t)c.bt;
    return bt[__builtin_amdgcn_readfirstlane(slot * c.bt_stride + pos / c.ps)];
  }
}

// ============================================================================
// Prefill (bf16): a workgroup = 8 wavefronts x 32 queries of one head of one
// sequence (256 queries: each K / V^T tile moved into LDS feeds 8
// wavefronts; workgroups of several heads of a GQA group x fewer queries, or
// of 128 queries, measured slower).  Key tiles of 64, K [64][hd] and V^T
// [hd][64] moved straight from global memory into LDS (global_load_lds_dwordx4:
// lane L writes 16 bytes at offset 16 L) two tiles ahead of the tile being
// computed, in a ring of three; v_mfma_f32_32x32x16_bf16 for both products.
// The bank swizzle of a tile (16-byte chunk c of row r stored at c ^ swz(r))
// is made by choosing which global chunk each lane loads.  Keys past the
// sequence load its last key (finite; their scores are masked).
// ============================================================================
constexpr int PK = 64;
constexpr int PREFILL_WAVES = 8;

// LDS row rho of a K tile holds key kappa(rho): bits 2 and 3 of the row index
// swapped.  The S^T = K Q^T accumulator puts rows {8a + 4 hl + 0..3} of a
// 16-row group in the half-wavefront hl (a = 0, 1), so with this order a
// lane's 8 probabilities of a k-step are 8 consecutive keys, and its V^T
// operand of the P V product is one 16-byte chunk (a single conflict-free LDS
// read instead of two 8-byte reads that share banks).  An involution.
AXON_DEV int kappa(int rho) { return (rho & ~12) | ((rho & 4) << 1) | ((rho & 8) >> 1); }

// physical 16-byte chunk of logical chunk c in row r of an LDS tile whose
// rows hold CH chunks: the 16 lanes of a read phase (16 consecutive rows,
// one logical chunk) hit distinct banks
template <int CH>
AXON_DEV int pswz(int r, int c) {
  if constexpr (CH == 16) return c ^ (r & 15);
  else return c ^ ((r >> 1) & 7);  // 8 chunks: rows r and r+1 share a 256-byte bank line
}

// Entries: the workgroups cover the entries listed in ``ents`` (all nseq
// entries in order when null).  Entry e holds tokens cu[e] .. cu[e+1]-1 of
// slot ent_slot[e] (e when null) at positions ent_base[e] .. (0 when null):
// queries attend to keys 0 .. their own position of that slot, the keys
// before ent_base[e] written by earlier calls (a chunked prefill).
template <int HD, bool PAGED>
__global__ void __launch_bounds__(64 * PREFILL_WAVES) attn_prefill_bf16_kernel(
    const bf16* __restrict__ q, KVView kv, bf16* __restrict__ o, int nseq, const int32_t* __restrict__ cu, int H,
    const int32_t* __restrict__ ents, const int32_t* __restrict__ ent_slot, const int32_t* __restrict__ ent_base,
    float* __restrict__ lse, int o_pair) {
  constexpr int NW = PREFILL_WAVES;      // wavefronts
  constexpr int KCH = HD / 8;            // 16-byte chunks per K row
  constexpr int VCH = PK / 8;            // chunks per V^T row (8)
  constexpr int KT = PK * KCH;           // chunks per K tile
  constexpr int VT = HD * VCH;           // chunks per V^T tile
  constexpr int BUF = KT + VT;           // chunks per buffer
  constexpr int TQ = 32 * NW;            // queries per workgroup
  constexpr int STG = 3;                 // tiles in the LDS ring: two in flight while one is used
  static_assert(KT % 64 == 0 && VT % 64 == 0, "tiles are whole load instructions");
  __shared__ bf16x8 lds[STG * BUF];

  // (entry, query tile, head) of this workgroup, in an XCD-aware order: the
  // workgroup id mod 8 picks the XCD, and each XCD walks a contiguous range
  // of (kv head, entry, query tile from the longest down, query head of the
  // group), so the workgroups that read one sequence's keys and values for
  // one kv head run together on one XCD and find them in its L2, and the
  // longest tiles start first
  const int group = H / kv.kv_heads;
  const int Gd = gridDim.x, ntl = Gd / H;  // ntl: query tiles over all entries
  int logical = blockIdx.x;
  const int full = Gd / 8 * 8;
  if (logical < full) logical = (logical % 8) * (full / 8) + logical / 8;
  const int hin = logical % group;
  const int rest = logical / group;
  int tile = rest % ntl;
  const int kvh = rest / ntl;
  const int head = kvh * group + hin;
  int li = 0, ent = 0;
  for (; li < nseq; ++li) {
    ent = ents ? ents[li] : li;
    const int nt = (cu[ent + 1] - cu[ent] + TQ - 1) / TQ;
    if (tile < nt) {
      tile = nt - 1 - tile;
      break;
    }
    tile -= nt;
  }
  const int S = cu[ent + 1] - cu[ent];         // this call's queries of the entry
  const int tok0 = cu[ent];
  const int seq = ent_slot ? ent_slot[ent] : ent;  // cache slot
  const int base = ent_base ? ent_base[ent] : 0;   // position of the entry's first query
  const int KL = base + S;                         // keys of the slot after this call
  const int q0 = tile * TQ;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qw0 = q0 + wave * 32;  // this wavefront's queries
  const int hl = lane >> 5;

  // Q^T fragments (B operand): column = query, k = head-dim (queries past S
  // read the last query; their outputs are not stored)
  bf16x8 qf[HD / 16];
  {
    const int myq = qw0 + (lane & 31);
    const bf16* qp = q + ((int64_t)(tok0 + min(myq, S - 1)) * H + head) * HD + hl * 8;
#pragma unroll
    for (int k = 0; k < HD / 16; ++k) qf[k] = *(const bf16x8*)(qp + k * 16);
  }

  // issue the loads of key tile kt into buffer b: instruction i of wavefront
  // w moves chunk slots (i NW + w) 64 + lane of the K tile, then of the V^T
  // tile.  A tile wholly inside the slot's keys takes the fast form: the
  // lane's offset inside a 16-key block is fixed per instruction, and the
  // four blocks' base addresses are wave-uniform (computed once per tile; in
  // a contiguous cache one tile base plus 16 hd per block, which measured 4-9%
  // faster than selecting among four per-block bases); the slot's last tile
  // clamps every key to the last one.
  const bf16* kb = (const bf16*)kv.k;
  const bf16* vb = (const bf16*)kv.v;
  // every wavefront issues the same number of load instructions per tile, so
  // the loads and their waits are free of (scalar) branches
  static_assert((KT / 64) % NW == 0 && (VT / 64) % NW == 0, "tiles split evenly over the wavefronts");
  constexpr int NKI = KT / 64 / NW, NVI = VT / 64 / NW;
  int koff[NKI], kgrp[NKI], voff[NVI], vgrp[NVI];
#pragma unroll
  for (int i = 0; i < NKI; ++i) {
    const int p = (i * NW + wave) * 64 + lane;
    const int r = p / KCH, c = pswz<KCH>(r, p % KCH);
    koff[i] = c * 128 + (kappa(r) & 15) * 8;
    kgrp[i] = __builtin_amdgcn_readfirstlane(kappa(r) >> 4);  // one 16-key block per instruction
  }
#pragma unroll
  for (int i = 0; i < NVI; ++i) {
    const int p = (i * NW + wave) * 64 + lane;
    const int d = p / VCH, c = pswz<VCH>(d, p % VCH);
    voff[i] = d * 16 + (c & 1) * 8;
    vgrp[i] = c >> 1;
  }
  auto issue = [&](int kt, int b) {
    const int j0 = kt * PK;
    if (!PAGED && j0 + PK <= KL) {
      // contiguous cache: the tile's four 16-key blocks are consecutive, so a
      // lane's block base is the tile's (wave-uniform) plus 16 hd per block
      const int64_t tb = (((int64_t)seq * kv.kv_heads + kvh) * kv.ps + j0) * HD;
#pragma unroll
      for (int i = 0; i < NKI; ++i) {
        __builtin_amdgcn_global_load_lds((const void*)(kb + tb + kgrp[i] * (16 * HD) + koff[i]),
                                         (__attribute__((address_space(3))) void*)(lds + b * BUF + (i * NW + wave) * 64),
                                         16, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < NVI; ++i) {
        __builtin_amdgcn_global_load_lds(
            (const void*)(vb + tb + vgrp[i] * (16 * HD) + voff[i]),
            (__attribute__((address_space(3))) void*)(lds + b * BUF + KT + (i * NW + wave) * 64), 16, 0, 0);
      }
      return;
    }
    if (PAGED && j0 + PK <= KL) {
      int64_t gb[4];
#pragma unroll
      for (int g = 0; g < 4; ++g)
        gb[g] = ((kv_page_of<PAGED>(kv, seq, j0 + g * 16) * kv.kv_heads + kvh) * kv.ps + (j0 + g * 16) % kv.ps) * HD;
#pragma unroll
      for (int i = 0; i < NKI; ++i) {
        const int g = kgrp[i];
        const int64_t base = g == 0 ? gb[0] : g == 1 ? gb[1] : g == 2 ? gb[2] : gb[3];
        __builtin_amdgcn_global_load_lds((const void*)(kb + base + koff[i]),
                                         (__attribute__((address_space(3))) void*)(lds + b * BUF + (i * NW + wave) * 64),
                                         16, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < NVI; ++i) {
        const int g = vgrp[i];
        const int64_t base = g == 0 ? gb[0] : g == 1 ? gb[1] : g == 2 ? gb[2] : gb[3];
        __builtin_amdgcn_global_load_lds(
            (const void*)(vb + base + voff[i]),
            (__attribute__((address_space(3))) void*)(lds + b * BUF + KT + (i * NW + wave) * 64), 16, 0, 0);
      }
      return;
    }
    int64_t pg[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) pg[g] = kv_page_of<PAGED>(kv, seq, min(j0 + g * 16, KL - 1) & ~15);
#pragma unroll
    for (int i = 0; i < NKI; ++i) {
      const int p = (i * NW + wave) * 64 + lane;
      const int r = p / KCH, c = pswz<KCH>(r, p % KCH);  // pswz is its own inverse
      const int key = min(j0 + kappa(r), KL - 1);         // in [j0, j0 + 64): j0 < KL
      const int64_t page = pg[(key - j0) >> 4];
      const int kp = key % kv.ps;
      const bf16* src = kb + ((page * kv.kv_heads + kvh) * kv.ps + (kp & ~15)) * HD + c * 128 + (kp & 15) * 8;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (__attribute__((address_space(3))) void*)(lds + b * BUF + (i * NW + wave) * 64),
                                       16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < NVI; ++i) {
      const int p = (i * NW + wave) * 64 + lane;
      const int d = p / VCH, c = pswz<VCH>(d, p % VCH);
      const int key = min(j0 + c * 8, (KL - 1) & ~7);  // 8 keys of one 16-key group, in [j0, j0 + 64)
      const int64_t page = pg[(key - j0) >> 4];
      const int kp = key % kv.ps;
      const bf16* src = vb + ((page * kv.kv_heads + kvh) * kv.ps + (kp & ~15)) * HD + d * 16 + (kp & 15);
      __builtin_amdgcn_global_load_lds(
          (const void*)src, (__attribute__((address_space(3))) void*)(lds + b * BUF + KT + (i * NW + wave) * 64), 16,
          0, 0);
    }
  };

  f32x16 acc_o[HD / 32];
#pragma unroll
  for (int d = 0; d < HD / 32; ++d) acc_o[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const float sc = LOG2E / sqrtf((float)HD);

  const int W = kv.window;
  const int kend = base + min(S, q0 + TQ);  // keys needed by the workgroup
  const int ntiles = (kend + PK - 1) / PK;
  // with a window, the first tile holding a key of the workgroup's first query
  const int kt0 = W ? max(0, base + q0 - W + 1) / PK : 0;
  issue(kt0, kt0 % STG);
  if (kt0 + 1 < ntiles) issue(kt0 + 1, (kt0 + 1) % STG);
  for (int kt = kt0; kt < ntiles; ++kt) {
    const int j0 = kt * PK, b = kt % STG;
    // tile kt landed for this wavefront (tile kt + 1, this wavefront's
    // NKI + NVI load instructions, may still be in flight)
    if (kt + 1 < ntiles) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(NKI + NVI) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();  // tile kt landed for every wavefront; the buffer of tile kt - 1 is free
    if (kt + 2 < ntiles) issue(kt + 2, (kt + 2) % STG);
    const bf16x8* ks = lds + b * BUF;
    const bf16* vsb = (const bf16*)(ks + KT);
    if (j0 > base + qw0 + 31 || qw0 >= S) continue;  // no key of the tile for this wavefront's queries
    if (W && j0 + PK - 1 <= base + qw0 - W) continue;         // every key of the tile is before their windows
    // ---- S^T = K Q^T
    f32x16 s[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      s[r] = f32x16{};
      const int row = r * 32 + (lane & 31);
#pragma unroll
      for (int k = 0; k < HD / 16; ++k) {
        const bf16x8 kf = ks[row * KCH + pswz<KCH>(row, k * 2 + hl)];
        s[r] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[k], s[r], 0, 0, 0);
      }
    }
    // ---- online softmax (lane = query column), on unscaled scores: the
    //      1/sqrt(hd) scale (log2 e folded in) enters the exponent's FMA.
    //      Masking only where the tile crosses the diagonal or the sequence
    //      end.  The reference maximum m_run is raised only when a score
    //      exceeds it by more than 8 (in log2 units): probabilities stay <= 2^8
    //      and the accumulator is rescaled rarely, not every tile (the sum and
    //      the accumulator always share the reference, so the result is exact).
    const bool masked = j0 + PK - 1 > base + qw0 || j0 + PK > KL || (W && j0 + W <= base + qw0 + 31);
    bf16x8 pb[2][2];
    {
      const int myq = qw0 + (lane & 31);
      float mloc = -INFINITY;
      if (masked) {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = j0 + r * 32 + (i / 8) * 16 + hl * 8 + ((i / 4) & 1) * 4 + (i % 4);  // kappa of the row
            const float v = (key <= base + myq && key < KL && (!W || key > base + myq - W)) ? s[r][i] : -INFINITY;
            s[r][i] = v;
            mloc = fmaxf(mloc, v);
          }
      } else {
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
          for (int i = 0; i < 16; ++i) mloc = fmaxf(mloc, s[r][i]);
      }
      mloc = fmaxf(mloc, lane_xor32(mloc)) * sc;  // scaled maximum of the tile
      // raise the reference when the tile's maximum exceeds it by > 8
      const bool raise = mloc > m_run + 8.f;
      if (__builtin_amdgcn_ballot_w64(raise) != 0) {  // wave-uniform: rare after the first tiles
        const float m_new = raise ? mloc : m_run;
        const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < HD / 32; ++d) acc_o[d] *= alpha;
      }
      const float m_ref = m_run == -INFINITY ? 0.f : m_run;
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[r][i], sc, -m_ref));
          l_run += p;
          pb[r][i / 8][i % 8] = (bf16)p;
        }
    }
    // ---- O^T += V^T P^T; the k index of block (r, h) in half-wavefront hl
    //      covers keys r*32 + h*16 + hl*8 + 0..7 (logical chunk r*4 + 2h + hl
    //      of the V^T row)
#pragma unroll
    for (int d = 0; d < HD / 32; ++d) {
      const int dd = d * 32 + (lane & 31);
      const bf16x8* vr = (const bf16x8*)(vsb + dd * PK);
#pragma unroll
      for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const bf16x8 va = vr[pswz<VCH>(dd, r * 4 + h * 2 + hl)];
          acc_o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[r][h], acc_o[d], 0, 0, 0);
        }
    }
  }
  const int myq = qw0 + (lane & 31);
  if (myq >= S) return;
  const float l_tot = l_run + lane_xor32(l_run);
  const float inv = 1.f / l_tot;
  // log2 of sum_k exp2(score_k * sc): what the backward pass recomputes its
  // probabilities from
  if (lse && hl == 0) lse[(int64_t)(tok0 + myq) * H + head] = (m_run == -INFINITY ? 0.f : m_run) + __log2f(l_tot);
  // 4 consecutive dims never cross a 32-dim slice of the row-pair layout
  const int64_t trow = tok0 + myq;
  bf16* op = o_pair ? o + xp_off(trow, (int64_t)head * HD, H * HD) : o + (trow * H + head) * HD;
#pragma unroll
  for (int d = 0; d < HD / 32; ++d)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int dd = g * 8 + hl * 4 + (o_pair ? d * 64 : d * 32);  // a 32-dim slice every 64 elements in a pair
      *(bf16x4*)(op + dd) = bf16x4{(bf16)(acc_o[d][g * 4 + 0] * inv), (bf16)(acc_o[d][g * 4 + 1] * inv),
                                   (bf16)(acc_o[d][g * 4 + 2] * inv), (bf16)(acc_o[d][g * 4 + 3] * inv)};
    }
}

// ============================================================================
// Decode (bf16): one query per slot.  Workgroup = (key split, kv head, slot)
// with DNW wavefronts; the group's query heads are the columns of
// v_mfma_f32_16x16x32_bf16 (up to 16 heads per group); the wavefronts take
// the split's 32-key chunks in turn, with K and V^T loaded straight from HBM
// into registers, NBUF chunks in flight per wavefront.  The
// wavefronts' (max, sum, o) are merged in LDS; with one split the normalized
// output is written directly, otherwise every split stores an unnormalized
// partial and the last split of its (slot, kv head) to finish, found with a
// counter in ``cnt`` (zero before the launch, left zero after it), merges
// them.
// ============================================================================

// Item b: query row rows[b] (b when null) of q / o, cache slot slots[b] (b
// when null), position len[b].
template <int HD, int DNW, bool PAGED, int NBUF>
__global__ void __launch_bounds__(DNW * 64) attn_decode_bf16_kernel(const bf16* __restrict__ q, KVView kv,
                                                                    bf16* __restrict__ o, float* __restrict__ part,
                                                                    int32_t* __restrict__ cnt, int H,
                                                                    const int32_t* __restrict__ len,
                                                                    int split_len, const int32_t* __restrict__ rows,
                                                                    const int32_t* __restrict__ slots, bool o_tiled) {
  extern __shared__ float dyn[];
  const int split = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int row = rows ? rows[b] : b, slot = slots ? slots[b] : b;
  const int nsplit = gridDim.x;
  const int ctx = len[b] + 1;
  // keys lo .. ctx-1 (a sliding window keeps the last W); the splits start at
  // lo rounded down to a 32-key chunk, and keys below lo are masked
  const int lo = kv.window ? max(0, ctx - kv.window) : 0;
  const int s0 = (lo & ~31) + split * split_len;
  const int s1 = min(ctx, s0 + split_len);
  const int group = H / kv.kv_heads;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = lane & 15, gq = lane >> 4;
  const float sc = LOG2E / sqrtf((float)HD);
  float* sm = dyn;                 // [DNW][16]
  float* sl = dyn + DNW * 16;      // [DNW][16]
  float* so = dyn + 2 * DNW * 16;  // [DNW][group][HD]

  // every load below is unconditional (a load under a lane condition makes
  // the compiler wait for all loads in flight where the branches join):
  // head columns past the group read the group's last head (never stored)
  bf16x8 qf[HD / 32];
  {
    const bf16* qp = q + ((int64_t)row * H + kvh * group + min(col, group - 1)) * HD + gq * 8;
#pragma unroll
    for (int k = 0; k < HD / 32; ++k) qf[k] = *(const bf16x8*)(qp + k * 32);
  }
  f32x4 acc[HD / 16];
#pragma unroll
  for (int d = 0; d < HD / 16; ++d) acc[d] = f32x4{};
  float m_run = -INFINITY, l_run = 0.f;
  const bf16* kb = (const bf16*)kv.k;
  const bf16* vb = (const bf16*)kv.v;
  struct Frag {
    bf16x8 k[2][HD / 32];
    bf16x4 vlo[HD / 16], vhi[HD / 16];
  };
  // issue the K and V^T loads of the 32 keys starting at j0, as two 16-key
  // blocks.  A block's page is looked up once, with a scalar load (a per-lane
  // load of the page table, on which the K/V addresses depend, would wait for
  // every load in flight).  A block at or past the context end reads the last
  // block of the context instead: keys past the context get probability 0
  // (their scores are masked), and the cached values they read are finite.
  auto load = [&](Frag& f, int j0) {
    int64_t kbase[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const int hs = min(j0 + blk * 16, (s1 - 1) & ~15);  // a 16-key block of the context
      const int64_t pg = kv_page_of<PAGED>(kv, slot, hs);
      kbase[blk] = ((pg * kv.kv_heads + kvh) * kv.ps + hs % kv.ps) * HD;
    }
    // K fragment (key col, dims 32k + 8gq ..): 16 bytes at lane * 16 of the
    // block's 1 KB run k; V^T fragment (dim 16d + col, keys 4gq ..): 8 bytes
    // of the block's 512-byte run d
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const bf16* kp = kb + kbase[blk] + lane * 8;
#pragma unroll
      for (int k = 0; k < HD / 32; ++k) f.k[blk][k] = *(const bf16x8*)(kp + k * 512);
    }
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
      const int64_t vo = (d * 16 + col) * 16 + gq * 4;
      f.vlo[d] = *(const bf16x4*)(vb + kbase[0] + vo);
      f.vhi[d] = *(const bf16x4*)(vb + kbase[1] + vo);
    }
  };
  // scores, online softmax update and P V for the 32 keys starting at j0
  auto step = [&](const Frag& f, int j0) {
    f32x4 s[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      s[blk] = f32x4{};
#pragma unroll
      for (int k = 0; k < HD / 32; ++k) s[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.k[blk][k], qf[k], s[blk], 0, 0, 0);
    }
    // s[blk][i]: key j0 + blk*16 + gq*4 + i, head column ``col``
    float mloc = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = j0 + blk * 16 + gq * 4 + i;
        const float v = key < s1 && key >= lo ? s[blk][i] * sc : -INFINITY;
        s[blk][i] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = fmaxf(mloc, lane_xor16(mloc));
    mloc = fmaxf(mloc, lane_xor32(mloc));
    const float m_new = fmaxf(m_run, mloc);  // finite: the first chunk holds a key in [lo, s1)
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) acc[d] *= alpha;
    bf16x8 pb;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = exp2f(s[blk][i] - m_new);
        l_run += p;
        pb[blk * 4 + i] = (bf16)p;
      }
    // O^T += V^T P^T; k index = {gq*4 + 0..3} of block 0, then of block 1
#pragma unroll
    for (int d = 0; d < HD / 16; ++d) {
      const bf16x8 vv = {f.vlo[d][0], f.vlo[d][1], f.vlo[d][2], f.vlo[d][3],
                         f.vhi[d][0], f.vhi[d][1], f.vhi[d][2], f.vhi[d][3]};
      acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vv, pb, acc[d], 0, 0, 0);
    }
  };
  // Wavefront w takes the 32-key chunks w, w + DNW, w + 2 DNW, ... of the
  // split, NBUF of them in flight (a chunk's registers are reloaded with the
  // chunk NBUF later as soon as it has been consumed).  The loop body is one
  // basic block: a load under a branch would be waited for where the branch
  // joins, or moved next to its use.  Chunks of the last round at or past the
  // context end are computed anyway: their keys are masked (probability 0;
  // the running maximum is already finite from the round's first chunk) and
  // their loads read the clamped block.
  auto chunk = [&](int i) { return s0 + (wave + i * DNW) * 32; };
  // Contiguous cache without a window: the first chunk's address does not
  // depend on the context length, so its loads are issued before that length
  // has arrived (one memory round trip less per workgroup), clamped to the
  // slot's positions (the cache is zeroed at allocation and holds only
  // finite values); a chunk that reaches past the context is loaded again
  // below with the context's clamping, so the result does not change.
  Frag f[NBUF];
  const bool spec = !PAGED && kv.window == 0;
  if (spec) {
    const int j0 = split * split_len + wave * 32;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      const int hs = min(j0 + blk * 16, kv.ps - 16);
      const int64_t kbase = (((int64_t)slot * kv.kv_heads + kvh) * kv.ps + hs) * HD;
      const bf16* kp = kb + kbase + lane * 8;
#pragma unroll
      for (int k = 0; k < HD / 32; ++k) f[0].k[blk][k] = *(const bf16x8*)(kp + k * 512);
#pragma unroll
      for (int d = 0; d < HD / 16; ++d) {
        const bf16x4 v = *(const bf16x4*)(vb + kbase + (d * 16 + col) * 16 + gq * 4);
        if (blk == 0) f[0].vlo[d] = v;
        else f[0].vhi[d] = v;
      }
    }
  }
  if (s0 >= ctx) return;
  if (chunk(0) < s1) {  // wave-uniform
    if (!spec || chunk(0) + 32 > s1) load(f[0], chunk(0));
#pragma unroll
    for (int j = 1; j < NBUF; ++j) load(f[j], chunk(j));
    int i = 0;
    for (; chunk(i + NBUF) < s1; i += NBUF) {  // another round follows this one
#pragma unroll
      for (int j = 0; j < NBUF; ++j) {
        step(f[j], chunk(i + j));
        load(f[j], chunk(i + NBUF + j));
      }
    }
#pragma unroll
    for (int j = 0; j < NBUF; ++j) step(f[j], chunk(i + j));  // the last round: chunk(i) < s1
  }
  // per-wave statistics: m uniform over the 4 lane groups of a column; l summed
  l_run += lane_xor16(l_run);
  l_run += lane_xor32(l_run);
  if (gq == 0) {
    sm[wave * 16 + col] = m_run;
    sl[wave * 16 + col] = l_run;
  }
  // acc[d][i]: head-dim d*16 + gq*4 + i, column ``col``
  if (col < group) {
#pragma unroll
    for (int d = 0; d < HD / 16; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) so[(wave * group + col) * HD + d * 16 + gq * 4 + i] = acc[d][i];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < group * HD; idx += DNW * 64) {
    const int c = idx / HD, d = idx % HD;
    float M = -INFINITY;
    for (int w = 0; w < DNW; ++w) M = fmaxf(M, sm[w * 16 + c]);
    float L = 0.f, O = 0.f;
    for (int w = 0; w < DNW; ++w) {
      const float mw = sm[w * 16 + c];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - M);
      L += f * sl[w * 16 + c];
      O += f * so[(w * group + c) * HD + d];
    }
    const int h = kvh * group + c;
    if (nsplit == 1) {
      o[o_tiled ? xt_off(row, h * HD + d) : ((int64_t)row * H + h) * HD + d] = (bf16)(O / L);
    } else {
      // system-scope stores: written through to memory, so the split that
      // merges (on any XCD) reads them without an L2 write-back
      float* pp = part + (((int64_t)b * H + h) * nsplit + split) * (HD + 2);
      __hip_atomic_store(pp + d, O, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      if (d == 0) {
        __hip_atomic_store(pp + HD, M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(pp + HD + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
    }
  }
  if (nsplit == 1) return;
  // The split that arrives last merges the active splits' partials (in split
  // order) and resets its (slot, kv head) counter for the next launch: every
  // thread's partial stores have completed before the workgroup's arrival is
  // counted.
  const int lo31 = lo & ~31;
  const int nact = min(nsplit, (ctx - lo31 + split_len - 1) / split_len);  // splits with s0 < ctx
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  int* flag = (int*)dyn;
  if (threadIdx.x == 0) {
    int32_t* cp = cnt + (int64_t)b * kv.kv_heads + kvh;
    const int arrived = __hip_atomic_fetch_add(cp, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = arrived == nact - 1;
    if (last) __hip_atomic_exchange(cp, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    flag[0] = last;
  }
  __syncthreads();
  if (!flag[0]) return;
  for (int idx = threadIdx.x; idx < group * HD; idx += DNW * 64) {
    const int c = idx / HD, d = idx % HD, h = kvh * group + c;
    const float* pp = part + ((int64_t)b * H + h) * nsplit * (HD + 2);
    // sums in split order.  Up to 8 splits: every partial's (max, sum, o) in
    // one round of independent loads, then the maximum and the sums from
    // registers (7B decode attention 21.6 -> 20.8 us per layer); more
    // splits: rounds of 8 for the maximum, then again for the sums
    float M = -INFINITY, L = 0.f, O = 0.f;
    if (nact <= 8) {
      float mv[8], lv[8], ov[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float* ps = pp + min(u, nact - 1) * (HD + 2);
        mv[u] = __hip_atomic_load(ps + HD, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        lv[u] = __hip_atomic_load(ps + HD + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        ov[u] = __hip_atomic_load(ps + d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (u < nact) M = fmaxf(M, mv[u]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (u < nact) {
          const float f = exp2f(mv[u] - M);
          L += f * lv[u];
          O += f * ov[u];
        }
    } else {
      for (int b0 = 0; b0 < nact; b0 += 8) {
        float mv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          mv[u] = __hip_atomic_load(pp + min(b0 + u, nact - 1) * (HD + 2) + HD, __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_SYSTEM);
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (b0 + u < nact) M = fmaxf(M, mv[u]);
      }
      for (int b0 = 0; b0 < nact; b0 += 8) {
        float mv[8], lv[8], ov[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float* ps = pp + min(b0 + u, nact - 1) * (HD + 2);
          mv[u] = __hip_atomic_load(ps + HD, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          lv[u] = __hip_atomic_load(ps + HD + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          ov[u] = __hip_atomic_load(ps + d, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (b0 + u < nact) {
            const float f = exp2f(mv[u] - M);
            L += f * lv[u];
            O += f * ov[u];
          }
      }
    }
    o[o_tiled ? xt_off(row, h * HD + d) : ((int64_t)row * H + h) * HD + d] = (bf16)(O / L);
  }
}

// ============================================================================
// float32 check mode: a wavefront per (query token, head).  Keys in chunks of
// 64, one per lane for the score; online softmax across the wavefront; lane d
// accumulates output dimensions d (and d + 64) over the chunk from the V^T
// rows.  Serves prefill (cu) and decode (len).
// ============================================================================
template <int HD>
__global__ void __launch_bounds__(64) attn_f32_kernel(const float* __restrict__ q, KVView kv, float* __restrict__ o,
                                                      int T_tokens, int nseq, const int32_t* __restrict__ cu,
                                                      const int32_t* __restrict__ len, int H,
                                                      const int32_t* __restrict__ ent_slot,
                                                      const int32_t* __restrict__ ent_base) {
  constexpr int DL = HD / 64;  // output dimensions per lane
  __shared__ float qs[HD];
  __shared__ float ps[64];
  const int t = blockIdx.x, head = blockIdx.y, lane = threadIdx.x;
  int slot, pos;
  if (len) {
    slot = t;
    pos = len[t];
  } else {
    const int e = seq_of_token(cu, nseq, t);
    slot = ent_slot ? ent_slot[e] : e;
    pos = (ent_base ? ent_base[e] : 0) + t - cu[e];
  }
  const int kvh = head / (H / kv.kv_heads);
  const float* qp = q + ((int64_t)t * H + head) * HD;
  for (int d = lane; d < HD; d += 64) qs[d] = qp[d];
  __syncthreads();
  const float sc = LOG2E / sqrtf((float)HD);
  const float* kb = (const float*)kv.k;
  const float* vb = (const float*)kv.v;
  float m = -INFINITY, l = 0.f, acc[DL] = {};
  const int lo = kv.window ? max(0, pos - kv.window + 1) : 0;  // keys lo .. pos
  for (int j0 = lo; j0 <= pos; j0 += 64) {
    // score of key j0 + lane
    const int j = j0 + lane;
    float sj = -INFINITY;
    if (j <= pos) {
      const float* kp = kb + k_el(kv, slot, kvh, j, 0);  // 8-dim chunks 128 elements apart
      float dot = 0.f;
      for (int d = 0; d < HD; d += 4) {
        const f32x4 kv4 = *(const f32x4*)(kp + (d >> 3) * 128 + (d & 7));
        dot = fmaf(qs[d], kv4[0], dot);
        dot = fmaf(qs[d + 1], kv4[1], dot);
        dot = fmaf(qs[d + 2], kv4[2], dot);
        dot = fmaf(qs[d + 3], kv4[3], dot);
      }
      sj = dot * sc;
    }
    const float m_new = fmaxf(m, wave_max(sj));  // finite: key j0 <= pos is valid
    const float alpha = exp2f(m - m_new);
    const float p = j <= pos ? exp2f(sj - m_new) : 0.f;
    l = l * alpha + wave_sum(p);
    m = m_new;
    ps[lane] = p;
    __syncthreads();
    const int nj = min(64, pos + 1 - j0);
#pragma unroll
    for (int i = 0; i < DL; ++i) {
      const int d = lane + i * 64;
      float a = acc[i] * alpha;
      for (int jj = 0; jj < nj; ++jj) a = fmaf(ps[jj], vb[v_el(kv, slot, kvh, j0 + jj, d)], a);
      acc[i] = a;
    }
    __syncthreads();
  }
  float* op = o + ((int64_t)t * H + head) * HD;
#pragma unroll
  for (int i = 0; i < DL; ++i) op[lane + i * 64] = acc[i] / l;
}

// ============================================================================
// float32 decode: one workgroup of 4 wavefronts per (query, kv head) serves the
// kv head's group of query heads (at most 8), so every key and value is read
// once per group.  Wavefront w takes the 64-key chunks w, w + 4, ...: lane j
// loads key j of the chunk (independent 16-byte loads) and scores it against
// each head of the group in turn, the online softmax runs per head across the
// wavefront, and lane d then accumulates output dimensions d (and d + 64)
// over the chunk's 64 keys from the V^T blocks (16 consecutive keys of a
// dimension are 64 contiguous bytes).  The per-head running state (maximum,
// sum, output accumulator) lives in the wavefront's own LDS rows, so the head
// loop needs no registers per head.  Keys past the context (or before a
// sliding window) get probability 0; their loads read the last key's block.
// The wavefronts' states are merged at the end.
// ============================================================================
constexpr int F32_DEC_MAXG = 8;

template <int HD>
__global__ void __launch_bounds__(256) attn_decode_f32_kernel(const float* __restrict__ q, KVView kv,
                                                              float* __restrict__ o, int H,
                                                              const int32_t* __restrict__ len) {
  constexpr int DL = HD / 64;  // output dimensions per lane
  __shared__ f32x4 qs[F32_DEC_MAXG][HD / 4];
  __shared__ f32x4 ps[4][F32_DEC_MAXG][16];  // probabilities of the chunk's 64 keys
  __shared__ float sm[4][F32_DEC_MAXG], sl[4][F32_DEC_MAXG], sa[4][F32_DEC_MAXG];
  __shared__ float so[4][F32_DEC_MAXG][HD];
  const int b = blockIdx.x, kvh = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = H / kv.kv_heads;  // <= F32_DEC_MAXG (checked by the launcher)
  const int pos = len[b], slot = b;
  const int lo = kv.window ? max(0, pos - kv.window + 1) : 0;  // keys lo .. pos
  const float sc = LOG2E / sqrtf((float)HD);
  const float* kb = (const float*)kv.k;
  const float* vb = (const float*)kv.v;
  // key j of a chunk (clamped into the context) and, at head_dim 64, the
  // chunk's V^T blocks of this lane's dimension: the loads of a chunk are
  // issued before anything waits (for the first chunk, before the query
  // staging), so they cost one memory round trip
  f32x4 kr[HD / 4], vr[16];
  auto load_k = [&](int j0) {
    const float* kp = kb + k_el(kv, slot, kvh, min(max(j0 + lane, lo), pos), 0);
#pragma unroll
    for (int d = 0; d < HD / 4; ++d) kr[d] = *(const f32x4*)(kp + (d >> 1) * 128 + (d & 1) * 4);
  };
  auto load_v = [&](int j0, int d) {
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      const float* vp = vb + v_el(kv, slot, kvh, min(j0 + blk * 16, pos & ~15), d);
#pragma unroll
      for (int c = 0; c < 4; ++c) vr[blk * 4 + c] = *(const f32x4*)(vp + c * 4);
    }
  };
  const int jfirst = (lo & ~63) + wave * 64;
  if (jfirst <= pos) {  // wave-uniform
    load_k(jfirst);
    if constexpr (DL == 1) load_v(jfirst, lane);
  }
  for (int i = tid; i < G * (HD / 4); i += 256)
    qs[i / (HD / 4)][i % (HD / 4)] =
        *(const f32x4*)(q + ((int64_t)b * H + kvh * G + i / (HD / 4)) * HD + 4 * (i % (HD / 4)));
  for (int i = lane; i < G * HD; i += 64) so[wave][i / HD][i % HD] = 0.f;
  if (lane < G) {
    sm[wave][lane] = -INFINITY;
    sl[wave][lane] = 0.f;
  }
  __syncthreads();
  for (int j0 = jfirst; j0 <= pos; j0 += 4 * 64) {
    const int j = j0 + lane;
    const bool valid = j >= lo && j <= pos;
    {
      for (int h = 0; h < G; ++h) {
        // 4 independent partial sums (a single chain waits on every FMA)
        float dp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int d = 0; d < HD / 4; ++d) {
          const f32x4 qv = qs[h][d];
#pragma unroll
          for (int e = 0; e < 4; ++e) dp[e] = fmaf(qv[e], kr[d][e], dp[e]);
        }
        const float dot = (dp[0] + dp[1]) + (dp[2] + dp[3]);
        const float s = valid ? dot * sc : -INFINITY;
        const float m_old = sm[wave][h];
        const float m_new = fmaxf(m_old, wave_max(s));  // finite: the chunk holds a key in [lo, pos]
        const float alpha = exp2f(m_old - m_new);
        const float p = valid ? exp2f(s - m_new) : 0.f;
        const float lsum = wave_sum(p);
        ((float*)ps[wave][h])[lane] = p;
        if (lane == 0) {
          sl[wave][h] = sl[wave][h] * alpha + lsum;
          sm[wave][h] = m_new;
          sa[wave][h] = alpha;
        }
      }
    }
    // o = alpha o + P V over the chunk: lane d reads the 4 16-key blocks of
    // dimension d (blocks past the context read the context's last block;
    // their keys have probability 0).  Only this wavefront touches its rows.
    const bool more = j0 + 4 * 64 <= pos;  // wave-uniform
    if (more) load_k(j0 + 4 * 64);
#pragma unroll
    for (int i = 0; i < DL; ++i) {
      const int d = lane + i * 64;
      if constexpr (DL > 1) load_v(j0, d);
      for (int h = 0; h < G; ++h) {
        float pa[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          const f32x4 pv = ps[wave][h][c];
#pragma unroll
          for (int e = 0; e < 4; ++e) pa[e] = fmaf(pv[e], vr[c][e], pa[e]);
        }
        so[wave][h][d] = so[wave][h][d] * sa[wave][h] + ((pa[0] + pa[1]) + (pa[2] + pa[3]));
      }
    }
    if constexpr (DL == 1) {
      if (more) load_v(j0 + 4 * 64, lane);
    }
  }
  __syncthreads();
  // merge the wavefronts (a wavefront without keys has m = -inf, l = 0)
  for (int idx = tid; idx < G * HD; idx += 256) {
    const int h = idx / HD, d = idx % HD;
    float M = -INFINITY;
    for (int w = 0; w < 4; ++w) M = fmaxf(M, sm[w][h]);
    float L = 0.f, O = 0.f;
    for (int w = 0; w < 4; ++w) {
      const float f = sm[w][h] == -INFINITY ? 0.f : exp2f(sm[w][h] - M);
      L += f * sl[w][h];
      O += f * so[w][h][d];
    }
    o[((int64_t)b * H + kvh * G + h) * HD + d] = O / L;
  }
}

// p[0 .. n) = 0 (a kernel, so that it may be recorded into a graph)
__global__ void __launch_bounds__(256) zero_i32_kernel(int32_t* __restrict__ p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

void launch_zero_i32(int32_t* p, int n, hipStream_t s) {
  if (n > 0) zero_i32_kernel<<<(n + 255) / 256, 256, 0, s>>>(p, n);
}

// ---------------------------------------------------------------- launchers

template <typename T>
void launch_attn_prefill(const T* q, KVView kv, T* o, int T_tokens, int nseq, const int32_t* cu,
                         const int32_t* h_cu, int H, hipStream_t s, const int32_t* ents, const int32_t* h_ents,
                         const int32_t* ent_slot, const int32_t* ent_base, float* lse, bool o_pair) {
  if (T_tokens <= 0 || nseq <= 0) return;
  if constexpr (sizeof(T) == 4) {
    dim3 grid(T_tokens, H);
    if (kv.hd == 64)
      attn_f32_kernel<64><<<grid, 64, 0, s>>>(q, kv, o, T_tokens, nseq, cu, nullptr, H, ent_slot, ent_base);
    else
      attn_f32_kernel<128><<<grid, 64, 0, s>>>(q, kv, o, T_tokens, nseq, cu, nullptr, H, ent_slot, ent_base);
  } else {
    constexpr int TQ = 32 * PREFILL_WAVES;
    int tiles = 0;
    for (int i = 0; i < nseq; ++i) {
      const int e = h_ents ? h_ents[i] : i;
      tiles += (h_cu[e + 1] - h_cu[e] + TQ - 1) / TQ;
    }
    const dim3 grid(tiles * H);  // the kernel maps the linear id to (tile, head)
    auto go = [&](auto kern) {
      kern<<<grid, 64 * PREFILL_WAVES, 0, s>>>(q, kv, o, nseq, cu, H, ents, ent_slot, ent_base, lse, o_pair ? 1 : 0);
    };
    if (kv.hd == 64) {
      if (kv.bt) go(attn_prefill_bf16_kernel<64, true>);
      else go(attn_prefill_bf16_kernel<64, false>);
    } else {
      if (kv.bt) go(attn_prefill_bf16_kernel<128, true>);
      else go(attn_prefill_bf16_kernel<128, false>);
    }
  }
}

// Decode workgroups have DECODE_WAVES wavefronts of 64 keys per iteration.
// Few (slot, kv head) pairs leave most CUs idle, so their keys are split
// towards ~256 workgroups with >= 512 keys per split; many pairs are split
// only for long contexts (<= 1536 keys per split), which bounds the time of the
// longest sequences of a ragged batch.  The last split of a (slot, kv head)
// to finish merges the partials (system-scope stores and loads carry them
// between XCDs without an L2 write-back).  Splitting short contexts further
// (128 keys per split on the 1B-shaped batch) measured slower.
constexpr int DECODE_WAVES = 8;

int plan_decode_splits(int B, int kv_heads, int max_ctx) {
  const int pairs = std::max(1, B * kv_heads);
  if (pairs >= 128) return std::max(1, std::min(16, (max_ctx + 1535) / 1536));  // <= 16 bounds the partials
  const int want = (256 + pairs - 1) / pairs;
  return std::max(1, std::min(want, max_ctx / 512));
}

template <int HD, int NW>
static void decode_launch(const bf16* q, KVView kv, bf16* o, float* part, int32_t* cnt, int B, int H,
                          const int32_t* len, int nsplit, int split_len, hipStream_t s, const int32_t* rows,
                          const int32_t* slots, bool o_tiled) {
  const int group = H / kv.kv_heads;
  const size_t lds = (size_t)(2 * NW * 16 + NW * group * HD) * sizeof(float);
  const dim3 grid(nsplit, kv.kv_heads, B);
  // chunks in flight per wavefront: 1 measured fastest on the 1B-, 7B- and
  // 32B-shaped batches (5.9 / 21.4 / 29.4 us against 6.5 / 22.3 / 29.8 with
  // 2; the 8 wavefronts of a workgroup already keep 8 chunks in flight)
  constexpr int NBUF = 1;
  if (kv.bt)
    attn_decode_bf16_kernel<HD, NW, true, NBUF>
        <<<grid, NW * 64, lds, s>>>(q, kv, o, part, cnt, H, len, split_len, rows, slots, o_tiled);
  else
    attn_decode_bf16_kernel<HD, NW, false, NBUF>
        <<<grid, NW * 64, lds, s>>>(q, kv, o, part, cnt, H, len, split_len, rows, slots, o_tiled);
}

template <typename T>
void launch_attn_decode(const T* q, KVView kv, T* o, float* part, int32_t* cnt, int B, int H, const int32_t* len,
                        int max_ctx, hipStream_t s, const int32_t* rows, const int32_t* slots, bool o_tiled) {
  if (B <= 0) return;
  if constexpr (sizeof(T) == 4) {
    // the float32 path takes rows / slots through launch_attn_prefill
    if (H / kv.kv_heads <= F32_DEC_MAXG) {
      const dim3 grid(B, kv.kv_heads);
      if (kv.hd == 64) attn_decode_f32_kernel<64><<<grid, 256, 0, s>>>(q, kv, o, H, len);
      else attn_decode_f32_kernel<128><<<grid, 256, 0, s>>>(q, kv, o, H, len);
    } else {
      const dim3 grid(B, H);
      if (kv.hd == 64) attn_f32_kernel<64><<<grid, 64, 0, s>>>(q, kv, o, B, 0, nullptr, len, H, nullptr, nullptr);
      else attn_f32_kernel<128><<<grid, 64, 0, s>>>(q, kv, o, B, 0, nullptr, len, H, nullptr, nullptr);
    }
  } else {
    if (kv.window) max_ctx = std::min(max_ctx, kv.window + 31);  // keys from the window's 32-key chunk
    const int nsplit = plan_decode_splits(B, kv.kv_heads, max_ctx);
    const int split_len = ((max_ctx + nsplit - 1) / nsplit + 63) / 64 * 64;
    if (kv.hd == 64)
      decode_launch<64, DECODE_WAVES>(q, kv, o, part, cnt, B, H, len, nsplit, split_len, s, rows, slots, o_tiled);
    else
      decode_launch<128, DECODE_WAVES>(q, kv, o, part, cnt, B, H, len, nsplit, split_len, s, rows, slots, o_tiled);
  }
}

template void launch_attn_prefill<float>(const float*, KVView, float*, int, int, const int32_t*, const int32_t*, int,
                                         hipStream_t, const int32_t*, const int32_t*, const int32_t*, const int32_t*,
                                         float*, bool);
template void launch_attn_prefill<bf16>(const bf16*, KVView, bf16*, int, int, const int32_t*, const int32_t*, int,
                                        hipStream_t, const int32_t*, const int32_t*, const int32_t*, const int32_t*,
                                        float*, bool);
template void launch_attn_decode<float>(const float*, KVView, float*, float*, int32_t*, int, int, const int32_t*,
                                        int, hipStream_t, const int32_t*, const int32_t*, bool);
template void launch_attn_decode<bf16>(const bf16*, KVView, bf16*, float*, int32_t*, int, int, const int32_t*, int,
                                       hipStream_t, const int32_t*, const int32_t*, bool);

}  // namespace axon
