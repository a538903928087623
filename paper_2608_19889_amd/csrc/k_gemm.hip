// Projection GEMMs: out[t][n] = sum_k X[t][k] * W[n][k] (the F.linear
// convention: W is [out, in], X is tokens x in).  bf16 W is fragment-tiled
// (wt_chunk), float W and both X row-major.
//
// Both operands are K-contiguous, so the kernels compute C^T = W X^T with W as
// the MFMA A operand (rows = output features) and X as the B operand (columns
// = tokens): every lane's operand fragment is 8 consecutive k values, one
// 16-byte load, from either operand.
#include "common.h"
#include "kernels.h"

namespace axon {

AXON_DEV float silu_f(float z) { return z / (1.f + __expf(-z)); }

// Store (or add, for the residual stream) four consecutive output columns of
// which ``left`` are inside the matrix.
template <bool ADD>
AXON_DEV void store_cols(float* p, f32x4 v, int left) {
  if (left >= 4) {
    if constexpr (ADD) v += *(const f32x4*)p;
    *(f32x4*)p = v;
  } else {
    for (int j = 0; j < left; ++j) p[j] = ADD ? p[j] + v[j] : v[j];
  }
}

// EPI_ROPE epilogue of one 32 x 32 accumulator block of the fused QKV
// projection: rows nb .. nb+31 (32-aligned, so inside one head), token t;
// v[i] = C[nb + (i/4)*8 + (lane/32)*4 + i%4][t].  Within a head the rows come
// in groups of 8: rotation-pair first halves i0 .. i0+3, then their partners
// i0+hd/2 .. i0+hd/2+3, so lane L < 32 holds first halves and lane L + 32 the
// partners for the same token, and one exchange across the half-wavefronts
// pairs them (both lanes of a pair share t, so they are active together).
// Bias first, then rotate-half RoPE at the token's position; q -> q_out, k ->
// its K page block, v (unrotated) -> its transposed V page block.
// The token's cache slot and position (rope_token) are looked up before the
// k-loop: the lookup is a chain of dependent loads (a binary search over the
// sequence offsets) whose latency the k-loop hides.
struct RopeTok {
  int slot, pos;
};
AXON_DEV RopeTok rope_token(const EpiArgs& ep, int t) {
  if (ep.len) return {t, ep.len[t]};
  const int e = seq_of_token(ep.cu, ep.nseq, t);
  return {ep.ent_slot ? ep.ent_slot[e] : e, (ep.ent_base ? ep.ent_base[e] : 0) + t - ep.cu[e]};
}
AXON_DEV void rope_block(const EpiArgs& ep, int nb, int t, RopeTok tok, const f32x16& v, int lane) {
  const int hd = ep.kv.hd, half = hd / 2, KVh = ep.kv.kv_heads;
  const int head = nb / hd;
  const bool first = lane < 32;
  const bool rotate = head < ep.H + KVh;  // q and k heads (v is stored unrotated)
  // every operand of the block is loaded before its first store: the stores
  // may alias the tables as far as the compiler knows, so loads issued
  // between them would cost one memory round trip per 8-row group
  bf16x4 bb[4];
  f32x4 cs[4], sn[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int i0 = ((nb % hd + g * 8) / 8) * 4;  // first rotation pair of the 8-row group
    const int e0 = first ? i0 : i0 + half;       // element index of this lane's first value
    bb[g] = ep.bias ? *(const bf16x4*)(ep.bias + head * hd + e0) : bf16x4{};
    cs[g] = f32x4{};
    sn[g] = f32x4{};
    if (rotate) {
      cs[g] = *(const f32x4*)(ep.cos_t + (int64_t)tok.pos * half + i0);
      sn[g] = *(const f32x4*)(ep.sin_t + (int64_t)tok.pos * half + i0);
    }
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int i0 = ((nb % hd + g * 8) / 8) * 4;
    const int e0 = first ? i0 : i0 + half;
    float x[4], xp[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = v[g * 4 + j] + (float)bb[g][j];
      xp[j] = lane_xor32(x[j]);
    }
    if (rotate) {
      bf16x4 y;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        y[j] = (bf16)(first ? x[j] * cs[g][j] - xp[j] * sn[g][j] : x[j] * cs[g][j] + xp[j] * sn[g][j]);
      if (head < ep.H) *(bf16x4*)(ep.q_out + ((int64_t)t * ep.H + head) * hd + e0) = y;
      else *(bf16x4*)((bf16*)ep.kv.k + k_el(ep.kv, tok.slot, head - ep.H, tok.pos, e0)) = y;  // 4 dims contiguous
    } else {
      bf16* vc = (bf16*)ep.kv.v;
#pragma unroll
      for (int j = 0; j < 4; ++j) vc[v_el(ep.kv, tok.slot, head - ep.H - KVh, tok.pos, e0 + j)] = (bf16)x[j];
    }
  }
}

// physical 16-byte chunk of logical chunk c in row r of an LDS panel with CH
// chunks per row.  The LDS serves 256 bytes (64 banks) per cycle, so the 16
// lanes of a ds_read_b128 phase (16 consecutive rows, one logical chunk) must
// land in 16 distinct 16-byte bank groups: with 128-byte rows two rows share
// a 256-byte bank line, so the XOR key is row / 2 (row / 4 for 64-byte rows).
template <int CH>
AXON_DEV int swz(int r, int c) {
  if constexpr (CH == 8) return c ^ ((r >> 1) & 7);
  else return c ^ ((r >> 2) & 3);
}

// ============================================================================
// Prefill GEMM: 128 (W rows) x 128 (tokens) x 64 (k) tiles, 4 wavefronts in a
// 2 x 2 arrangement, each owning a 64 x 64 sub-tile = 2 x 2 blocks of
// v_mfma_f32_32x32x16_bf16.  Tiles are staged through LDS, double-buffered;
// a row of 64 k values is 8 chunks of 16 bytes, stored swizzled (swz)
// so that the 16-byte fragment reads of 16 consecutive rows hit distinct banks.
// ============================================================================
namespace pf {
constexpr int BN = 128, BM = 128, BK = 64, CH = BK / 8;
}

template <int EPI>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(const bf16* __restrict__ W, const bf16* __restrict__ X,
                                                        int N, int M, int K, EpiArgs ep) {
  using namespace pf;
  __shared__ bf16x8 lds[2][2][BN * CH];  // [buffer][0 = W, 1 = X][row * 8 + swizzled chunk]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave >> 1, wc = wave & 1;
  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;

  // global -> register staging: 4 chunks of W and 4 of X per thread
  bf16x8 ra[4], rb[4];
  const bf16x8 zero8 = {};
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + i * 256, row = idx >> 3, ch = idx & 7;
      const int n = n0 + row, m = m0 + row;
      ra[i] = n < N ? *(const bf16x8*)(W + wt_chunk(n, (k0 >> 3) + ch, K)) : zero8;
      rb[i] = m < M ? *(const bf16x8*)(X + (ep.xpair ? xp_off(m, k0 + ch * 8, K) : (int64_t)m * K + k0 + ch * 8))
                    : zero8;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + i * 256, row = idx >> 3, ch = idx & 7;
      lds[buf][0][row * CH + swz<8>(row, ch)] = ra[i];
      lds[buf][1][row * CH + swz<8>(row, ch)] = rb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
  RopeTok tok[2] = {};

  const int nk = K / BK;
  gload(0);
  if constexpr (EPI == EPI_ROPE) {  // behind the first tile's loads
#pragma unroll
    for (int b = 0; b < 2; ++b) tok[b] = rope_token(ep, min(m0 + wc * 64 + b * 32 + (lane & 31), M - 1));
  }
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = ks * 2 + (lane >> 5);
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int ra_row = wr * 64 + r * 32 + (lane & 31);
        const int rb_row = wc * 64 + r * 32 + (lane & 31);
        fa[r] = lds[buf][0][ra_row * CH + swz<8>(ra_row, ch)];
        fb[r] = lds[buf][1][rb_row * CH + swz<8>(rb_row, ch)];
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b], acc[a][b], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // epilogue: acc[a][b][i] = C[n][t] with
  //   n = n0 + wr*64 + a*32 + (i/4)*8 + (lane/32)*4 + i%4,  t = m0 + wc*64 + b*32 + lane%32
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int t = m0 + wc * 64 + b * 32 + (lane & 31);
    if (t >= M) continue;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int nb = n0 + wr * 64 + a * 32;  // 32-aligned row block
      if (nb >= N) continue;
      if constexpr (EPI == EPI_ROPE) {
        rope_block(ep, nb, t, tok[b], acc[a][b], lane);
      } else if constexpr (EPI == EPI_SILU) {
        // rows nb..nb+15 are gate rows, nb+16..nb+31 the matching up rows
        // (features (nb / 32) * 16 .. +15: inside one 32-feature slice)
        const int64_t f0 = (nb / 32) * 16;
        bf16* out = (bf16*)ep.out_t + (ep.opair ? xp_off(t, f0, ep.ldo) : (int64_t)t * ep.ldo + f0);
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int f = g * 8 + (lane >> 5) * 4;
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)(silu_f(acc[a][b][g * 4 + j]) * acc[a][b][8 + g * 4 + j]);
          *(bf16x4*)(out + f) = v;
        }
      } else if constexpr (EPI == EPI_GELU) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = nb + g * 8 + (lane >> 5) * 4;  // N % 32 == 0: all 4 rows exist
          const bf16x4 bb = *(const bf16x4*)(ep.bias + n);
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)gelu_tanh_f(acc[a][b][g * 4 + j] + (float)bb[j]);
          *(bf16x4*)((bf16*)ep.out_t + (int64_t)t * ep.ldo + n) = v;
        }
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = nb + g * 8 + (lane >> 5) * 4;
          if (n >= N) continue;
          float* p = ep.out_f32 + (int64_t)t * ep.ldo + n;
          f32x4 v = {acc[a][b][g * 4 + 0], acc[a][b][g * 4 + 1], acc[a][b][g * 4 + 2], acc[a][b][g * 4 + 3]};
          if (ep.bias) {
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] += (float)ep.bias[min(n + j, N - 1)];
          }
          store_cols<EPI == EPI_RESID>(p, v, N - n);
        }
      }
    }
  }
}

// ============================================================================
// Large prefill GEMM: 256 (W rows) x 256 (tokens) tiles, k-tiles of 32, 8
// wavefronts run as two groups that take turns on the matrix cores
// ("ping-pong").  Group g = wave / 4 owns W rows g*128 .. g*128+127 of the
// tile; wave (g, c) owns tokens c*64 .. c*64+63: 4 x 2 blocks of
// v_mfma_f32_32x32x16_bf16.  Waves w and w + 4 share a SIMD, and the groups
// run one phase apart: while one group issues a k-tile's 16 MFMAs, the other
// reads its next fragments from LDS and issues its share of the global->LDS
// loads, then a barrier swaps the roles.  The matrix core of every SIMD thus
// always has one wavefront's uninterrupted MFMA run in flight, and LDS
// latency and load issue are hidden behind it.
// Operands go straight from global memory to LDS (global_load_lds_dwordx4:
// lane L of an instruction writes 16 bytes at LDS offset 16 L) into a ring of
// STAGES k-tiles (32 KB each), issued STAGES-1 tiles ahead; the bank swizzle
// of the 64-byte panel rows is produced by choosing which global chunk each
// lane loads.
// Workgroups are renumbered so that each XCD (workgroup id mod 8) receives a
// contiguous range of tiles, walked in groups of 8 token tiles so that
// neighbouring tiles share operand panels in that XCD's L2.
// ============================================================================
namespace pf2 {
constexpr int BN = 256, BM = 256, BK = 32, STAGES = 4;
constexpr int CH = BK / 8;            // 16-byte chunks per panel row
constexpr int PANEL = BN * CH;        // chunks per operand panel
constexpr int STAGE = 2 * PANEL;      // W panel + X panel
constexpr int LPT = PANEL / 512;      // load instructions per operand per wave per k-tile
constexpr int ROWSTEP = 512 / CH;     // panel rows between a lane's consecutive chunks
constexpr int LDS_BYTES = STAGES * STAGE * 16;
}

AXON_DEV void tile_order(int bid, int gx, int gy, int& pn, int& pm) {
  const int G = gx * gy;
  int logical = bid;
  const int full = G / 8 * 8;
  if (bid < full) logical = (bid % 8) * (full / 8) + bid / 8;
  constexpr int GROUP = 8;
  const int per_group = GROUP * gx;
  const int gid = logical / per_group;
  const int first_m = gid * GROUP;
  const int gsize = min(gy - first_m, GROUP);
  pm = first_m + (logical % per_group) % gsize;
  pn = (logical % per_group) / gsize;
}

// Wait until at most ``after`` k-tiles' loads of this wavefront are in flight
// (2 * LPT load instructions per k-tile).
AXON_DEV void wait_tiles(int after) {
  using namespace pf2;
  static_assert(2 * 2 * LPT <= 63, "vmcnt range");
  if (after >= 2) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * 2 * LPT) : "memory");
  else if (after == 1) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPT) : "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// a workgroup barrier the compiler schedules nothing across
AXON_DEV void phase_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// GROUPED: the mixture-of-experts form (EpiArgs::g_*): workgroup L takes n-tile
// L % gx of m-tile L / gx in the experts' tile sequence; that m-tile belongs to
// expert e (g_toff[e] <= L / gx < g_toff[e+1]), covers its local rows
// m0 .. m0+255 of M = g_off[e+1] - g_off[e], reads X row g_xrow[g_off[e] +
// row] and writes output row g_off[e] + row.
// XP: X in the row-pair layout (xp_off), so a k-tile's two 64-byte pieces of a
// row pair are one 128-byte line.
template <int EPI, bool GROUPED = false, bool XP = false>
__global__ void __launch_bounds__(512, 1) gemm_bf16_256_kernel(const bf16* __restrict__ W,
                                                               const bf16* __restrict__ X, int N, int M, int K,
                                                               EpiArgs ep) {
  using namespace pf2;
  static_assert(STAGES >= 3 && STAGES - 2 <= 2, "wait_tiles covers up to 2 later tiles");
  static_assert(CH == 4, "the W chunk address below assumes one 32-wide tile per k-tile");
  extern __shared__ bf16x8 lds2[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar branches only
  const int grp = wave >> 2, wc = wave & 3;
  const int gx = (N + BN - 1) / BN;
  int pn, pm, n0, m0, rowbase = 0;
  if constexpr (GROUPED) {
    const int mt = blockIdx.x / gx;
    if (mt >= ep.g_toff[ep.g_E]) return;  // surplus workgroup: exits before any barrier
    int lo = 0, hi = ep.g_E - 1;          // the expert: largest e with g_toff[e] <= mt
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (ep.g_toff[mid] <= mt) lo = mid; else hi = mid - 1;
    }
    const int e = lo;
    pn = blockIdx.x % gx;
    pm = mt - ep.g_toff[e];
    rowbase = ep.g_off[e];
    M = ep.g_off[e + 1] - rowbase;  // this expert's rows (>= 1: it has an m-tile)
    W += (int64_t)e * ep.g_wstride;
  } else {
    tile_order(blockIdx.x, gx, (M + BM - 1) / BM, pn, pm);
  }
  n0 = pn * BN;
  m0 = pm * BM;

  // this lane's chunks of a stage: q = (i * 8 + wave) * 64 + lane, i < LPT,
  // row q / CH, logical chunk swz(row, q % CH) (swz is its own inverse)
  const int lrow0 = (wave * 64 + lane) / CH, lch = lane % CH;
  const int64_t rowblk = (int64_t)(K >> 5) * 512;  // elements per 16-row block of tiled W
  auto issue = [&](int stage, int k0) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int row = lrow0 + i * ROWSTEP;
      const int c = swz<CH>(row, lch);
      const int n = min(n0 + row, N - 1), m = min(m0 + row, M - 1);  // rows past the edge: any valid row
      // wt_chunk(n, k0 / 8 + c, K) with k0 a multiple of 32
      const bf16* ws = W + ((int64_t)(n >> 4) * rowblk + (int64_t)k0 * 16 + ((n & 15) + 16 * c) * 8);
      int64_t xr = m;
      if constexpr (GROUPED) xr = ep.g_xrow ? ep.g_xrow[rowbase + m] : rowbase + m;
      const bf16* xs = XP ? X + xp_off(xr, k0 + c * 8, K) : X + xr * K + k0 + c * 8;
      bf16x8* base = lds2 + stage * STAGE + (i * 8 + wave) * 64;
      __builtin_amdgcn_global_load_lds((const void*)ws, (__attribute__((address_space(3))) void*)base, 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)xs, (__attribute__((address_space(3))) void*)(base + PANEL),
                                       16, 0, 0);
    }
  };

  f32x16 acc[4][2];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
  RopeTok tok[2] = {};

  // split K (gridDim.y > 1, float32 partials): this workgroup's share of
  // the k-tiles (gridDim.y divides K / BK)
  const int nk = K / BK / (int)gridDim.y;
  const int kbase = (int)blockIdx.y * nk * BK;
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < nk) issue(st, kbase + st * BK);
  if constexpr (EPI == EPI_ROPE) {  // behind the first stages' loads
#pragma unroll
    for (int b = 0; b < 2; ++b) tok[b] = rope_token(ep, rowbase + min(m0 + wc * 64 + b * 32 + (lane & 31), M - 1));
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (grp == 1) phase_barrier();  // group 1 runs one phase behind group 0

  bf16x8 fa[2][4], fb[2][2];
  // one k-tile: do_issue -- issue the loads of k-tile kt + STAGES - 1;
  // after -- k-tiles of this wavefront's loads left in flight by its wait
  auto ktile = [&](int kt, bool do_issue, int after) {
    // ---- memory phase: fragments of k-tile kt, loads of k-tile kt+STAGES-1
    // into the buffer of k-tile kt-1, which both groups have read (group 1
    // in the phase that just ended)
    const bf16x8* la = lds2 + (kt % STAGES) * STAGE;
    const bf16x8* lb = la + PANEL;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ch = ks * 2 + (lane >> 5);
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int r = grp * 128 + a * 32 + (lane & 31);
        fa[ks][a] = la[r * CH + swz<CH>(r, ch)];
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int r = wc * 64 + b * 32 + (lane & 31);
        fb[ks][b] = lb[r * CH + swz<CH>(r, ch)];
      }
    }
    const int kn = kt + STAGES - 1;
    if (do_issue) issue(kn % STAGES, kbase + kn * BK);
    // group 1's share of k-tile kt+1 must land before group 0 reads it in
    // the phase after the coming barrier; group 0 waits for its own share at
    // the end of its compute phase
    if (grp == 1) wait_tiles(after);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    phase_barrier();
    // ---- compute phase
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks][a], fb[ks][b], acc[a][b], 0, 0, 0);
    __builtin_amdgcn_s_setprio(0);
    if (grp == 0) wait_tiles(after);
    phase_barrier();
  };
  // steady state with constant arguments (no scalar branches around the
  // loads and waits: 1-3% on the 7B shapes), then the last STAGES - 1
  // k-tiles, which issue nothing and leave fewer k-tiles in flight
  static_assert(STAGES == 4, "the tail below peels STAGES - 1 k-tiles");
  int kt = 0;
  for (; kt + STAGES - 1 < nk; ++kt) ktile(kt, true, STAGES - 2);
#pragma unroll
  for (int j = 0; j < STAGES - 1; ++j)
    if (kt < nk) {
      ktile(kt, false, min(STAGES - 2, nk - 2 - kt));
      ++kt;
    }
  if (grp == 0) phase_barrier();  // same barrier count in both groups

  // SiLU epilogue staged through LDS (the ring is idle: every load has landed
  // and, after the barrier, every fragment has been read), so that global
  // memory sees 256-byte rows instead of 8-byte pieces (gate/up GEMM on the
  // 7B shape: 3% faster)
  if constexpr (EPI == EPI_SILU) {
    // 256 tokens x 128 gated features in bf16, rows 272 bytes apart (a
    // half-wavefront's 32 tokens hit distinct bank pairs), then 256-byte rows
    constexpr int LD = 136;
    bf16* st = (bf16*)lds2;
    __syncthreads();
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int tl = wc * 64 + b * 32 + (lane & 31);
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)(silu_f(acc[a][b][g * 4 + j]) * acc[a][b][8 + g * 4 + j]);
          *(bf16x4*)(st + tl * LD + grp * 64 + a * 16 + g * 8 + (lane >> 5) * 4) = v;
        }
    }
    __syncthreads();
    const int nf = min(128, (N - n0) / 2);  // N % 32 == 0
    for (int idx = tid; idx < 256 * 16; idx += 512) {
      // row-major output: 16 chunks of a token row in consecutive lanes; the
      // row-pair layout: 8 lanes fill one 128-byte line (4 chunks of 32
      // features of each row of a pair), then the pair's next 32 features
      const int tl = ep.opair ? ((idx >> 5) << 1) | ((idx >> 2) & 1) : idx >> 4;
      const int ch = ep.opair ? (((idx >> 3) & 3) << 2) | (idx & 3) : idx & 15;
      if (m0 + tl < M && ch * 8 < nf) {
        const int64_t t = rowbase + m0 + tl, f = n0 / 2 + ch * 8;
        *(bf16x8*)((bf16*)ep.out_t + (ep.opair ? xp_off(t, f, ep.ldo) : t * ep.ldo + f)) =
            *(const bf16x8*)(st + tl * LD + ch * 8);
      }
    }
    return;
  }
  // epilogue: acc[a][b][i] = C[n][t],
  //   n = n0 + grp*128 + a*32 + (i/4)*8 + (lane/32)*4 + i%4,  t = m0 + wc*64 + b*32 + lane%32
  // (grouped: output row rowbase + t)
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int tl = m0 + wc * 64 + b * 32 + (lane & 31);
    if (tl >= M) continue;
    const int t = rowbase + tl;
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int nb = n0 + grp * 128 + a * 32;
      if (nb >= N) continue;
      if constexpr (EPI == EPI_ROPE) {
        rope_block(ep, nb, t, tok[b], acc[a][b], lane);
      } else if constexpr (EPI == EPI_SILU) {
        bf16* out = (bf16*)ep.out_t + (int64_t)t * ep.ldo + (nb / 32) * 16;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int f = g * 8 + (lane >> 5) * 4;
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)(silu_f(acc[a][b][g * 4 + j]) * acc[a][b][8 + g * 4 + j]);
          *(bf16x4*)(out + f) = v;
        }
      } else if constexpr (EPI == EPI_GELU) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = nb + g * 8 + (lane >> 5) * 4;  // N % 32 == 0: all 4 rows exist
          const bf16x4 bb = *(const bf16x4*)(ep.bias + n);
          bf16x4 v;
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = (bf16)gelu_tanh_f(acc[a][b][g * 4 + j] + (float)bb[j]);
          *(bf16x4*)((bf16*)ep.out_t + (int64_t)t * ep.ldo + n) = v;
        }
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int n = nb + g * 8 + (lane >> 5) * 4;
          if (n >= N) continue;
          float* p = ep.out_f32 + (int64_t)blockIdx.y * ep.part_stride + (int64_t)t * ep.ldo + n;
          f32x4 v = {acc[a][b][g * 4 + 0], acc[a][b][g * 4 + 1], acc[a][b][g * 4 + 2], acc[a][b][g * 4 + 3]};
          if (ep.bias) {
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] += (float)ep.bias[min(n + j, N - 1)];
          }
          store_cols<EPI == EPI_RESID>(p, v, N - n);
        }
      }
    }
  }
}

// the 256 x 256 kernel instance, its LDS size raised at first use
template <int EPI, bool GROUPED, bool XP>
static auto kern_256() {
  static bool attr = false;
  auto kern = gemm_bf16_256_kernel<EPI, GROUPED, XP>;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, pf2::LDS_BYTES);
    attr = true;
  }
  return kern;
}

template <int EPI, bool XP = false>
static void launch_256(const bf16* W, const bf16* X, int N, int M, int K, const EpiArgs& ep, hipStream_t s) {
  if constexpr (!XP) {
    if (ep.xpair) {
      if constexpr (EPI != EPI_GELU) launch_256<EPI, true>(W, X, N, M, K, ep, s);  // GELU: GPT-2, row-major only
      return;
    }
  }
  const int tiles = ((N + pf2::BN - 1) / pf2::BN) * ((M + pf2::BM - 1) / pf2::BM);
  klaunch(kern_256<EPI, false, XP>(), dim3(tiles), dim3(512), pf2::LDS_BYTES, s, W, X, N, M, K, ep);
}

template <int EPI>
static void launch_grouped(const bf16* W, const bf16* X, int N, int K, int max_rows, const EpiArgs& ep,
                           hipStream_t s) {
  // sum over experts of ceil(rows_e / 256) <= ceil(max_rows / 256) + E
  const int64_t mtiles = (max_rows + pf2::BM - 1) / pf2::BM + ep.g_E;
  const int64_t tiles = mtiles * ((N + pf2::BN - 1) / pf2::BN);
  klaunch(kern_256<EPI, true, false>(), dim3((unsigned)tiles), dim3(512), pf2::LDS_BYTES, s, W, X, N, 0, K, ep);
}

void launch_gemm_bf16_split(const bf16* W, const bf16* X, int N, int M, int K, int ksplit, float* part,
                            int64_t part_stride, hipStream_t s, bool xpair) {
  if (M <= 0) return;
  EpiArgs ep{};
  ep.out_f32 = part;
  ep.ldo = N;
  ep.part_stride = part_stride;
  const int tiles = ((N + pf2::BN - 1) / pf2::BN) * ((M + pf2::BM - 1) / pf2::BM);
  const dim3 grid(tiles, ksplit);
  if (xpair) klaunch(kern_256<EPI_F32, false, true>(), grid, dim3(512), pf2::LDS_BYTES, s, W, X, N, M, K, ep);
  else klaunch(kern_256<EPI_F32, false, false>(), grid, dim3(512), pf2::LDS_BYTES, s, W, X, N, M, K, ep);
}

int gemm_ksplit(int N, int M, int K) {
  if (M < 256 || N < 256) return 1;
  const int tiles = ((N + 255) / 256) * ((M + 255) / 256);
  if (tiles >= 160) return 1;
  const int nk = K / 32;
  for (int ks : {2, 4})
    if (tiles * ks >= 200 && nk % ks == 0 && nk / ks >= 8) return ks;
  return nk % 2 == 0 && nk / 2 >= 8 ? 2 : 1;
}

void launch_gemm_bf16_grouped(const bf16* W, const bf16* X, int N, int K, int max_rows, int epi, const EpiArgs& ep,
                              hipStream_t s) {
  if (max_rows <= 0) return;
  if (epi == EPI_SILU) launch_grouped<EPI_SILU>(W, X, N, K, max_rows, ep, s);
  else launch_grouped<EPI_F32>(W, X, N, K, max_rows, ep, s);
}

void launch_gemm_bf16(const bf16* W, const bf16* X, int N, int M, int K, int epi, const EpiArgs& ep,
                      hipStream_t s) {
  if (M <= 0) return;
  // 256 x 256 tiles unless that leaves most CUs idle (fewer than 160 tiles)
  const int64_t tiles256 = (int64_t)((N + 255) / 256) * ((M + 255) / 256);
  if (M >= 256 && N >= 256 && tiles256 >= 160) {
    switch (epi) {
      case EPI_F32: launch_256<EPI_F32>(W, X, N, M, K, ep, s); return;
      case EPI_RESID: launch_256<EPI_RESID>(W, X, N, M, K, ep, s); return;
      case EPI_SILU: launch_256<EPI_SILU>(W, X, N, M, K, ep, s); return;
      case EPI_ROPE: launch_256<EPI_ROPE>(W, X, N, M, K, ep, s); return;
      case EPI_GELU: launch_256<EPI_GELU>(W, X, N, M, K, ep, s); return;
      default: break;
    }
  }
  dim3 grid((N + pf::BN - 1) / pf::BN, (M + pf::BM - 1) / pf::BM);
  switch (epi) {
    case EPI_F32: klaunch(gemm_bf16_kernel<EPI_F32>, grid, dim3(256), 0, s, W, X, N, M, K, ep); break;
    case EPI_RESID: klaunch(gemm_bf16_kernel<EPI_RESID>, grid, dim3(256), 0, s, W, X, N, M, K, ep); break;
    case EPI_SILU: klaunch(gemm_bf16_kernel<EPI_SILU>, grid, dim3(256), 0, s, W, X, N, M, K, ep); break;
    case EPI_ROPE: klaunch(gemm_bf16_kernel<EPI_ROPE>, grid, dim3(256), 0, s, W, X, N, M, K, ep); break;
    case EPI_GELU: klaunch(gemm_bf16_kernel<EPI_GELU>, grid, dim3(256), 0, s, W, X, N, M, K, ep); break;
    default: break;
  }
}

// ============================================================================
// float32 check-mode GEMM: 64 x 64 tiles, k-step 16, 256 threads with a 4 x 4
// register block each, operands staged k-major in LDS.  Dot products use
// compensated (Kahan) float32 summation, so their error does not grow with K.
// ============================================================================
template <int EPI>
__global__ void __launch_bounds__(256) gemm_f32_kernel(const float* __restrict__ W, const float* __restrict__ X,
                                                       int N, int M, int K, EpiArgs ep) {
  __shared__ float ws[16][68], xs[16][68];
  const int tid = threadIdx.x;
  const int n0 = blockIdx.x * 64, m0 = blockIdx.y * 64;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const int tf = tid & 15, tt = tid >> 4;
  float acc[4][4] = {}, comp[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    {
      const int n = n0 + lr, m = m0 + lr;
      f32x4 wv = {}, xv = {};
      if (n < N) {
        for (int j = 0; j < 4; ++j) wv[j] = (k0 + lk + j < K) ? W[(int64_t)n * K + k0 + lk + j] : 0.f;
      }
      if (m < M) {
        for (int j = 0; j < 4; ++j) xv[j] = (k0 + lk + j < K) ? X[(int64_t)m * K + k0 + lk + j] : 0.f;
      }
      for (int j = 0; j < 4; ++j) { ws[lk + j][lr] = wv[j]; xs[lk + j][lr] = xv[j]; }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
      for (int i = 0; i < 4; ++i) { a[i] = ws[kk][tf * 4 + i]; b[i] = xs[kk][tt * 4 + i]; }
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) {
          const float y = fmaf(a[i], b[j], -comp[i][j]);
          const float t = acc[i][j] + y;
          comp[i][j] = (t - acc[i][j]) - y;
          acc[i][j] = t;
        }
    }
    __syncthreads();
  }
  for (int j = 0; j < 4; ++j) {
    const int t = m0 + tt * 4 + j;
    if (t >= M) continue;
    for (int i = 0; i < 4; ++i) {
      const int n = n0 + tf * 4 + i;
      if (n >= N) continue;
      float* p = ep.out_f32 + (int64_t)t * ep.ldo + n;
      if constexpr (EPI == EPI_RESID) *p += acc[i][j];
      else *p = acc[i][j];
    }
  }
}

// ============================================================================
// float32 check mode, one token (M <= MT): a wavefront per weight row, lanes
// along K with 16-byte loads, compensated (Kahan) per-lane sums reduced across
// the wavefront by shuffles.  K % 4 == 0.
// ============================================================================
template <int EPI, int MT>
__global__ void __launch_bounds__(256) gemv_f32_kernel(const float* __restrict__ W, const float* __restrict__ X,
                                                       int N, int M, int K, EpiArgs ep) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;  // whole wavefronts only: no barrier follows
  float acc[MT], comp[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = comp[t] = 0.f;
  const float* wr = W + (int64_t)n * K;
  for (int k = lane * 4; k < K; k += 256) {
    const f32x4 w = *(const f32x4*)(wr + k);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      if (t >= M) break;
      const f32x4 x = *(const f32x4*)(X + (int64_t)t * K + k);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float y = fmaf(w[j], x[j], -comp[t]);
        const float u = acc[t] + y;
        comp[t] = (u - acc[t]) - y;
        acc[t] = u;
      }
    }
  }
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    if (t >= M) break;
    const float v = wave_sum(acc[t]);
    if (lane == 0) {
      float* p = ep.out_f32 + (int64_t)t * ep.ldo + n;
      if constexpr (EPI == EPI_RESID) *p += v;
      else *p = v;
    }
  }
}

// ============================================================================
// float32 check mode, 2..32 tokens: the token rows are staged through LDS in
// k-chunks of 256 (double-buffered; the next chunk's loads are issued before
// the current chunk is used and stored after it), and each wavefront computes two weight rows for
// every token, lanes along K with compensated (Kahan) per-lane sums and a
// butterfly sum across the wavefront: the token operand is read from HBM once
// per workgroup instead of once per weight row.  Workgroup = 8 rows x MT
// tokens (token groups along gridDim.y, so that there are enough wavefronts
// for the compensated sums).  K % 4 == 0.
// ============================================================================
template <int EPI, int MT>
__global__ void __launch_bounds__(256) gemv_f32_lds_kernel(const float* __restrict__ W, const float* __restrict__ X,
                                                           int N, int M, int K, EpiArgs ep) {
  constexpr int KC = 256;
  __shared__ f32x4 xs[2][MT][KC / 4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // token group blockIdx.y: tokens MT y .. MT y + MT - 1
  X += (int64_t)blockIdx.y * MT * K;
  ep.out_f32 += (int64_t)blockIdx.y * MT * ep.ldo;
  M = min(MT, M - (int)blockIdx.y * MT);
  const int n0 = blockIdx.x * 8 + 2 * w, n1 = n0 + 1;
  const float* w0 = W + (int64_t)min(n0, N - 1) * K;
  const float* w1 = W + (int64_t)min(n1, N - 1) * K;
  float acc0[MT], cmp0[MT], acc1[MT], cmp1[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc0[t] = cmp0[t] = acc1[t] = cmp1[t] = 0.f;
  const int nch = (K + KC - 1) / KC;
  // chunk c of the token rows: loaded into registers (MT * KC / 1024 16-byte
  // pieces per thread), then written to xs[c & 1] (zeros past K and past M)
  constexpr int SP = MT * (KC / 4) / 256;
  f32x4 sv[SP];
  auto stage_load = [&](int c) {
#pragma unroll
    for (int r = 0; r < SP; ++r) {
      const int i = tid + r * 256, t = i / (KC / 4), k = c * KC + 4 * (i % (KC / 4));
      sv[r] = *(const f32x4*)(X + (int64_t)min(t, M - 1) * K + min(k, K - 4));
    }
  };
  auto stage_store = [&](int c) {
#pragma unroll
    for (int r = 0; r < SP; ++r) {
      const int i = tid + r * 256, t = i / (KC / 4), q = i % (KC / 4), k = c * KC + 4 * q;
      xs[c & 1][t][q] = t < M && k < K ? sv[r] : f32x4{};
    }
  };
  stage_load(0);
  stage_store(0);
  f32x4 wv0 = *(const f32x4*)(w0 + min(lane * 4, K - 4)), wv1 = *(const f32x4*)(w1 + min(lane * 4, K - 4));
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    if (c + 1 < nch) stage_load(c + 1);
    const int k = c * KC + lane * 4;
    const f32x4 a0 = wv0, a1 = wv1;
    if (c + 1 < nch) {
      const int kn = min(k + KC, K - 4);
      wv0 = *(const f32x4*)(w0 + kn);
      wv1 = *(const f32x4*)(w1 + kn);
    }
    if (k < K) {
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const f32x4 x = xs[c & 1][t][lane];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float y = fmaf(a0[j], x[j], -cmp0[t]);
          float u = acc0[t] + y;
          cmp0[t] = (u - acc0[t]) - y;
          acc0[t] = u;
          y = fmaf(a1[j], x[j], -cmp1[t]);
          u = acc1[t] + y;
          cmp1[t] = (u - acc1[t]) - y;
          acc1[t] = u;
        }
      }
    }
    // the buffer of chunk c + 1 was last read in chunk c - 1, before the
    // barrier that ended it
    if (c + 1 < nch) stage_store(c + 1);
    __syncthreads();
  }
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    if (t >= M) break;
    const float v0 = wave_sum(acc0[t] - cmp0[t]), v1 = wave_sum(acc1[t] - cmp1[t]);
    if (lane == 0) {
      float* p = ep.out_f32 + (int64_t)t * ep.ldo;
      if (n0 < N) p[n0] = EPI == EPI_RESID ? p[n0] + v0 : v0;
      if (n1 < N) p[n1] = EPI == EPI_RESID ? p[n1] + v1 : v1;
    }
  }
}

void launch_gemm_f32(const float* W, const float* X, int N, int M, int K, int epi, const EpiArgs& ep,
                     hipStream_t s) {
  if (M <= 0) return;
  if (M <= 32 && K % 4 == 0) {
    const bool r = epi == EPI_RESID;
    if (M <= 1) {
      const dim3 g((N + 3) / 4);
      r ? klaunch(gemv_f32_kernel<EPI_RESID, 1>, g, dim3(256), 0, s, W, X, N, M, K, ep)
        : klaunch(gemv_f32_kernel<EPI_F32, 1>, g, dim3(256), 0, s, W, X, N, M, K, ep);
      return;
    }
    const dim3 g((N + 7) / 8, (M + 7) / 8);
    r ? klaunch(gemv_f32_lds_kernel<EPI_RESID, 8>, g, dim3(256), 0, s, W, X, N, M, K, ep)
      : klaunch(gemv_f32_lds_kernel<EPI_F32, 8>, g, dim3(256), 0, s, W, X, N, M, K, ep);
    return;
  }
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  if (epi == EPI_RESID) klaunch(gemm_f32_kernel<EPI_RESID>, grid, dim3(256), 0, s, W, X, N, M, K, ep);
  else klaunch(gemm_f32_kernel<EPI_F32>, grid, dim3(256), 0, s, W, X, N, M, K, ep);
}

// ============================================================================
// split-K reductions
// ============================================================================
// out[i] (accumulate ? += : =) sum over s of parts[s * stride + i], in order
__global__ void __launch_bounds__(256) sum_parts_kernel(float* __restrict__ out, const float* __restrict__ parts,
                                                        int nparts, int64_t stride, int64_t n4, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  f32x4 v = accumulate ? *(const f32x4*)(out + i * 4) : f32x4{};
  for (int p = 0; p < nparts; ++p) v += *(const f32x4*)(parts + p * stride + i * 4);
  *(f32x4*)(out + i * 4) = v;
}

void launch_sum_parts(float* out, const float* parts, int nparts, int64_t stride, int64_t n, int accumulate,
                      hipStream_t s) {
  const int64_t n4 = n / 4;
  if (n4 > 0) sum_parts_kernel<<<(unsigned)((n4 + 255) / 256), 256, 0, s>>>(out, parts, nparts, stride, n4, accumulate);
}
template <typename T>
__global__ void silu_reduce_kernel(const float* __restrict__ parts, int nparts, int64_t part_stride,
                                   T* __restrict__ a, int M, int I) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)M * I) return;
  const int t = (int)(idx / I), f = (int)(idx % I);
  const int rg = (f / 16) * 32 + (f % 16);  // gate row in the interleaved layout; up row = rg + 16
  const float* p = parts + (int64_t)t * 2 * I;
  float g = 0.f, u = 0.f;
  for (int s = 0; s < nparts; ++s) {
    g += p[s * part_stride + rg];
    u += p[s * part_stride + rg + 16];
  }
  a[idx] = from_f32<T>(silu_f(g) * u);
}

template <typename T>
void launch_silu_reduce(const float* parts, int nparts, int64_t part_stride, T* a, int M, int I, hipStream_t s) {
  const int64_t n = (int64_t)M * I;
  if (n <= 0) return;
  silu_reduce_kernel<T><<<(unsigned)((n + 255) / 256), 256, 0, s>>>(parts, nparts, part_stride, a, M, I);
}
template void launch_silu_reduce<float>(const float*, int, int64_t, float*, int, int, hipStream_t);
template void launch_silu_reduce<bf16>(const float*, int, int64_t, bf16*, int, int, hipStream_t);

}  // namespace axon
