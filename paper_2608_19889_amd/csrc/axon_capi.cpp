// C ABI and runtime of the decoder forward pass: configuration and weight-map
// validation (all on the host, before any HIP call), weight repacking, KV
// cache, work buffers, the prefill and decode kernel sequences, and the
// per-(batch, pointers) HIP graph of the decode step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <unordered_map>
#include <vector>

#include "axon.h"
#include "kernels.h"

using namespace axon;

thread_local axon::TimingSlot axon::g_timing_slot;

// Work memory of axon_decode_step_noalloc: one array per GPU, reserved when
// the code object is loaded and held until the process ends.  Host code never
// passes ``scratch`` itself to a kernel (in host code the name is only a
// stand-in); it uses the device address that hipGetSymbolAddress returns for
// the current device, looked up once per device by axon_init_model.
static __device__ __align__(256) unsigned char scratch[AXON_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;

// device id -> address of that device's ``scratch`` (or the lookup's error)
std::mutex g_scratch_mu;
std::map<int, std::pair<void*, std::string>> g_scratch_addr;

void scratch_of_current_device(void** ptr, std::string* err) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *ptr = nullptr;
    *err = std::string("hipGetDevice: ") + hipGetErrorString(e);
    return;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_addr.find(dev);
  if (it == g_scratch_addr.end()) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    std::string msg;
    if (e != hipSuccess) {
      p = nullptr;
      msg = std::string("hipGetSymbolAddress of the no-allocation work array: ") + hipGetErrorString(e);
      (void)hipGetLastError();
    }
    it = g_scratch_addr.emplace(dev, std::make_pair(p, msg)).first;
  }
  *ptr = it->second.first;
  *err = it->second.second;
}

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(AXON_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

std::string shape_str(int ndim, const int64_t* s) {
  if (ndim == 1) return "[" + std::to_string(s[0]) + "]";
  return "[" + std::to_string(s[0]) + ", " + std::to_string(s[1]) + "]";
}

struct Expected {
  int ndim;
  int64_t shape[2];
};

// The weight names and shapes implied by a configuration.
std::vector<std::pair<std::string, Expected>> expected_weights(const axon_config& c) {
  const int64_t D = c.hidden, H = c.n_heads, KV = c.n_kv_heads, hd = c.head_dim, I = c.intermediate,
                V = c.vocab;
  std::vector<std::pair<std::string, Expected>> w;
  if (c.arch == AXON_ARCH_GPT2) {
    // the GPT-2 checkpoint layout: Conv1D weights stored [in, out]
    w.push_back({"transformer.wte.weight", {2, {V, D}}});
    w.push_back({"transformer.wpe.weight", {2, {c.max_positions, D}}});
    for (int i = 0; i < c.n_layers; ++i) {
      const std::string p = "transformer.h." + std::to_string(i) + ".";
      w.push_back({p + "ln_1.weight", {1, {D, 0}}});
      w.push_back({p + "ln_1.bias", {1, {D, 0}}});
      w.push_back({p + "attn.c_attn.weight", {2, {D, 3 * D}}});
      w.push_back({p + "attn.c_attn.bias", {1, {3 * D, 0}}});
      w.push_back({p + "attn.c_proj.weight", {2, {D, D}}});
      w.push_back({p + "attn.c_proj.bias", {1, {D, 0}}});
      w.push_back({p + "ln_2.weight", {1, {D, 0}}});
      w.push_back({p + "ln_2.bias", {1, {D, 0}}});
      w.push_back({p + "mlp.c_fc.weight", {2, {D, I}}});
      w.push_back({p + "mlp.c_fc.bias", {1, {I, 0}}});
      w.push_back({p + "mlp.c_proj.weight", {2, {I, D}}});
      w.push_back({p + "mlp.c_proj.bias", {1, {D, 0}}});
    }
    w.push_back({"transformer.ln_f.weight", {1, {D, 0}}});
    w.push_back({"transformer.ln_f.bias", {1, {D, 0}}});
    return w;
  }
  w.push_back({"model.embed_tokens.weight", {2, {V, D}}});
  for (int i = 0; i < c.n_layers; ++i) {
    const std::string p = "model.layers." + std::to_string(i) + ".";
    w.push_back({p + "input_layernorm.weight", {1, {D, 0}}});
    w.push_back({p + "self_attn.q_proj.weight", {2, {H * hd, D}}});
    w.push_back({p + "self_attn.k_proj.weight", {2, {KV * hd, D}}});
    w.push_back({p + "self_attn.v_proj.weight", {2, {KV * hd, D}}});
    if (c.qkv_bias) {
      w.push_back({p + "self_attn.q_proj.bias", {1, {H * hd, 0}}});
      w.push_back({p + "self_attn.k_proj.bias", {1, {KV * hd, 0}}});
      w.push_back({p + "self_attn.v_proj.bias", {1, {KV * hd, 0}}});
    }
    w.push_back({p + "self_attn.o_proj.weight", {2, {D, H * hd}}});
    w.push_back({p + "post_attention_layernorm.weight", {1, {D, 0}}});
    if (c.n_experts > 0 && i >= c.first_moe_layer) {
      const int64_t Ie = c.moe_intermediate, Is = (int64_t)c.n_shared_experts * Ie;
      w.push_back({p + "mlp.gate.weight", {2, {c.n_experts, D}}});
      for (int e = 0; e < c.n_experts; ++e) {
        const std::string q = p + "mlp.experts." + std::to_string(e) + ".";
        w.push_back({q + "gate_proj.weight", {2, {Ie, D}}});
        w.push_back({q + "up_proj.weight", {2, {Ie, D}}});
        w.push_back({q + "down_proj.weight", {2, {D, Ie}}});
      }
      if (Is > 0) {
        w.push_back({p + "mlp.shared_experts.gate_proj.weight", {2, {Is, D}}});
        w.push_back({p + "mlp.shared_experts.up_proj.weight", {2, {Is, D}}});
        w.push_back({p + "mlp.shared_experts.down_proj.weight", {2, {D, Is}}});
      }
      continue;
    }
    w.push_back({p + "mlp.gate_proj.weight", {2, {I, D}}});
    w.push_back({p + "mlp.up_proj.weight", {2, {I, D}}});
    w.push_back({p + "mlp.down_proj.weight", {2, {D, I}}});
  }
  w.push_back({"model.norm.weight", {1, {D, 0}}});
  if (!c.tie_embeddings) w.push_back({"lm_head.weight", {2, {V, D}}});
  return w;
}

int validate_config(const axon_config& c) {
  auto bad = [](const std::string& m) { return fail(AXON_E_INVALID, "invalid config: " + m); };
  if (c.hidden <= 0 || c.hidden % 64) return bad("hidden must be a positive multiple of 64");
  if (c.n_layers <= 0) return bad("n_layers must be >= 1");
  if (c.n_heads <= 0 || c.n_kv_heads <= 0) return bad("n_heads and n_kv_heads must be >= 1");
  if (c.n_heads % c.n_kv_heads) return bad("n_heads must be a multiple of n_kv_heads");
  if (c.n_heads / c.n_kv_heads > 16) return bad("n_heads / n_kv_heads must be <= 16");
  if (c.n_heads / c.n_kv_heads * c.head_dim > 1536) return bad("(n_heads / n_kv_heads) * head_dim must be <= 1536");
  if (c.head_dim != 64 && c.head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c.intermediate <= 0 || c.intermediate % 64) return bad("intermediate must be a positive multiple of 64");
  if (c.vocab <= 0) return bad("vocab must be >= 1");
  if (!(c.rms_eps > 0.f) || !std::isfinite(c.rms_eps)) return bad("rms_eps must be finite and > 0");
  if (c.arch != AXON_ARCH_LLAMA && c.arch != AXON_ARCH_GPT2) return bad("arch must be AXON_ARCH_LLAMA or AXON_ARCH_GPT2");
  const bool gpt2 = c.arch == AXON_ARCH_GPT2;
  if (!gpt2 && (!(c.rope_theta > 1.0) || !std::isfinite(c.rope_theta))) return bad("rope_theta must be finite and > 1");
  if (c.sliding_window < 0) return bad("sliding_window must be >= 0");
  if (c.qkv_bias != 0 && c.qkv_bias != 1) return bad("qkv_bias must be 0 or 1");
  if (c.tie_embeddings != 0 && c.tie_embeddings != 1) return bad("tie_embeddings must be 0 or 1");
  if (c.dtype != AXON_BF16 && c.dtype != AXON_F32) return bad("dtype must be AXON_BF16 or AXON_F32");
  if (c.max_batch < 1 || c.max_batch > 1024) return bad("max_batch must be in [1, 1024]");
  if (c.max_seq < 1 || c.max_seq > (1 << 20)) return bad("max_seq must be in [1, 2^20]");
  if (c.max_tokens < 0) return bad("max_tokens must be >= 0");
  if (c.kv_page_size < 0 || c.kv_page_size % 16) return bad("kv_page_size must be 0 or a multiple of 16");
  if (c.kv_page_size > 0 && c.kv_num_pages < 1) return bad("kv_num_pages must be >= 1 for a paged cache");
  if (c.n_experts != 0) {
    if (c.n_experts < 2 || c.n_experts > 256) return bad("n_experts must be 0 or in [2, 256]");
    if (c.top_k < 1 || c.top_k > 8 || c.top_k > c.n_experts) return bad("top_k must be in [1, min(n_experts, 8)]");
    if (c.moe_intermediate <= 0 || c.moe_intermediate % 64) return bad("moe_intermediate must be a positive multiple of 64");
    if (c.n_shared_experts < 0) return bad("n_shared_experts must be >= 0");
    if (c.first_moe_layer < 0 || c.first_moe_layer > c.n_layers) return bad("first_moe_layer must be in [0, n_layers]");
    if (c.norm_topk_prob != 0 && c.norm_topk_prob != 1) return bad("norm_topk_prob must be 0 or 1");
    if (c.dtype != AXON_BF16) return bad("mixture-of-experts layers need dtype AXON_BF16");
  }
  if (gpt2) {
    if (c.n_kv_heads != c.n_heads) return bad("GPT-2 attention has n_kv_heads == n_heads");
    if (c.qkv_bias != 1 || c.tie_embeddings != 1) return bad("GPT-2 has qkv_bias == 1 and tie_embeddings == 1");
    if (c.dtype != AXON_BF16) return bad("the GPT-2 family needs dtype AXON_BF16");
    if (c.n_experts != 0) return bad("the GPT-2 family has no mixture-of-experts layers (n_experts 0)");
    if (c.max_positions < 1 || c.max_seq > c.max_positions) return bad("GPT-2 needs 1 <= max_seq <= max_positions");
    if (c.hidden > 8192) return bad("GPT-2 hidden must be <= 8192");
  }
  return AXON_OK;
}

struct LayerW {
  void* wqkv;   // [(H+2KV)hd, D]
  void* bqkv;   // [(H+2KV)hd] or null
  void* wo;     // [D, H hd]
  void* wgu;    // [2I, D], 16 gate rows then the 16 matching up rows, repeated
  void* wd;     // [D, I]
  void* gin;    // [D]
  void* gpost;  // [D]
  // mixture-of-experts layer: the router [E rounded up to 32, D] (padding rows
  // zero), every expert's interleaved gate/up [2 Ie, D] and down [D, Ie]
  // stacked expert after expert; wgu / wd then hold the shared experts (a
  // dense MLP of n_shared * Ie), or are null
  // GPT-2: LayerNorm biases, O and MLP biases (wgu then holds c_fc [I, D]
  // and wd c_proj [D, I]; bqkv the c_attn bias)
  void* gin_b = nullptr;
  void* gpost_b = nullptr;
  void* bo = nullptr;
  void* bfc = nullptr;
  void* bd = nullptr;
  bool moe = false;
  void* wrouter = nullptr;
  void* wgu_e = nullptr;
  void* wd_e = nullptr;
};

struct TimingRec {
  int cls, d0, d1, d2;
  hipEvent_t a, b;
};

struct GraphKey {
  int batch;
  const void* tok;
  const void* logits;
  const void* next;
  const void* cu = nullptr;  // decode-only continuous-batching step: its cu_seqlens
  bool operator<(const GraphKey& o) const {
    return std::tie(batch, tok, logits, next, cu) < std::tie(o.batch, o.tok, o.logits, o.next, o.cu);
  }
};

// Backward-pass state, allocated by the first axon_loss_and_grads call: the
// activations the forward pass keeps per layer, the weights transposed and
// tiled (the B operand of dX = dY W), and the gradient work buffers.
struct TrainLayer {
  float *xin, *xmid, *lse, *gu;  // layer input, residual after attention, log2-sum-exp [T][H], gate/up [T][2I]
  bf16 *h1, *h2, *q, *o, *a;     // normed inputs, rotated q, attention output, gated activation
  bf16 *wqkvT, *woT, *wguT, *wdT;
};
struct TrainBufs {
  bool ready = false;
  int Tc = 0, Tp = 0, Vp = 0;
  int SP = 0;       // positions per sequence in the attention backward's packed copies
  int64_t W = 0;    // max_batch * SP
  bf16 *kr, *vr, *kt, *qt, *dot;
  std::vector<TrainLayer> L;
  float *xfin, *logits, *rowloss, *valid, *lserow, *scal, *dx, *dtmp, *dgrow, *dqf, *dkf, *dvf, *dsum, *dqkvf,
      *colpart, *gtmp, *dkh, *dvh;
  float* statp;     // attention backward: log2-sum-exp and D in packed per-head rows [2][H][W]
  bf16 *hf, *dlog, *dxb, *dgu, *dob, *dqkv, *tra, *trs, *trb, *headT;
};

// Per-step work buffers of the bf16 decode step: the model's own (allocated
// at init), or carved from the no-allocation array.
struct DecodeWs {
  float* x;          // residual rows [B][D]
  bf16* xg;          // bf16(x * g) [B][D]
  float* ss;         // sums-of-squares partials [D / 8][B]
  bf16* q;           // rotated queries [B][H hd]
  bf16* o;           // attention output [B][H hd]
  bf16* a;           // gated activation [B][I]
  float* attn_part;  // decode attention split partials
  int32_t* attn_cnt; // decode attention split arrival counters [B][KV], zero between launches
  float* gemv_part;  // split-K partials of the projections
  float* am_val;     // head argmax partials [B][V / rows of the head tile]
  int32_t* am_idx;
};

}  // namespace

struct axon_model {
  axon_config cfg{};
  int esz = 2;
  bool bf = true;
  std::vector<void*> dev_allocs;
  void* embed = nullptr;
  void* lm_head = nullptr;
  void* gfinal = nullptr;
  void* gfinal_b = nullptr;  // GPT-2: final LayerNorm bias
  void* wpe = nullptr;       // GPT-2: learned positions [max_positions][D], row-major
  std::vector<LayerW> layers;
  TrainBufs train;
  // KV cache
  void* kcache = nullptr;
  void* vcache = nullptr;
  int64_t kv_layer_elems = 0;
  int ps = 0;
  int bt_stride = 0;
  int32_t* d_bt = nullptr;
  int32_t* h_bt = nullptr;  // pinned host copy of the page table
  hipEvent_t bt_copied = nullptr;
  float* rope_cos = nullptr;
  float* rope_sin = nullptr;
  // work buffers
  int rows = 0;
  float* x = nullptr;
  void* h = nullptr;
  float* qkv = nullptr;
  void* q = nullptr;
  void* o = nullptr;
  void* a = nullptr;
  void* hlast = nullptr;
  float* gu_f32 = nullptr;
  float* logits_int = nullptr;
  float* attn_part = nullptr;
  int32_t* attn_cnt = nullptr;  // [max_batch][KV], zero between decode attention launches
  float* gemv_part = nullptr;  // split-K partial sums of the decode projections
  float* gemm_part = nullptr;  // split-K partial sums of the narrow prefill / training GEMMs
  int64_t gemm_part_floats = 0;
  float* ss = nullptr;       // per-workgroup sums of squares of x rows
  void* xg = nullptr;        // bf16(x * g) for the next normalized projection
  int ss_n = 0;              // number of partials currently in ss
  float* am_val = nullptr;   // per-workgroup argmax partials of the head
  int32_t* am_idx = nullptr;
  int32_t* d_len = nullptr;
  std::vector<int> h_len;
  // this device's no-allocation work array (or why it is unavailable)
  void* scratch_ptr = nullptr;
  std::string scratch_err;
  DecodeWs own_ws() const {
    return DecodeWs{x, (bf16*)xg, ss, (bf16*)q, (bf16*)o, (bf16*)a, attn_part, attn_cnt, gemv_part, am_val, am_idx};
  }
  // per-entry arrays of a continuous-batching step (6 x max_batch int32):
  // slot, base position, chunk entries, single-token rows / slots / positions
  // mixture-of-experts work buffers (sized for the most tokens of a call)
  float* moe_logits = nullptr;  // [rows][E rounded up to 32]
  int32_t* moe_topi = nullptr;  // [rows][k]
  float* moe_topw = nullptr;
  int32_t* moe_cnt = nullptr;   // [E], then row / tile offsets [E+1] each
  int32_t* moe_off = nullptr;
  int32_t* moe_toff = nullptr;
  int32_t* moe_xrow = nullptr;  // [rows * k]
  int32_t* moe_inv = nullptr;
  void* moe_a = nullptr;        // [rows * k][Ie] bf16 gated expert activations
  float* moe_y = nullptr;       // [rows * k][D] expert outputs
  bool moe_model() const { return cfg.n_experts > 0; }
  bool gpt2() const { return cfg.arch == AXON_ARCH_GPT2; }
  // keys a query at context length ctx attends to (timing records)
  int keys_read(int ctx) const { return cfg.sliding_window > 0 ? std::min(ctx, cfg.sliding_window) : ctx; }
  int moe_ep() const { return (cfg.n_experts + 31) / 32 * 32; }
  int32_t* d_step = nullptr;
  int32_t* h_step = nullptr;  // pinned staging copy
  hipEvent_t step_copied = nullptr;
  int active = 0;
  hipStream_t cap_stream = nullptr;
  std::map<GraphKey, hipGraphExec_t> graphs;
  bool use_graphs = true;
  std::string enqueue_err;  // set while enqueueing a step when a launch had no kernel
  // kernel timing (measurement mode)
  bool timing = false;
  std::vector<TimingRec> trecs;
  std::vector<hipEvent_t> tpool;
  size_t tnext = 0;

  hipEvent_t tevent() {
    if (tnext == tpool.size()) {
      hipEvent_t e = nullptr;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      tpool.push_back(e);
    }
    return tpool[tnext++];
  }
  // Time ``launch`` when timing is on.  Single-kernel classes (projections)
  // carry the events in their own dispatch; multi-kernel ones are bracketed
  // by event records on s.
  template <typename F>
  void timed(int cls, int d0, int d1, int d2, hipStream_t s, F&& launch) {
    if (!timing) {
      launch();
      return;
    }
    TimingRec r{cls, d0, d1, d2, tevent(), tevent()};
    if (!r.a || !r.b) {
      launch();
      return;
    }
    if (cls == 0 || cls == 1) {
      axon::g_timing_slot = axon::TimingSlot{r.a, r.b};
      launch();
      const bool used = axon::g_timing_slot.start == nullptr;
      axon::g_timing_slot = axon::TimingSlot{};
      if (used) trecs.push_back(r);
      return;
    }
    (void)hipEventRecord(r.a, s);
    launch();
    (void)hipEventRecord(r.b, s);
    trecs.push_back(r);
  }

  int D() const { return cfg.hidden; }
  int H() const { return cfg.n_heads; }
  int KVh() const { return cfg.n_kv_heads; }
  int hd() const { return cfg.head_dim; }
  int I() const { return cfg.intermediate; }
  int V() const { return cfg.vocab; }
  int nqkv() const { return (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim; }

  KVView kv(int l, bool paged_table) const {
    KVView v;
    v.k = (char*)kcache + (int64_t)l * kv_layer_elems * esz;
    v.v = (char*)vcache + (int64_t)l * kv_layer_elems * esz;
    v.bt = paged_table ? d_bt : nullptr;
    v.bt_stride = bt_stride;
    v.ps = ps;
    v.kv_heads = cfg.n_kv_heads;
    v.hd = cfg.head_dim;
    v.window = cfg.sliding_window;
    return v;
  }
  bool paged() const { return cfg.kv_page_size > 0; }
};

namespace {

int dev_alloc(axon_model* m, void** p, size_t bytes) {
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? AXON_E_OOM : AXON_E_HIP,
                "device allocation of " + std::to_string(bytes) + " bytes failed: " + hipGetErrorString(e));
  }
  m->dev_allocs.push_back(*p);
  return AXON_OK;
}

void release(axon_model* m) {
  for (hipEvent_t e : m->tpool) (void)hipEventDestroy(e);
  for (auto& kv : m->graphs) (void)hipGraphExecDestroy(kv.second);
  m->graphs.clear();
  for (void* p : m->dev_allocs) (void)hipFree(p);
  m->dev_allocs.clear();
  if (m->h_bt) (void)hipHostFree(m->h_bt);
  if (m->bt_copied) (void)hipEventDestroy(m->bt_copied);
  if (m->h_step) (void)hipHostFree(m->h_step);
  if (m->step_copied) (void)hipEventDestroy(m->step_copied);
  if (m->cap_stream) (void)hipStreamDestroy(m->cap_stream);
  delete m;
}

// ------------------------------------------------------------------ forward
// xpair / opair: X / the bf16 output out_t in the row-pair layout (bf16 only)
template <typename T>
void gemm_many(axon_model* m, const void* W, const void* X, int N, int M, int K, int epi, float* out_f32,
               void* out_t, int ldo, hipStream_t s, const EpiArgs* rope = nullptr, const void* bias = nullptr,
               bool xpair = false, bool opair = false) {
  EpiArgs ep = rope ? *rope : EpiArgs{};
  if (bias) ep.bias = (const bf16*)bias;
  ep.out_f32 = out_f32;
  ep.out_t = out_t;
  ep.ldo = ldo;
  ep.xpair = xpair ? 1 : 0;
  ep.opair = opair ? 1 : 0;
  m->timed(1, N, M, K, s, [&] {
    if constexpr (sizeof(T) == 2)
      launch_gemm_bf16((const bf16*)W, (const bf16*)X, N, M, K, epi, ep, s);
    else
      launch_gemm_f32((const float*)W, (const float*)X, N, M, K, epi, ep, s);
  });
}

// Split-K choice for a bf16 GEMM with a float32 result: the split
// gemm_ksplit takes when its partials fit m->gemm_part, else 1.
int split_for(axon_model* m, int N, int M, int K) {
  const int ks = gemm_ksplit(N, M, K);
  return ks > 1 && (int64_t)ks * M * N <= m->gemm_part_floats ? ks : 1;
}

// out (accumulate ? += : =) X W^T (float32 [M][N], rows N apart), split over
// K when the output has few 256-tiles (partials summed in order)
void gemm_f32_out(axon_model* m, const void* W, const void* X, int N, int M, int K, float* out, bool accumulate,
                  hipStream_t s) {
  const int ks = split_for(m, N, M, K);
  if (ks > 1) {
    m->timed(1, N, M, K, s, [&] {
      launch_gemm_bf16_split((const bf16*)W, (const bf16*)X, N, M, K, ks, m->gemm_part, (int64_t)M * N, s);
    });
    launch_sum_parts(out, m->gemm_part, ks, (int64_t)M * N, (int64_t)M * N, accumulate ? 1 : 0, s);
  } else {
    gemm_many<bf16>(m, W, X, N, M, K, accumulate ? EPI_RESID : EPI_F32, out, nullptr, N, s);
  }
}

// Split of an inference prefill's residual projection (O, dense down): by
// its shape alone, never by the token count, so that a prompt fed in chunks
// takes the same k-order as the whole prompt and gives the same bits.  Narrow
// outputs (hidden <= 2048: too few 256-tiles at any prompt length) split K in
// two.
int prefill_split(axon_model* m, int N, int M, int K) {
  const int nk = K / 32;
  if (N > 2048 || K < 1024 || nk % 2 || (int64_t)2 * M * N > m->gemm_part_floats) return 1;
  return 2;
}

// x += X W^T, then h = RMSNorm(x) g for ``rows`` rows (the last row of each
// sequence when cu_last is set): a split-K GEMM's partials are summed into x
// by the normalization kernel itself.  xpair / hpair: X / h in the row-pair
// layout.
void gemm_resid_norm(axon_model* m, const void* W, const bf16* X, int T, int K, const bf16* g, bf16* h, int rows,
                     const int32_t* cu_last, hipStream_t s, bool by_shape = false, bool xpair = false,
                     bool hpair = false) {
  const int D = m->D(), ks = by_shape ? prefill_split(m, D, T, K) : split_for(m, D, T, K);
  if (ks > 1) {
    m->timed(1, D, T, K, s, [&] {
      launch_gemm_bf16_split((const bf16*)W, X, D, T, K, ks, m->gemm_part, (int64_t)T * D, s, xpair);
    });
    launch_resid_rmsnorm<bf16>(m->x, m->gemm_part, ks, (int64_t)T * D, g, h, rows, D, m->cfg.rms_eps, cu_last, s,
                               hpair);
  } else {
    gemm_many<bf16>(m, W, X, D, T, K, EPI_RESID, m->x, nullptr, D, s, nullptr, nullptr, xpair);
    launch_resid_rmsnorm<bf16>(m->x, nullptr, 0, 0, g, h, rows, D, m->cfg.rms_eps, cu_last, s, hpair);
  }
}

// Few-token projection in float32 check mode.
void gemm_few_f32(axon_model* m, const void* W, const void* X, int N, int M, int K, int epi, float* out,
                  int ldo, hipStream_t s) {
  EpiArgs ep{out, nullptr, ldo, 0};
  m->timed(0, N, M, K, s, [&] { launch_gemm_f32((const float*)W, (const float*)X, N, M, K, epi, ep, s); });
}

// Fused few-token projection; a shape with no kernel is recorded in
// m->enqueue_err (checked by the caller once the step is enqueued).
void gemv_step(axon_model* m, const GemvArgs& a, int epi, hipStream_t s) {
  bool ok = true;
  m->timed(0, a.N, a.M, a.K, s, [&] { ok = launch_gemv_fused(a, epi, s); });
  if (!ok && m->enqueue_err.empty())
    m->enqueue_err = "no fused projection kernel for N=" + std::to_string(a.N) + " K=" + std::to_string(a.K) +
                     " M=" + std::to_string(a.M) + " epilogue " + std::to_string(epi);
}

// Routed experts of a mixture-of-experts layer over T rows of normed
// activations h (bf16): router logits (float) -> top-k routing -> grouped plan
// -> grouped gate/up with the SiLU gate over the gathered token rows ->
// grouped down, one float row per (token, choice) in m->moe_y.  Up to 64
// tokens (decode) the experts' weights are streamed once by the grouped
// few-token projection (a workgroup per 64-row block and expert, the
// expert's rows gathered from h); wider batches take the grouped GEMM.
void moe_routed(axon_model* m, const LayerW& w, const bf16* h, int T, hipStream_t s) {
  const axon_config& c = m->cfg;
  const int D = m->D(), E = c.n_experts, k = c.top_k, Ie = c.moe_intermediate, Ep = m->moe_ep();
  if (T <= GEMV_MAX_M) {
    GemvArgs ra{};
    ra.W = (const bf16*)w.wrouter; ra.N = Ep; ra.K = D; ra.M = T; ra.X = h;
    ra.out_f32 = m->moe_logits; ra.ldo = Ep; ra.part = m->gemv_part;
    gemv_step(m, ra, GV_F32, s);
  } else {
    gemm_many<bf16>(m, w.wrouter, h, Ep, T, D, EPI_F32, m->moe_logits, nullptr, Ep, s);
  }
  launch_moe_route(m->moe_logits, Ep, T, E, k, c.norm_topk_prob, m->moe_topi, m->moe_topw, s);
  launch_moe_plan(m->moe_topi, T, E, k, m->moe_cnt, m->moe_off, m->moe_toff, m->moe_xrow, m->moe_inv, s);
  if (T <= GEMV_MAX_M) {
    GemvArgs ga{};
    ga.W = (const bf16*)w.wgu_e; ga.N = 2 * Ie; ga.K = D; ga.M = T; ga.X = h;
    ga.out_t = (bf16*)m->moe_a; ga.ldo = Ie;
    ga.g_off = m->moe_off; ga.g_xrow = m->moe_xrow; ga.g_wstride = (int64_t)2 * Ie * D;
    m->timed(4, 2 * Ie, T, D, s, [&] { launch_gemv_grouped(ga, GV_SILU, E, s); });
    GemvArgs da{};
    da.W = (const bf16*)w.wd_e; da.N = D; da.K = Ie; da.M = T; da.X = (const bf16*)m->moe_a;
    da.out_f32 = m->moe_y; da.ldo = D;
    da.g_off = m->moe_off; da.g_xrow = nullptr; da.g_wstride = (int64_t)D * Ie;
    m->timed(4, D, T, Ie, s, [&] { launch_gemv_grouped(da, GV_F32, E, s); });
    return;
  }
  // the token rows in grouped order, contiguous, in moe_y's memory (free
  // until the down projection writes it, after gate/up has read them)
  bf16* xg = (bf16*)m->moe_y;
  launch_moe_gather(h, m->moe_xrow, T * k, D, xg, s);
  EpiArgs g{};
  g.g_off = m->moe_off;
  g.g_toff = m->moe_toff;
  g.g_E = E;
  g.g_xrow = nullptr;
  g.g_wstride = (int64_t)2 * Ie * D;
  g.out_t = m->moe_a;
  g.ldo = Ie;
  m->timed(1, 2 * Ie, T * k, D, s, [&] {
    launch_gemm_bf16_grouped((const bf16*)w.wgu_e, xg, 2 * Ie, D, T * k, EPI_SILU, g, s);
  });
  g.g_xrow = nullptr;
  g.g_wstride = (int64_t)D * Ie;
  g.out_t = nullptr;
  g.out_f32 = m->moe_y;
  g.ldo = D;
  m->timed(1, D, T * k, Ie, s, [&] {
    launch_gemm_bf16_grouped((const bf16*)w.wd_e, (const bf16*)m->moe_a, D, Ie, T * k, EPI_F32, g, s);
  });
}

// Mixture-of-experts MLP of a layer over T rows of normed activations h,
// added to the residual stream x: routed experts, shared experts (dense,
// residual epilogue), then the weighted combine of each token's k expert
// rows into x.
void enqueue_moe(axon_model* m, const LayerW& w, const bf16* h, int T, hipStream_t s) {
  const int D = m->D(), Is = m->cfg.n_shared_experts * m->cfg.moe_intermediate;
  moe_routed(m, w, h, T, s);
  if (Is > 0) {
    gemm_many<bf16>(m, w.wgu, h, 2 * Is, T, D, EPI_SILU, nullptr, m->a, Is, s);
    gemm_many<bf16>(m, w.wd, m->a, D, T, Is, EPI_RESID, m->x, nullptr, D, s);
  }
  launch_moe_combine(m->x, m->moe_y, m->moe_inv, m->moe_topw, T, D, m->cfg.top_k, s);
}


// A continuous-batching step: entry e appends tokens cu[e] .. cu[e+1]-1 to
// slot slot[e] from position base[e].  Entries of >= 2 tokens (prompt chunks)
// go through the prefill attention kernel, single tokens through the decode
// attention kernel (one workgroup per (item, kv head) reads the slot's keys
// once for the head group).
struct StepPlan {
  int n = 0;
  const int32_t* d_slot = nullptr;
  const int32_t* d_base = nullptr;
  int nc = 0;                          // chunk entries
  const int32_t* d_chunks = nullptr;
  const int32_t* h_chunks = nullptr;
  int nd = 0;                          // single-token entries
  const int32_t* d_drow = nullptr;     // token row
  const int32_t* d_dslot = nullptr;
  const int32_t* d_dpos = nullptr;
  int dctx = 0;                        // summed keys attended by the single-token entries
};

// Epilogue arguments of the bf16 QKV GEMM with bias + RoPE + KV write fused:
// prefill positions from cu (nseq sequences), decode positions from len.
EpiArgs rope_epi(axon_model* m, const LayerW& w, const KVView& kv, const int32_t* cu, int nseq, const int32_t* len) {
  EpiArgs e{};
  e.bias = (const bf16*)w.bqkv;
  e.cos_t = m->rope_cos;
  e.sin_t = m->rope_sin;
  e.q_out = (bf16*)m->q;
  e.kv = kv;
  e.cu = cu;
  e.nseq = nseq;
  e.len = len;
  e.H = m->H();
  return e;
}

// Prefill of B fresh sequences in slots 0..B-1, or (plan != nullptr) a
// continuous-batching step of B entries.
template <typename T>
void enqueue_prefill(axon_model* m, int B, int Ttok, const int32_t* d_tokens, const int32_t* d_cu,
                     const int32_t* h_cu, int all_logits, float* d_logits, int32_t* d_next, hipStream_t s,
                     const StepPlan* plan = nullptr) {
  const int D = m->D(), H = m->H(), hd = m->hd(), I = m->I(), V = m->V(), nq = m->nqkv();
  const float eps = m->cfg.rms_eps;
  T* h = (T*)m->h;
  const int32_t* ent_slot = plan ? plan->d_slot : nullptr;
  const int32_t* ent_base = plan ? plan->d_base : nullptr;
  if (plan) launch_set_step_lengths(d_cu, ent_slot, ent_base, m->d_len, B, s);
  else launch_set_lengths(d_cu, m->d_len, B, s);
  const bool gpt2 = m->gpt2();  // bf16 only (checked at init)
  // dense Llama-family bf16 models pass the GEMMs' token operands (h, o, a) in
  // the row-pair layout; o only when no single-token entry (decode attention
  // writes row-major rows) shares the step
  const bool xp = sizeof(T) == 2 && !gpt2 && !m->moe_model();
  const bool o_pair = xp && !(plan && plan->nd > 0);
  if (gpt2)
    launch_embed_pos_ln(d_tokens, (const bf16*)m->embed, (const bf16*)m->wpe, (const bf16*)m->layers[0].gin,
                        (const bf16*)m->layers[0].gin_b, m->x, (bf16*)h, Ttok, D, V, m->cfg.max_positions, eps, d_cu,
                        B, ent_base, nullptr, s);
  else
    launch_embed_rmsnorm<T>(d_tokens, (const T*)m->embed, (const T*)m->layers[0].gin, m->x, h, Ttok, D, V, eps, s,
                            xp);
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const LayerW& w = m->layers[l];
    KVView kv = m->kv(l, m->paged());
    if constexpr (sizeof(T) == 2) {
      // bias, RoPE (GPT-2: the identity) and the KV-cache write in the QKV
      // GEMM's epilogue
      EpiArgs re = rope_epi(m, w, kv, d_cu, B, nullptr);
      re.ent_slot = ent_slot;
      re.ent_base = ent_base;
      gemm_many<T>(m, w.wqkv, h, nq, Ttok, D, EPI_ROPE, nullptr, nullptr, nq, s, &re, nullptr, xp);
    } else {
      gemm_many<T>(m, w.wqkv, h, nq, Ttok, D, EPI_F32, m->qkv, nullptr, nq, s);
      launch_rope_kv<T>(m->qkv, 1, 0, (const T*)w.bqkv, m->rope_cos, m->rope_sin, (T*)m->q, kv, Ttok, B, d_cu,
                        nullptr, H, s, ent_slot, ent_base);
    }
    if (plan && sizeof(T) == 2) {
      if (plan->nc > 0)
        m->timed(3, H, plan->nc, Ttok, s, [&] {
          launch_attn_prefill<T>((const T*)m->q, kv, (T*)m->o, Ttok, plan->nc, d_cu, h_cu, H, s, plan->d_chunks,
                                 plan->h_chunks, ent_slot, ent_base, nullptr, o_pair);
        });
      if (plan->nd > 0)
        m->timed(2, H, plan->nd, plan->dctx, s, [&] {
          launch_attn_decode<T>((const T*)m->q, kv, (T*)m->o, m->attn_part, m->attn_cnt, plan->nd, H, plan->d_dpos,
                                m->cfg.max_seq, s, plan->d_drow, plan->d_dslot);
        });
    } else {
      // prefill, and every entry of a float32 step (its kernel is per token)
      m->timed(3, H, B, Ttok, s, [&] {
        launch_attn_prefill<T>((const T*)m->q, kv, (T*)m->o, Ttok, B, d_cu, h_cu, H, s, nullptr, nullptr, ent_slot,
                               ent_base, nullptr, o_pair);
      });
    }
    const bool llama_bf16 = sizeof(T) == 2 && !gpt2;
    if (llama_bf16) {
      gemm_resid_norm(m, w.wo, (const bf16*)m->o, Ttok, H * hd, (const bf16*)w.gpost, (bf16*)h, Ttok, nullptr, s, true,
                      o_pair, xp);
    } else {
      gemm_many<T>(m, w.wo, m->o, D, Ttok, H * hd, EPI_RESID, m->x, nullptr, D, s, nullptr, w.bo);
      if (gpt2)
        launch_layernorm(m->x, (const bf16*)w.gpost, (const bf16*)w.gpost_b, (bf16*)h, Ttok, D, eps, nullptr, s);
      else
        launch_resid_rmsnorm<T>(m->x, nullptr, 0, 0, (const T*)w.gpost, h, Ttok, D, eps, nullptr, s);
    }
    const bool last = l + 1 == m->cfg.n_layers;
    const T* gnext = (const T*)(last ? m->gfinal : m->layers[l + 1].gin);
    bool normed = false;  // the dense down projection also ran the next normalization
    if (gpt2) {
      gemm_many<T>(m, w.wgu, h, I, Ttok, D, EPI_GELU, nullptr, m->a, I, s, nullptr, w.bfc);
      gemm_many<T>(m, w.wd, m->a, D, Ttok, I, EPI_RESID, m->x, nullptr, D, s, nullptr, w.bd);
    } else if (w.moe) {
      enqueue_moe(m, w, (const bf16*)h, Ttok, s);  // bf16 only (checked at init)
    } else {
      if constexpr (sizeof(T) == 2) {
        gemm_many<T>(m, w.wgu, h, 2 * I, Ttok, D, EPI_SILU, nullptr, m->a, I, s, nullptr, nullptr, xp, xp);
        const bool to_last = last && !all_logits;  // hlast: row-major rows for the head projection
        gemm_resid_norm(m, w.wd, (const bf16*)m->a, Ttok, I, (const bf16*)gnext, (bf16*)(to_last ? m->hlast : h),
                        to_last ? B : Ttok, to_last ? d_cu : nullptr, s, true, xp, xp && !to_last);
        normed = true;
      } else {
        gemm_many<T>(m, w.wgu, h, 2 * I, Ttok, D, EPI_F32, m->gu_f32, nullptr, 2 * I, s);
        launch_silu_reduce<T>(m->gu_f32, 1, 0, (T*)m->a, Ttok, I, s);
        gemm_many<T>(m, w.wd, m->a, D, Ttok, I, EPI_RESID, m->x, nullptr, D, s);
      }
    }
    if (normed) continue;
    if (gpt2) {
      const bf16* bnext = (const bf16*)(last ? m->gfinal_b : m->layers[l + 1].gin_b);
      if (!last || all_logits)
        launch_layernorm(m->x, (const bf16*)gnext, bnext, (bf16*)h, Ttok, D, eps, nullptr, s);
      else
        launch_layernorm(m->x, (const bf16*)gnext, bnext, (bf16*)m->hlast, B, D, eps, d_cu, s);
    } else if (!last || all_logits) {
      launch_resid_rmsnorm<T>(m->x, nullptr, 0, 0, gnext, h, Ttok, D, eps, nullptr, s);
    } else {
      launch_resid_rmsnorm<T>(m->x, nullptr, 0, 0, gnext, (T*)m->hlast, B, D, eps, d_cu, s);
    }
  }
  if (all_logits) {
    gemm_many<T>(m, m->lm_head, h, V, Ttok, D, EPI_F32, d_logits, nullptr, V, s, nullptr, nullptr, xp);
    launch_argmax_rows(d_logits, B, V, d_next, d_cu, s);
  } else if (sizeof(T) == 2 && B <= GEMV_MAX_M) {
    GemvArgs ha{};
    ha.W = (const bf16*)m->lm_head; ha.N = V; ha.K = D; ha.M = B; ha.X = (const bf16*)m->hlast;
    ha.out_f32 = d_logits; ha.ldo = V; ha.am_val = m->am_val; ha.am_idx = m->am_idx;
    gemv_step(m, ha, GV_HEAD, s);
    const int hr = gemv_rows(V, D, B, GV_HEAD);
    launch_argmax_final(m->am_val, m->am_idx, (V + hr - 1) / hr, B, d_next, nullptr, s);
  } else {
    float* dst = d_logits ? d_logits : m->logits_int;
    if constexpr (sizeof(T) == 2) gemm_many<T>(m, m->lm_head, m->hlast, V, B, D, EPI_F32, dst, nullptr, V, s);
    else gemm_few_f32(m, m->lm_head, m->hlast, V, B, D, EPI_F32, dst, V, s);
    launch_argmax(dst, B, V, d_next, nullptr, s);
  }
}

// Decode step as separate GEMM, RoPE/KV, attention and normalization kernels:
// the float32 check mode, and bf16 batches wider than one fused projection.
template <typename T>
void enqueue_decode_many(axon_model* m, int B, const int32_t* d_tokens, float* d_logits, int32_t* d_next,
                         hipStream_t s) {
  const int D = m->D(), H = m->H(), hd = m->hd(), I = m->I(), V = m->V(), nq = m->nqkv();
  const float eps = m->cfg.rms_eps;
  T* h = (T*)m->h;
  launch_embed_rmsnorm<T>(d_tokens, (const T*)m->embed, (const T*)m->layers[0].gin, m->x, h, B, D, V, eps, s);
  // projection: bf16 prefill GEMM, or the float32 GEMM of the check mode
  auto proj = [&](const void* W, const void* X, int N, int K, int epi, float* out_f32, void* out_t, int ldo) {
    if constexpr (sizeof(T) == 2) gemm_many<T>(m, W, X, N, B, K, epi, out_f32, out_t, ldo, s);
    else gemm_few_f32(m, W, X, N, B, K, epi, out_f32, ldo, s);
  };
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const LayerW& w = m->layers[l];
    KVView kv = m->kv(l, m->paged());
    if constexpr (sizeof(T) == 2) {
      const EpiArgs re = rope_epi(m, w, kv, nullptr, 0, m->d_len);
      gemm_many<T>(m, w.wqkv, h, nq, B, D, EPI_ROPE, nullptr, nullptr, nq, s, &re);
    } else {
      proj(w.wqkv, h, nq, D, EPI_F32, m->qkv, nullptr, nq);
      launch_rope_kv<T>(m->qkv, 1, 0, (const T*)w.bqkv, m->rope_cos, m->rope_sin, (T*)m->q, kv, B, 0, nullptr,
                        m->d_len, H, s);
    }
    launch_attn_decode<T>((const T*)m->q, kv, (T*)m->o, m->attn_part, m->attn_cnt, B, H, m->d_len, m->cfg.max_seq, s);
    proj(w.wo, m->o, D, H * hd, EPI_RESID, m->x, nullptr, D);
    launch_resid_rmsnorm<T>(m->x, nullptr, 0, 0, (const T*)w.gpost, h, B, D, eps, nullptr, s);
    if (w.moe) {
      enqueue_moe(m, w, (const bf16*)h, B, s);
    } else {
      if constexpr (sizeof(T) == 2) {
        proj(w.wgu, h, 2 * I, D, EPI_SILU, nullptr, m->a, I);
      } else {
        proj(w.wgu, h, 2 * I, D, EPI_F32, m->gu_f32, nullptr, 2 * I);
        launch_silu_reduce<T>(m->gu_f32, 1, 0, (T*)m->a, B, I, s);
      }
      proj(w.wd, m->a, D, I, EPI_RESID, m->x, nullptr, D);
    }
    const bool last = l + 1 == m->cfg.n_layers;
    const T* gnext = (const T*)(last ? m->gfinal : m->layers[l + 1].gin);
    launch_resid_rmsnorm<T>(m->x, nullptr, 0, 0, gnext, h, B, D, eps, nullptr, s);
  }
  float* dst = d_logits ? d_logits : m->logits_int;
  proj(m->lm_head, h, V, D, EPI_F32, dst, nullptr, V);
  launch_argmax(dst, B, V, d_next, m->d_len, s);
}

// Decode step, bf16: five fused weight-streaming projections per layer.
//   embed: x = E[tok], sum of squares
//   per layer: QKV (RMSNorm on load; bias + RoPE + KV write) -> attention ->
//              O (x += ; sums of squares) -> gate/up (RMSNorm on load; SiLU) ->
//              down (x += ; sums of squares)
//   head (RMSNorm on load; logits + argmax partials) -> argmax
//   plan != nullptr: a step of single-token entries: item b is at position
//   plan->d_dpos[b] of slot plan->d_dslot[b]; lengths are set at the end.
void enqueue_decode_bf16(axon_model* m, int B, const int32_t* d_tokens, float* d_logits, int32_t* d_next,
                         hipStream_t s, const StepPlan* plan = nullptr, const int32_t* d_cu = nullptr,
                         const DecodeWs* wsp = nullptr) {
  const int D = m->D(), H = m->H(), hd = m->hd(), I = m->I(), V = m->V(), nq = m->nqkv();
  const DecodeWs ws = wsp ? *wsp : m->own_ws();
  const int32_t* pos = plan ? plan->d_dpos : m->d_len;
  const int32_t* slot = plan ? plan->d_dslot : nullptr;
  const float eps = m->cfg.rms_eps;
  bf16* xg = ws.xg;
  // up to 16 tokens of a dense model: the token operands of every projection
  // (xg, the attention output, the gated activation) pass in the tile order
  // of the one-block fused kernel, written so by their producers
  const int xt = B <= XT_ROWS && !m->moe_model() ? 1 : 0;
  launch_embed_ss(d_tokens, (const bf16*)m->embed, (const bf16*)m->layers[0].gin, ws.x, xg, ws.ss, B, D, V, s, xt);
  int ss_n = 1;
  auto gemv = [&](GemvArgs& a, int epi) { gemv_step(m, a, epi, s); };
  auto ss_count = [&](int K) {
    const int rr = gemv_rows(D, K, B, GV_RESID);
    return (D + rr - 1) / rr;
  };
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const LayerW& w = m->layers[l];
    KVView kv = m->kv(l, m->paged());
    const bool last = l + 1 == m->cfg.n_layers;
    GemvArgs qa{};
    qa.W = (const bf16*)w.wqkv; qa.N = nq; qa.K = D; qa.M = B;
    qa.X = xg; qa.ss_in = ws.ss; qa.ss_n = ss_n; qa.eps = eps;
    qa.bias = (const bf16*)w.bqkv; qa.cos_t = m->rope_cos; qa.sin_t = m->rope_sin; qa.q_out = ws.q;
    qa.kv = kv; qa.len = pos; qa.slot = slot; qa.H = H; qa.part = ws.gemv_part;
    qa.x_tiled = xt;
    gemv(qa, GV_ROPE);
    int ctx_sum = 0;
    if (plan) ctx_sum = plan->dctx;
    else for (int b = 0; b < B; ++b) ctx_sum += m->keys_read(m->h_len[b] + 1);
    m->timed(2, H, B, ctx_sum, s, [&] {
      launch_attn_decode<bf16>(ws.q, kv, ws.o, ws.attn_part, ws.attn_cnt, B, H, pos, m->cfg.max_seq, s, nullptr, slot,
                               xt);
    });
    GemvArgs oa{};
    oa.W = (const bf16*)w.wo; oa.N = D; oa.K = H * hd; oa.M = B; oa.X = ws.o;
    oa.out_f32 = ws.x; oa.ldo = D; oa.ss_out = ws.ss; oa.xg_out = xg; oa.gain_next = (const bf16*)w.gpost;
    oa.part = ws.gemv_part;
    oa.x_tiled = oa.out_tiled = xt;
    gemv(oa, GV_RESID);
    ss_n = ss_count(H * hd);
    const bf16* gnext = (const bf16*)(last ? m->gfinal : m->layers[l + 1].gin);
    // dense MLP, or the shared experts of a mixture-of-experts layer
    const int Id = w.moe ? m->cfg.n_shared_experts * m->cfg.moe_intermediate : I;
    if (w.moe) {
      // the router and the routed experts read normed rows h; x gains the
      // routed rows before the shared experts' down projection (which then
      // leaves the next layer's xg and sums of squares), or, without shared
      // experts, the combine leaves them
      launch_resid_rmsnorm<bf16>(ws.x, nullptr, 0, 0, (const bf16*)w.gpost, (bf16*)m->h, B, D, eps, nullptr, s);
      moe_routed(m, w, (const bf16*)m->h, B, s);
    }
    if (Id > 0) {
      GemvArgs ga{};
      ga.W = (const bf16*)w.wgu; ga.N = 2 * Id; ga.K = D; ga.M = B;
      ga.X = xg; ga.ss_in = ws.ss; ga.ss_n = ss_n; ga.eps = eps;
      ga.out_t = ws.a; ga.ldo = Id; ga.part = ws.gemv_part;
      ga.x_tiled = ga.out_tiled = xt;
      gemv(ga, GV_SILU);
    }
    if (w.moe) {
      const bool fold = Id == 0;  // no shared experts: the combine leaves xg
      launch_moe_combine(ws.x, m->moe_y, m->moe_inv, m->moe_topw, B, D, m->cfg.top_k, s, fold ? gnext : nullptr,
                         fold ? xg : nullptr, fold ? ws.ss : nullptr);
      if (fold) ss_n = moe_combine_blocks(D);
    }
    if (Id > 0) {
      GemvArgs da{};
      da.W = (const bf16*)w.wd; da.N = D; da.K = Id; da.M = B; da.X = ws.a;
      da.out_f32 = ws.x; da.ldo = D; da.ss_out = ws.ss; da.xg_out = xg; da.part = ws.gemv_part;
      da.gain_next = gnext;
      da.x_tiled = da.out_tiled = xt;
      gemv(da, GV_RESID);
      ss_n = ss_count(Id);
    }
  }
  GemvArgs ha{};
  ha.W = (const bf16*)m->lm_head; ha.N = V; ha.K = D; ha.M = B;
  ha.X = xg; ha.ss_in = ws.ss; ha.ss_n = ss_n; ha.eps = eps;
  ha.out_f32 = d_logits; ha.ldo = V; ha.am_val = ws.am_val; ha.am_idx = ws.am_idx;
  ha.x_tiled = xt;
  gemv(ha, GV_HEAD);
  const int hr = gemv_rows(V, D, B, GV_HEAD);
  launch_argmax_final(ws.am_val, ws.am_idx, (V + hr - 1) / hr, B, d_next, plan ? nullptr : m->d_len, s);
  if (plan) launch_set_step_lengths(d_cu, plan->d_slot, plan->d_base, m->d_len, B, s);
}

// Decode step of a float32 model (Llama family) over at most 16 tokens: the
// float32 fused projections, 5 kernels per layer (4 when the contexts are
// short enough for every O workgroup to compute the attention itself).
//   embed: x = E[tok], xg = x * g, sum of squares
//   per layer: QKV (RMSNorm on load; bias + RoPE + KV write) -> attention ->
//              O (x += ; xg, sums of squares) -> gate/up (RMSNorm on load;
//              SiLU) -> down (x += ; xg, sums of squares)
//   head (RMSNorm on load; logits + argmax partials) -> argmax
void enqueue_decode_f32(axon_model* m, int B, const int32_t* d_tokens, float* d_logits, int32_t* d_next,
                        hipStream_t s) {
  const int D = m->D(), H = m->H(), hd = m->hd(), I = m->I(), V = m->V(), nq = m->nqkv();
  const float eps = m->cfg.rms_eps;
  float* xg = (float*)m->xg;
  // contexts never exceed the capacity max_seq
  const bool fused_attn = attn_o_f32_fits(B, H, m->KVh(), hd, m->cfg.max_seq);
  launch_embed_ss_f32(d_tokens, (const float*)m->embed, (const float*)m->layers[0].gin, m->x, xg, m->ss, B, D, V, s);
  int ss_n = 1;
  auto proj = [&](GemvF32Args& a, int epi) {
    bool ok = true;
    m->timed(0, a.N, a.M, a.K, s, [&] { ok = launch_gemv_f32_fused(a, epi, s); });
    if (!ok && m->enqueue_err.empty())
      m->enqueue_err = "no float32 projection kernel for N=" + std::to_string(a.N) + " K=" + std::to_string(a.K) +
                       " M=" + std::to_string(a.M) + " epilogue " + std::to_string(epi);
  };
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const LayerW& w = m->layers[l];
    KVView kv = m->kv(l, m->paged());
    const bool last = l + 1 == m->cfg.n_layers;
    GemvF32Args qa{};
    qa.W = (const float*)w.wqkv; qa.N = nq; qa.K = D; qa.M = B;
    qa.X = xg; qa.ss_in = m->ss; qa.ss_n = ss_n; qa.eps = eps;
    qa.bias = (const float*)w.bqkv; qa.cos_t = m->rope_cos; qa.sin_t = m->rope_sin; qa.q_out = (float*)m->q;
    qa.kv = kv; qa.len = m->d_len; qa.H = H;
    proj(qa, GV_ROPE);
    GemvF32Args oa{};
    oa.W = (const float*)w.wo; oa.N = D; oa.K = H * hd; oa.M = B; oa.X = (const float*)m->o;
    oa.out = m->x; oa.ldo = D; oa.xg_out = xg; oa.gain_next = (const float*)w.gpost; oa.ss_out = m->ss;
    if (fused_attn) {
      // short contexts: every O workgroup computes the attention itself
      oa.len = m->d_len; oa.H = H;
      bool ok = true;
      m->timed(0, D, B, H * hd, s, [&] { ok = launch_attn_o_f32(oa, (const float*)m->q, kv, s); });
      if (!ok && m->enqueue_err.empty()) m->enqueue_err = "no fused attention + O projection kernel";
    } else {
      m->timed(2, H, B, 0, s, [&] {
        launch_attn_decode<float>((const float*)m->q, kv, (float*)m->o, m->attn_part, m->attn_cnt, B, H, m->d_len,
                                  m->cfg.max_seq, s);
      });
      proj(oa, GV_RESID);
    }
    ss_n = gemv_f32_parts(D, GV_RESID);
    GemvF32Args ga{};
    ga.W = (const float*)w.wgu; ga.N = 2 * I; ga.K = D; ga.M = B;
    ga.X = xg; ga.ss_in = m->ss; ga.ss_n = ss_n; ga.eps = eps; ga.out = (float*)m->a; ga.ldo = I;
    proj(ga, GV_SILU);
    GemvF32Args da{};
    da.W = (const float*)w.wd; da.N = D; da.K = I; da.M = B; da.X = (const float*)m->a;
    da.out = m->x; da.ldo = D; da.xg_out = xg; da.ss_out = m->ss;
    da.gain_next = (const float*)(last ? m->gfinal : m->layers[l + 1].gin);
    proj(da, GV_RESID);
  }
  GemvF32Args ha{};
  ha.W = (const float*)m->lm_head; ha.N = V; ha.K = D; ha.M = B;
  ha.X = xg; ha.ss_in = m->ss; ha.ss_n = ss_n; ha.eps = eps;
  ha.out = d_logits; ha.ldo = V; ha.am_val = m->am_val; ha.am_idx = m->am_idx;
  proj(ha, GV_HEAD);
  launch_argmax_final(m->am_val, m->am_idx, gemv_f32_parts(V, GV_HEAD), B, d_next, m->d_len, s);
}

// Decode step of the GPT-2 family: embedding + learned position + the first
// LayerNorm, then per layer QKV (bias, identity rotation, KV write) ->
// attention -> c_proj (+ bias, residual) -> LayerNorm -> c_fc (+ bias, GELU)
// -> c_proj (+ bias, residual) -> the next LayerNorm; the tied head + argmax.
// Up to 64 tokens the projections are the fused weight-streaming kernels,
// else the GEMMs.  plan: as enqueue_decode_bf16.
void enqueue_decode_gpt2(axon_model* m, int B, const int32_t* d_tokens, float* d_logits, int32_t* d_next,
                         hipStream_t s, const StepPlan* plan = nullptr, const int32_t* d_cu = nullptr) {
  const int D = m->D(), H = m->H(), hd = m->hd(), I = m->I(), V = m->V(), nq = m->nqkv();
  const int32_t* pos = plan ? plan->d_dpos : m->d_len;
  const int32_t* slot = plan ? plan->d_dslot : nullptr;
  const float eps = m->cfg.rms_eps;
  const bool few = B <= GEMV_MAX_M;  // plan implies few
  bf16* h = (bf16*)m->h;
  launch_embed_pos_ln(d_tokens, (const bf16*)m->embed, (const bf16*)m->wpe, (const bf16*)m->layers[0].gin,
                      (const bf16*)m->layers[0].gin_b, m->x, h, B, D, V, m->cfg.max_positions, eps, nullptr, 0,
                      nullptr, pos, s);
  // x += X W^T + bias, or a = gelu(X W^T + bias)
  auto proj = [&](const void* W, const bf16* X, int N, int K, int epi, const void* bias) {
    if (few) {
      GemvArgs a{};
      a.W = (const bf16*)W; a.N = N; a.K = K; a.M = B; a.X = X; a.bias = (const bf16*)bias;
      a.part = m->gemv_part;
      if (epi == GV_GELU) { a.out_t = (bf16*)m->a; a.ldo = I; }
      else { a.out_f32 = m->x; a.ldo = D; }
      gemv_step(m, a, epi, s);
    } else if (epi == GV_GELU) {
      gemm_many<bf16>(m, W, X, N, B, K, EPI_GELU, nullptr, m->a, I, s, nullptr, bias);
    } else {
      gemm_many<bf16>(m, W, X, N, B, K, EPI_RESID, m->x, nullptr, D, s, nullptr, bias);
    }
  };
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const LayerW& w = m->layers[l];
    KVView kv = m->kv(l, m->paged());
    if (few) {
      GemvArgs qa{};
      qa.W = (const bf16*)w.wqkv; qa.N = nq; qa.K = D; qa.M = B; qa.X = h;
      qa.bias = (const bf16*)w.bqkv; qa.cos_t = m->rope_cos; qa.sin_t = m->rope_sin; qa.q_out = (bf16*)m->q;
      qa.kv = kv; qa.len = pos; qa.slot = slot; qa.H = H; qa.part = m->gemv_part;
      gemv_step(m, qa, GV_ROPE, s);
    } else {
      const EpiArgs re = rope_epi(m, w, kv, nullptr, 0, pos);
      gemm_many<bf16>(m, w.wqkv, h, nq, B, D, EPI_ROPE, nullptr, nullptr, nq, s, &re);
    }
    int ctx_sum = 0;
    if (plan) ctx_sum = plan->dctx;
    else for (int b = 0; b < B; ++b) ctx_sum += m->keys_read(m->h_len[b] + 1);
    m->timed(2, H, B, ctx_sum, s, [&] {
      launch_attn_decode<bf16>((const bf16*)m->q, kv, (bf16*)m->o, m->attn_part, m->attn_cnt, B, H, pos, m->cfg.max_seq, s,
                               nullptr, slot);
    });
    proj(w.wo, (const bf16*)m->o, D, H * hd, GV_RESID, w.bo);
    launch_layernorm(m->x, (const bf16*)w.gpost, (const bf16*)w.gpost_b, h, B, D, eps, nullptr, s);
    proj(w.wgu, h, I, D, GV_GELU, w.bfc);
    proj(w.wd, (const bf16*)m->a, D, I, GV_RESID, w.bd);
    const bool last = l + 1 == m->cfg.n_layers;
    launch_layernorm(m->x, (const bf16*)(last ? m->gfinal : m->layers[l + 1].gin),
                     (const bf16*)(last ? m->gfinal_b : m->layers[l + 1].gin_b), h, B, D, eps, nullptr, s);
  }
  if (few) {
    GemvArgs ha{};
    ha.W = (const bf16*)m->lm_head; ha.N = V; ha.K = D; ha.M = B; ha.X = h;
    ha.out_f32 = d_logits; ha.ldo = V; ha.am_val = m->am_val; ha.am_idx = m->am_idx;
    gemv_step(m, ha, GV_HEAD, s);
    const int hr = gemv_rows(V, D, B, GV_HEAD);
    launch_argmax_final(m->am_val, m->am_idx, (V + hr - 1) / hr, B, d_next, plan ? nullptr : m->d_len, s);
  } else {
    float* dst = d_logits ? d_logits : m->logits_int;
    gemm_many<bf16>(m, m->lm_head, h, V, B, D, EPI_F32, dst, nullptr, V, s);
    launch_argmax(dst, B, V, d_next, m->d_len, s);
  }
  if (plan) launch_set_step_lengths(d_cu, plan->d_slot, plan->d_base, m->d_len, B, s);
}

void enqueue_decode(axon_model* m, int B, const int32_t* d_tokens, float* d_logits, int32_t* d_next, hipStream_t s) {
  if (m->gpt2()) enqueue_decode_gpt2(m, B, d_tokens, d_logits, d_next, s);
  else if (m->bf && B <= GEMV_MAX_M) enqueue_decode_bf16(m, B, d_tokens, d_logits, d_next, s);
  else if (m->bf) enqueue_decode_many<bf16>(m, B, d_tokens, d_logits, d_next, s);
  else if (B <= GEMV_F32_MAX_M) enqueue_decode_f32(m, B, d_tokens, d_logits, d_next, s);
  else enqueue_decode_many<float>(m, B, d_tokens, d_logits, d_next, s);
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(AXON_E_HIP, std::string(what) + ": kernel launch failed: " + hipGetErrorString(e));
  return AXON_OK;
}

// A projection shape without a kernel (never produced by a validated model):
// reported, and cleared for the next call.
int take_enqueue_err(axon_model* m, const char* what) {
  if (m->enqueue_err.empty()) return AXON_OK;
  std::string e;
  e.swap(m->enqueue_err);
  return fail(AXON_E_INVALID, std::string(what) + ": " + e);
}

}  // namespace

// ====================================================================== ABI

extern "C" const char* axon_last_error(void) { return g_err.c_str(); }

extern "C" int axon_init_model(const axon_config* cfg, const axon_weight* weights, int32_t n_weights, void* stream,
                               axon_model** out) {
  g_err.clear();
  if (!out) return fail(AXON_E_INVALID, "out is NULL");
  *out = nullptr;
  if (!cfg) return fail(AXON_E_INVALID, "cfg is NULL");
  if (n_weights < 0 || (n_weights > 0 && !weights)) return fail(AXON_E_INVALID, "weights is NULL or n_weights < 0");
  int rc = validate_config(*cfg);
  if (rc) return rc;
  const axon_config& c = *cfg;

  // ---- weight map (host only)
  auto expected = expected_weights(c);
  std::unordered_map<std::string, size_t> index;
  for (size_t i = 0; i < expected.size(); ++i) index[expected[i].first] = i;
  std::vector<const axon_weight*> found(expected.size(), nullptr);
  for (int i = 0; i < n_weights; ++i) {
    const axon_weight& w = weights[i];
    if (!w.name) return fail(AXON_E_INVALID, "weight " + std::to_string(i) + " has a NULL name");
    auto it = index.find(w.name);
    if (it == index.end()) {
      std::string why = std::string(w.name) == "lm_head.weight" ? " (tie_embeddings is set)" : "";
      return fail(AXON_E_MISSING, std::string("unknown weight '") + w.name + "'" + why);
    }
    if (found[it->second]) return fail(AXON_E_MISSING, std::string("duplicate weight '") + w.name + "'");
    const Expected& e = expected[it->second].second;
    if (w.dtype != c.dtype)
      return fail(AXON_E_DTYPE, std::string("weight '") + w.name + "' has dtype " + std::to_string(w.dtype) +
                                    ", the model dtype is " + std::to_string(c.dtype));
    if (w.ndim != e.ndim || w.shape[0] != e.shape[0] || (e.ndim == 2 && w.shape[1] != e.shape[1]))
      return fail(AXON_E_SHAPE, std::string("weight '") + w.name + "' has shape " +
                                    (w.ndim == 1 || w.ndim == 2 ? shape_str(w.ndim, w.shape) : "ndim=" + std::to_string(w.ndim)) +
                                    ", expected " + shape_str(e.ndim, e.shape));
    if (!w.data) return fail(AXON_E_INVALID, std::string("weight '") + w.name + "' has NULL data");
    found[it->second] = &w;
  }
  for (size_t i = 0; i < expected.size(); ++i)
    if (!found[i]) return fail(AXON_E_MISSING, "missing weight '" + expected[i].first + "'");

  // ---- device state
  axon_model* m = new axon_model();
  m->cfg = c;
  m->bf = c.dtype == AXON_BF16;
  m->esz = m->bf ? 2 : 4;
  if (const char* e = std::getenv("AXON_NO_GRAPH")) m->use_graphs = std::atoi(e) == 0;
  hipStream_t s = (hipStream_t)stream;
  const int64_t D = c.hidden, H = c.n_heads, KV = c.n_kv_heads, hd = c.head_dim, I = c.intermediate, V = c.vocab;
  const int64_t esz = m->esz, nq = (H + 2 * KV) * hd;
  auto get = [&](const std::string& n) -> const axon_weight* { return found[index.at(n)]; };
  auto kind = [](const axon_weight* w) { return w->on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice; };

#define TRY(expr)          \
  do {                     \
    int r_ = (expr);       \
    if (r_) {              \
      (void)hipStreamSynchronize(s); \
      release(m);          \
      return r_;           \
    }                      \
  } while (0)
#define HTRY(expr)                                                                                 \
  do {                                                                                             \
    hipError_t e_ = (expr);                                                                        \
    if (e_ != hipSuccess) {                                                                        \
      std::string msg_ = std::string(#expr) + ": " + hipGetErrorString(e_);                        \
      (void)hipStreamSynchronize(s);                                                               \
      release(m);                                                                                  \
      return fail(AXON_E_HIP, msg_);                                                               \
    }                                                                                              \
  } while (0)

  auto copy_in = [&](void** dst, const axon_weight* w) -> int {
    const size_t bytes = (size_t)w->shape[0] * (w->ndim == 2 ? (size_t)w->shape[1] : 1) * esz;
    int r = dev_alloc(m, dst, bytes);
    if (r) return r;
    hipError_t e = hipMemcpyAsync(*dst, w->data, bytes, kind(w), s);
    if (e != hipSuccess) return fail(AXON_E_HIP, std::string("copy of '") + w->name + "': " + hipGetErrorString(e));
    return AXON_OK;
  };

  // Weight matrices.  ``fill`` writes the row-major (permuted) matrix; float
  // models keep it as is, bf16 models stage it in ``stage`` and store it
  // fragment-tiled (every bf16 projection kernel and the embedding gather
  // read that layout).
  struct StageBuf {
    void* p = nullptr;
    ~StageBuf() {
      if (p) (void)hipFree(p);  // waits for the tiling kernels that read it
    }
  } stage;
  if (m->bf) {
    const int64_t Ie = c.moe_intermediate, Is = (int64_t)c.n_shared_experts * Ie;
    const int64_t most = std::max({V * D, nq * D, D * H * hd, 2 * I * D, 2 * Ie * D, 2 * Is * D,
                                   (int64_t)m->moe_ep() * D});
    hipError_t e = hipMalloc(&stage.p, (size_t)most * esz);
    if (e != hipSuccess) {
      stage.p = nullptr;
      (void)hipGetLastError();
      release(m);
      return fail(e == hipErrorOutOfMemory ? AXON_E_OOM : AXON_E_HIP,
                  std::string("staging allocation failed: ") + hipGetErrorString(e));
    }
  }
  auto matrix = [&](void** dst, int64_t N, int64_t K, const std::function<int(void*)>& fill) -> int {
    if (!m->bf) {
      int r = dev_alloc(m, dst, (size_t)N * K * esz);
      return r ? r : fill(*dst);
    }
    int r = dev_alloc(m, dst, (size_t)(N + 15) / 16 * 16 * K * esz);
    if (!r) r = fill(stage.p);
    if (r) return r;
    launch_tile_weight((const bf16*)stage.p, (bf16*)*dst, N, (int)K, s);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? AXON_OK : fail(AXON_E_HIP, std::string("weight tiling: ") + hipGetErrorString(e));
  };
  // fill the staging buffer, tile it into dst (bf16 only)
  auto tile_into = [&](void* dst, int64_t N, int64_t K, const std::function<int(void*)>& fill) -> int {
    int r = fill(stage.p);
    if (r) return r;
    launch_tile_weight((const bf16*)stage.p, (bf16*)dst, N, (int)K, s);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? AXON_OK : fail(AXON_E_HIP, std::string("weight tiling: ") + hipGetErrorString(e));
  };
  // gate/up of an MLP of intermediate ii interleaved in blocks of 16 rows:
  // [g0..g15, u0..u15, g16..g31, u16..u31, ...]
  auto gate_up = [&](const axon_weight* wg, const axon_weight* wu, int64_t ii) {
    return [&, wg, wu, ii](void* dst) -> int {
      const size_t blk = 16 * D * esz;
      hipError_t e = hipMemcpy2DAsync(dst, 2 * blk, wg->data, blk, blk, ii / 16, kind(wg), s);
      if (e == hipSuccess) e = hipMemcpy2DAsync((char*)dst + blk, 2 * blk, wu->data, blk, blk, ii / 16, kind(wu), s);
      return e == hipSuccess ? AXON_OK : fail(AXON_E_HIP, std::string("gate/up repack: ") + hipGetErrorString(e));
    };
  };
  auto copy_to = [&](const axon_weight* w) {
    return [&, w](void* dst) -> int {
      const size_t bytes = (size_t)w->shape[0] * (size_t)w->shape[1] * esz;
      hipError_t e = hipMemcpyAsync(dst, w->data, bytes, kind(w), s);
      return e == hipSuccess ? AXON_OK
                             : fail(AXON_E_HIP, std::string("copy of '") + w->name + "': " + hipGetErrorString(e));
    };
  };

  if (m->gpt2()) {
    // Conv1D weights arrive [in][out]: copied to a second staging buffer, then
    // transposed into the first (the fused QKV rows also permuted into the
    // rotation-pair grouping every QKV kernel expects; GPT-2 rotates by the
    // identity), then tiled
    struct Stage2 {
      void* p = nullptr;
      ~Stage2() {
        if (p) (void)hipFree(p);
      }
    } st2;
    HTRY(hipMalloc(&st2.p, (size_t)std::max(3 * D * D, I * D) * esz));
    std::vector<int32_t> perm(nq);
    for (int64_t hh = 0; hh < 3 * H; ++hh)
      for (int64_t r = 0; r < hd; ++r) {
        const int64_t g = r / 8, j = r % 8;
        perm[hh * hd + r] = (int32_t)(hh * hd + (j < 4 ? 4 * g + j : hd / 2 + 4 * g + j - 4));
      }
    int32_t* d_perm = nullptr;
    TRY(dev_alloc(m, (void**)&d_perm, perm.size() * sizeof(int32_t)));
    HTRY(hipMemcpy(d_perm, perm.data(), perm.size() * sizeof(int32_t), hipMemcpyHostToDevice));
    auto tposed = [&](const axon_weight* w, int64_t K, int64_t N, const int32_t* pm) {
      return [&, w, K, N, pm](void* dst) -> int {
        hipError_t e = hipMemcpyAsync(st2.p, w->data, (size_t)K * N * esz, kind(w), s);
        if (e == hipSuccess) {
          launch_transpose_rows((const bf16*)st2.p, (bf16*)dst, (int)K, (int)N, pm, s);
          e = hipGetLastError();
        }
        return e == hipSuccess ? AXON_OK
                               : fail(AXON_E_HIP, std::string("transpose of '") + w->name + "': " + hipGetErrorString(e));
      };
    };
    TRY(matrix(&m->embed, V, D, copy_to(get("transformer.wte.weight"))));
    m->lm_head = m->embed;
    TRY(copy_in(&m->wpe, get("transformer.wpe.weight")));
    TRY(copy_in(&m->gfinal, get("transformer.ln_f.weight")));
    TRY(copy_in(&m->gfinal_b, get("transformer.ln_f.bias")));
    m->layers.resize(c.n_layers);
    for (int l = 0; l < c.n_layers; ++l) {
      const std::string p = "transformer.h." + std::to_string(l) + ".";
      LayerW& w = m->layers[l];
      TRY(copy_in(&w.gin, get(p + "ln_1.weight")));
      TRY(copy_in(&w.gin_b, get(p + "ln_1.bias")));
      TRY(copy_in(&w.gpost, get(p + "ln_2.weight")));
      TRY(copy_in(&w.gpost_b, get(p + "ln_2.bias")));
      TRY(matrix(&w.wqkv, nq, D, tposed(get(p + "attn.c_attn.weight"), D, 3 * D, d_perm)));
      TRY(copy_in(&w.bqkv, get(p + "attn.c_attn.bias")));
      TRY(matrix(&w.wo, D, D, tposed(get(p + "attn.c_proj.weight"), D, D, nullptr)));
      TRY(copy_in(&w.bo, get(p + "attn.c_proj.bias")));
      TRY(matrix(&w.wgu, I, D, tposed(get(p + "mlp.c_fc.weight"), D, I, nullptr)));
      TRY(copy_in(&w.bfc, get(p + "mlp.c_fc.bias")));
      TRY(matrix(&w.wd, D, I, tposed(get(p + "mlp.c_proj.weight"), I, D, nullptr)));
      TRY(copy_in(&w.bd, get(p + "mlp.c_proj.bias")));
    }
    HTRY(hipStreamSynchronize(s));  // the transposes read the second staging buffer
  } else {
    TRY(matrix(&m->embed, V, D, copy_to(get("model.embed_tokens.weight"))));
    TRY(copy_in(&m->gfinal, get("model.norm.weight")));
    if (c.tie_embeddings) m->lm_head = m->embed;
    else TRY(matrix(&m->lm_head, V, D, copy_to(get("lm_head.weight"))));
    m->layers.resize(c.n_layers);
    for (int l = 0; l < c.n_layers; ++l) {
      const std::string p = "model.layers." + std::to_string(l) + ".";
      LayerW& w = m->layers[l];
      TRY(copy_in(&w.gin, get(p + "input_layernorm.weight")));
      TRY(copy_in(&w.gpost, get(p + "post_attention_layernorm.weight")));
      TRY(matrix(&w.wo, D, H * hd, copy_to(get(p + "self_attn.o_proj.weight"))));
      w.moe = c.n_experts > 0 && l >= c.first_moe_layer;
      if (!w.moe) TRY(matrix(&w.wd, D, I, copy_to(get(p + "mlp.down_proj.weight"))));
      // fused QKV: heads q, then k, then v; within each head, rows in groups of
      // 8 = 4 first-half rows i and their rotation partners i + hd/2
      const axon_weight* wq = get(p + "self_attn.q_proj.weight");
      const axon_weight* wk = get(p + "self_attn.k_proj.weight");
      const axon_weight* wv = get(p + "self_attn.v_proj.weight");
      TRY(matrix(&w.wqkv, nq, D, [&](void* dst) -> int {
        const size_t row = (size_t)D * esz;
        for (int64_t hh = 0; hh < H + 2 * KV; ++hh) {
          const axon_weight* src = hh < H ? wq : (hh < H + KV ? wk : wv);
          const int64_t hs = hh < H ? hh : (hh < H + KV ? hh - H : hh - H - KV);
          const char* sbase = (const char*)src->data + hs * hd * row;
          char* dbase = (char*)dst + hh * hd * row;
          hipError_t e = hipMemcpy2DAsync(dbase, 8 * row, sbase, 4 * row, 4 * row, hd / 8, kind(src), s);
          if (e == hipSuccess)
            e = hipMemcpy2DAsync(dbase + 4 * row, 8 * row, sbase + (hd / 2) * row, 4 * row, 4 * row, hd / 8,
                                 kind(src), s);
          if (e != hipSuccess) return fail(AXON_E_HIP, std::string("QKV repack: ") + hipGetErrorString(e));
        }
        return AXON_OK;
      }));
      w.bqkv = nullptr;
      if (c.qkv_bias) {
        TRY(dev_alloc(m, &w.bqkv, (size_t)nq * esz));
        const axon_weight* bq = get(p + "self_attn.q_proj.bias");
        const axon_weight* bk = get(p + "self_attn.k_proj.bias");
        const axon_weight* bv = get(p + "self_attn.v_proj.bias");
        HTRY(hipMemcpyAsync(w.bqkv, bq->data, H * hd * esz, kind(bq), s));
        HTRY(hipMemcpyAsync((char*)w.bqkv + H * hd * esz, bk->data, KV * hd * esz, kind(bk), s));
        HTRY(hipMemcpyAsync((char*)w.bqkv + (H + KV) * hd * esz, bv->data, KV * hd * esz, kind(bv), s));
      }
      if (!w.moe) {
        TRY(matrix(&w.wgu, 2 * I, D, gate_up(get(p + "mlp.gate_proj.weight"), get(p + "mlp.up_proj.weight"), I)));
        continue;
      }
      // mixture of experts (bf16 only): router rows padded with zeros to a
      // multiple of 32, experts stacked, shared experts as a dense MLP
      const int64_t E = c.n_experts, Ep = m->moe_ep(), Ie = c.moe_intermediate;
      const int64_t Is = (int64_t)c.n_shared_experts * Ie;
      const axon_weight* wr = get(p + "mlp.gate.weight");
      TRY(matrix(&w.wrouter, Ep, D, [&](void* dst) -> int {
        hipError_t e = hipMemcpyAsync(dst, wr->data, (size_t)E * D * esz, kind(wr), s);
        if (e == hipSuccess && Ep > E) e = hipMemsetAsync((char*)dst + E * D * esz, 0, (size_t)(Ep - E) * D * esz, s);
        return e == hipSuccess ? AXON_OK : fail(AXON_E_HIP, std::string("router copy: ") + hipGetErrorString(e));
      }));
      TRY(dev_alloc(m, &w.wgu_e, (size_t)E * 2 * Ie * D * esz));
      TRY(dev_alloc(m, &w.wd_e, (size_t)E * D * Ie * esz));
      for (int64_t e = 0; e < E; ++e) {
        const std::string q = p + "mlp.experts." + std::to_string(e) + ".";
        TRY(tile_into((char*)w.wgu_e + e * 2 * Ie * D * esz, 2 * Ie, D,
                      gate_up(get(q + "gate_proj.weight"), get(q + "up_proj.weight"), Ie)));
        TRY(tile_into((char*)w.wd_e + e * D * Ie * esz, D, Ie, copy_to(get(q + "down_proj.weight"))));
      }
      w.wgu = w.wd = nullptr;
      if (Is > 0) {
        TRY(matrix(&w.wgu, 2 * Is, D,
                   gate_up(get(p + "mlp.shared_experts.gate_proj.weight"), get(p + "mlp.shared_experts.up_proj.weight"), Is)));
        TRY(matrix(&w.wd, D, Is, copy_to(get(p + "mlp.shared_experts.down_proj.weight"))));
      }
    }
  }  // Llama-family weights

  // ---- KV cache
  if (m->paged()) {
    m->ps = c.kv_page_size;
    const int64_t pages = c.kv_num_pages;
    m->kv_layer_elems = pages * KV * m->ps * hd;
    m->bt_stride = (c.max_seq + m->ps - 1) / m->ps;
    TRY(dev_alloc(m, (void**)&m->d_bt, (size_t)c.max_batch * m->bt_stride * sizeof(int32_t)));
    HTRY(hipHostMalloc((void**)&m->h_bt, (size_t)c.max_batch * m->bt_stride * sizeof(int32_t), hipHostMallocDefault));
    for (int64_t i = 0; i < (int64_t)c.max_batch * m->bt_stride; ++i) m->h_bt[i] = -1;
    HTRY(hipEventCreateWithFlags(&m->bt_copied, hipEventDisableTiming));
  } else {
    m->ps = (c.max_seq + 15) / 16 * 16;
    m->kv_layer_elems = (int64_t)c.max_batch * KV * m->ps * hd;
  }
  const size_t kv_bytes = (size_t)c.n_layers * m->kv_layer_elems * esz;
  TRY(dev_alloc(m, &m->kcache, kv_bytes));
  TRY(dev_alloc(m, &m->vcache, kv_bytes));
  HTRY(hipMemsetAsync(m->kcache, 0, kv_bytes, s));
  HTRY(hipMemsetAsync(m->vcache, 0, kv_bytes, s));

  // ---- rotary table, computed in double precision, stored as float
  {
    const int half = (int)hd / 2;
    std::vector<float> cs((size_t)c.max_seq * half), sn((size_t)c.max_seq * half);
    for (int p = 0; p < c.max_seq; ++p)
      for (int i = 0; i < half; ++i) {
        // GPT-2 has learned positions instead: the QKV epilogue rotates by 0
        const double ang = m->gpt2() ? 0.0 : (double)p * std::pow(c.rope_theta, -2.0 * i / (double)hd);
        cs[(size_t)p * half + i] = (float)std::cos(ang);
        sn[(size_t)p * half + i] = (float)std::sin(ang);
      }
    TRY(dev_alloc(m, (void**)&m->rope_cos, cs.size() * sizeof(float)));
    TRY(dev_alloc(m, (void**)&m->rope_sin, sn.size() * sizeof(float)));
    HTRY(hipMemcpy(m->rope_cos, cs.data(), cs.size() * sizeof(float), hipMemcpyHostToDevice));
    HTRY(hipMemcpy(m->rope_sin, sn.data(), sn.size() * sizeof(float), hipMemcpyHostToDevice));
  }

  // ---- work buffers
  {
    int64_t tmax = c.max_tokens > 0 ? c.max_tokens : (int64_t)c.max_batch * c.max_seq;
    tmax = std::max<int64_t>(tmax, c.max_batch);
    m->rows = (int)tmax;
    TRY(dev_alloc(m, (void**)&m->x, tmax * D * 4));
    // h, o and a may hold the row-pair layout: an even number of rows
    const int64_t tpair = (tmax + 1) & ~(int64_t)1;
    TRY(dev_alloc(m, &m->h, tpair * D * esz));
    if (!m->bf) TRY(dev_alloc(m, (void**)&m->qkv, tmax * nq * 4));  // bf16: RoPE is the QKV GEMM's epilogue
    TRY(dev_alloc(m, &m->q, tmax * H * hd * esz));
    // o, a and xg hold at least the 16 token rows of the tile order
    const int64_t trows = std::max<int64_t>(tpair, XT_ROWS);
    TRY(dev_alloc(m, &m->o, trows * H * hd * esz));
    const int64_t Ishared = (int64_t)c.n_shared_experts * c.moe_intermediate;
    TRY(dev_alloc(m, &m->a, trows * std::max<int64_t>(I, Ishared) * esz));
    if (m->moe_model()) {
      const int64_t E = c.n_experts, k = c.top_k;
      TRY(dev_alloc(m, (void**)&m->moe_logits, tmax * m->moe_ep() * 4));
      TRY(dev_alloc(m, (void**)&m->moe_topi, tmax * k * 4));
      TRY(dev_alloc(m, (void**)&m->moe_topw, tmax * k * 4));
      TRY(dev_alloc(m, (void**)&m->moe_cnt, (size_t)(3 * E + 2) * 4));
      m->moe_off = m->moe_cnt + E;
      m->moe_toff = m->moe_off + E + 1;
      TRY(dev_alloc(m, (void**)&m->moe_xrow, tmax * k * 4));
      TRY(dev_alloc(m, (void**)&m->moe_inv, tmax * k * 4));
      TRY(dev_alloc(m, &m->moe_a, tmax * k * c.moe_intermediate * esz));
      TRY(dev_alloc(m, (void**)&m->moe_y, tmax * k * D * 4));
    }
    TRY(dev_alloc(m, &m->hlast, (int64_t)c.max_batch * D * esz));
    TRY(dev_alloc(m, (void**)&m->logits_int, (int64_t)c.max_batch * V * 4));
    if (!m->bf) TRY(dev_alloc(m, (void**)&m->gu_f32, tmax * 2 * I * 4));
    int64_t bsplits = 1;
    for (int b = 1; b <= c.max_batch; ++b)
      bsplits = std::max<int64_t>(bsplits, (int64_t)b * plan_decode_splits(b, c.n_kv_heads, c.max_seq));
    TRY(dev_alloc(m, (void**)&m->attn_part, bsplits * H * (hd + 2) * 4));
    TRY(dev_alloc(m, (void**)&m->attn_cnt, (size_t)c.max_batch * KV * sizeof(int32_t)));
    HTRY(hipMemsetAsync(m->attn_cnt, 0, (size_t)c.max_batch * KV * sizeof(int32_t), s));
    if (m->bf) {
      int64_t wsf = 0;
      const int Is = c.n_shared_experts * c.moe_intermediate;
      for (int b = 1; b <= std::min<int>(c.max_batch, GEMV_MAX_M); ++b) {
        wsf = std::max({wsf, gemv_workspace_floats((int)nq, (int)D, b, GV_ROPE),
                        gemv_workspace_floats((int)D, (int)(H * hd), b, GV_RESID),
                        gemv_workspace_floats(2 * (int)I, (int)D, b, GV_SILU),
                        gemv_workspace_floats((int)I, (int)D, b, GV_GELU),
                        gemv_workspace_floats((int)D, (int)I, b, GV_RESID)});
        if (m->moe_model()) wsf = std::max(wsf, gemv_workspace_floats(m->moe_ep(), (int)D, b, GV_F32));
        if (Is > 0)
          wsf = std::max({wsf, gemv_workspace_floats(2 * Is, (int)D, b, GV_SILU),
                          gemv_workspace_floats((int)D, Is, b, GV_RESID)});
      }
      if (wsf > 0) TRY(dev_alloc(m, (void**)&m->gemv_part, (size_t)wsf * 4));
      // two K halves of the narrow prefill residual projections (hidden <= 2048)
      if (!m->gpt2() && D <= 2048) {
        m->gemm_part_floats = 2 * tmax * D;
        TRY(dev_alloc(m, (void**)&m->gemm_part, (size_t)m->gemm_part_floats * 4));
      }
    }
    TRY(dev_alloc(m, (void**)&m->ss, (int64_t)std::max<int64_t>(D / 8, 1) * c.max_batch * 4));
    TRY(dev_alloc(m, &m->xg, (int64_t)std::max(c.max_batch, XT_ROWS) * D * esz));
    const int64_t nam = (V + 7) / 8;  // argmax partials per token (8-row float32 head tiles)
    TRY(dev_alloc(m, (void**)&m->am_val, nam * c.max_batch * 4));
    TRY(dev_alloc(m, (void**)&m->am_idx, nam * c.max_batch * 4));
    TRY(dev_alloc(m, (void**)&m->d_len, (size_t)c.max_batch * sizeof(int32_t)));
    HTRY(hipMemsetAsync(m->d_len, 0, (size_t)c.max_batch * sizeof(int32_t), s));
    TRY(dev_alloc(m, (void**)&m->d_step, (size_t)6 * c.max_batch * sizeof(int32_t)));
    HTRY(hipHostMalloc((void**)&m->h_step, (size_t)6 * c.max_batch * sizeof(int32_t), hipHostMallocDefault));
    HTRY(hipEventCreateWithFlags(&m->step_copied, hipEventDisableTiming));
  }
  m->h_len.assign(c.max_batch, 0);
  // this device's no-allocation work array (a failed lookup only disables
  // axon_decode_step_noalloc)
  scratch_of_current_device(&m->scratch_ptr, &m->scratch_err);
  HTRY(hipStreamCreateWithFlags(&m->cap_stream, hipStreamNonBlocking));
  HTRY(hipStreamSynchronize(s));
#undef TRY
#undef HTRY
  *out = m;
  return AXON_OK;
}

extern "C" int axon_prefill(axon_model* m, int32_t batch, const int32_t* d_tokens, const int32_t* d_cu_seqlens,
                            const int32_t* h_cu_seqlens, const int32_t* h_block_table, int32_t block_table_stride,
                            int32_t all_logits, float* d_logits, int32_t* d_next_tokens, void* stream) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  const axon_config& c = m->cfg;
  if (batch < 1) return fail(AXON_E_INVALID, "batch must be >= 1");
  if (batch > c.max_batch)
    return fail(AXON_E_CAPACITY, "batch " + std::to_string(batch) + " exceeds max_batch " + std::to_string(c.max_batch));
  if (!d_tokens || !d_cu_seqlens || !h_cu_seqlens || !d_next_tokens)
    return fail(AXON_E_INVALID, "d_tokens, d_cu_seqlens, h_cu_seqlens and d_next_tokens must be non-NULL");
  if (all_logits != 0 && all_logits != 1) return fail(AXON_E_INVALID, "all_logits must be 0 or 1");
  if (all_logits && !d_logits) return fail(AXON_E_INVALID, "all_logits requires d_logits");
  if (h_cu_seqlens[0] != 0) return fail(AXON_E_INVALID, "cu_seqlens[0] must be 0");
  int64_t total = 0;
  for (int b = 0; b < batch; ++b) {
    const int64_t sb = (int64_t)h_cu_seqlens[b + 1] - h_cu_seqlens[b];
    if (sb < 1) return fail(AXON_E_INVALID, "sequence " + std::to_string(b) + " has length " + std::to_string(sb) + " (must be >= 1)");
    if (sb > c.max_seq)
      return fail(AXON_E_CAPACITY, "sequence " + std::to_string(b) + " has length " + std::to_string(sb) +
                                       " > max_seq " + std::to_string(c.max_seq));
    total += sb;
  }
  if (total > m->rows)
    return fail(AXON_E_CAPACITY, "prefill of " + std::to_string(total) + " tokens exceeds max_tokens " + std::to_string(m->rows));
  hipStream_t s = (hipStream_t)stream;
  if (m->paged()) {
    if (!h_block_table) return fail(AXON_E_INVALID, "a paged cache needs h_block_table");
    if (block_table_stride < 1) return fail(AXON_E_INVALID, "block_table_stride must be >= 1");
    const int cols = std::min(block_table_stride, m->bt_stride);
    std::vector<char> used(c.kv_num_pages, 0);
    for (int b = 0; b < batch; ++b) {
      const int sb = h_cu_seqlens[b + 1] - h_cu_seqlens[b];
      const int need = (sb + m->ps - 1) / m->ps;
      if (need > cols)
        return fail(AXON_E_CAPACITY, "page table row " + std::to_string(b) + " has " + std::to_string(cols) +
                                         " columns, the prompt needs " + std::to_string(need));
      for (int j = 0; j < cols; ++j) {
        const int p = h_block_table[(int64_t)b * block_table_stride + j];
        if (p < 0) {
          if (j < need)
            return fail(AXON_E_CAPACITY, "page table row " + std::to_string(b) + " has no page for block " + std::to_string(j));
          continue;
        }
        if (p >= c.kv_num_pages)
          return fail(AXON_E_CAPACITY, "page id " + std::to_string(p) + " out of range [0, " + std::to_string(c.kv_num_pages) + ")");
        if (used[p]) return fail(AXON_E_INVALID, "page id " + std::to_string(p) + " appears twice");
        used[p] = 1;
      }
    }
    // the previous upload must have left the pinned staging copy
    HIP_TRY(hipEventSynchronize(m->bt_copied));
    for (int b = 0; b < c.max_batch; ++b)
      for (int j = 0; j < m->bt_stride; ++j)
        m->h_bt[(int64_t)b * m->bt_stride + j] =
            (b < batch && j < cols) ? h_block_table[(int64_t)b * block_table_stride + j] : -1;
    HIP_TRY(hipMemcpyAsync(m->d_bt, m->h_bt, (size_t)c.max_batch * m->bt_stride * sizeof(int32_t),
                           hipMemcpyHostToDevice, s));
    HIP_TRY(hipEventRecord(m->bt_copied, s));
  } else if (h_block_table) {
    return fail(AXON_E_INVALID, "h_block_table given for a contiguous cache");
  }
  if (m->bf)
    enqueue_prefill<bf16>(m, batch, (int)total, d_tokens, d_cu_seqlens, h_cu_seqlens, all_logits, d_logits,
                          d_next_tokens, s);
  else
    enqueue_prefill<float>(m, batch, (int)total, d_tokens, d_cu_seqlens, h_cu_seqlens, all_logits, d_logits,
                           d_next_tokens, s);
  int rc = check_launch("prefill");
  if (!rc) rc = take_enqueue_err(m, "prefill");
  if (rc) return rc;
  for (int b = 0; b < c.max_batch; ++b) m->h_len[b] = b < batch ? h_cu_seqlens[b + 1] - h_cu_seqlens[b] : 0;
  m->active = batch;
  return AXON_OK;
}

// Record ``enqueue`` (launching onto the stream it is given) once per key as a
// HIP graph and replay it on s; run it eagerly when graphs are off or kernel
// timing is on.  The graph reads every per-call input through pointers that
// are part of the key or owned by the model.
template <typename F>
int replay_or_run(axon_model* m, const GraphKey& key, hipStream_t s, const char* what, F&& enqueue) {
  if (m->use_graphs && !m->timing) {
    auto it = m->graphs.find(key);
    if (it == m->graphs.end()) {
      hipGraph_t g = nullptr;
      HIP_TRY(hipStreamBeginCapture(m->cap_stream, hipStreamCaptureModeThreadLocal));
      enqueue(m->cap_stream);
      hipError_t le = hipGetLastError();
      hipError_t ce = hipStreamEndCapture(m->cap_stream, &g);
      if (le != hipSuccess || ce != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        m->enqueue_err.clear();
        return fail(AXON_E_HIP, std::string(what) + " graph capture failed: " +
                                    hipGetErrorString(le != hipSuccess ? le : ce));
      }
      if (int rc = take_enqueue_err(m, what)) {
        (void)hipGraphDestroy(g);
        return rc;
      }
      hipGraphExec_t ex = nullptr;
      hipError_t ie = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
      (void)hipGraphDestroy(g);
      if (ie != hipSuccess) return fail(AXON_E_HIP, std::string(what) + " graph instantiate: " + hipGetErrorString(ie));
      it = m->graphs.emplace(key, ex).first;
    }
    HIP_TRY(hipGraphLaunch(it->second, s));
    return AXON_OK;
  }
  enqueue(s);
  int rc = check_launch(what);
  if (!rc) rc = take_enqueue_err(m, what);
  return rc;
}

namespace {

// Host checks shared by the decode entry points.
int check_decode(const axon_model* m, int32_t batch, const int32_t* d_tokens, const int32_t* d_next_tokens) {
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  if (!d_tokens || !d_next_tokens) return fail(AXON_E_INVALID, "d_tokens and d_next_tokens must be non-NULL");
  if (batch < 1) return fail(AXON_E_INVALID, "batch must be >= 1");
  if (batch > m->active)
    return fail(AXON_E_CAPACITY, "batch " + std::to_string(batch) + " exceeds the " + std::to_string(m->active) +
                                     " active slots of the last prefill");
  for (int b = 0; b < batch; ++b) {
    const int pos = m->h_len[b];
    if (pos < 1) return fail(AXON_E_INVALID, "slot " + std::to_string(b) + " holds no sequence");
    if (pos + 1 > m->cfg.max_seq)
      return fail(AXON_E_CAPACITY, "slot " + std::to_string(b) + " is full (max_seq " + std::to_string(m->cfg.max_seq) + ")");
    if (m->paged() && m->h_bt[(int64_t)b * m->bt_stride + pos / m->ps] < 0)
      return fail(AXON_E_CAPACITY, "slot " + std::to_string(b) + " has no page for position " + std::to_string(pos));
  }
  return AXON_OK;
}

// Bytes of the per-step work buffers of a bf16 decode step over B tokens,
// each buffer 256-byte aligned; with ``base`` set, *ws receives the buffers
// laid out from it.
size_t decode_ws_layout(const axon_model* m, int B, char* base, DecodeWs* ws) {
  const int64_t D = m->D(), H = m->H(), hd = m->hd(), I = m->I(), V = m->V();
  size_t off = 0;
  auto take = [&](int64_t bytes) -> char* {
    const size_t at = off;
    off += (size_t)(bytes + 255) / 256 * 256;
    return base ? base + at : nullptr;
  };
  DecodeWs w{};
  w.attn_cnt = (int32_t*)take((int64_t)B * m->KVh() * 4);  // first, cleared by every call
  const int64_t trows = std::max(B, XT_ROWS);  // the tile order's 16 token rows
  w.x = (float*)take(B * D * 4);
  w.xg = (bf16*)take(trows * D * 2);
  w.ss = (float*)take(std::max<int64_t>(D / 8, 1) * B * 4);
  w.q = (bf16*)take(B * H * hd * 2);
  w.o = (bf16*)take(trows * H * hd * 2);
  w.a = (bf16*)take(trows * I * 2);
  w.attn_part = (float*)take((int64_t)B * plan_decode_splits(B, m->KVh(), m->cfg.max_seq) * H * (hd + 2) * 4);
  const int64_t wsf = std::max({gemv_workspace_floats(m->nqkv(), (int)D, B, GV_ROPE),
                                gemv_workspace_floats((int)D, (int)(H * hd), B, GV_RESID),
                                gemv_workspace_floats(2 * (int)I, (int)D, B, GV_SILU),
                                gemv_workspace_floats((int)D, (int)I, B, GV_RESID), (int64_t)1});
  w.gemv_part = (float*)take(wsf * 4);
  const int64_t nam = (V + 15) / 16;
  w.am_val = (float*)take(nam * B * 4);
  w.am_idx = (int32_t*)take(nam * B * 4);
  if (ws) *ws = w;
  return off;
}

}  // namespace

extern "C" int axon_decode_step_noalloc(axon_model* m, int32_t batch, const int32_t* d_tokens, float* d_logits,
                                        int32_t* d_next_tokens, void* stream) {
  g_err.clear();
  if (int rc = check_decode(m, batch, d_tokens, d_next_tokens)) return rc;
  if (!m->bf || m->gpt2() || m->moe_model())
    return fail(AXON_E_INVALID, "the no-allocation decode step serves dense Llama-family bf16 models only");
  if (batch > GEMV_MAX_M)
    return fail(AXON_E_CAPACITY, "the no-allocation decode step takes at most " + std::to_string(GEMV_MAX_M) +
                                     " sequences, got " + std::to_string(batch));
  if (!m->scratch_ptr) return fail(AXON_E_HIP, "no-allocation work array unavailable: " + m->scratch_err);
  const size_t need = decode_ws_layout(m, batch, nullptr, nullptr);
  if (need > (size_t)AXON_NOALLOC_SCRATCH_BYTES)
    return fail(AXON_E_CAPACITY, "a decode step of " + std::to_string(batch) + " sequences of this model needs " +
                                     std::to_string(need) + " bytes of work memory, more than the " +
                                     std::to_string((size_t)AXON_NOALLOC_SCRATCH_BYTES) + " of the fixed array");
  DecodeWs ws{};
  decode_ws_layout(m, batch, (char*)m->scratch_ptr, &ws);
  hipStream_t s = (hipStream_t)stream;
  // launched directly: no graph is recorded (instantiation allocates) and no
  // timing events are created
  const bool timing = m->timing;
  m->timing = false;
  // the split counters must start at zero; the array keeps whatever the last
  // call on this GPU left there
  launch_zero_i32(ws.attn_cnt, batch * m->KVh(), s);
  enqueue_decode_bf16(m, batch, d_tokens, d_logits, d_next_tokens, s, nullptr, nullptr, &ws);
  m->timing = timing;
  int rc = check_launch("decode (no allocation)");
  if (!rc) rc = take_enqueue_err(m, "decode (no allocation)");
  if (rc) return rc;
  for (int b = 0; b < batch; ++b) m->h_len[b] += 1;
  return AXON_OK;
}

extern "C" int axon_decode_step(axon_model* m, int32_t batch, const int32_t* d_tokens, float* d_logits,
                                int32_t* d_next_tokens, void* stream) {
  g_err.clear();
  if (int rc = check_decode(m, batch, d_tokens, d_next_tokens)) return rc;
  hipStream_t s = (hipStream_t)stream;
  if (int rc = replay_or_run(m, GraphKey{batch, d_tokens, d_logits, d_next_tokens}, s, "decode",
                             [&](hipStream_t st) { enqueue_decode(m, batch, d_tokens, d_logits, d_next_tokens, st); }))
    return rc;
  for (int b = 0; b < batch; ++b) m->h_len[b] += 1;
  return AXON_OK;
}

extern "C" int axon_step(axon_model* m, int32_t n, const int32_t* h_slots, const int32_t* h_fresh,
                         const int32_t* d_tokens, const int32_t* d_cu_seqlens, const int32_t* h_cu_seqlens,
                         const int32_t* h_block_table, int32_t block_table_stride, float* d_logits,
                         int32_t* d_next_tokens, void* stream) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  const axon_config& c = m->cfg;
  if (n < 1) return fail(AXON_E_INVALID, "n must be >= 1");
  if (n > c.max_batch)
    return fail(AXON_E_CAPACITY, "n " + std::to_string(n) + " exceeds max_batch " + std::to_string(c.max_batch));
  if (!h_slots || !d_tokens || !d_cu_seqlens || !h_cu_seqlens || !d_next_tokens)
    return fail(AXON_E_INVALID, "h_slots, d_tokens, d_cu_seqlens, h_cu_seqlens and d_next_tokens must be non-NULL");
  if (h_cu_seqlens[0] != 0) return fail(AXON_E_INVALID, "cu_seqlens[0] must be 0");
  std::vector<char> seen(c.max_batch, 0);
  std::vector<int> base(n), cnt(n);
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    const int sl = h_slots[i];
    if (sl < 0 || sl >= c.max_batch)
      return fail(AXON_E_INVALID, "entry " + std::to_string(i) + ": slot " + std::to_string(sl) + " out of range [0, " +
                                      std::to_string(c.max_batch) + ")");
    if (seen[sl]) return fail(AXON_E_INVALID, "slot " + std::to_string(sl) + " appears twice");
    seen[sl] = 1;
    const int fr = h_fresh ? h_fresh[i] : 0;
    if (fr != 0 && fr != 1) return fail(AXON_E_INVALID, "h_fresh entries must be 0 or 1");
    const int64_t ni = (int64_t)h_cu_seqlens[i + 1] - h_cu_seqlens[i];
    if (ni < 1) return fail(AXON_E_INVALID, "entry " + std::to_string(i) + " has " + std::to_string(ni) + " tokens (must be >= 1)");
    base[i] = fr ? 0 : m->h_len[sl];
    cnt[i] = (int)ni;
    if (base[i] + ni > c.max_seq)
      return fail(AXON_E_CAPACITY, "slot " + std::to_string(sl) + ": " + std::to_string(base[i]) + " + " +
                                       std::to_string(ni) + " tokens exceed max_seq " + std::to_string(c.max_seq));
    total += ni;
  }
  if (total > m->rows)
    return fail(AXON_E_CAPACITY, "step of " + std::to_string(total) + " tokens exceeds max_tokens " + std::to_string(m->rows));
  hipStream_t s = (hipStream_t)stream;
  if (m->paged()) {
    const int cols = h_block_table ? std::min(block_table_stride, m->bt_stride) : m->bt_stride;
    if (h_block_table && block_table_stride < 1) return fail(AXON_E_INVALID, "block_table_stride must be >= 1");
    // the rows each entry's slot will have after the call
    auto row_of = [&](int i, int j) -> int {
      if (h_block_table) return j < cols ? h_block_table[(int64_t)i * block_table_stride + j] : -1;
      return m->h_bt[(int64_t)h_slots[i] * m->bt_stride + j];
    };
    std::vector<char> used(c.kv_num_pages, 0);
    // pages of the slots this call leaves alone
    for (int sl = 0; sl < c.max_batch; ++sl) {
      if (seen[sl]) continue;
      for (int j = 0; j < m->bt_stride; ++j) {
        const int p = m->h_bt[(int64_t)sl * m->bt_stride + j];
        if (p >= 0) used[p] = 1;
      }
    }
    for (int i = 0; i < n; ++i) {
      const int sl = h_slots[i];
      const int need = (base[i] + cnt[i] + m->ps - 1) / m->ps;
      const int kept = (base[i] + m->ps - 1) / m->ps;  // pages holding the slot's cached positions
      if (need > cols)
        return fail(AXON_E_CAPACITY, "entry " + std::to_string(i) + " needs " + std::to_string(need) +
                                         " pages, the page table has " + std::to_string(cols) + " columns");
      for (int j = 0; j < m->bt_stride; ++j) {
        const int p = row_of(i, j);
        if (j < kept && p != m->h_bt[(int64_t)sl * m->bt_stride + j])
          return fail(AXON_E_INVALID, "entry " + std::to_string(i) + " changes page " + std::to_string(j) +
                                          " that holds cached positions of slot " + std::to_string(sl));
        if (p < 0) {
          if (j < need)
            return fail(AXON_E_CAPACITY, "slot " + std::to_string(sl) + " has no page for block " + std::to_string(j));
          continue;
        }
        if (p >= c.kv_num_pages)
          return fail(AXON_E_CAPACITY, "page id " + std::to_string(p) + " out of range [0, " + std::to_string(c.kv_num_pages) + ")");
        if (used[p]) return fail(AXON_E_INVALID, "page id " + std::to_string(p) + " appears twice");
        used[p] = 1;
      }
    }
    if (h_block_table) {
      HIP_TRY(hipEventSynchronize(m->bt_copied));
      for (int i = 0; i < n; ++i)
        for (int j = 0; j < m->bt_stride; ++j) m->h_bt[(int64_t)h_slots[i] * m->bt_stride + j] = row_of(i, j);
      HIP_TRY(hipMemcpyAsync(m->d_bt, m->h_bt, (size_t)c.max_batch * m->bt_stride * sizeof(int32_t),
                             hipMemcpyHostToDevice, s));
      HIP_TRY(hipEventRecord(m->bt_copied, s));
    }
  } else if (h_block_table) {
    return fail(AXON_E_INVALID, "h_block_table given for a contiguous cache");
  }
  // per-entry arrays: staged in pinned memory (after the previous step's copy
  // has left it), copied in one transfer
  HIP_TRY(hipEventSynchronize(m->step_copied));
  StepPlan plan;
  const int MB = c.max_batch;
  int32_t* hs = m->h_step;
  int nc = 0, nd = 0;
  for (int i = 0; i < n; ++i) {
    hs[i] = h_slots[i];
    hs[MB + i] = base[i];
    if (cnt[i] > 1 || !m->bf) {
      hs[2 * MB + nc++] = i;
    } else {
      hs[3 * MB + nd] = h_cu_seqlens[i];
      hs[4 * MB + nd] = h_slots[i];
      hs[5 * MB + nd] = base[i];
      ++nd;
      plan.dctx += m->keys_read(base[i] + 1);
    }
  }
  HIP_TRY(hipMemcpyAsync(m->d_step, hs, (size_t)6 * MB * sizeof(int32_t), hipMemcpyHostToDevice, s));
  HIP_TRY(hipEventRecord(m->step_copied, s));
  plan.n = n;
  plan.d_slot = m->d_step;
  plan.d_base = m->d_step + MB;
  plan.nc = nc;
  plan.d_chunks = m->d_step + 2 * MB;
  plan.h_chunks = hs + 2 * MB;
  plan.nd = nd;
  plan.d_drow = m->d_step + 3 * MB;
  plan.d_dslot = m->d_step + 4 * MB;
  plan.d_dpos = m->d_step + 5 * MB;
  if (m->bf && nd == n && n <= GEMV_MAX_M) {
    // decode tokens only: the fused weight-streaming decode step, recorded as
    // a graph per (n, buffers); the per-entry arrays are read from d_step
    if (int rc = replay_or_run(m, GraphKey{n, d_tokens, d_logits, d_next_tokens, d_cu_seqlens}, s, "step",
                               [&](hipStream_t st) {
                                 if (m->gpt2())
                                   enqueue_decode_gpt2(m, n, d_tokens, d_logits, d_next_tokens, st, &plan, d_cu_seqlens);
                                 else
                                   enqueue_decode_bf16(m, n, d_tokens, d_logits, d_next_tokens, st, &plan, d_cu_seqlens);
                               }))
      return rc;
  } else {
    if (m->bf)
      enqueue_prefill<bf16>(m, n, (int)total, d_tokens, d_cu_seqlens, h_cu_seqlens, 0, d_logits, d_next_tokens, s,
                            &plan);
    else
      enqueue_prefill<float>(m, n, (int)total, d_tokens, d_cu_seqlens, h_cu_seqlens, 0, d_logits, d_next_tokens, s,
                             &plan);
    int rc = check_launch("step");
    if (!rc) rc = take_enqueue_err(m, "step");
    if (rc) return rc;
  }
  int top = 0;
  for (int i = 0; i < n; ++i) {
    m->h_len[h_slots[i]] = base[i] + cnt[i];
    top = std::max(top, h_slots[i] + 1);
  }
  m->active = std::max(m->active, top);
  return AXON_OK;
}

// ------------------------------------------------------------------ training

namespace {

// Allocate the backward-pass state for up to m->rows tokens and build the
// transposed weight tiles (once per model).
int train_setup(axon_model* m, hipStream_t s) {
  TrainBufs& tb = m->train;
  if (tb.ready) return AXON_OK;
  const axon_config& c = m->cfg;
  const int64_t D = c.hidden, H = c.n_heads, KV = c.n_kv_heads, hd = c.head_dim, I = c.intermediate, V = c.vocab;
  const int64_t nq = (H + 2 * KV) * hd, Hhd = H * hd;
  tb.Tc = m->rows;
  tb.Tp = (tb.Tc + 31) / 32 * 32;
  tb.Vp = (int)((V + 31) / 32 * 32);
  const int64_t T = tb.Tc, Tp = tb.Tp, Vp = tb.Vp;
  auto tiled = [](int64_t rows, int64_t cols) { return (rows + 15) / 16 * 16 * cols; };
  auto fa = [&](float** p, int64_t n) { return dev_alloc(m, (void**)p, (size_t)n * 4); };
  auto ba = [&](bf16** p, int64_t n) { return dev_alloc(m, (void**)p, (size_t)n * 2); };
  int r = 0;
  tb.L.resize(c.n_layers);
  for (auto& l : tb.L) {
    if (!r) r = fa(&l.xin, T * D);
    if (!r) r = fa(&l.xmid, T * D);
    if (!r) r = fa(&l.lse, T * H);
    if (!r) r = fa(&l.gu, T * 2 * I);
    if (!r) r = ba(&l.h1, T * D);
    if (!r) r = ba(&l.h2, T * D);
    if (!r) r = ba(&l.q, T * Hhd);
    if (!r) r = ba(&l.o, T * Hhd);
    if (!r) r = ba(&l.a, T * I);
    if (!r) r = ba(&l.wqkvT, tiled(D, nq));
    if (!r) r = ba(&l.woT, tiled(Hhd, D));
    if (!r) r = ba(&l.wguT, tiled(D, 2 * I));
    if (!r) r = ba(&l.wdT, tiled(I, D));
  }
  const int64_t maxN = std::max({Vp, 2 * I, nq, D}), maxK = std::max({D, I, Hhd});
  if (!r) r = fa(&tb.xfin, T * D);
  if (!r) r = fa(&tb.logits, T * Vp);
  if (!r) r = fa(&tb.rowloss, T);
  if (!r) r = fa(&tb.valid, T);
  if (!r) r = fa(&tb.lserow, T);
  if (!r) r = fa(&tb.scal, 4);
  if (!r) r = fa(&tb.dx, T * D);
  if (!r) r = fa(&tb.dtmp, T * std::max({D, I, Hhd}));
  if (!r) r = fa(&tb.dgrow, T * D);
  if (!r) r = fa(&tb.dqf, T * Hhd);
  if (!r) r = fa(&tb.dkf, T * KV * hd);
  if (!r) r = fa(&tb.dvf, T * KV * hd);
  if (!r) r = fa(&tb.dkh, T * Hhd);
  if (!r) r = fa(&tb.dvh, T * Hhd);
  if (!r) r = fa(&tb.dsum, T * H);
  if (!r) r = fa(&tb.dqkvf, T * nq);
  if (!r) r = fa(&tb.colpart, (int64_t)colsum_chunks((int)T) * std::max(nq, D));
  if (!r) r = fa(&tb.gtmp, std::max(nq, 2 * I) * D);
  if (!r) r = ba(&tb.hf, T * D);
  if (!r) r = ba(&tb.dlog, T * Vp);
  if (!r) r = ba(&tb.dxb, T * D);
  if (!r) r = ba(&tb.dgu, T * 2 * I);
  if (!r) r = ba(&tb.dob, T * Hhd);
  if (!r) r = ba(&tb.dqkv, T * nq);
  if (!r) r = ba(&tb.tra, maxN * Tp);
  if (!r) r = ba(&tb.trs, maxK * Tp);
  if (!r) r = ba(&tb.trb, tiled(maxK, Tp));
  if (!r) r = ba(&tb.headT, tiled(D, Vp));
  // split-K partials of the narrow training GEMMs: up to 4 splits of an
  // output as large as T x max(D, I) or one weight's gradient
  const int64_t want = 4 * std::max({T * D, T * I, T * Hhd, nq * D, 2 * I * D});
  if (m->gemm_part_floats < want) {  // the inference buffer (if any) stays allocated until axon_free
    float* p = nullptr;
    if (!r) r = fa(&p, want);
    if (!r) {
      m->gemm_part = p;
      m->gemm_part_floats = want;
    }
  }
  tb.SP = (c.max_seq + 31) / 32 * 32 + 32;
  tb.W = (int64_t)c.max_batch * tb.SP;
  if (!r) r = fa(&tb.statp, 2 * H * tb.W);
  if (!r) r = ba(&tb.kr, tb.W * KV * hd);
  if (!r) r = ba(&tb.vr, tb.W * KV * hd);
  if (!r) r = ba(&tb.kt, tb.W * KV * hd);
  if (!r) r = ba(&tb.qt, tb.W * Hhd);
  if (!r) r = ba(&tb.dot, tb.W * Hhd);
  if (r) return r;
  // the packed copies' padding is read (masked) past each sequence's end: finite from the start
  for (bf16* p : {tb.kr, tb.vr, tb.kt}) (void)hipMemsetAsync(p, 0, (size_t)tb.W * KV * hd * 2, s);
  for (bf16* p : {tb.qt, tb.dot}) (void)hipMemsetAsync(p, 0, (size_t)tb.W * Hhd * 2, s);
  // W [N][K] (tiled) -> W^T [K][Np] tiled, through a row-major staging copy
  // whose columns N .. Np-1 are zero
  bf16* stage = nullptr;
  const int64_t most = std::max({D * nq, Hhd * D, D * 2 * I, I * D, D * Vp});
  hipError_t e = hipMalloc((void**)&stage, (size_t)most * 2);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? AXON_E_OOM : AXON_E_HIP,
                std::string("training staging allocation: ") + hipGetErrorString(e));
  }
  auto wt = [&](const void* W, int64_t N, int64_t K, int64_t Np, bf16* dst) {
    if (Np > N) (void)hipMemsetAsync(stage, 0, (size_t)K * Np * 2, s);
    launch_untile_transpose((const bf16*)W, N, (int)K, stage, Np, s);
    launch_tile_weight(stage, dst, K, (int)Np, s);
  };
  for (int l = 0; l < c.n_layers; ++l) {
    const LayerW& w = m->layers[l];
    TrainLayer& t = tb.L[l];
    wt(w.wqkv, nq, D, nq, t.wqkvT);
    wt(w.wo, D, Hhd, D, t.woT);
    wt(w.wgu, 2 * I, D, 2 * I, t.wguT);
    wt(w.wd, D, I, D, t.wdT);
  }
  wt(m->lm_head, V, D, Vp, tb.headT);
  e = hipGetLastError();
  const hipError_t e2 = hipStreamSynchronize(s);
  (void)hipFree(stage);
  if (e != hipSuccess || e2 != hipSuccess)
    return fail(AXON_E_HIP, std::string("weight transposes: ") + hipGetErrorString(e != hipSuccess ? e : e2));
  tb.ready = true;
  return AXON_OK;
}

// Forward over B fresh sequences keeping every activation the backward pass
// reads, the loss, and the reverse pass into the caller's gradient buffers
// (g: one float pointer per expected weight, in expected_weights order).
void enqueue_train(axon_model* m, int B, int T, const int32_t* d_tokens, const int32_t* d_cu, const int32_t* h_cu,
                   const int32_t* d_targets, float* d_loss, const std::vector<float*>& g,
                   const std::unordered_map<std::string, size_t>& gi, hipStream_t s) {
  const axon_config& c = m->cfg;
  TrainBufs& tb = m->train;
  const int D = c.hidden, H = c.n_heads, KV = c.n_kv_heads, hd = c.head_dim, I = c.intermediate, V = c.vocab;
  const int nq = (H + 2 * KV) * hd, Hhd = H * hd, Tp = tb.Tp, Vp = tb.Vp, L = c.n_layers;
  const float eps = c.rms_eps;
  auto G = [&](const std::string& n) { return g[gi.at(n)]; };
  // ---- forward, keeping activations
  launch_set_lengths(d_cu, m->d_len, B, s);
  launch_embed_rmsnorm<bf16>(d_tokens, (const bf16*)m->embed, (const bf16*)m->layers[0].gin, m->x, tb.L[0].h1, T, D,
                             V, eps, s);
  for (int l = 0; l < L; ++l) {
    const LayerW& w = m->layers[l];
    TrainLayer& t = tb.L[l];
    KVView kv = m->kv(l, false);
    (void)hipMemcpyAsync(t.xin, m->x, (size_t)T * D * 4, hipMemcpyDeviceToDevice, s);
    EpiArgs re = rope_epi(m, w, kv, d_cu, B, nullptr);
    re.q_out = t.q;
    gemm_many<bf16>(m, w.wqkv, t.h1, nq, T, D, EPI_ROPE, nullptr, nullptr, nq, s, &re);
    m->timed(3, H, B, T, s, [&] {
      launch_attn_prefill<bf16>(t.q, kv, t.o, T, B, d_cu, h_cu, H, s, nullptr, nullptr, nullptr, nullptr, t.lse);
    });
    gemm_resid_norm(m, w.wo, t.o, T, Hhd, (const bf16*)w.gpost, t.h2, T, nullptr, s);
    (void)hipMemcpyAsync(t.xmid, m->x, (size_t)T * D * 4, hipMemcpyDeviceToDevice, s);
    gemm_many<bf16>(m, w.wgu, t.h2, 2 * I, T, D, EPI_F32, t.gu, nullptr, 2 * I, s);
    launch_silu_reduce<bf16>(t.gu, 1, 0, t.a, T, I, s);
    if (l + 1 < L) {
      gemm_resid_norm(m, w.wd, t.a, T, I, (const bf16*)m->layers[l + 1].gin, tb.L[l + 1].h1, T, nullptr, s);
    } else {
      gemm_resid_norm(m, w.wd, t.a, T, I, (const bf16*)m->gfinal, tb.hf, T, nullptr, s);
      (void)hipMemcpyAsync(tb.xfin, m->x, (size_t)T * D * 4, hipMemcpyDeviceToDevice, s);
    }
  }
  gemm_many<bf16>(m, m->lm_head, tb.hf, V, T, D, EPI_F32, tb.logits, nullptr, Vp, s);
  // ---- loss and its gradient at the logits
  launch_ce_loss(tb.logits, Vp, V, d_targets, T, tb.rowloss, tb.valid, tb.lserow, d_loss, tb.scal, tb.dlog, s);
  // ---- backward
  // dX = dY W: [T][K] float from dY [T][N] and the tiled W^T [K][N]
  auto dX = [&](const bf16* WT, const bf16* dY, int N, int K, float* out) {
    gemm_f32_out(m, WT, dY, K, T, N, out, false, s);
  };
  // dW = dY^T X: [N][K] float from dY [T][N] (rows ldy apart) and X [T][K]
  auto dW = [&](const bf16* dY, int ldy, int N, const bf16* X, int K, float* out) {
    launch_transpose_pad(dY, ldy, T, N, tb.tra, Tp, s);
    launch_transpose_pad(X, K, T, K, tb.trs, Tp, s);
    launch_tile_weight(tb.trs, tb.trb, K, Tp, s);
    gemm_f32_out(m, tb.trb, tb.tra, K, N, Tp, out, false, s);
  };
  const bool tied = c.tie_embeddings;
  float* g_embed = G("model.embed_tokens.weight");
  dW(tb.dlog, Vp, V, tb.hf, D, tied ? g_embed : G("lm_head.weight"));
  dX(tb.headT, tb.dlog, Vp, D, tb.dtmp);
  launch_rmsnorm_bwd(tb.xfin, (const bf16*)m->gfinal, tb.dtmp, D, T, D, eps, tb.dx, 0, tb.dgrow, s);
  launch_colsum(tb.dgrow, D, T, D, tb.colpart, G("model.norm.weight"), s);
  for (int l = L - 1; l >= 0; --l) {
    const LayerW& w = m->layers[l];
    TrainLayer& t = tb.L[l];
    KVView kv = m->kv(l, false);
    const std::string p = "model.layers." + std::to_string(l) + ".";
    // MLP
    launch_to_bf16(tb.dx, tb.dxb, (int64_t)T * D, s);
    dW(tb.dxb, D, D, t.a, I, G(p + "mlp.down_proj.weight"));
    dX(t.wdT, tb.dxb, D, I, tb.dtmp);
    launch_swiglu_bwd(t.gu, tb.dtmp, tb.dgu, T, I, s);
    dW(tb.dgu, 2 * I, 2 * I, t.h2, D, tb.gtmp);
    launch_scatter_rows(tb.gtmp, 2 * I, D, 1, hd, H, KV, G(p + "mlp.gate_proj.weight"), G(p + "mlp.up_proj.weight"),
                        nullptr, s);
    dX(t.wguT, tb.dgu, 2 * I, D, tb.dtmp);
    launch_rmsnorm_bwd(t.xmid, (const bf16*)w.gpost, tb.dtmp, D, T, D, eps, tb.dx, 1, tb.dgrow, s);
    launch_colsum(tb.dgrow, D, T, D, tb.colpart, G(p + "post_attention_layernorm.weight"), s);
    // attention
    launch_to_bf16(tb.dx, tb.dxb, (int64_t)T * D, s);
    dW(tb.dxb, D, D, t.o, Hhd, G(p + "self_attn.o_proj.weight"));
    dX(t.woT, tb.dxb, D, Hhd, tb.dtmp);
    launch_to_bf16(tb.dtmp, tb.dob, (int64_t)T * Hhd, s);
    m->timed(5, H, B, T, s, [&] {
      if (!launch_attn_bwd(t.q, kv, t.o, tb.dob, t.lse, tb.dsum, tb.statp, d_cu, h_cu, B, T, H, tb.SP, tb.W, tb.kr, tb.vr, tb.kt,
                      tb.qt, tb.dot, tb.dqf, tb.dkh, tb.dvh, tb.dkf, tb.dvf, s) &&
          m->enqueue_err.empty())
        m->enqueue_err = "attention backward: packed layout does not fit the shape";
    });
    launch_rope_bwd(tb.dqf, tb.dkf, tb.dvf, m->rope_cos, m->rope_sin, d_cu, B, T, H, KV, hd, tb.dqkv,
                    c.qkv_bias ? tb.dqkvf : nullptr, s);
    dW(tb.dqkv, nq, nq, t.h1, D, tb.gtmp);
    launch_scatter_rows(tb.gtmp, nq, D, 0, hd, H, KV, G(p + "self_attn.q_proj.weight"),
                        G(p + "self_attn.k_proj.weight"), G(p + "self_attn.v_proj.weight"), s);
    if (c.qkv_bias) {
      launch_colsum(tb.dqkvf, nq, T, Hhd, tb.colpart, G(p + "self_attn.q_proj.bias"), s);
      launch_colsum(tb.dqkvf + Hhd, nq, T, KV * hd, tb.colpart, G(p + "self_attn.k_proj.bias"), s);
      launch_colsum(tb.dqkvf + Hhd + KV * hd, nq, T, KV * hd, tb.colpart, G(p + "self_attn.v_proj.bias"), s);
    }
    dX(t.wqkvT, tb.dqkv, nq, D, tb.dtmp);
    launch_rmsnorm_bwd(t.xin, (const bf16*)w.gin, tb.dtmp, D, T, D, eps, tb.dx, 1, tb.dgrow, s);
    launch_colsum(tb.dgrow, D, T, D, tb.colpart, G(p + "input_layernorm.weight"), s);
  }
  if (!tied) (void)hipMemsetAsync(g_embed, 0, (size_t)V * D * 4, s);
  launch_embed_bwd(d_tokens, tb.dx, T, D, V, g_embed, s);
}

}  // namespace

extern "C" int axon_loss_and_grads(axon_model* m, int32_t batch, const int32_t* d_tokens,
                                   const int32_t* d_cu_seqlens, const int32_t* h_cu_seqlens,
                                   const int32_t* d_targets, float* d_loss, const axon_weight* grads,
                                   int32_t n_grads, void* stream) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  const axon_config& c = m->cfg;
  if (!m->bf || m->gpt2() || m->moe_model() || c.sliding_window > 0 || m->paged())
    return fail(AXON_E_INVALID, "the backward pass covers dense Llama-family bf16 models with a contiguous cache "
                                "and no sliding window");
  if (batch < 1) return fail(AXON_E_INVALID, "batch must be >= 1");
  if (batch > c.max_batch)
    return fail(AXON_E_CAPACITY, "batch " + std::to_string(batch) + " exceeds max_batch " + std::to_string(c.max_batch));
  if (!d_tokens || !d_cu_seqlens || !h_cu_seqlens || !d_targets || !d_loss || !grads)
    return fail(AXON_E_INVALID, "d_tokens, d_cu_seqlens, h_cu_seqlens, d_targets, d_loss and grads must be non-NULL");
  if (h_cu_seqlens[0] != 0) return fail(AXON_E_INVALID, "cu_seqlens[0] must be 0");
  int64_t total = 0;
  for (int b = 0; b < batch; ++b) {
    const int64_t sb = (int64_t)h_cu_seqlens[b + 1] - h_cu_seqlens[b];
    if (sb < 1) return fail(AXON_E_INVALID, "sequence " + std::to_string(b) + " has length " + std::to_string(sb) + " (must be >= 1)");
    if (sb > c.max_seq)
      return fail(AXON_E_CAPACITY, "sequence " + std::to_string(b) + " has length " + std::to_string(sb) +
                                       " > max_seq " + std::to_string(c.max_seq));
    total += sb;
  }
  if (total > m->rows)
    return fail(AXON_E_CAPACITY, std::to_string(total) + " tokens exceed max_tokens " + std::to_string(m->rows));
  // the gradient map: exactly the weight map's names and shapes, float32, on the device
  const auto expected = expected_weights(c);
  std::unordered_map<std::string, size_t> index;
  for (size_t i = 0; i < expected.size(); ++i) index[expected[i].first] = i;
  std::vector<float*> g(expected.size(), nullptr);
  if (n_grads < 0) return fail(AXON_E_INVALID, "n_grads must be >= 0");
  for (int i = 0; i < n_grads; ++i) {
    const axon_weight& w = grads[i];
    if (!w.name) return fail(AXON_E_INVALID, "gradient " + std::to_string(i) + " has a NULL name");
    auto it = index.find(w.name);
    if (it == index.end()) return fail(AXON_E_MISSING, std::string("unknown gradient '") + w.name + "'");
    if (g[it->second]) return fail(AXON_E_MISSING, std::string("duplicate gradient '") + w.name + "'");
    const Expected& ex = expected[it->second].second;
    if (w.dtype != AXON_F32) return fail(AXON_E_DTYPE, std::string("gradient '") + w.name + "' must be AXON_F32");
    if (w.ndim != ex.ndim || w.shape[0] != ex.shape[0] || (ex.ndim == 2 && w.shape[1] != ex.shape[1]))
      return fail(AXON_E_SHAPE, std::string("gradient '") + w.name + "' has shape " + shape_str(w.ndim, w.shape) +
                                    ", expected " + shape_str(ex.ndim, ex.shape));
    if (!w.data || !w.on_device)
      return fail(AXON_E_INVALID, std::string("gradient '") + w.name + "' needs a device buffer");
    g[it->second] = (float*)w.data;
  }
  for (size_t i = 0; i < g.size(); ++i)
    if (!g[i]) return fail(AXON_E_MISSING, "missing gradient '" + expected[i].first + "'");
  hipStream_t s = (hipStream_t)stream;
  if (int r = train_setup(m, s)) return r;
  if (!attn_bwd_layout_ok(m->H(), m->KVh(), m->hd(), m->train.SP, m->train.W))
    return fail(AXON_E_INVALID, "attention backward: the packed layout needs H*hd, KV*hd, the packed width and the "
                                "per-sequence stride to be multiples of 32 (hd 64 or 128)");
  enqueue_train(m, batch, (int)total, d_tokens, d_cu_seqlens, h_cu_seqlens, d_targets, d_loss, g, index, s);
  if (int r = check_launch("backward pass")) return r;
  if (int r = take_enqueue_err(m, "backward pass")) return r;
  for (int b = 0; b < c.max_batch; ++b) m->h_len[b] = b < batch ? h_cu_seqlens[b + 1] - h_cu_seqlens[b] : 0;
  m->active = batch;
  return AXON_OK;
}

extern "C" int axon_reset_slot(axon_model* m, int32_t slot) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  if (slot < 0 || slot >= m->cfg.max_batch)
    return fail(AXON_E_INVALID, "slot " + std::to_string(slot) + " out of range [0, " + std::to_string(m->cfg.max_batch) + ")");
  m->h_len[slot] = 0;
  if (m->paged()) {
    // host view only: the device row is rewritten when the slot is next given pages
    HIP_TRY(hipEventSynchronize(m->bt_copied));
    for (int j = 0; j < m->bt_stride; ++j) m->h_bt[(int64_t)slot * m->bt_stride + j] = -1;
  }
  return AXON_OK;
}

extern "C" int axon_slot_lengths(const axon_model* m, int32_t* lens, int32_t n) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  if (n > 0 && !lens) return fail(AXON_E_INVALID, "lens is NULL");
  for (int i = 0; i < n && i < m->cfg.max_batch; ++i) lens[i] = m->h_len[i];
  return m->active;
}

extern "C" int axon_timing_enable(axon_model* m, int32_t enable) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  if (enable != 0 && enable != 1) return fail(AXON_E_INVALID, "enable must be 0 or 1");
  m->timing = enable == 1;
  m->trecs.clear();
  m->tnext = 0;
  return AXON_OK;
}

extern "C" int axon_timing_records(axon_model* m, int32_t* cls, int32_t* dims, float* ms, int32_t cap) {
  g_err.clear();
  if (!m) return fail(AXON_E_INVALID, "model is NULL");
  if (cap > 0 && (!cls || !dims || !ms)) return fail(AXON_E_INVALID, "output arrays are NULL");
  for (int i = 0; i < (int)m->trecs.size() && i < cap; ++i) {
    const TimingRec& r = m->trecs[i];
    HIP_TRY(hipEventSynchronize(r.b));
    float t = 0.f;
    HIP_TRY(hipEventElapsedTime(&t, r.a, r.b));
    cls[i] = r.cls;
    dims[3 * i] = r.d0;
    dims[3 * i + 1] = r.d1;
    dims[3 * i + 2] = r.d2;
    ms[i] = t;
  }
  return (int)m->trecs.size();
}

extern "C" void axon_free(axon_model* m) {
  if (m) release(m);
}
