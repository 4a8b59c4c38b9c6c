// HIP runtime side of the C ABI: contexts with a ladder of CU-masked stream
// pairs, argument checks, metadata staging and the per-layer launch sequence.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "hs_kernels.h"
#include "plan.h"

namespace {

// Pinned staging slots for the per-call metadata image.  Calls on different
// streams (the two stages of a co-run) must not wait for each other's queued
// work, so a call takes any slot whose copy has completed and adds a slot when
// all are still pending, up to kMaxStagingSlots; only then does it wait for
// the oldest.
constexpr int kStagingSlots = 4;
constexpr int kMaxStagingSlots = 64;
// The no-allocation entry point stages through a ring of its own, allocated
// with the context and never grown: a call waits for the oldest slot's copy
// when every slot is still pending.
constexpr int kFixedSlots = 4;
constexpr size_t kFixedSlotBytes = size_t(1) << 20;

struct Level {
  int budget = 0;
  uint32_t shared[8] = {0};
  uint32_t down[8] = {0};
  hipStream_t s_shared = nullptr;
  hipStream_t s_down = nullptr;
};

struct Slot {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
  uint64_t used = 0;  // call counter at the last use (oldest = smallest)
};

int popcount8(const uint32_t m[8]) {
  int n = 0;
  for (int i = 0; i < 8; ++i) n += __builtin_popcount(m[i]);
  return n;
}

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return hs::fail(HS_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

}  // namespace

struct hs_context {
  int device = 0;
  int n_cus = 0;
  hs_topology topo{};
  std::vector<Level> levels;
  std::vector<Slot> slots;
  std::vector<Slot> fixed_slots;  // staging of the no-allocation entry point
  uint64_t calls = 0;
  void* scratch = nullptr;        // this device's static scratch (device address)
  // Optional per-launch event timing.
  struct TimingRec {
    int kind;
    hipEvent_t a, b;
  };
  bool timing = false;
  uint64_t* clock_buf = nullptr;  // device, four launch counters per record (see LaunchClock)
  std::vector<hipEvent_t> ev_pool;
  size_t ev_next = 0;
  std::vector<TimingRec> recs;
};

// A captured decode step (see hs_decode_graph_create).
struct hs_decode_graph {
  hs_context* ctx = nullptr;
  hs_layer_cfg cfg{};
  std::vector<hs_layer_weights> w;
  std::vector<void*> k, v;  // copies of the caller's per-layer cache pointer arrays
  hs_kv_cache kv{};
  int32_t n_layers = 0, batch = 0, budget = 0;
  const void* x_in = nullptr;
  void* x_out = nullptr;
  void* ws = nullptr;
  hs::WsLayout lay{};
  hs::PlanCapacity cap{};
  bool paged = false;
  size_t image_bytes = 0;   // the fixed layout's image size (every launch's plan has it)
  hipStream_t stream = nullptr;
  hipGraphExec_t exec = nullptr;
};

namespace {

const Level* find_level(const hs_context* ctx, int budget) {
  for (const Level& l : ctx->levels)
    if (l.budget == budget) return &l;
  return nullptr;
}

void destroy_context(hs_context* ctx) {
  if (!ctx) return;
  hipSetDevice(ctx->device);
  for (Level& l : ctx->levels) {
    if (l.s_shared) hipStreamDestroy(l.s_shared);
    if (l.s_down) hipStreamDestroy(l.s_down);
  }
  for (hipEvent_t e : ctx->ev_pool) hipEventDestroy(e);
  if (ctx->clock_buf) hipFree(ctx->clock_buf);
  for (std::vector<Slot>* ring : {&ctx->slots, &ctx->fixed_slots})
    for (Slot& s : *ring) {
      if (s.ev) {
        hipEventSynchronize(s.ev);
        hipEventDestroy(s.ev);
      }
      if (s.host) hipHostFree(s.host);
    }
  delete ctx;
}

// Copy the plan's metadata image to the workspace through a pinned slot.
hs_status stage_metadata(hs_context* ctx, const hs::Plan& plan, void* dst, hipStream_t s) {
  Slot* free_slot = nullptr;
  Slot* oldest = nullptr;
  for (Slot& sl : ctx->slots) {
    if (sl.pending) {
      const hipError_t q = hipEventQuery(sl.ev);
      if (q == hipSuccess) {
        sl.pending = false;
      } else if (q != hipErrorNotReady) {
        return hs::fail(HS_ERR_HIP, "hipEventQuery failed: %s", hipGetErrorString(q));
      }
    }
    if (!sl.pending && !free_slot) free_slot = &sl;
    if (!oldest || sl.used < oldest->used) oldest = &sl;
  }
  if (!free_slot && ctx->slots.size() < size_t(kMaxStagingSlots)) {
    Slot fresh;
    HIP_TRY(hipEventCreateWithFlags(&fresh.ev, hipEventDisableTiming));
    ctx->slots.push_back(fresh);
    free_slot = &ctx->slots.back();
  }
  if (!free_slot) {
    HIP_TRY(hipEventSynchronize(oldest->ev));
    oldest->pending = false;
    free_slot = oldest;
  }
  Slot& slot = *free_slot;
  slot.used = ++ctx->calls;
  const size_t bytes = plan.image.size();
  if (slot.cap < bytes) {
    if (slot.host) HIP_TRY(hipHostFree(slot.host));
    slot.host = nullptr;
    slot.cap = 0;
    const size_t cap = hs::align_up(bytes, size_t(1) << 20);
    HIP_TRY(hipHostMalloc(&slot.host, cap, hipHostMallocDefault));
    slot.cap = cap;
  }
  memcpy(slot.host, plan.image.data(), bytes);
  HIP_TRY(hipMemcpyAsync(dst, slot.host, bytes, hipMemcpyHostToDevice, s));
  HIP_TRY(hipEventRecord(slot.ev, s));
  slot.pending = true;
  return HS_OK;
}

// The same through the fixed ring: no allocation, no growth.  The image must
// fit a slot (checked by the caller before anything is enqueued).
hs_status stage_metadata_fixed(hs_context* ctx, const hs::Plan& plan, void* dst, hipStream_t s) {
  Slot* slot = nullptr;
  for (Slot& sl : ctx->fixed_slots) {
    if (sl.pending) {
      const hipError_t q = hipEventQuery(sl.ev);
      if (q == hipSuccess) {
        sl.pending = false;
      } else if (q != hipErrorNotReady) {
        return hs::fail(HS_ERR_HIP, "hipEventQuery failed: %s", hipGetErrorString(q));
      }
    }
    if (!sl.pending && !slot) slot = &sl;
  }
  if (!slot) {
    for (Slot& sl : ctx->fixed_slots)
      if (!slot || sl.used < slot->used) slot = &sl;
    HIP_TRY(hipEventSynchronize(slot->ev));
    slot->pending = false;
  }
  slot->used = ++ctx->calls;
  memcpy(slot->host, plan.image.data(), plan.image.size());
  HIP_TRY(hipMemcpyAsync(dst, slot->host, plan.image.size(), hipMemcpyHostToDevice, s));
  HIP_TRY(hipEventRecord(slot->ev, s));
  slot->pending = true;
  return HS_OK;
}

// Resolve the stream for (budget, role) and check that its mask carries the budget.
hs_status resolve_stream(hs_context* ctx, int32_t budget, int role, void* stream, hipStream_t* out) {
  if (budget < 1 || budget > ctx->n_cus)
    return hs::fail(HS_ERR_BUDGET, "CU budget %d outside [1, %d]", budget, ctx->n_cus);
  if (!stream) {
    const int level_budget = role == HS_ROLE_SHARED ? budget : ctx->n_cus - budget;
    const Level* l = find_level(ctx, level_budget);
    if (!l) return hs::fail(HS_ERR_BUDGET, "no ladder level for a %s budget of %d CUs",
                            role == HS_ROLE_SHARED ? "shared" : "downstream", budget);
    *out = role == HS_ROLE_SHARED ? l->s_shared : l->s_down;
    if (!*out) return hs::fail(HS_ERR_BUDGET, "ladder level %d has no downstream stream", level_budget);
    return HS_OK;
  }
  uint32_t mask[8] = {0};
  HIP_TRY(hipExtStreamGetCUMask(reinterpret_cast<hipStream_t>(stream), 8, mask));
  const int n = popcount8(mask);
  if (n != budget)
    return hs::fail(HS_ERR_BUDGET, "stream carries %d CUs, budget is %d", n, budget);
  *out = reinterpret_cast<hipStream_t>(stream);
  return HS_OK;
}

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<uint8_t*>(base) + off);
}

constexpr size_t kTimingPairs = 8192;

void timing_begin(hs_context* ctx, hipStream_t s, hipEvent_t* a, hipEvent_t* b) {
  *a = *b = nullptr;
  if (!ctx->timing || ctx->ev_next + 2 > ctx->ev_pool.size()) return;
  *a = ctx->ev_pool[ctx->ev_next++];
  *b = ctx->ev_pool[ctx->ev_next++];
  hipEventRecord(*a, s);
}

void timing_end(hs_context* ctx, hipStream_t s, int kind, hipEvent_t a, hipEvent_t b) {
  if (!a) return;
  hipEventRecord(b, s);
  ctx->recs.push_back({kind, a, b});
}

// Clock counters of the launch the next TIMED record brackets (record i
// owns counters 4i .. 4i + 3), or null when it will not be recorded.
uint64_t* clock_slot(const hs_context* ctx) {
  if (!ctx->timing || !ctx->clock_buf || ctx->ev_next + 2 > ctx->ev_pool.size()) return nullptr;
  return ctx->clock_buf + 4 * (ctx->ev_next / 2);
}

#define TIMED(kind, expr)                              \
  do {                                                 \
    hipEvent_t ta_, tb_;                               \
    timing_begin(ctx, s, &ta_, &tb_);                  \
    HIP_TRY(expr);                                     \
    timing_end(ctx, s, kind, ta_, tb_);                \
  } while (0)

// Large persistent GEMM, or the skinny variant for decode-sized batches.
hipError_t gemm(int epi, const hs::GemmArgs& a, int grid_cap, hipStream_t s) {
  if (hs::skinny_supported(epi, a)) return hs::launch_gemm_skinny(epi, a, s);
  return hs::launch_gemm(epi, a, grid_cap, s);
}

// Residual GEMM a also produces the next RMSNorm's input: its output times
// gain in fp16 (into n_buf) and per-row partial sums of squares (into sumsq).
void fold_norm(hs::GemmArgs& a, float* sumsq, uint16_t* n_buf, const void* gain) {
  a.sumsq_out = sumsq;
  a.scaled_out = n_buf;
  a.gain = static_cast<const uint16_t*>(gain);
}

// The next projection scales its rows from those partial sums.
void use_norm(hs::GemmArgs& a, const float* sumsq, int parts, float eps) {
  a.row_sumsq = sumsq;
  a.row_parts = parts;
  a.eps = eps;
}

// The kernel launches of one call (everything after the metadata copy and
// the RoPE table): the layer loop of the shared-stage forward and the decode
// step.  With L.fixed the plan has a fixed layout and single-row attention is
// launched over the layout's capacity, reading the call's work item count from
// the metadata image, so the launches can be captured once and replayed.
struct LaunchSet {
  const hs_layer_cfg* cfg;
  const hs_layer_weights* w;
  int32_t n_layers;
  const void* x_in;
  void* x_out;
  const hs_kv_cache* kv;
  bool cache;
  void* ws;
  hs::WsLayout lay;
  const hs::Plan* plan_ptr;
  int32_t budget;
  bool pos3;
  bool fixed;
};

hs_status launch_layers(hs_context* ctx, const LaunchSet& L, hipStream_t s) {
  const hs_layer_cfg* cfg = L.cfg;
  const hs_layer_weights* w = L.w;
  const int32_t n_layers = L.n_layers;
  const hs::Plan& plan = *L.plan_ptr;
  const hs::WsLayout& lay = L.lay;
  void* ws = L.ws;
  const hs_kv_cache* kv = L.kv;
  const int32_t T = plan.T, budget = L.budget;
  const int d = cfg->hidden, hq = cfg->n_q_heads, hkv = cfg->n_kv_heads, dh = cfg->head_dim, f = cfg->ffn;
  uint8_t* meta = at<uint8_t>(ws, lay.meta);
  const int32_t* d_pos = reinterpret_cast<const int32_t*>(meta + plan.pos);
  const int64_t* d_koff = reinterpret_cast<const int64_t*>(meta + plan.k_off);
  const int64_t* d_voff = reinterpret_cast<const int64_t*>(meta + plan.v_off);
  float2* rope = at<float2>(ws, lay.rope);
  uint16_t* n_buf = at<uint16_t>(ws, lay.n);
  uint16_t* q_buf = at<uint16_t>(ws, lay.q);
  uint16_t* o_buf = at<uint16_t>(ws, lay.o);
  float* h_buf = at<float>(ws, lay.h);
  uint16_t* a_buf = at<uint16_t>(ws, lay.a);
  float* xtmp = at<float>(ws, lay.xtmp);
  float* sk_part = lay.part_bytes ? at<float>(ws, lay.part) : nullptr;
  int32_t* sk_count = plan.n_counters ? reinterpret_cast<int32_t*>(meta + plan.counters) : nullptr;
  // Decode-sized layers (every GEMM on the skinny path) fold RMSNorm into the
  // GEMMs around it after layer 0's: each residual GEMM writes its output
  // times the next norm's gain (fp16, into n_buf) and per-row partial sums of
  // squares over its 32-column strips; the next projection scales its rows by
  // rsqrt(mean square + eps).  Larger batches keep the norm kernel.
  float* sumsq = at<float>(ws, lay.sumsq);
  const int norm_parts = d / 32;
  bool folded = false;  // n_buf holds x * gain, sumsq its partial sums
  // Decode-sized batches keep the GEMM inputs (normed rows, attention output,
  // SwiGLU output) k-group-major, the skinny GEMM's operand layout.
  const int k8 = T <= hs::kSkinnyMaxRows ? hs::skinny_k8_rows(T) : 0;

  const int grid_cap = budget;  // persistent GEMM: one block per CU of the budget
  const float scale_log2 = 1.4426950408889634f / sqrtf(float(dh));
  // The residual stream is bf16 only at the input; every layer writes fp32.
  const uint16_t* x_cur = static_cast<const uint16_t*>(L.x_in);
  const float* x_cur_f32 = nullptr;
  for (int l = 0; l < n_layers; ++l) {
    // The last layer writes x_out; earlier layers alternate so that no layer
    // reads and writes the same buffer.
    const int remaining = n_layers - 1 - l;
    float* x_next = (remaining % 2 == 0) ? static_cast<float*>(L.x_out) : xtmp;
    uint16_t* kstore = L.cache ? static_cast<uint16_t*>(kv->k[l]) : at<uint16_t>(ws, lay.kpack);
    uint16_t* vstore = L.cache ? static_cast<uint16_t*>(kv->v[l]) : at<uint16_t>(ws, lay.vpack);

    if (!folded)
      TIMED(HS_KERNEL_RMSNORM, hs::launch_rmsnorm(x_cur, x_cur_f32, static_cast<const uint16_t*>(w[l].ln1), n_buf,
                                                  T, d, cfg->rms_eps, k8, 4 * budget, s));
    hs::GemmArgs g{};
    g.part = sk_part;
    g.counters = sk_count;
    g.A = n_buf;
    g.W = static_cast<const uint16_t*>(w[l].w_qkv);
    g.w_f16 = w[l].format == HS_WEIGHTS_F16;
    g.M = T;
    g.K = d;
    g.n_tiles_n = (hq + 2 * hkv) * dh / 256;
    g.q = q_buf;
    g.kstore = kstore;
    g.vstore = vstore;
    // RoPE positions: the plain row positions, or the three multimodal components.
    g.pos = L.pos3 ? reinterpret_cast<const int32_t*>(meta + plan.pos3) : d_pos;
    g.pos_stride = L.pos3 ? T : 0;
    g.sec1 = L.pos3 ? cfg->mrope_sections[0] : dh / 2;
    g.sec2 = L.pos3 ? cfg->mrope_sections[0] + cfg->mrope_sections[1] : dh / 2;
    g.k_off = d_koff;
    g.v_off = d_voff;
    g.kv_head_stride = plan.kv_head_stride;
    g.rope = rope;
    g.bias = static_cast<const uint16_t*>(w[l].b_qkv);
    g.hq = hq;
    g.hkv = hkv;
    g.dh = dh;
    g.k8_rows = k8;
    if (folded) use_norm(g, sumsq, norm_parts, cfg->rms_eps);
    g.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_QKV, gemm(hs::EPI_QKV, g, grid_cap, s));

    hs::AttnArgs at_args{};
    at_args.q = q_buf;
    at_args.kstore = kstore;
    at_args.vstore = vstore;
    at_args.o = o_buf;
    at_args.o_k8_rows = k8;
    at_args.items = reinterpret_cast<const int32_t*>(meta + plan.att_items);
    at_args.n_items = plan.n_att_items;
    at_args.seq_start = reinterpret_cast<const int32_t*>(meta + plan.seq_start);
    at_args.seq_len = reinterpret_cast<const int32_t*>(meta + plan.seq_len);
    at_args.seq_ctx = reinterpret_cast<const int32_t*>(meta + plan.seq_ctx);
    at_args.seq_page0 = reinterpret_cast<const int32_t*>(meta + plan.seq_page0);
    at_args.page_base = reinterpret_cast<const int64_t*>(meta + plan.page_base);
    at_args.page_keys = plan.page_keys;
    at_args.kv_head_stride = plan.kv_head_stride;
    at_args.hq = hq;
    at_args.hkv = hkv;
    at_args.dh = dh;
    at_args.scale_log2 = scale_log2;
    at_args.clock = clock_slot(ctx);
    if (plan.n_att_items > 0) TIMED(HS_KERNEL_ATTENTION, hs::launch_attention(at_args, s));

    hs::DecodeAttnArgs da{};
    da.q = q_buf;
    da.kstore = kstore;
    da.vstore = vstore;
    da.o = o_buf;
    da.o_k8_rows = k8;
    da.items = reinterpret_cast<const hs::DecItem*>(meta + plan.dec_items);
    da.n_items = L.fixed ? int(plan.cap_dec_items) : plan.n_dec_items;
    da.n_items_dev = L.fixed ? reinterpret_cast<const int32_t*>(meta + plan.dec_n) : nullptr;
    da.part = lay.dec_part_bytes ? at<float>(ws, lay.dec_part) : nullptr;
    da.counters = reinterpret_cast<int32_t*>(meta + plan.dec_count);
    da.kv_head_stride = plan.kv_head_stride;
    da.page_keys = plan.page_keys;
    da.unit_keys = plan.unit_keys;
    da.hq = hq;
    da.hkv = hkv;
    da.dh = dh;
    da.scale_log2 = scale_log2;
    if (plan.n_dec_rows > 0 || L.fixed) TIMED(HS_KERNEL_DECODE_ATTN, hs::launch_decode_attention(da, s));

    hs::GemmArgs go{};
    go.part = sk_part;
    go.counters = sk_count;
    go.A = o_buf;
    go.W = static_cast<const uint16_t*>(w[l].w_o);
    go.w_f16 = w[l].format == HS_WEIGHTS_F16;
    go.M = T;
    go.K = hq * dh;
    go.n_tiles_n = d / 256;
    go.out_f32 = h_buf;
    go.ldo = d;
    go.resid = x_cur;
    go.resid_f32 = x_cur_f32;
    go.k8_rows = k8;
    // Fold when every GEMM of the layer takes the skinny path (gate/up and
    // down share M, and their K are multiples of 64) and a consumer can
    // prefetch a row's partial sums.
    const bool fold = hs::skinny_supported(hs::EPI_QKV, g) && hs::skinny_supported(hs::EPI_RESID, go) &&
                      norm_parts <= hs::kSkinnyMaxNormParts;
    if (fold) fold_norm(go, sumsq, n_buf, w[l].ln2);
    go.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_O_PROJ, gemm(hs::EPI_RESID, go, grid_cap, s));
    if (!fold)
      TIMED(HS_KERNEL_RMSNORM, hs::launch_rmsnorm(nullptr, h_buf, static_cast<const uint16_t*>(w[l].ln2), n_buf, T,
                                                  d, cfg->rms_eps, k8, 4 * budget, s));

    hs::GemmArgs gu{};
    gu.part = sk_part;
    gu.counters = sk_count;
    gu.A = n_buf;
    gu.W = static_cast<const uint16_t*>(w[l].w_gate_up);
    gu.w_f16 = w[l].format == HS_WEIGHTS_F16;
    gu.M = T;
    gu.K = d;
    gu.n_tiles_n = f / 128;
    gu.out = a_buf;
    gu.ldo = f;
    gu.ffn = f;
    gu.k8_rows = k8;
    if (fold) use_norm(gu, sumsq, norm_parts, cfg->rms_eps);
    gu.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_GATE_UP, gemm(hs::EPI_SWIGLU, gu, grid_cap, s));

    hs::GemmArgs gd{};
    gd.part = sk_part;
    gd.counters = sk_count;
    gd.A = a_buf;
    gd.W = static_cast<const uint16_t*>(w[l].w_down);
    gd.w_f16 = w[l].format == HS_WEIGHTS_F16;
    gd.M = T;
    gd.K = f;
    gd.n_tiles_n = d / 256;
    gd.out_f32 = x_next;
    gd.ldo = d;
    gd.resid_f32 = h_buf;
    gd.k8_rows = k8;
    folded = fold && l + 1 < n_layers;
    if (folded) fold_norm(gd, sumsq, n_buf, w[l + 1].ln1);
    gd.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_DOWN, gemm(hs::EPI_RESID, gd, grid_cap, s));
    x_cur = nullptr;
    x_cur_f32 = x_next;
  }
  return HS_OK;
}

// Shared body of the prefill forward and the decode step.
// noalloc: the workspace is the context's static scratch (ws and ws_bytes are
// ignored), laid out without the packed key/value slot (a cache is required),
// and the metadata goes through the fixed staging ring.
hs_status run_stack(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w, int32_t n_layers,
                    const void* x_in, void* x_out, const int32_t* seq_offsets, const int32_t* ctx_lens,
                    int32_t n_seqs, const hs_kv_cache* kv, int32_t budget, int role, void* stream,
                    void* ws, size_t ws_bytes, const int32_t* pos3 = nullptr, bool noalloc = false) {
  hs::clear_error();
  hs_status st = hs::validate_cfg(cfg);
  if (st != HS_OK) return st;
  if (!w || n_layers < 1) return hs::fail(HS_ERR_INVALID_ARG, "weights missing or n_layers %d < 1", n_layers);
  for (int l = 0; l < n_layers; ++l) {
    if (!w[l].ln1 || !w[l].w_qkv || !w[l].w_o || !w[l].ln2 || !w[l].w_gate_up || !w[l].w_down)
      return hs::fail(HS_ERR_INVALID_ARG, "layer %d has a null weight pointer", l);
    if (w[l].format != HS_WEIGHTS_BF16 && w[l].format != HS_WEIGHTS_F16)
      return hs::fail(HS_ERR_INVALID_ARG, "layer %d has weight format %d", l, w[l].format);
  }
  if (!x_in || !x_out) return hs::fail(HS_ERR_INVALID_ARG, "x_in / x_out is null");
  if (x_in == x_out) return hs::fail(HS_ERR_INVALID_ARG, "x_in and x_out must not alias");
  int32_t T = 0, max_pos = 0;
  st = hs::validate_batch(seq_offsets, ctx_lens, n_seqs, &T, &max_pos);
  if (st != HS_OK) return st;
  st = hs::check_32bit_extents(*cfg, T, kv ? kv->max_ctx : 0);
  if (st != HS_OK) return st;
  hs::KvPlacement place;
  if (kv) {
    if (!ctx_lens) return hs::fail(HS_ERR_INVALID_ARG, "a key/value cache needs ctx_lens");
    if (!kv->k || !kv->v) return hs::fail(HS_ERR_INVALID_ARG, "cache pointer arrays are null");
    for (int l = 0; l < n_layers; ++l)
      if (!kv->k[l] || !kv->v[l]) return hs::fail(HS_ERR_INVALID_ARG, "cache of layer %d is null", l);
    if (kv->max_ctx < 64 || kv->max_ctx % 64 != 0)
      return hs::fail(HS_ERR_INVALID_ARG, "max_ctx %d must be a positive multiple of 64", kv->max_ctx);
    if (kv->block_table) {
      st = hs::check_block_table(kv->block_table, kv->pages_per_seq, kv->n_slots, kv->max_ctx, seq_offsets,
                                 ctx_lens, n_seqs);
      if (st != HS_OK) return st;
      place.table = kv->block_table;
      place.pages_per_seq = kv->pages_per_seq;
    } else {
      if (n_seqs > kv->n_slots)
        return hs::fail(HS_ERR_INVALID_ARG, "%d sequences but only %d cache slots", n_seqs, kv->n_slots);
      if (max_pos > kv->max_ctx)
        return hs::fail(HS_ERR_INVALID_ARG, "position %d exceeds max_ctx %d", max_pos - 1, kv->max_ctx);
    }
    place.cache = true;
    place.max_ctx = kv->max_ctx;
  } else if (ctx_lens) {
    for (int b = 0; b < n_seqs; ++b)
      if (ctx_lens[b] != 0)
        return hs::fail(HS_ERR_INVALID_ARG, "ctx_lens[%d] = %d but no cache holds the prefix", b, ctx_lens[b]);
  }
  if (pos3) {
    const int32_t* sec = cfg->mrope_sections;
    if (!(sec[0] || sec[1] || sec[2]))
      return hs::fail(HS_ERR_INVALID_ARG, "multimodal positions need non-zero mrope_sections");
    for (int64_t i = 0; i < 3 * int64_t(T); ++i)
      if (pos3[i] < 0 || pos3[i] >= max_pos)
        return hs::fail(HS_ERR_INVALID_ARG, "multimodal position %d (entry %lld) outside [0, %d)", pos3[i],
                        (long long)i, max_pos);
  }
  if (!ctx) return hs::fail(HS_ERR_INVALID_ARG, "context is null");
  hipStream_t s = nullptr;
  st = resolve_stream(ctx, budget, role, stream, &s);
  if (st != HS_OK) return st;
  if (noalloc) {
    if (!place.cache) return hs::fail(HS_ERR_INVALID_ARG, "the no-allocation call needs a key/value cache");
    if (!ctx->scratch) return hs::fail(HS_ERR_INTERNAL, "the context has no static scratch");
    ws = ctx->scratch;
    ws_bytes = hs::noalloc_scratch_bytes();
  }
  if (!ws) return hs::fail(HS_ERR_WORKSPACE, "workspace is null");
  const hs::WsLayout lay = hs::ws_layout(*cfg, T, n_seqs, max_pos, place.table ? place.max_ctx : 0, !noalloc);
  if (ws_bytes < lay.total) {
    if (noalloc)
      return hs::fail(HS_ERR_WORKSPACE, "the call needs %zu bytes of scratch; the static scratch holds %zu",
                      lay.total, ws_bytes);
    return hs::fail(HS_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, lay.total);
  }
  place.packed_ctx = lay.packed_ctx;
  hs::Plan plan;
  st = hs::build_plan(*cfg, seq_offsets, ctx_lens, n_seqs, place, &plan, pos3);
  if (st != HS_OK) return st;
  if (plan.image.size() > lay.meta_bytes) return hs::fail(HS_ERR_INTERNAL, "metadata image exceeds its region");
  if (noalloc && plan.image.size() > kFixedSlotBytes)
    return hs::fail(HS_ERR_WORKSPACE, "metadata of %zu bytes exceeds the %zu-byte staging slot of the "
                    "no-allocation call", plan.image.size(), kFixedSlotBytes);

  HIP_TRY(hipSetDevice(ctx->device));
  // An error left by an earlier, unrelated runtime call has been reported to
  // its caller; clear it so the launch checks below see only this call's.
  (void)hipGetLastError();
  st = noalloc ? stage_metadata_fixed(ctx, plan, at<void>(ws, lay.meta), s)
               : stage_metadata(ctx, plan, at<void>(ws, lay.meta), s);
  if (st != HS_OK) return st;
  TIMED(HS_KERNEL_ROPE_TABLE,
        hs::launch_rope_table(at<float2>(ws, lay.rope), max_pos, cfg->head_dim, cfg->rope_base, s));
  LaunchSet L{cfg, w, n_layers, x_in, x_out, kv, place.cache, ws, lay, &plan, budget, pos3 != nullptr, false};
  return launch_layers(ctx, L, s);
}

}  // namespace

extern "C" {

hs_status hs_context_create(int32_t device, const int32_t* budgets, int32_t n_budgets, const hs_topology* topo,
                            hs_context** out) {
  hs::clear_error();
  if (!out) return hs::fail(HS_ERR_INVALID_ARG, "output pointer is null");
  *out = nullptr;
  if (n_budgets < 0 || (n_budgets > 0 && !budgets))
    return hs::fail(HS_ERR_INVALID_ARG, "budget list is null");
  int n_dev = 0;
  HIP_TRY(hipGetDeviceCount(&n_dev));
  if (device < 0 || device >= n_dev) return hs::fail(HS_ERR_INVALID_ARG, "device %d of %d", device, n_dev);
  HIP_TRY(hipSetDevice(device));
  hipDeviceProp_t prop;
  HIP_TRY(hipGetDeviceProperties(&prop, device));
  const int n_cus = prop.multiProcessorCount;
  if (n_cus < 1 || n_cus > 256) return hs::fail(HS_ERR_UNSUPPORTED, "%d compute units", n_cus);

  hs_context* ctx = new hs_context();
  ctx->device = device;
  ctx->n_cus = n_cus;
  if (topo) {
    if (topo->n_cus != n_cus) {
      delete ctx;
      return hs::fail(HS_ERR_INVALID_ARG, "topology has %d CUs, device has %d", topo->n_cus, n_cus);
    }
    ctx->topo = *topo;
  } else {
    const int n_xcc = (n_cus % 8 == 0) ? 8 : 1;
    hs_status st = hs_default_topology(n_cus, n_xcc, &ctx->topo);
    if (st != HS_OK) {
      delete ctx;
      return st;
    }
  }
  std::vector<int32_t> want(budgets, budgets + n_budgets);
  bool has_full = false;
  for (int32_t b : want) has_full |= (b == n_cus);
  if (!has_full) want.push_back(n_cus);
  for (int32_t b : want) {
    if (find_level(ctx, b)) continue;
    Level l;
    l.budget = b;
    hs_status st = hs_cu_partition(&ctx->topo, b, l.shared, l.down);
    if (st != HS_OK) {
      destroy_context(ctx);
      return st;
    }
    hipError_t e;
    if (b == n_cus) {
      e = hipStreamCreateWithFlags(&l.s_shared, hipStreamNonBlocking);
    } else {
      e = hipExtStreamCreateWithCUMask(&l.s_shared, 8, l.shared);
      if (e == hipSuccess) e = hipExtStreamCreateWithCUMask(&l.s_down, 8, l.down);
    }
    if (e != hipSuccess) {
      ctx->levels.push_back(l);
      destroy_context(ctx);
      return hs::fail(HS_ERR_HIP, "stream creation for budget %d failed: %s", b, hipGetErrorString(e));
    }
    ctx->levels.push_back(l);
  }
  ctx->slots.resize(kStagingSlots);
  for (Slot& s : ctx->slots) {
    hipError_t e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming);
    if (e != hipSuccess) {
      destroy_context(ctx);
      return hs::fail(HS_ERR_HIP, "event creation failed: %s", hipGetErrorString(e));
    }
  }
  // The no-allocation entry point's resources: this device's static scratch
  // (its address resolved once per device, with the device current) and a
  // fixed ring of pinned staging slots.
  {
    hipError_t e = hs::noalloc_scratch_resolve(device, &ctx->scratch);
    if (e != hipSuccess) {
      destroy_context(ctx);
      return hs::fail(HS_ERR_HIP, "resolving the static scratch of device %d failed: %s", device,
                      hipGetErrorString(e));
    }
    ctx->fixed_slots.resize(kFixedSlots);
    for (Slot& s : ctx->fixed_slots) {
      e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming);
      if (e == hipSuccess) e = hipHostMalloc(&s.host, kFixedSlotBytes, hipHostMallocDefault);
      if (e != hipSuccess) {
        destroy_context(ctx);
        return hs::fail(HS_ERR_HIP, "no-allocation staging setup failed: %s", hipGetErrorString(e));
      }
      s.cap = kFixedSlotBytes;
    }
  }
  *out = ctx;
  return HS_OK;
}

hs_status hs_context_topology(const hs_context* ctx, hs_topology* out) {
  if (!ctx || !out) return hs::fail(HS_ERR_INVALID_ARG, "null argument");
  *out = ctx->topo;
  return HS_OK;
}

hs_status hs_context_stream(hs_context* ctx, int32_t cu_budget, int32_t role, void** stream_out) {
  if (!ctx || !stream_out) return hs::fail(HS_ERR_INVALID_ARG, "null argument");
  if (role != HS_ROLE_SHARED && role != HS_ROLE_DOWN) return hs::fail(HS_ERR_INVALID_ARG, "role %d", role);
  const Level* l = find_level(ctx, cu_budget);
  if (!l) return hs::fail(HS_ERR_BUDGET, "budget %d is not on the ladder", cu_budget);
  hipStream_t s = role == HS_ROLE_SHARED ? l->s_shared : l->s_down;
  if (!s) return hs::fail(HS_ERR_BUDGET, "the full budget has no downstream stream");
  *stream_out = s;
  return HS_OK;
}

hs_status hs_context_masks(const hs_context* ctx, int32_t cu_budget, uint32_t shared_mask[8], uint32_t down_mask[8]) {
  if (!ctx) return hs::fail(HS_ERR_INVALID_ARG, "null context");
  const Level* l = find_level(ctx, cu_budget);
  if (!l) return hs::fail(HS_ERR_BUDGET, "budget %d is not on the ladder", cu_budget);
  if (shared_mask) memcpy(shared_mask, l->shared, sizeof(l->shared));
  if (down_mask) memcpy(down_mask, l->down, sizeof(l->down));
  return HS_OK;
}

hs_status hs_context_destroy(hs_context* ctx) {
  destroy_context(ctx);
  return HS_OK;
}

hs_status hs_shared_stage_forward(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                  int32_t n_layers, const void* x_in, void* x_out, const int32_t* seq_offsets,
                                  const int32_t* ctx_lens, int32_t n_seqs, const hs_kv_cache* kv,
                                  int32_t cu_budget, void* stream, void* workspace, size_t ws_bytes) {
  return run_stack(ctx, cfg, w, n_layers, x_in, x_out, seq_offsets, ctx_lens, n_seqs, kv, cu_budget,
                   HS_ROLE_SHARED, stream, workspace, ws_bytes);
}

hs_status hs_shared_stage_forward_mrope(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                        int32_t n_layers, const void* x_in, void* x_out, const int32_t* seq_offsets,
                                        const int32_t* ctx_lens, int32_t n_seqs, const hs_kv_cache* kv,
                                        const int32_t* positions3, int32_t cu_budget, void* stream, void* workspace,
                                        size_t ws_bytes) {
  if (!positions3) {
    hs::clear_error();
    return hs::fail(HS_ERR_INVALID_ARG, "positions3 is null");
  }
  return run_stack(ctx, cfg, w, n_layers, x_in, x_out, seq_offsets, ctx_lens, n_seqs, kv, cu_budget,
                   HS_ROLE_SHARED, stream, workspace, ws_bytes, positions3);
}

hs_status hs_downstream_decode_step(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                    int32_t n_layers, const void* x_in, void* x_out, const hs_kv_cache* kv,
                                    const int32_t* kv_lens, int32_t batch, int32_t cu_budget, void* stream,
                                    void* workspace, size_t ws_bytes) {
  hs::clear_error();
  if (!kv) return hs::fail(HS_ERR_INVALID_ARG, "decode needs a key/value cache");
  if (!kv_lens) return hs::fail(HS_ERR_INVALID_ARG, "kv_lens is null");
  if (batch < 1) return hs::fail(HS_ERR_INVALID_ARG, "batch %d < 1", batch);
  std::vector<int32_t> off(batch + 1);
  for (int32_t b = 0; b <= batch; ++b) off[b] = b;
  return run_stack(ctx, cfg, w, n_layers, x_in, x_out, off.data(), kv_lens, batch, kv, cu_budget,
                   HS_ROLE_DOWN, stream, workspace, ws_bytes);
}

hs_status hs_downstream_decode_step_noalloc(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                            int32_t n_layers, const void* x_in, void* x_out, const hs_kv_cache* kv,
                                            const int32_t* kv_lens, int32_t batch, int32_t cu_budget, void* stream) {
  hs::clear_error();
  if (!kv) return hs::fail(HS_ERR_INVALID_ARG, "decode needs a key/value cache");
  if (!kv_lens) return hs::fail(HS_ERR_INVALID_ARG, "kv_lens is null");
  if (batch < 1) return hs::fail(HS_ERR_INVALID_ARG, "batch %d < 1", batch);
  if (batch > hs::kNoAllocMaxBatch)
    return hs::fail(HS_ERR_UNSUPPORTED, "batch %d exceeds the no-allocation call's %d rows", batch,
                    hs::kNoAllocMaxBatch);
  int32_t off[hs::kNoAllocMaxBatch + 1];
  for (int32_t b = 0; b <= batch; ++b) off[b] = b;
  return run_stack(ctx, cfg, w, n_layers, x_in, x_out, off, kv_lens, batch, kv, cu_budget, HS_ROLE_DOWN, stream,
                   nullptr, 0, nullptr, true);
}

hs_status hs_decode_graph_create(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                 int32_t n_layers, const void* x_in, void* x_out, const hs_kv_cache* kv,
                                 int32_t batch, int32_t cu_budget, void* stream, void* workspace, size_t ws_bytes,
                                 hs_decode_graph** out) {
  hs::clear_error();
  if (!out) return hs::fail(HS_ERR_INVALID_ARG, "output pointer is null");
  *out = nullptr;
  if (!ctx) return hs::fail(HS_ERR_INVALID_ARG, "context is null");
  hs_status st = hs::validate_cfg(cfg);
  if (st != HS_OK) return st;
  if (!w || n_layers < 1) return hs::fail(HS_ERR_INVALID_ARG, "weights missing or n_layers %d < 1", n_layers);
  for (int l = 0; l < n_layers; ++l) {
    if (!w[l].ln1 || !w[l].w_qkv || !w[l].w_o || !w[l].ln2 || !w[l].w_gate_up || !w[l].w_down)
      return hs::fail(HS_ERR_INVALID_ARG, "layer %d has a null weight pointer", l);
    if (w[l].format != HS_WEIGHTS_BF16 && w[l].format != HS_WEIGHTS_F16)
      return hs::fail(HS_ERR_INVALID_ARG, "layer %d has weight format %d", l, w[l].format);
  }
  if (!x_in || !x_out) return hs::fail(HS_ERR_INVALID_ARG, "x_in / x_out is null");
  if (x_in == x_out) return hs::fail(HS_ERR_INVALID_ARG, "x_in and x_out must not alias");
  if (batch < 1) return hs::fail(HS_ERR_INVALID_ARG, "batch %d < 1", batch);
  if (!kv || !kv->k || !kv->v) return hs::fail(HS_ERR_INVALID_ARG, "decode needs a key/value cache");
  for (int l = 0; l < n_layers; ++l)
    if (!kv->k[l] || !kv->v[l]) return hs::fail(HS_ERR_INVALID_ARG, "cache of layer %d is null", l);
  if (kv->max_ctx < 64 || kv->max_ctx % 64 != 0)
    return hs::fail(HS_ERR_INVALID_ARG, "max_ctx %d must be a positive multiple of 64", kv->max_ctx);
  if (kv->n_slots < 1) return hs::fail(HS_ERR_INVALID_ARG, "the cache has %d slots", kv->n_slots);
  const bool paged = kv->block_table != nullptr;
  if (paged && kv->pages_per_seq < 1)
    return hs::fail(HS_ERR_INVALID_ARG, "pages_per_seq %d must be >= 1", kv->pages_per_seq);
  if (!paged && batch > kv->n_slots)
    return hs::fail(HS_ERR_INVALID_ARG, "batch %d but only %d cache slots", batch, kv->n_slots);
  st = hs::check_32bit_extents(*cfg, batch, kv->max_ctx);
  if (st != HS_OK) return st;
  hs::PlanCapacity cap;
  cap.page_keys = paged ? kv->max_ctx : 0;
  const int64_t max_pos = paged ? int64_t(kv->pages_per_seq) * kv->max_ctx : int64_t(kv->max_ctx);
  if (max_pos > (int64_t(1) << 30)) return hs::fail(HS_ERR_UNSUPPORTED, "%lld positions per sequence", (long long)max_pos);
  cap.max_pos = int32_t(max_pos);
  hipStream_t s = nullptr;
  st = resolve_stream(ctx, cu_budget, HS_ROLE_DOWN, stream, &s);
  if (st != HS_OK) return st;
  if (!workspace) return hs::fail(HS_ERR_WORKSPACE, "workspace is null");
  const hs::WsLayout lay = hs::ws_layout(*cfg, batch, batch, cap.max_pos, cap.page_keys, false);
  if (ws_bytes < lay.total) return hs::fail(HS_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, lay.total);

  // The launches are captured from a plan of empty caches in the fixed
  // layout: its offsets, and so every kernel argument, are those of any
  // later call; the contents are staged per launch.
  std::vector<int32_t> off(batch + 1), zero(batch, 0), table;
  for (int32_t b = 0; b <= batch; ++b) off[b] = b;
  hs::KvPlacement place;
  place.cache = true;
  place.max_ctx = kv->max_ctx;
  if (paged) {
    table.assign(size_t(batch) * kv->pages_per_seq, 0);
    place.table = table.data();
    place.pages_per_seq = kv->pages_per_seq;
  }
  hs::Plan plan;
  st = hs::build_plan(*cfg, off.data(), zero.data(), batch, place, &plan, nullptr, &cap);
  if (st != HS_OK) return st;
  if (plan.image.size() > lay.meta_bytes) return hs::fail(HS_ERR_INTERNAL, "metadata image exceeds its region");

  hs_decode_graph* g = new hs_decode_graph();
  g->ctx = ctx;
  g->cfg = *cfg;
  g->w.assign(w, w + n_layers);
  g->k.assign(kv->k, kv->k + n_layers);
  g->v.assign(kv->v, kv->v + n_layers);
  g->kv = *kv;
  g->kv.k = g->k.data();
  g->kv.v = g->v.data();
  g->kv.block_table = nullptr;
  g->n_layers = n_layers;
  g->batch = batch;
  g->budget = cu_budget;
  g->x_in = x_in;
  g->x_out = x_out;
  g->ws = workspace;
  g->lay = lay;
  g->cap = cap;
  g->paged = paged;
  g->image_bytes = plan.image.size();
  g->stream = s;

  auto fail_hip = [&](const char* what, hipError_t e) {
    delete g;
    return hs::fail(HS_ERR_HIP, "%s failed: %s", what, hipGetErrorString(e));
  };
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return fail_hip("hipSetDevice", e);
  (void)hipGetLastError();
  // The RoPE table for every position the layout holds, once, on the stream.
  e = hs::launch_rope_table(at<float2>(workspace, lay.rope), cap.max_pos, cfg->head_dim, cfg->rope_base, s);
  if (e != hipSuccess) return fail_hip("the RoPE table launch", e);
  const bool timing = ctx->timing;
  ctx->timing = false;  // no event records inside the capture
  e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    ctx->timing = timing;
    return fail_hip("hipStreamBeginCapture", e);
  }
  LaunchSet L{&g->cfg, g->w.data(), n_layers, x_in, x_out, &g->kv, true, workspace, lay, &plan, cu_budget, false, true};
  st = launch_layers(ctx, L, s);
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(s, &graph);
  ctx->timing = timing;
  if (st != HS_OK) {
    if (graph) hipGraphDestroy(graph);
    delete g;
    return st;
  }
  if (e != hipSuccess) {
    if (graph) hipGraphDestroy(graph);
    return fail_hip("hipStreamEndCapture", e);
  }
  e = hipGraphInstantiate(&g->exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (e != hipSuccess) return fail_hip("hipGraphInstantiate", e);
  *out = g;
  return HS_OK;
}

hs_status hs_decode_graph_launch(hs_decode_graph* g, const int32_t* kv_lens, const int32_t* block_table) {
  hs::clear_error();
  if (!g) return hs::fail(HS_ERR_INVALID_ARG, "graph is null");
  if (!kv_lens) return hs::fail(HS_ERR_INVALID_ARG, "kv_lens is null");
  if (g->paged != (block_table != nullptr))
    return hs::fail(HS_ERR_INVALID_ARG, g->paged ? "the graph was captured for a paged cache: block_table is required"
                                                 : "the graph was captured for cache slots: block_table must be null");
  std::vector<int32_t> off(g->batch + 1);
  for (int32_t b = 0; b <= g->batch; ++b) off[b] = b;
  for (int32_t b = 0; b < g->batch; ++b)
    if (kv_lens[b] < 0 || int64_t(kv_lens[b]) + 1 > g->cap.max_pos)
      return hs::fail(HS_ERR_INVALID_ARG, "kv_lens[%d] = %d: the new row must sit below position %d", b, kv_lens[b],
                      g->cap.max_pos);
  hs::KvPlacement place;
  place.cache = true;
  place.max_ctx = g->kv.max_ctx;
  if (g->paged) {
    hs_status st = hs::check_block_table(block_table, g->kv.pages_per_seq, g->kv.n_slots, g->kv.max_ctx,
                                         off.data(), kv_lens, g->batch);
    if (st != HS_OK) return st;
    place.table = block_table;
    place.pages_per_seq = g->kv.pages_per_seq;
  }
  hs::Plan plan;
  hs_status st = hs::build_plan(g->cfg, off.data(), kv_lens, g->batch, place, &plan, nullptr, &g->cap);
  if (st != HS_OK) return st;
  if (plan.image.size() != g->image_bytes) return hs::fail(HS_ERR_INTERNAL, "metadata layout changed since capture");
  hs_context* ctx = g->ctx;
  HIP_TRY(hipSetDevice(ctx->device));
  (void)hipGetLastError();
  st = stage_metadata(ctx, plan, at<void>(g->ws, g->lay.meta), g->stream);
  if (st != HS_OK) return st;
  HIP_TRY(hipGraphLaunch(g->exec, g->stream));
  return HS_OK;
}

hs_status hs_decode_graph_destroy(hs_decode_graph* g) {
  hs::clear_error();
  if (!g) return HS_OK;
  if (g->exec) {
    hipSetDevice(g->ctx->device);
    hipStreamSynchronize(g->stream);
    hipGraphExecDestroy(g->exec);
  }
  delete g;
  return HS_OK;
}

}  // extern "C"

namespace {

hs_status validate_dit_cfg(const hs_dit_cfg* c) {
  if (!c) return hs::fail(HS_ERR_INVALID_ARG, "DiT config is null");
  if (c->hidden <= 0 || c->hidden % 256 != 0 || c->hidden > 8192)
    return hs::fail(HS_ERR_UNSUPPORTED, "hidden %d must be a positive multiple of 256, at most 8192", c->hidden);
  if (c->head_dim != 64 && c->head_dim != 128)
    return hs::fail(HS_ERR_UNSUPPORTED, "head_dim %d must be 64 or 128", c->head_dim);
  if (c->n_heads <= 0 || c->n_heads * c->head_dim != c->hidden)
    return hs::fail(HS_ERR_INVALID_ARG, "n_heads %d * head_dim %d must equal hidden %d", c->n_heads, c->head_dim,
                    c->hidden);
  if (c->mlp <= 0 || c->mlp % 256 != 0)
    return hs::fail(HS_ERR_UNSUPPORTED, "mlp %d must be a positive multiple of 256", c->mlp);
  if (!(c->ln_eps > 0.0f)) return hs::fail(HS_ERR_INVALID_ARG, "ln_eps must be > 0");
  return HS_OK;
}

// The decoder-layer shape the shared buffers and checks are sized by: the
// MLP width in the FFN's place, Hq = Hkv.
hs_layer_cfg dit_as_layer(const hs_dit_cfg& c) {
  hs_layer_cfg l{};
  l.hidden = c.hidden;
  l.n_q_heads = c.n_heads;
  l.n_kv_heads = c.n_heads;
  l.head_dim = c.head_dim;
  l.ffn = c.mlp;
  l.rms_eps = c.ln_eps;
  l.rope_base = 10000.0f;
  return l;
}

struct DitLayout {
  hs::WsLayout base;
  size_t silu, mod, total;
};

DitLayout dit_layout(const hs_dit_cfg& c, int32_t T, int32_t B, int32_t max_pos) {
  DitLayout L;
  L.base = hs::ws_layout(dit_as_layer(c), T, B, max_pos, 0, true);
  L.silu = hs::align_up(L.base.total, hs::kAlign);
  L.mod = hs::align_up(L.silu + size_t(B) * c.hidden * 4, hs::kAlign);
  // The modulation of up to kDitModLayers layers, computed in one launch.
  L.total = hs::align_up(L.mod + size_t(hs::kDitModLayers) * B * 6 * c.hidden * 4, hs::kAlign);
  return L;
}

}  // namespace

extern "C" {

hs_status hs_dit_workspace_size(const hs_dit_cfg* cfg, int32_t max_tokens, int32_t max_seqs, size_t* bytes) {
  hs::clear_error();
  hs_status st = validate_dit_cfg(cfg);
  if (st != HS_OK) return st;
  if (!bytes) return hs::fail(HS_ERR_INVALID_ARG, "bytes output is null");
  if (max_tokens < 0 || max_seqs < 1) return hs::fail(HS_ERR_INVALID_ARG, "max_tokens %d, max_seqs %d", max_tokens,
                                                      max_seqs);
  *bytes = dit_layout(*cfg, max_tokens, max_seqs, std::max(max_tokens, 1)).total;
  return HS_OK;
}

hs_status hs_dit_forward(hs_context* ctx, const hs_dit_cfg* cfg, const hs_dit_weights* w, int32_t n_layers,
                         const void* x_in, void* x_out, const float* cond, const int32_t* seq_offsets,
                         int32_t n_seqs, int32_t cu_budget, void* stream, void* workspace, size_t ws_bytes) {
  hs::clear_error();
  hs_status st = validate_dit_cfg(cfg);
  if (st != HS_OK) return st;
  if (!w || n_layers < 1) return hs::fail(HS_ERR_INVALID_ARG, "weights missing or n_layers %d < 1", n_layers);
  for (int l = 0; l < n_layers; ++l) {
    const hs_dit_weights& lw = w[l];
    if (!lw.w_ada || !lw.b_ada || !lw.w_qkv || !lw.b_qkv || !lw.w_o || !lw.b_o || !lw.w_fc1 || !lw.b_fc1 ||
        !lw.w_fc2 || !lw.b_fc2)
      return hs::fail(HS_ERR_INVALID_ARG, "block %d has a null weight pointer", l);
    if (lw.format != HS_WEIGHTS_BF16 && lw.format != HS_WEIGHTS_F16)
      return hs::fail(HS_ERR_INVALID_ARG, "block %d has weight format %d", l, lw.format);
  }
  if (!x_in || !x_out || !cond) return hs::fail(HS_ERR_INVALID_ARG, "x_in / x_out / cond is null");
  if (x_in == x_out) return hs::fail(HS_ERR_INVALID_ARG, "x_in and x_out must not alias");
  int32_t T = 0, max_pos = 0;
  st = hs::validate_batch(seq_offsets, nullptr, n_seqs, &T, &max_pos);
  if (st != HS_OK) return st;
  const hs_layer_cfg lcfg = dit_as_layer(*cfg);
  st = hs::check_32bit_extents(lcfg, T, 0);
  if (st != HS_OK) return st;
  if (int64_t(6) * cfg->hidden * cfg->hidden * 2 >= (int64_t(1) << 32))
    return hs::fail(HS_ERR_UNSUPPORTED, "w_ada of %d x %d exceeds 2^32 bytes", 6 * cfg->hidden, cfg->hidden);
  if (!ctx) return hs::fail(HS_ERR_INVALID_ARG, "context is null");
  hipStream_t s = nullptr;
  st = resolve_stream(ctx, cu_budget, HS_ROLE_DOWN, stream, &s);
  if (st != HS_OK) return st;
  if (!workspace) return hs::fail(HS_ERR_WORKSPACE, "workspace is null");
  const DitLayout DL = dit_layout(*cfg, T, n_seqs, std::max(max_pos, 1));
  if (ws_bytes < DL.total) return hs::fail(HS_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, DL.total);
  const hs::WsLayout& lay = DL.base;
  hs::KvPlacement place;
  place.packed_ctx = lay.packed_ctx;
  hs::Plan plan;
  st = hs::build_plan(lcfg, seq_offsets, nullptr, n_seqs, place, &plan, nullptr, nullptr, true);
  if (st != HS_OK) return st;
  if (plan.image.size() > lay.meta_bytes) return hs::fail(HS_ERR_INTERNAL, "metadata image exceeds its region");

  HIP_TRY(hipSetDevice(ctx->device));
  (void)hipGetLastError();
  st = stage_metadata(ctx, plan, at<void>(workspace, lay.meta), s);
  if (st != HS_OK) return st;
  if (T == 0) return HS_OK;

  const int d = cfg->hidden, H = cfg->n_heads, dh = cfg->head_dim, mlp = cfg->mlp;
  void* ws = workspace;
  uint8_t* meta = at<uint8_t>(ws, lay.meta);
  const int32_t* row_seq = reinterpret_cast<const int32_t*>(meta + plan.row_seq);
  uint16_t* n_buf = at<uint16_t>(ws, lay.n);
  uint16_t* q_buf = at<uint16_t>(ws, lay.q);
  uint16_t* o_buf = at<uint16_t>(ws, lay.o);
  float* h_buf = at<float>(ws, lay.h);
  uint16_t* a_buf = at<uint16_t>(ws, lay.a);
  float* xtmp = at<float>(ws, lay.xtmp);
  float* s_buf = at<float>(ws, DL.silu);
  float* mod_all = at<float>(ws, DL.mod);
  uint16_t* kstore = at<uint16_t>(ws, lay.kpack);
  uint16_t* vstore = at<uint16_t>(ws, lay.vpack);
  const int grid_cap = cu_budget;
  const float scale_log2 = 1.4426950408889634f / sqrtf(float(dh));

  TIMED(HS_KERNEL_MODULATION, hs::launch_silu_rows(cond, s_buf, n_seqs * d, s));
  const uint16_t* x_cur = static_cast<const uint16_t*>(x_in);
  const float* x_cur_f32 = nullptr;
  for (int l = 0; l < n_layers; ++l) {
    const int remaining = n_layers - 1 - l;
    float* x_next = (remaining % 2 == 0) ? static_cast<float*>(x_out) : xtmp;
    const bool f16 = w[l].format == HS_WEIGHTS_F16;
    if (l % hs::kDitModLayers == 0) {
      // Every block's modulation depends on the conditioning only: up to
      // kDitModLayers layers' at once, one slot of B x 6d floats per layer.
      hs::DitModArgs mp{};
      mp.n_layers = std::min(hs::kDitModLayers, n_layers - l);
      for (int i = 0; i < mp.n_layers; ++i) {
        mp.w[i] = static_cast<const uint16_t*>(w[l + i].w_ada);
        mp.bias[i] = static_cast<const uint16_t*>(w[l + i].b_ada);
      }
      TIMED(HS_KERNEL_MODULATION, hs::launch_dit_modulation(mp, s_buf, mod_all, n_seqs, d, s));
    }
    float* const mod = mod_all + size_t(l % hs::kDitModLayers) * n_seqs * 6 * d;
    TIMED(HS_KERNEL_LN_MOD, hs::launch_ln_modulate(x_cur, x_cur_f32, mod, row_seq, n_buf, T, d, cfg->ln_eps, 0, d,
                                                   4 * cu_budget, s));
    hs::GemmArgs g{};
    g.A = n_buf;
    g.W = static_cast<const uint16_t*>(w[l].w_qkv);
    g.w_f16 = f16;
    g.M = T;
    g.K = d;
    g.n_tiles_n = 3 * d / 256;
    g.q = q_buf;
    g.kstore = kstore;
    g.vstore = vstore;
    g.pos = reinterpret_cast<const int32_t*>(meta + plan.pos);
    g.sec1 = g.sec2 = dh / 2;
    g.k_off = reinterpret_cast<const int64_t*>(meta + plan.k_off);
    g.v_off = reinterpret_cast<const int64_t*>(meta + plan.v_off);
    g.kv_head_stride = plan.kv_head_stride;
    g.rope = nullptr;  // positions enter with the token embeddings
    g.bias = static_cast<const uint16_t*>(w[l].b_qkv);
    g.hq = H;
    g.hkv = H;
    g.dh = dh;
    g.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_QKV, hs::launch_gemm(hs::EPI_QKV, g, grid_cap, s));

    hs::AttnArgs at_args{};
    at_args.q = q_buf;
    at_args.kstore = kstore;
    at_args.vstore = vstore;
    at_args.o = o_buf;
    at_args.items = reinterpret_cast<const int32_t*>(meta + plan.att_items);
    at_args.n_items = plan.n_att_items;
    at_args.seq_start = reinterpret_cast<const int32_t*>(meta + plan.seq_start);
    at_args.seq_len = reinterpret_cast<const int32_t*>(meta + plan.seq_len);
    at_args.seq_ctx = reinterpret_cast<const int32_t*>(meta + plan.seq_ctx);
    at_args.seq_page0 = reinterpret_cast<const int32_t*>(meta + plan.seq_page0);
    at_args.page_base = reinterpret_cast<const int64_t*>(meta + plan.page_base);
    at_args.page_keys = plan.page_keys;
    at_args.kv_head_stride = plan.kv_head_stride;
    at_args.hq = H;
    at_args.hkv = H;
    at_args.dh = dh;
    at_args.scale_log2 = scale_log2;
    at_args.bidirectional = 1;
    at_args.clock = clock_slot(ctx);
    if (plan.n_att_items > 0) TIMED(HS_KERNEL_ATTENTION, hs::launch_attention(at_args, s));
    if (plan.n_dec_rows > 0) {
      // One-row sequences: attention over the row itself.
      hs::DecodeAttnArgs da{};
      da.q = q_buf;
      da.kstore = kstore;
      da.vstore = vstore;
      da.o = o_buf;
      da.items = reinterpret_cast<const hs::DecItem*>(meta + plan.dec_items);
      da.n_items = plan.n_dec_items;
      da.part = lay.dec_part_bytes ? at<float>(ws, lay.dec_part) : nullptr;
      da.counters = reinterpret_cast<int32_t*>(meta + plan.dec_count);
      da.kv_head_stride = plan.kv_head_stride;
      da.page_keys = plan.page_keys;
      da.unit_keys = plan.unit_keys;
      da.hq = H;
      da.hkv = H;
      da.dh = dh;
      da.scale_log2 = scale_log2;
      TIMED(HS_KERNEL_DECODE_ATTN, hs::launch_decode_attention(da, s));
    }

    hs::GemmArgs go{};
    go.A = o_buf;
    go.W = static_cast<const uint16_t*>(w[l].w_o);
    go.w_f16 = f16;
    go.M = T;
    go.K = d;
    go.n_tiles_n = d / 256;
    go.out_f32 = h_buf;
    go.ldo = d;
    go.resid = x_cur;
    go.resid_f32 = x_cur_f32;
    go.bias = static_cast<const uint16_t*>(w[l].b_o);
    go.gate = mod + 2 * d;
    go.gate_stride = 6 * d;
    go.row_seq = row_seq;
    go.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_O_PROJ, hs::launch_gemm(hs::EPI_GATED, go, grid_cap, s));

    TIMED(HS_KERNEL_LN_MOD, hs::launch_ln_modulate(nullptr, h_buf, mod, row_seq, n_buf, T, d, cfg->ln_eps, 3 * d,
                                                   4 * d, 4 * cu_budget, s));
    hs::GemmArgs g1{};
    g1.A = n_buf;
    g1.W = static_cast<const uint16_t*>(w[l].w_fc1);
    g1.w_f16 = f16;
    g1.M = T;
    g1.K = d;
    g1.n_tiles_n = mlp / 256;
    g1.out = a_buf;
    g1.ldo = mlp;
    g1.bias = static_cast<const uint16_t*>(w[l].b_fc1);
    g1.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_MLP_UP, hs::launch_gemm(hs::EPI_GELU, g1, grid_cap, s));

    hs::GemmArgs g2{};
    g2.A = a_buf;
    g2.W = static_cast<const uint16_t*>(w[l].w_fc2);
    g2.w_f16 = f16;
    g2.M = T;
    g2.K = mlp;
    g2.n_tiles_n = d / 256;
    g2.out_f32 = x_next;
    g2.ldo = d;
    g2.resid_f32 = h_buf;
    g2.bias = static_cast<const uint16_t*>(w[l].b_fc2);
    g2.gate = mod + 5 * d;
    g2.gate_stride = 6 * d;
    g2.row_seq = row_seq;
    g2.clock = clock_slot(ctx);
    TIMED(HS_KERNEL_MLP_DOWN, hs::launch_gemm(hs::EPI_GATED, g2, grid_cap, s));
    x_cur = nullptr;
    x_cur_f32 = x_next;
  }
  return HS_OK;
}

hs_status hs_downstream_decode_step_mrope(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                          int32_t n_layers, const void* x_in, void* x_out, const hs_kv_cache* kv,
                                          const int32_t* kv_lens, const int32_t* positions3, int32_t batch,
                                          int32_t cu_budget, void* stream, void* workspace, size_t ws_bytes) {
  hs::clear_error();
  if (!positions3) return hs::fail(HS_ERR_INVALID_ARG, "positions3 is null");
  if (!kv) return hs::fail(HS_ERR_INVALID_ARG, "decode needs a key/value cache");
  if (!kv_lens) return hs::fail(HS_ERR_INVALID_ARG, "kv_lens is null");
  if (batch < 1) return hs::fail(HS_ERR_INVALID_ARG, "batch %d < 1", batch);
  std::vector<int32_t> off(batch + 1);
  for (int32_t b = 0; b <= batch; ++b) off[b] = b;
  return run_stack(ctx, cfg, w, n_layers, x_in, x_out, off.data(), kv_lens, batch, kv, cu_budget, HS_ROLE_DOWN,
                   stream, workspace, ws_bytes, positions3);
}

hs_status hs_convert_weights_f16(hs_context* ctx, const void* src, void* dst, int64_t rows, int64_t cols,
                                 void* stream) {
  hs::clear_error();
  if (!ctx || !src || !dst) return hs::fail(HS_ERR_INVALID_ARG, "null argument");
  if (rows < 1 || cols < 32 || cols % 32 != 0)
    return hs::fail(HS_ERR_INVALID_ARG, "shape [%lld, %lld]: need rows >= 1 and cols a positive multiple of 32",
                    (long long)rows, (long long)cols);
  if ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 4 != 0)
    return hs::fail(HS_ERR_INVALID_ARG, "pointers must be 4-byte aligned");
  const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
  const uintptr_t bytes = uintptr_t(rows) * uintptr_t(cols) * 2;
  if (s0 < d0 + bytes && d0 < s0 + bytes) return hs::fail(HS_ERR_INVALID_ARG, "source and destination overlap");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (!s) s = find_level(ctx, ctx->n_cus)->s_shared;
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(hs::launch_convert_bf16_f16(static_cast<const uint16_t*>(src), static_cast<uint16_t*>(dst), rows, cols, s));
  return HS_OK;
}

hs_status hs_timing_enable(hs_context* ctx, int32_t enable) {
  hs::clear_error();
  if (!ctx) return hs::fail(HS_ERR_INVALID_ARG, "null context");
  HIP_TRY(hipSetDevice(ctx->device));
  if (enable && ctx->ev_pool.empty()) {
    ctx->ev_pool.reserve(2 * kTimingPairs);
    for (size_t i = 0; i < 2 * kTimingPairs; ++i) {
      hipEvent_t e;
      HIP_TRY(hipEventCreate(&e));
      ctx->ev_pool.push_back(e);
    }
  }
  if (enable && !ctx->clock_buf) HIP_TRY(hipMalloc(&ctx->clock_buf, kTimingPairs * 4 * sizeof(uint64_t)));
  // Finish outstanding records before their events can be recorded again.
  for (const auto& r : ctx->recs) HIP_TRY(hipEventSynchronize(r.b));
  ctx->recs.clear();
  ctx->ev_next = 0;
  if (enable) HIP_TRY(hipMemset(ctx->clock_buf, 0, kTimingPairs * 4 * sizeof(uint64_t)));
  ctx->timing = enable != 0;
  return HS_OK;
}

hs_status hs_timing_read_clock(hs_context* ctx, int32_t kind, double* mhz, int32_t* n_launches) {
  hs::clear_error();
  if (!ctx || !mhz || !n_launches) return hs::fail(HS_ERR_INVALID_ARG, "null argument");
  if (kind < 0 || kind >= HS_KERNEL_KINDS) return hs::fail(HS_ERR_INVALID_ARG, "kernel kind %d", kind);
  *mhz = 0.0;
  *n_launches = 0;
  if (!ctx->clock_buf || ctx->recs.empty()) return HS_OK;
  HIP_TRY(hipSetDevice(ctx->device));
  for (const auto& r : ctx->recs) HIP_TRY(hipEventSynchronize(r.b));
  std::vector<uint64_t> c(4 * ctx->recs.size());
  HIP_TRY(hipMemcpy(c.data(), ctx->clock_buf, c.size() * sizeof(uint64_t), hipMemcpyDeviceToHost));
  int wall_khz = 0;
  HIP_TRY(hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, ctx->device));
  double cycles = 0.0, ticks = 0.0;
  int32_t n = 0;
  for (size_t i = 0; i < ctx->recs.size(); ++i) {
    const uint64_t* v = &c[4 * i];
    if (ctx->recs[i].kind != kind || v[3] <= v[1] || v[2] <= v[0]) continue;
    cycles += double(v[2] - v[0]);
    ticks += double(v[3] - v[1]);
    ++n;
  }
  if (n && ticks > 0.0) *mhz = cycles / ticks * (double(wall_khz) / 1e3);
  *n_launches = n;
  return HS_OK;
}

hs_status hs_timing_read(hs_context* ctx, int32_t kind, double* total_ms, int32_t* n_launches) {
  hs::clear_error();
  if (!ctx || !total_ms || !n_launches) return hs::fail(HS_ERR_INVALID_ARG, "null argument");
  if (kind < 0 || kind >= HS_KERNEL_KINDS) return hs::fail(HS_ERR_INVALID_ARG, "kernel kind %d", kind);
  double total = 0.0;
  int32_t n = 0;
  for (const auto& r : ctx->recs) {
    if (r.kind != kind) continue;
    HIP_TRY(hipEventSynchronize(r.b));
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, r.a, r.b));
    total += ms;
    ++n;
  }
  *total_ms = total;
  *n_launches = n;
  return HS_OK;
}

hs_status hs_probe_hw_ids(hs_context* ctx, void* stream, int32_t n_groups, void* out_ids) {
  hs::clear_error();
  if (!ctx || !out_ids || n_groups < 1) return hs::fail(HS_ERR_INVALID_ARG, "bad probe arguments");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (!s) {
    const Level* l = find_level(ctx, ctx->n_cus);
    s = l->s_shared;
  }
  HIP_TRY(hipSetDevice(ctx->device));
  HIP_TRY(hs::launch_probe(static_cast<uint32_t*>(out_ids), n_groups, s));
  return HS_OK;
}

}  // extern "C"
