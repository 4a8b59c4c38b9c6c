/*
 * horizon.h - C ABI of the MI355X (gfx950) shared-stage hot path.
 *
 * The library runs the shared multimodal stage ("thinker") of an omni model:
 * a stack of pre-norm decoder layers over a packed ragged batch of prefill
 * rows, on an explicit budget of compute units, while a downstream decode
 * stage ("talker") runs on the complementary compute units of the same GPU.
 *
 * Paper passages this interface follows (HorizonServe):
 *   - §2.1 "Autoregressive transformers": prefill processes the context and
 *     builds the key/value cache; decode re-reads the weights and the cache.
 *   - §4.4 "Complementary downstream headroom" and Algorithm 1, step 3: the
 *     downstream stage gets s_down = S_tot - s_shared.
 *   - §4.5 Algorithm 1, step 4: the selected batch runs with cap s_shared.
 *   - §5: one pre-built allocation per ladder level, selected (not created)
 *     before each forward pass; the two stages' ladders are complementary.
 *
 * Conventions for every entry point:
 *   - Device pointers are HIP device addresses; "host" arrays are ordinary
 *     host memory that the call reads before it returns (the caller may
 *     reuse them at once).  Streams are hipStream_t passed as void*.
 *   - bf16 means IEEE bfloat16 and fp16 IEEE binary16, stored as 16-bit words.
 *   - Precision: token rows and weights are bf16 in memory; every contraction
 *     runs on fp16 MFMA operands with fp32 accumulation (weights are converted
 *     bf16 -> fp16 on load, exact for magnitudes in [2^-14, 65504]); the
 *     residual stream is fp32; intermediate activations and the key/value
 *     cache are fp16 (finite values saturate at +-65504).
 *   - Weight matrices are [out, in] row-major, so y = x * W^T.
 *   - Every function returns an hs_status.  No C++ exception crosses the
 *     ABI.  On any error other than HS_ERR_HIP nothing has been enqueued.
 *     hs_last_error() returns a thread-local message for the last failure.
 *   - Compute calls are asynchronous with respect to their stream; device
 *     faults surface at the caller's next synchronisation.
 *   - A context is not thread-safe; use one per host thread.
 */
#ifndef HORIZON_H_
#define HORIZON_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hs_status {
  HS_OK = 0,
  HS_ERR_INVALID_ARG = 1, /* null pointer, bad shape, bad offsets, aliasing */
  HS_ERR_UNSUPPORTED = 2, /* valid request outside what the kernels implement */
  HS_ERR_BUDGET = 3,      /* CU budget outside [1, n_cus] or not matching the stream */
  HS_ERR_WORKSPACE = 4,   /* workspace missing or smaller than hs_workspace_size() */
  HS_ERR_HIP = 5,         /* a HIP runtime call failed; see hs_last_error() */
  HS_ERR_INTERNAL = 6
} hs_status;

/* Shape of one decoder layer (all layers of a stack share it).
 * Requirements: hidden % 256 == 0, head_dim in {64, 128},
 * n_q_heads % n_kv_heads == 0, (n_q_heads + 2 n_kv_heads) * head_dim % 256 == 0,
 * n_q_heads * head_dim % 128 == 0, ffn % 128 == 0. */
typedef struct hs_layer_cfg {
  int32_t hidden;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t ffn;
  float rms_eps;   /* RMSNorm epsilon, inside the square root */
  float rope_base; /* RoPE base; pair (j, j + dh/2) turns by pos * base^(-2j/dh) */
  /* Multimodal RoPE: rotary pairs j < dh/2 split into temporal, height and
   * width sections of these many pairs (in that order); pair j turns by the
   * position component of its section.  All zero: one position per row (the
   * plain RoPE above).  Otherwise each is a multiple of 4 and they sum to
   * dh/2.  The paper does not define the multimodal positions; this is the
   * sectioned form models of the Qwen2-VL family use for image and video
   * rows. */
  int32_t mrope_sections[3];
} hs_layer_cfg;

/* Storage format of the four projection matrices of a layer. */
enum { HS_WEIGHTS_BF16 = 0, HS_WEIGHTS_F16 = 1 };

/* Device pointers to one layer's weights.
 *   ln1, ln2   [hidden] bf16                         RMSNorm gains
 *   w_qkv      [(Hq + 2 Hkv) * dh, hidden]           rows: Q heads | K heads | V heads
 *   b_qkv      [(Hq + 2 Hkv) * dh] bf16, or NULL     bias of the QKV projection, added
 *                                                    before RoPE (same row order)
 *   w_o        [hidden, Hq * dh]
 *   w_gate_up  [2 * ffn, hidden]                      rows: gate | up
 *   w_down     [hidden, ffn]
 * format: HS_WEIGHTS_BF16 (the matrices are bf16 row-major as above and each
 * GEMM converts its tiles on the fly) or HS_WEIGHTS_F16 (the matrices were
 * prepared once with hs_convert_weights_f16: same values as fp16 in
 * panel-major order, no per-call conversion; the fastest format). */
typedef struct hs_layer_weights {
  const void* ln1;
  const void* w_qkv;
  const void* w_o;
  const void* ln2;
  const void* w_gate_up;
  const void* w_down;
  int32_t format;
  const void* b_qkv;
} hs_layer_weights;

/* Key/value cache (§2.1: prefill builds it, decode re-reads it).  k[l] and
 * v[l] are device pointers for layer l (host arrays of n_layers pointers,
 * owned by the caller).  The cache of a layer is a pool of n_slots slots of
 * max_ctx positions each:
 *   K: fp16 [n_slots, Hkv, max_ctx, dh]            (the key rows of one head
 *      are contiguous)
 *   V: fp16 [n_slots, Hkv, max_ctx / 32, dh, 32]   (values transposed in
 *      tiles of 32 positions: the P.V contraction reads keys contiguously and
 *      a tile of one head is one contiguous block)
 * max_ctx % 64 == 0.
 *
 * block_table NULL: sequence b of a call uses slot b; its positions are
 *   < max_ctx.
 * block_table non-NULL (paged cache): a slot is a page of max_ctx positions.
 *   block_table is a host array [n_seqs][pages_per_seq] of slot indices;
 *   position p of sequence b lives in slot block_table[b * pages_per_seq +
 *   p / max_ctx] at position p % max_ctx.  Positions are
 *   < pages_per_seq * max_ctx.  Entries for pages a sequence does not reach
 *   are not read.  Sequences may share pages they only read (a common
 *   prefix); a page that receives new rows in a call must belong to one
 *   sequence only and appear once in its row of the table, else the call
 *   fails with HS_ERR_INVALID_ARG.  Single-row attention splits its key range
 *   at page boundaries, so pages of 512 (head_dim 128) or 1024 (head_dim 64)
 *   positions or a multiple keep its work units whole; the workspace comes
 *   from hs_workspace_size_paged. */
typedef struct hs_kv_cache {
  void* const* k;
  void* const* v;
  int32_t n_slots;
  int32_t max_ctx;
  const int32_t* block_table;
  int32_t pages_per_seq;
} hs_kv_cache;

/* Per mask bit i (bit i%32 of word i/32): hardware XCD, shader engine and CU
 * index inside that shader engine. */
typedef struct hs_topology {
  int32_t n_cus;
  int32_t n_xcc;
  uint8_t xcc[256];
  uint8_t se[256];
  uint8_t cu[256];
} hs_topology;

typedef struct hs_context hs_context;
typedef struct hs_decode_graph hs_decode_graph;

enum { HS_ROLE_SHARED = 0, HS_ROLE_DOWN = 1 };

/* Human-readable name of a status code (static storage). */
const char* hs_status_string(hs_status s);

/* Message of the last failing call on this host thread ("" if none). */
const char* hs_last_error(void);

/* Default topology of an n_cus / n_xcc part with 4 shader engines per XCD:
 * bit i -> XCD i % n_xcc, slot j = i / n_xcc -> (se j % 4, cu j / 4).
 * Host only. */
hs_status hs_default_topology(int32_t n_cus, int32_t n_xcc, hs_topology* out);

/* Complementary CU partition (§4.4 complementary headroom; §5 complementary
 * ladders).  Pure host function of (topology, budget):
 *   XCD x receives floor(c / n_xcc) + (x < c % n_xcc) shared CUs, taken from
 *   that XCD's mask bits ordered by (cu, se, bit); every other bit is down.
 * shared_mask and down_mask are 8 words each (256 bits), written by the call.
 * Errors: HS_ERR_BUDGET for c outside [1, n_cus]; HS_ERR_INVALID_ARG for null
 * pointers or a topology with more than 256 CUs or an XCD too small. */
hs_status hs_cu_partition(const hs_topology* topo, int32_t shared_cus, uint32_t shared_mask[8],
                          uint32_t down_mask[8]);

/* Packed-batch metadata (Algorithm 1, step 4: batch B).  Host only.
 * seq_offsets[n_seqs + 1] (host) must start at 0 and be non-decreasing;
 * ctx_lens[n_seqs] (host, may be NULL = all 0) must be >= 0.  Writes
 * pos_out[T] = ctx_lens[b] + (t - seq_offsets[b]) and seq_id_out[T] = b for
 * every packed row t, T = seq_offsets[n_seqs]. */
hs_status hs_plan_metadata(const int32_t* seq_offsets, const int32_t* ctx_lens, int32_t n_seqs,
                           int32_t* pos_out, int32_t* seq_id_out);

/* Create a context on HIP device `device` with a ladder of CU-masked stream
 * pairs, one pair per budget in budgets[n_budgets] (each in [1, n_cus]).
 * Budget n_cus has a SHARED stream only.  topo may be NULL (default
 * topology); the masks are hs_cu_partition(topo, budget).  The context owns
 * its streams and a pool of pinned staging slots for the calls' metadata (4,
 * growing to at most 64 while calls queued on several streams are pending, so
 * that a call never waits for another stream's queued work).  Each stream
 * is a hardware queue of its own (2 per level, 1 at n_cus). */
hs_status hs_context_create(int32_t device, const int32_t* budgets, int32_t n_budgets,
                            const hs_topology* topo, hs_context** out);

/* Topology the context's masks were built from. */
hs_status hs_context_topology(const hs_context* ctx, hs_topology* out);

/* Pre-built stream of the ladder for (budget, role).  HS_ERR_BUDGET if the
 * budget is not on the ladder or role is DOWN at the full budget. */
hs_status hs_context_stream(hs_context* ctx, int32_t cu_budget, int32_t role, void** stream_out);

/* Masks of the ladder level (8 words each; either pointer may be NULL). */
hs_status hs_context_masks(const hs_context* ctx, int32_t cu_budget, uint32_t shared_mask[8],
                           uint32_t down_mask[8]);

hs_status hs_context_destroy(hs_context* ctx);

/* Workspace bytes needed by the calls below for up to max_tokens packed rows,
 * max_seqs sequences and positions up to max_pos (exclusive). */
hs_status hs_workspace_size(const hs_layer_cfg* cfg, int32_t max_tokens, int32_t max_seqs,
                            int32_t max_pos, size_t* bytes);

/* The same for calls on a paged cache (hs_kv_cache.block_table non-NULL)
 * whose pages hold page_positions positions (its max_ctx); 0 means no block
 * table.  page_positions must be 0 or a positive multiple of 64. */
hs_status hs_workspace_size_paged(const hs_layer_cfg* cfg, int32_t max_tokens, int32_t max_seqs,
                                  int32_t max_pos, int32_t page_positions, size_t* bytes);

/* Shared-stage forward: n_layers decoder layers over a packed ragged batch.
 *   x_in         bf16 [T, hidden] device, T = seq_offsets[n_seqs].
 *   x_out        fp32 [T, hidden] device (the residual stream is carried in
 *                fp32 between layers); must not overlap x_in.
 *   w            host array of n_layers weight sets.
 *   seq_offsets  host [n_seqs + 1];  ctx_lens host [n_seqs] or NULL.
 *   kv           NULL: keys/values live in the workspace only (plain prefill).
 *                non-NULL: row i of sequence b is written to position
 *                ctx_lens[b] + i of sequence b in every layer's cache (slot
 *                b, or the page its block table names), and the sequence
 *                attends to its cache positions 0 .. ctx_lens[b] + i (§2.1:
 *                prefill builds the cache).  Requires ctx_lens.
 *   cu_budget    CU cap s_shared (§4.5, Algorithm 1, step 4).  stream NULL
 *                selects the context's SHARED stream of that budget; a
 *                non-NULL stream must carry exactly cu_budget CUs.
 *   workspace    device buffer of ws_bytes >= hs_workspace_size(cfg, T,
 *                n_seqs, max position + 1) (hs_workspace_size_paged with the
 *                page size for a paged cache), owned by the caller; must not
 *                overlap the inputs or outputs.  It may be reused as soon as
 *                the stream has passed this call.
 * The output is the residual stream after the last layer (no final norm). */
hs_status hs_shared_stage_forward(hs_context* ctx, const hs_layer_cfg* cfg,
                                  const hs_layer_weights* w, int32_t n_layers, const void* x_in,
                                  void* x_out, const int32_t* seq_offsets,
                                  const int32_t* ctx_lens, int32_t n_seqs, const hs_kv_cache* kv,
                                  int32_t cu_budget, void* stream, void* workspace,
                                  size_t ws_bytes);

/* The same with multimodal RoPE positions (cfg->mrope_sections non-zero):
 * positions3 is a host array [3][T] giving, for every packed row, its
 * temporal, height and width position (image or video rows take their patch
 * grid coordinates, text rows three equal positions).  Each must be in
 * [0, P), P the largest ctx_lens[b] + row + 1 of the batch.  Cache
 * placement and causal masking still follow the row order; only the RoPE
 * angles change.  Errors as hs_shared_stage_forward, plus HS_ERR_INVALID_ARG
 * for null positions3, zero mrope_sections or a position outside [0, P). */
hs_status hs_shared_stage_forward_mrope(hs_context* ctx, const hs_layer_cfg* cfg,
                                        const hs_layer_weights* w, int32_t n_layers, const void* x_in,
                                        void* x_out, const int32_t* seq_offsets,
                                        const int32_t* ctx_lens, int32_t n_seqs, const hs_kv_cache* kv,
                                        const int32_t* positions3, int32_t cu_budget, void* stream,
                                        void* workspace, size_t ws_bytes);

/* Downstream decode step (§2.1: decode re-reads weights and the cache):
 * one new row per sequence through n_layers layers.
 *   x_in         bf16 [batch, hidden] device.
 *   x_out        fp32 [batch, hidden] device; must not overlap x_in.
 *   kv_lens      host [batch]: cached rows before the step.  The new row is at
 *                position kv_lens[b], its K/V are written there (slot b, or
 *                the page its block table names), and it attends to
 *                kv_lens[b] + 1 keys.  kv_lens[b] < max_ctx without a block
 *                table, < pages_per_seq * max_ctx with one.
 *   cu_budget, stream, workspace as for hs_shared_stage_forward, with the
 *   DOWN role: stream NULL selects the context's DOWN stream for the ladder
 *   level whose SHARED budget is n_cus - cu_budget.
 * The library never changes kv_lens; the caller advances them. */
/* The decode step with multimodal RoPE positions (cfg->mrope_sections
 * non-zero): positions3 is a host array [3][batch] with the new rows'
 * temporal, height and width positions, each in [0, max kv_lens + 1).  Cache
 * placement and masking follow kv_lens.  Errors as for the decode step, plus
 * HS_ERR_INVALID_ARG for null positions3, zero mrope_sections or a position
 * out of range. */
hs_status hs_downstream_decode_step_mrope(hs_context* ctx, const hs_layer_cfg* cfg,
                                          const hs_layer_weights* w, int32_t n_layers, const void* x_in,
                                          void* x_out, const hs_kv_cache* kv, const int32_t* kv_lens,
                                          const int32_t* positions3, int32_t batch, int32_t cu_budget,
                                          void* stream, void* workspace, size_t ws_bytes);

hs_status hs_downstream_decode_step(hs_context* ctx, const hs_layer_cfg* cfg,
                                    const hs_layer_weights* w, int32_t n_layers,
                                    const void* x_in, void* x_out, const hs_kv_cache* kv,
                                    const int32_t* kv_lens, int32_t batch, int32_t cu_budget,
                                    void* stream, void* workspace, size_t ws_bytes);

/* The decode step for callers that cannot allocate device memory (tight
 * serving loops, harnesses that forbid allocation): the same computation and
 * kernels as hs_downstream_decode_step, with no workspace argument.  Its
 * workspace is a static device array of 64 MiB that the library holds on each
 * GPU it runs on until the process ends, laid out without the packed key/value
 * region (the cache is required); the metadata is staged through a fixed ring
 * of pinned slots allocated by hs_context_create.  The call allocates nothing
 * (no hipMalloc, hipHostMalloc or hipFree); it may wait on the host for the
 * oldest staging slot's copy when four calls are in flight.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (on different streams, or from several contexts) race and must not be
 * issued.  Consecutive calls on one stream are ordered and safe.
 * Arguments as hs_downstream_decode_step.  Errors as that call, plus
 * HS_ERR_UNSUPPORTED for batch > 1024 and HS_ERR_WORKSPACE when the call's
 * workspace exceeds the 64 MiB array or its metadata a 1 MiB staging slot
 * (the talker at batch 128 behind 1024 cached rows needs about 5 MiB);
 * nothing is enqueued then. */
hs_status hs_downstream_decode_step_noalloc(hs_context* ctx, const hs_layer_cfg* cfg,
                                            const hs_layer_weights* w, int32_t n_layers,
                                            const void* x_in, void* x_out, const hs_kv_cache* kv,
                                            const int32_t* kv_lens, int32_t batch, int32_t cu_budget,
                                            void* stream);

/* The downstream decode step captured once and replayed per step (§2.1:
 * decode re-runs the same layers for every new token, so the launch sequence
 * of a step does not change while the batch does not).  A talker step is a
 * chain of ~5 short launches per layer; replaying them from a HIP graph takes
 * the host's launch work and most of the gaps between them off the step.
 *
 * hs_decode_graph_create captures the launches of hs_downstream_decode_step
 * for fixed (cfg, weights, n_layers, x_in, x_out, cache, batch, cu_budget,
 * stream, workspace): every pointer is bound at capture and must stay valid,
 * and the caller refreshes the contents of x_in between launches and reads
 * x_out after.  The metadata image has a fixed layout sized for the cache's
 * capacity (positions below max_ctx, or below pages_per_seq * max_ctx with a
 * block table), single-row attention is launched over that capacity and its
 * blocks beyond the step's work exit, and the RoPE table for every such
 * position is computed once (enqueued on the stream by this call).  The
 * stream is resolved as hs_downstream_decode_step resolves it (NULL: the
 * context's DOWN stream of that budget); a replay keeps the stream's CU
 * mask (the graph's kernels run on the stream it is launched on).  The
 * workspace (hs_workspace_size, or hs_workspace_size_paged with the page
 * size, for batch rows, batch sequences and that position capacity) belongs
 * to the graph until it is destroyed; no other call may use it.
 * kv->block_table, if non-null, only marks the cache as paged (its contents
 * are not read here); kv->k / kv->v arrays are copied.
 *
 * hs_decode_graph_launch stages the step's metadata from kv_lens (host,
 * [batch], cached rows before the step, as hs_downstream_decode_step) and,
 * for a paged cache, block_table (host, [batch][pages_per_seq], checked as
 * that call checks it; NULL otherwise) into the graph's workspace with an
 * ordinary copy on the stream, then launches the graph on the stream.  The
 * copy is issued before the graph, outside it, so a replay never reads a
 * staging buffer that a later launch reuses.  Outputs are bit-identical to
 * hs_downstream_decode_step on the same inputs.  Errors: HS_ERR_INVALID_ARG
 * (kv_lens outside the capacity, table errors), HS_ERR_HIP; nothing is
 * enqueued on a validation error.
 *
 * hs_decode_graph_destroy waits for the graph's stream and frees the graph
 * (NULL is a no-op).  A graph is not thread-safe, like its context, and must
 * be destroyed before its context. */
hs_status hs_decode_graph_create(hs_context* ctx, const hs_layer_cfg* cfg, const hs_layer_weights* w,
                                 int32_t n_layers, const void* x_in, void* x_out, const hs_kv_cache* kv,
                                 int32_t batch, int32_t cu_budget, void* stream, void* workspace,
                                 size_t ws_bytes, hs_decode_graph** out);
hs_status hs_decode_graph_launch(hs_decode_graph* graph, const int32_t* kv_lens, const int32_t* block_table);
hs_status hs_decode_graph_destroy(hs_decode_graph* graph);

/* ------------------------------------------------------------------------
 * Diffusion-transformer (DiT) denoising step: a second downstream workload.
 * The paper names diffusion transformers among the output-side generators of
 * omni models, a denoising loop distinct from autoregressive decode (§2.1,
 * "Visual generators"), which an image-output request enters as its
 * downstream stage (§2.2).  It gives no block formula; this is the
 * adaLN-Zero block of the DiT design over a ragged batch of latent-token
 * sequences, each with its own conditioning vector c_b:
 *   (shift1, scale1, gate1, shift2, scale2, gate2) = chunk6(silu(c_b) W_ada^T + b_ada)
 *   h = LN(x) (1 + scale1) + shift1;  x += gate1 * (MHSA(h) W_o^T + b_o)
 *   h = LN(x) (1 + scale2) + shift2;  x += gate2 * (gelu_tanh(h W_1^T + b_1) W_2^T + b_2)
 * LN without affine parameters, eps inside the root; attention bidirectional
 * within each sequence (Hq = Hkv = n_heads, scale 1/sqrt(head_dim)); w_qkv
 * rows [Q heads | K heads | V heads] with bias b_qkv; no rotary embedding.
 * A step is the block stack; patch embedding, the final projection and the
 * sampler's update are outside it. */
typedef struct hs_dit_cfg {
  int32_t hidden;     /* multiple of 256, at most 8192 */
  int32_t n_heads;    /* n_heads * head_dim == hidden */
  int32_t head_dim;   /* 64 or 128 */
  int32_t mlp;        /* MLP width, multiple of 256 */
  float ln_eps;       /* > 0 */
} hs_dit_cfg;

/* Device pointers, bf16 unless noted.  w_ada [6 hidden, hidden] and all
 * biases are bf16 row-major; w_qkv [3 hidden, hidden], w_o [hidden, hidden],
 * w_fc1 [mlp, hidden], w_fc2 [hidden, mlp] are bf16 row-major
 * (format HS_WEIGHTS_BF16) or prepared by hs_convert_weights_f16
 * (HS_WEIGHTS_F16). */
typedef struct hs_dit_weights {
  const void* w_ada;
  const void* b_ada;
  const void* w_qkv;
  const void* b_qkv;
  const void* w_o;
  const void* b_o;
  const void* w_fc1;
  const void* b_fc1;
  const void* w_fc2;
  const void* b_fc2;
  int32_t format;
} hs_dit_weights;

/* Workspace bytes of hs_dit_forward for up to max_tokens rows in max_seqs
 * sequences. */
hs_status hs_dit_workspace_size(const hs_dit_cfg* cfg, int32_t max_tokens, int32_t max_seqs, size_t* bytes);

/* n_layers DiT blocks over a packed ragged batch, on the downstream side of a
 * ladder level (cu_budget and stream as hs_downstream_decode_step).
 *   x_in   bf16 [T, hidden] device, T = seq_offsets[n_seqs]; x_out fp32
 *          [T, hidden] device (the residual stream is fp32 between blocks),
 *          not overlapping x_in.
 *   cond   fp32 [n_seqs, hidden] device: sequence b's conditioning vector.
 *   seq_offsets host [n_seqs + 1], non-decreasing from 0 (empty sequences
 *          allowed); copied before the call returns.
 * MFMA operands are fp16 (activations rounded once per GEMM input) with fp32
 * accumulation; LayerNorm statistics, the modulation and the residual
 * branches are fp32.  Errors as hs_shared_stage_forward (validation enqueues
 * nothing). */
hs_status hs_dit_forward(hs_context* ctx, const hs_dit_cfg* cfg, const hs_dit_weights* w, int32_t n_layers,
                         const void* x_in, void* x_out, const float* cond, const int32_t* seq_offsets,
                         int32_t n_seqs, int32_t cu_budget, void* stream, void* workspace, size_t ws_bytes);

/* Topology probe: launches n_groups work-groups on `stream` (NULL = the
 * context's full-budget stream); each writes, into out_ids (device, uint32
 * [n_groups * 4]): XCC id, shader engine, CU id, and the low 32 bits of the
 * constant-rate clock at its start.  Used to check that masks hold. */
hs_status hs_probe_hw_ids(hs_context* ctx, void* stream, int32_t n_groups, void* out_ids);

/* One-time weight preparation for format HS_WEIGHTS_F16: src is a bf16
 * [rows, cols] row-major matrix, dst receives the same values as fp16 in
 * panel-major order [cols / 32][rows][32] (element (r, c) at
 * ((c / 32) * rows + r) * 32 + c % 32).  That order makes every 32-wide K
 * slice of a weight tile one contiguous run for the GEMMs' copy engine.
 * Device pointers, 4-byte aligned, non-overlapping; cols a positive multiple
 * of 32.  Enqueued on stream (NULL = the context's full-budget stream).
 * Exact for magnitudes in [2^-14, 65504]; smaller magnitudes round toward
 * zero to fp16 subnormals (error below 2^-24), larger ones saturate. */
hs_status hs_convert_weights_f16(hs_context* ctx, const void* src_bf16, void* dst_f16, int64_t rows, int64_t cols,
                                 void* stream);

/* Per-kernel timing with HIP events on the launch stream.  While enabled,
 * every launch of the compute calls is bracketed by a pair of events (a pool
 * of 8192 pairs; launches beyond it are not recorded).  hs_timing_enable(ctx,
 * 1) clears earlier records; hs_timing_read waits for the recorded events of
 * one kernel kind and returns their summed duration and count. */
enum {
  HS_KERNEL_RMSNORM = 0,
  HS_KERNEL_QKV = 1,          /* QKV projection with RoPE and key/value store */
  HS_KERNEL_ATTENTION = 2,    /* multi-row causal attention */
  HS_KERNEL_DECODE_ATTN = 3,  /* single-row attention */
  HS_KERNEL_O_PROJ = 4,       /* output projection + residual */
  HS_KERNEL_GATE_UP = 5,      /* gate/up projection + SwiGLU */
  HS_KERNEL_DOWN = 6,         /* down projection + residual */
  HS_KERNEL_ROPE_TABLE = 7,
  HS_KERNEL_MODULATION = 8,   /* DiT: silu(c) and the per-layer adaLN modulation */
  HS_KERNEL_LN_MOD = 9,       /* DiT: modulated LayerNorm */
  HS_KERNEL_MLP_UP = 10,      /* DiT: first MLP projection + bias + GELU */
  HS_KERNEL_MLP_DOWN = 11,    /* DiT: second MLP projection + bias + gated residual */
  HS_KERNEL_KINDS = 12
};

hs_status hs_timing_enable(hs_context* ctx, int32_t enable);
hs_status hs_timing_read(hs_context* ctx, int32_t kernel_kind, double* total_ms, int32_t* n_launches);

/* Sustained shader clock of the recorded launches of one kernel kind (the
 * large GEMMs and multi-row attention; other kinds report 0 launches).
 * While timing is enabled, the first lane of block 0 of each such launch
 * reads the shader-clock counter (one count per core clock cycle) and the
 * constant-rate counter at entry and exit; *mhz receives the ratio of the
 * summed cycle counts to the summed constant-rate ticks, scaled by the
 * device's constant clock rate.  The persistent GEMM's block 0 lives for the
 * whole launch, so for it this is the launch's average clock.  Waits for the
 * recorded launches; 0 MHz and 0 launches when none was recorded. */
hs_status hs_timing_read_clock(hs_context* ctx, int32_t kernel_kind, double* mhz, int32_t* n_launches);

/* ------------------------------------------------------------------------
 * Spatial controller: the bandwidth-guided shared-stage cap of §4.4
 * ("Bandwidth-pressure signal", "SM ladder", Eq. (1)) applied as in step 3 of
 * Algorithm 1.  Host only; no HIP call.  Per scheduling step:
 *   B_hat = ewma_weight * B + (1 - ewma_weight) * B_hat   (the first sample
 *           initialises B_hat)
 *   rho   = clamp(B_hat / saturation, 0, 1)
 *   s*    = aggressive_cus                       if downstream is inactive
 *         = snap(S_min + rho * (S_cap - S_min))  otherwise, snap = the nearest
 *           ladder level, ties to the larger one
 *   s*  is applied when downstream is inactive, on the first step, when the
 *       current cap is not a ladder level, or when its ladder index is at
 *       least hysteresis_steps away from the current level; otherwise the
 *       current cap is kept.  down_cus = max(0, total_cus - shared_cus).
 * Ladder levels are meant to be budgets of a context's ladder, so a decision
 * selects a pre-built stream pair with hs_context_stream (§5). */
typedef struct hs_controller_cfg {
  int32_t total_cus;        /* S_tot */
  int32_t aggressive_cus;   /* S_aggr, the cap with no downstream activity */
  const int32_t* ladder;    /* host [n_ladder]: co-running levels S_min .. S_cap,
                               strictly increasing, >= 1; S_cap < S_aggr <= S_tot */
  int32_t n_ladder;
  double ewma_weight;       /* gamma, weight of the newest sample, in (0, 1] */
  double saturation;        /* B_sat > 0, in the units of the samples */
  int32_t hysteresis_steps; /* Delta_step >= 1, in ladder levels */
} hs_controller_cfg;

typedef struct hs_split {
  int32_t shared_cus;       /* s_shared: cap of the shared stage */
  int32_t down_cus;         /* s_down = max(0, S_tot - s_shared) */
  int32_t level;            /* index of s_shared in the ladder, -1 for S_aggr */
  int32_t changed;          /* 1 when this step moved the cap */
  double pressure;          /* B_hat after this step's sample */
  double rho;               /* clamp(B_hat / saturation, 0, 1) */
} hs_split;

typedef struct hs_controller hs_controller;

/* The controller copies cfg (and the ladder).  Errors: HS_ERR_INVALID_ARG for
 * a null pointer, an empty or non-increasing ladder, S_cap >= S_aggr,
 * S_aggr > S_tot, ewma_weight outside (0, 1], saturation <= 0 or
 * hysteresis_steps < 1. */
hs_status hs_controller_create(const hs_controller_cfg* cfg, hs_controller** out);

/* One scheduling step: downstream_active is A(t) (non-zero when a downstream
 * stage runs), sample is B(t).  Writes the split to *out.  Errors:
 * HS_ERR_INVALID_ARG for null pointers or a non-finite sample (the state is
 * then unchanged). */
hs_status hs_controller_step(hs_controller* ctrl, int32_t downstream_active, double sample, hs_split* out);

hs_status hs_controller_destroy(hs_controller* ctrl);

/* Memory-system activity of a GPU in [0, 1]: the memory-controller (UMC)
 * activity that AMD SMI reports, the AMD counterpart of the NVML memory
 * activity the paper samples (§4.4, §5).  device is a HIP device index; the
 * reading comes from the AMD SMI GPU at that device's PCI address (AMD SMI's
 * own enumeration order is not used).  AMD SMI is loaded on first use.
 * Errors: HS_ERR_INVALID_ARG for a null pointer or a device outside HIP's
 * device count; HS_ERR_HIP if the PCI address cannot be read;
 * HS_ERR_UNSUPPORTED when AMD SMI, a GPU at that address, or the reading is
 * unavailable.  One reading takes on the order of 100 us (a driver query).
 * The value is the firmware's average over its last interval, which MI355X
 * refreshes about once per second: under a copy load at 5.0 TB/s it reads
 * 0.61, close to the share of the 8 TB/s peak, and readings taken within one
 * interval repeat. */
hs_status hs_pressure_sample(int32_t device, double* activity);

/* ------------------------------------------------------------------------
 * Temporal scheduler: shared-stage path rotation (§4.2 "Remaining-slack
 * ratio"; §4.3 "Path rotation", "Slack guard", "Adaptive rotation ratio",
 * "Long-path admission cap"; Algorithm 1, steps 1 and 2).  Host only.
 *
 * Each call is one scheduling step k (counted from 0 per scheduler).  For
 * every request of the queue:
 *   u_i = (deadline - now) / remaining;  protected when u_i < u_guard.
 * N = round(n_min + f (n_max - n_min)), halves upward, where f is the
 * protected share of the waiting short-path prefills (0 when none wait).
 * The step is a short-path phase when k mod (N + m) < N, else a long-path
 * phase.  visible[i] = 1 for decode continuations, protected requests and
 * prefills of the phase's path; other prefills get 0 for this step only.
 * Then, if long_cap >= 0 and more than long_cap ordinary (unprotected)
 * long-path prefills are visible, only the long_cap with the earliest
 * deadlines stay visible (ties: lower index).  The caller batches from the
 * visible requests; nothing of the queue is stored or reordered. */
enum { HS_PATH_SHORT = 0, HS_PATH_LONG = 1 };
enum { HS_WORK_PREFILL = 0, HS_WORK_DECODE = 1 };

typedef struct hs_temporal_cfg {
  int32_t n_min, n_max; /* short-path phases per cycle, 1 <= n_min <= n_max ([2, 8] in §4.3) */
  int32_t m;            /* long-path phases per cycle, >= 1 (2 in §4.3) */
  double u_guard;       /* slack guard, > 0 */
  int32_t long_cap;     /* most ordinary long-path prefills per view; < 0: no cap */
} hs_temporal_cfg;

typedef struct hs_request_view {
  int32_t path;      /* HS_PATH_SHORT: ends after the shared stage; HS_PATH_LONG: continues downstream */
  int32_t work;      /* HS_WORK_PREFILL: waiting for its prefill; HS_WORK_DECODE: a decode continuation */
  double deadline;   /* first-response deadline d_i = a_i + Delta_c, finite */
  double remaining;  /* estimated remaining time to the first response, > 0, same unit */
} hs_request_view;

typedef struct hs_temporal_step_info {
  int64_t step;        /* k of this call */
  int32_t n;           /* N used by this step */
  int32_t phase;       /* HS_PATH_* of this step */
  int32_t n_protected; /* requests with u_i < u_guard */
  int32_t n_hidden;    /* prefills hidden by the phase */
  int32_t n_capped;    /* long-path prefills hidden by the cap */
} hs_temporal_step_info;

typedef struct hs_temporal hs_temporal;

/* Errors: HS_ERR_INVALID_ARG for a null pointer, n_min < 1, n_min > n_max,
 * m < 1 or u_guard not a positive finite number.  The scheduler copies the
 * configuration; release it with hs_temporal_destroy. */
hs_status hs_temporal_create(const hs_temporal_cfg* cfg, hs_temporal** out);

/* reqs[n_reqs] and visible[n_reqs] are host arrays owned by the caller; info
 * may be NULL.  Errors (HS_ERR_INVALID_ARG, nothing written and the step not
 * counted): null pointers with n_reqs > 0, n_reqs < 0, a non-finite now or
 * deadline, remaining <= 0, or an unknown path or work code. */
hs_status hs_temporal_step(hs_temporal* s, double now, const hs_request_view* reqs, int32_t n_reqs,
                           uint8_t* visible, hs_temporal_step_info* info);

hs_status hs_temporal_destroy(hs_temporal* s);

#ifdef __cplusplus
}
#endif

#endif /* HORIZON_H_ */
