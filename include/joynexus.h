/*
 * joynexus.h -- C ABI of the MI355X (gfx950) group-batched step.
 *
 * The step follows the multi-tenant group batching of JoyNexus
 * (Sec. 4.3 "Multi-Tenant Group Batching", its figure of the pipeline;
 * App. A.3 "Inference Queue Composition"; Sec. 5.2 "Multi-Tenant
 * Group-Batched Execution"):
 *
 *   jn_pack_group          canonicalize + pad: concatenate compatible tenant
 *                          requests into one physical batch and record the
 *                          slices that partition it again
 *   jn_backbone_forward    one frozen shared-backbone forward over that batch
 *                          (the "encode" of App. A.3), attention confined to
 *                          each sample
 *   jn_tenant_heads_fwd_bwd split the shared features by tenant; per tenant:
 *                          action-head forward, loss, weight gradients (the
 *                          tenant-private decode / loss / backward of Sec. 5.2;
 *                          nothing is averaged across tenants)
 *   jn_tenant_experts_fwd_bwd the same for tenants whose action module is a
 *                          transformer expert reading each sample's backbone rows
 *   jn_tenant_adamw_step   per-tenant AdamW update of the tenants' parameters
 *   jn_unpack              scatter packed rows back to the requests' own
 *                          padded buffers (the "split" by slices, App. A.3)
 *   jn_collector_*         the inference queue's FIFO-compatible-prefix
 *                          batching under a maximum batch size and a timeout
 *   jn_infer_plan_*        a resident decode-only step over one physical
 *                          batch, launchable eagerly or as a HIP graph
 *
 * Conventions
 *   - bf16 is the IEEE-754 binary32 upper half (bfloat16), stored as 2 bytes.
 *   - Every device buffer is owned by the caller.  The library allocates no
 *     device memory after jn_ctx_create; scratch comes from the caller's
 *     workspace.  It keeps no pointer after a call returns.
 *   - Calls are asynchronous on the context's HIP stream.  All validation is
 *     done before anything is enqueued: a non-OK status means nothing was
 *     written to any output.  jn_last_error() holds a message for the last
 *     non-OK status of that context.
 *   - "host" arrays are read during the call and may be reused on return.
 *   - One context per stream and per host thread; contexts share nothing.
 *   - Weight matrices are row-major [out][in].
 */
#ifndef JOYNEXUS_H
#define JOYNEXUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum jn_status {
  JN_OK = 0,
  JN_EINVAL = 1,        /* null pointer, bad option or count                    */
  JN_EINCOMPAT = 2,     /* tenants do not share the backbone's prefix interface */
  JN_ESHAPE = 3,        /* a length, size or index out of its range             */
  JN_ENOSPACE = 4,      /* a caller buffer or workspace is too small            */
  JN_EHIP = 5,          /* the HIP runtime reported an error                    */
  JN_EUNSUPPORTED = 6   /* a shape the kernels do not implement                 */
} jn_status;

typedef struct jn_ctx jn_ctx;

/* Create a context bound to `hip_stream` (a hipStream_t, borrowed; NULL = the
 * null stream) on the current HIP device.  Allocates pinned host staging for
 * index-map uploads. */
jn_status jn_ctx_create(jn_ctx** out, void* hip_stream);
void jn_ctx_destroy(jn_ctx* ctx);
/* Rebind the context to another stream of the same device. */
jn_status jn_ctx_set_stream(jn_ctx* ctx, void* hip_stream);
/* Message for the last non-OK status returned on this context ("" if none). */
const char* jn_last_error(const jn_ctx* ctx);

/* ------------------------------------------------------- measurement --- */

/* Kernel classes reported by the launch trace. */
typedef enum jn_op {
  JN_OP_PACK = 1, JN_OP_RMSNORM = 2, JN_OP_GEMM_QKV = 3, JN_OP_ATTENTION = 4, JN_OP_GEMM_O = 5,
  JN_OP_GEMM_UP = 6, JN_OP_GEMM_DOWN = 7, JN_OP_POOL = 8, JN_OP_HEAD_FWD = 9, JN_OP_LOSS = 10,
  JN_OP_HEAD_BWD = 11, JN_OP_UNPACK = 12, JN_OP_EXPERT_GEMM = 13, JN_OP_EXPERT_ATTENTION = 14,
  JN_OP_EXPERT_OTHER = 15, JN_OP_OPTIMIZER = 16, JN_OP_ROPE = 17
} jn_op;

/* One traced kernel launch.  For GEMMs (M, N, K) is the launch shape
 * (N counts gate and up rows for GeGLU); for the other kernels M is the
 * number of rows touched and N the row width. */
typedef struct jn_trace_entry {
  int32_t op, M, N, K;
  float ms;               /* device time between the bracketing events */
  int32_t reserved;
} jn_trace_entry;

/* Enable (1) or disable (0) the launch trace: while enabled, every kernel the
 * context enqueues is bracketed by a pair of HIP timing events on its stream.
 * Enabling clears previously collected entries. */
jn_status jn_ctx_set_trace(jn_ctx* ctx, int32_t enable);
/* Wait for the traced launches to finish and copy up to `cap` entries (in
 * launch order) to `out`; `*n` receives the number collected.  Clears the
 * trace.  Synchronizes with the context stream. */
jn_status jn_ctx_trace_read(jn_ctx* ctx, jn_trace_entry* out, int32_t cap, int32_t* n);

/* Context options (jn_ctx_set_option), for verification; a context starts
 * with every option 0.
 *   JN_OPT_EXPERT_TRANSPOSES: 1 = the action-expert gradient GEMMs (the
 *     weight gradients dY^T X over a tenant's rows, the data gradients dY W)
 *     read materialised, zero-padded transposes of their operands -- the
 *     path the library takes by itself only where a problem's offsets exceed
 *     the 32-bit ones of its transposed operand loads; 0 = they read the row
 *     buffers and weights transposed inside the GEMM.  Both issue the same
 *     MFMA sequence per output element, so results are bitwise identical.
 * Sec. 5.2 (tenant-private backward of the action modules).  Returns
 * JN_EINVAL for an unknown option or a value other than 0 / 1; takes effect
 * for calls enqueued after it. */
#define JN_OPT_EXPERT_TRANSPOSES 1
jn_status jn_ctx_set_option(jn_ctx* ctx, int32_t option, int32_t value);

/* ---------------------------------------------------------------- pack --- */

/* One inference / training request of one tenant (App. A.3: a request carries
 * the tenant identity, its schema signature and a batch of observations; here
 * the observations are already embedded by the tenant's front end). */
typedef struct jn_request {
  int32_t tenant;          /* slot in the tenant table                       */
  int32_t n_samples;       /* >= 1                                           */
  int32_t max_len;         /* rows per sample in `embeds` (canonical length) */
  int32_t reserved;
  const void* embeds;      /* device bf16 [n_samples][max_len][d]            */
  const int32_t* lengths;  /* host int32 [n_samples]: valid rows, 1..max_len */
} jn_request;

/* A tenant taking part in the group.  Compatibility is decided at the shared
 * frozen-prefix boundary, not by tenant identity (App. A.3): every tenant in
 * the table must carry the same `prefix_sig` and consume features of the
 * backbone's width. */
typedef struct jn_tenant {
  uint64_t prefix_sig;     /* signature of the shared-prefix interface */
  int32_t d_model;         /* feature width the tenant expects         */
  int32_t reserved;
} jn_tenant;

typedef struct jn_pack_opts {
  int32_t d_model;         /* backbone width d (row width of embeds)            */
  int32_t align;           /* each sample occupies roundup(len, align) rows, >=1 */
} jn_pack_opts;

typedef struct jn_pack_sizes {
  int32_t N;               /* samples                                   */
  int32_t T;               /* packed rows (sum of aligned lengths)      */
  int32_t max_seqlen;      /* longest valid length                      */
  int32_t reserved;
  int64_t map_bytes;       /* size of the index-map buffer to allocate  */
  int64_t token_bytes;     /* size of the packed-token buffer: T*d*2    */
} jn_pack_sizes;

/* The physical batch: sizes plus device pointers into the caller's buffers.
 * Filled by jn_pack_group; read by the later calls.  Map meaning (all int32):
 *   seqlens[N]            valid rows of sample i
 *   cu_seqlens[N+1]       first packed row of sample i (aligned prefix sums)
 *   sample_request[N]     request of sample i (arrival order: requests in the
 *                         order given, samples in order inside a request)
 *   sample_local[N]       index of sample i inside its request
 *   sample_tenant[N]      tenant slot of sample i
 *   tenant_sample_off[G+1] first tenant-order position of tenant g
 *   tenant_perm[N]        sample at tenant-order position k (stable by tenant)
 *   sample_tenant_rank[N] tenant-order position of sample i (inverse of perm)
 *   token_sample[T]       sample of packed row t, -1 for an alignment row
 *   token_pos[T]          row of that sample, -1 for an alignment row      */
typedef struct jn_packed {
  int32_t R, G, N, T, d, max_seqlen, align;
  int32_t req_sig;         /* signature of the requests' (n_samples, max_len)
                              list, checked by jn_unpack                     */
  int32_t max_tenant_n;    /* most samples of any one tenant (sizes the
                              per-tenant launches; 0 = unknown, N is used)   */
  void* tokens;            /* device bf16 [T][d]; alignment rows are zero */
  int32_t* seqlens;
  int32_t* cu_seqlens;
  int32_t* sample_request;
  int32_t* sample_local;
  int32_t* sample_tenant;
  int32_t* tenant_sample_off;
  int32_t* tenant_perm;
  int32_t* sample_tenant_rank;
  int32_t* token_sample;
  int32_t* token_pos;
  void* req_table;         /* library-internal request table [R] (32 B each) */
} jn_packed;

/* Sizes of the physical batch (host only, touches no device). */
jn_status jn_pack_plan(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                       const jn_pack_opts* opts, jn_pack_sizes* out);

/* The same index maps, computed on the host into `host_maps` (map_bytes from
 * jn_pack_plan), in the layout jn_pack_group uses on the device:
 *   seqlens | cu_seqlens | sample_request | sample_local | sample_tenant |
 *   tenant_sample_off | tenant_perm | sample_tenant_rank | token_sample |
 *   token_pos | request table (32 B per request, library-internal), each
 *   array starting on a 256-byte boundary of the buffer.
 * `out` receives host pointers into `host_maps` (tokens = NULL). */
jn_status jn_pack_maps_host(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                            const jn_pack_opts* opts, void* host_maps, size_t map_bytes,
                            jn_packed* out);

/* Build the physical batch on the device: index maps into `maps`
 * (map_bytes), packed rows into `tokens` (token_bytes).  Row
 * cu_seqlens[i] + j of `tokens` is row j of sample i for j < seqlens[i];
 * alignment rows are zero.  Bit-exact copy. */
jn_status jn_pack_group(jn_ctx* ctx, const jn_request* req, int32_t R, const jn_tenant* ten,
                        int32_t G, const jn_pack_opts* opts, void* maps, size_t map_bytes,
                        void* tokens, size_t token_bytes, jn_packed* out);

/* ------------------------------------------------------------ backbone --- */

typedef struct jn_layer {
  const void* wqkv;        /* bf16 [(H + 2 Hkv) hd][d]: q rows, then k rows,
                              then v rows (Hkv = H unless grouped); head h
                              uses rows h*hd .. h*hd+hd-1 of each            */
  const void* wo;          /* bf16 [d][d]                                     */
  const void* w_up;        /* bf16 [f][d]                                     */
  const void* w_gate;      /* bf16 [f][d] for a GeGLU MLP, NULL for GELU MLP  */
  const void* w_down;      /* bf16 [d][f]                                     */
  const void* g1;          /* bf16 [d] pre-attention RMSNorm gain             */
  const void* g2;          /* bf16 [d] pre-MLP RMSNorm gain                   */
} jn_layer;

/* Frozen shared backbone: pre-RMSNorm transformer blocks
 *   h = RMS(x) g1; q,k,v = h Wqkv^T; x += Attn(q,k,v) Wo^T;
 *   h = RMS(x) g2; x += Wdown gelu(Wup h)   or   Wdown (gelu(Wgate h) * Wup h)
 * then z = RMS(x) gf.  Attention never crosses samples; it is bidirectional
 * within a sample, or causal (row j sees rows 0..j of its sample) when
 * `causal` is set.  RMS(x) = x / sqrt(mean(x^2) + eps); gelu is the tanh form.
 * Variants of the VLM families the paper's tenants build on (Sec. 5.2):
 *   n_kv_heads    0 (= n_heads) or a divisor of n_heads: query head h reads
 *                 key/value head h / (n_heads / n_kv_heads); wqkv then has
 *                 (n_heads + 2 n_kv_heads) * hd rows (q, then k, then v)
 *   rope_theta    > 0: rotary embedding of q and k after the projection --
 *                 for i < hd/2 the pair (x_i, x_{i+hd/2}) of a row at
 *                 position p (its row inside its own sample, from 0) is
 *                 rotated by p * rope_theta^(-2i/hd); 0: no positions
 * Arithmetic: bf16 GEMM / attention operands with fp32 accumulation, fp32
 * residual stream, fp32 norm / softmax / rotation math, bf16 stored
 * activations (q and k are stored rotated, rounded once more).
 * Supported sizes: d a multiple of 128 in [128, 4096], ffn a multiple of 128,
 * head dim d / n_heads in {32, 64, 128, 256}; other sizes fail with
 * JN_EUNSUPPORTED before anything is enqueued. */
typedef struct jn_backbone {
  int32_t n_layers, d, n_heads, ffn;
  float eps;
  int32_t n_kv_heads;      /* 0 = n_heads                               */
  const jn_layer* layers;  /* host array [n_layers] of device pointers */
  const void* gf;          /* bf16 [d] final RMSNorm gain              */
  int32_t causal;          /* 0 bidirectional, 1 causal                */
  float rope_theta;        /* 0 = no rotary embedding                  */
} jn_backbone;

/* Workspace bytes jn_backbone_forward needs for a batch of T rows. */
jn_status jn_backbone_workspace_size(const jn_backbone* bb, int32_t T, size_t* bytes);

/* hidden: device bf16 [T][d], written for every row (alignment rows zero). */
jn_status jn_backbone_forward(jn_ctx* ctx, const jn_backbone* bb, const jn_packed* p,
                              void* hidden, void* ws, size_t ws_bytes);

/* --------------------------------------------------------------- heads --- */

/* A tenant-private MLP action head: y = W_L gelu(... gelu(W_1 p + b_1) ...) + b_L
 * with p the mean of the sample's valid rows of the shared feature. */
typedef struct jn_head {
  int32_t n_layers;            /* >= 1                                       */
  int32_t action_dim, chunk;   /* dims[n_layers] == action_dim * chunk       */
  int32_t reserved;
  const int32_t* dims;         /* host [n_layers+1], dims[0] == d            */
  const float* const* W;       /* host [n_layers] of device fp32 [dims[k+1]][dims[k]] */
  const float* const* b;       /* host [n_layers] of device fp32 [dims[k+1]] */
} jn_head;

/* Per-tenant inputs and outputs.  Rows follow the tenant's own arrival order
 * (the order of its samples in the request list). */
typedef struct jn_head_io {
  const float* targets;        /* device fp32 [n_g][chunk][action_dim]       */
  float* actions;              /* out: device fp32 [n_g][chunk*action_dim]   */
  float* loss;                 /* out: device fp32 [1], mean squared error   */
  float* const* dW;            /* host [n_layers] of device fp32 outputs [out][in] */
  float* const* db;            /* host [n_layers] of device fp32 outputs [out]     */
} jn_head_io;

jn_status jn_heads_workspace_size(const jn_packed* p, const jn_head* heads, int32_t G, size_t* bytes);

/* Pool, then per tenant g (heads[g], io[g]): forward, loss
 * L_g = mean((y - t)^2), and dL_g/dW, dL_g/db of every head layer (fp32).
 * No gradient flows into the frozen backbone.  `pooled` (optional, may be
 * NULL): device fp32 [N][d] receives the pooled features in tenant order. */
jn_status jn_tenant_heads_fwd_bwd(jn_ctx* ctx, const jn_packed* p, const void* hidden,
                                  const jn_head* heads, const jn_head_io* io, int32_t G,
                                  void* ws, size_t ws_bytes, float* pooled);

/* Allocation-free variant of jn_tenant_heads_fwd_bwd, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments (minus the
 * workspace), same kernels, same results bit for bit.  The workspace is a
 * library-owned device array of JN_HEADS_SCRATCH_BYTES per GPU, created with
 * the library and held until the process ends; its index tables are staged
 * through a fixed 1 MiB pinned buffer that jn_ctx_create allocates.  The call
 * allocates nothing (no hipMalloc / hipFree / pinned allocation).  Nothing in
 * the array needs to start at zero: every value a call reads was written by
 * that call.
 * Errors (nothing enqueued): JN_ENOSPACE when jn_heads_workspace_size exceeds
 * JN_HEADS_SCRATCH_BYTES or the tables exceed 1 MiB; the other statuses as
 * for jn_tenant_heads_fwd_bwd.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * GPU (other streams or contexts) race and must be ordered by the caller. */
#define JN_HEADS_SCRATCH_BYTES (64u << 20)
jn_status jn_tenant_heads_fwd_bwd_noalloc(jn_ctx* ctx, const jn_packed* p, const void* hidden,
                                          const jn_head* heads, const jn_head_io* io, int32_t G,
                                          float* pooled);

/* ------------------------------------------------------- action expert --- */

/* Per-tenant sample counts and valid prefix rows of a group (host only): the
 * sizes jn_tenant_experts_fwd_bwd needs, from the same tables jn_pack_group
 * takes.  samples[G], rows[G]. */
jn_status jn_pack_tenant_sizes(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                               const jn_pack_opts* opts, int32_t* samples, int64_t* rows);

/* A tenant-private action expert (the GR00T / pi0.5-style action module of a
 * tenant, Sec. 5.2): per sample, `chunk` noisy action tokens embedded by W_in,
 * n_layers blocks of [RMSNorm -> self-attention over the sample's action
 * tokens -> RMSNorm -> cross-attention whose keys / values are projected
 * (W_kv_c) from that sample's own valid backbone rows -> RMSNorm -> GELU MLP],
 * residual each, final RMSNorm and W_out.  No biases.  Weights bf16 [out][in]. */
typedef struct jn_expert_layer {
  const void* wqkv_s;   /* [3d][d]  self-attention q | k | v            */
  const void* wo_s;     /* [d][d]                                        */
  const void* wq_c;     /* [d][d]   cross-attention queries             */
  const void* wkv_c;    /* [2d][d_prefix] cross-attention keys | values */
  const void* wo_c;     /* [d][d]                                        */
  const void* w_up;     /* [ffn][d]                                      */
  const void* w_down;   /* [d][ffn]                                      */
  const void* g1;       /* [d] gains of the three pre-norms              */
  const void* g2;
  const void* g3;
} jn_expert_layer;

typedef struct jn_expert {
  int32_t n_layers, d, n_heads, ffn;
  int32_t action_dim;   /* <= 32 */
  int32_t chunk;        /* action tokens per sample, <= 64 */
  int32_t d_prefix;     /* backbone width */
  float eps;
  const void* w_in;     /* [d][action_dim] */
  const void* w_out;    /* [action_dim][d] */
  const void* gf;       /* [d]             */
  const jn_expert_layer* layers;  /* host [n_layers] */
  /* Flow matching (the GR00T / pi0.5-style objective of such experts): with
   * w_time set, the expert reads the point x = t*noise + (1-t)*actions of the
   * straight path from the clean actions to the noise, every action token's
   * embedding receives w_time phi(t), phi(t) = [sin(1000 t w_j) | cos(1000 t
   * w_j)], w_j = 10000^(-j/(d_time/2)), j < d_time/2, and the regression
   * target is the path's velocity noise - actions.  NULL: plain regression
   * of `targets` from `noisy`. */
  const void* w_time;   /* [d][d_time] or NULL                     */
  int32_t d_time;       /* even, a multiple of 64, when w_time set */
  int32_t reserved;
} jn_expert;

/* fp32 gradient outputs, same shapes as the weights they belong to. */
typedef struct jn_expert_layer_grads {
  float *wqkv_s, *wo_s, *wq_c, *wkv_c, *wo_c, *w_up, *w_down, *g1, *g2, *g3;
} jn_expert_layer_grads;

typedef struct jn_expert_io {
  int32_t n_samples;      /* the tenant's samples in the packed batch      */
  int32_t reserved;
  int64_t prefix_rows;    /* sum of their valid lengths (jn_pack_tenant_sizes) */
  const float* noisy;     /* device fp32 [n][chunk][action_dim], tenant arrival order */
  const float* targets;   /* device fp32 [n][chunk][action_dim]            */
  float* pred;            /* out: device fp32 [n][chunk][action_dim]       */
  float* loss;            /* out: device fp32 [1], mean squared error      */
  float* dw_in;           /* out: fp32 [d][action_dim]                     */
  float* dw_out;          /* out: fp32 [action_dim][d]                     */
  float* dgf;             /* out: fp32 [d]                                 */
  const jn_expert_layer_grads* layers;  /* host [n_layers] of device outputs */
  /* flow matching (expert w_time set): `noisy` holds the noise, `targets` the
   * clean actions, flow_t the per-sample flow times; dw_time receives the
   * gradient of w_time.  Both NULL otherwise. */
  const float* flow_t;    /* device fp32 [n], tenant arrival order         */
  float* dw_time;         /* out: fp32 [d][d_time]                         */
} jn_expert_io;

jn_status jn_experts_workspace_size(const jn_packed* p, const jn_expert* ex, const jn_expert_io* io, int32_t G,
                                    size_t* bytes);

/* The tenant stage for action-expert tenants: for every tenant g of the packed
 * batch (ex[g], io[g]; all experts share n_layers, d, n_heads, ffn, chunk and
 * d_prefix) the expert forward over its samples, its loss
 * L_g = mean((pred - target)^2) and dL_g / d(every expert weight and gain).
 * `hidden` is jn_backbone_forward's output; no gradient flows into it.
 * Precision: GEMM operands bf16 (activations rounded where they are stored for
 * a GEMM, incoming gradients rounded before a GEMM), fp32 accumulation, fp32
 * residual, norms, attention, GELU derivative and loss.  Gradient outputs must
 * be 16-byte aligned. */
jn_status jn_tenant_experts_fwd_bwd(jn_ctx* ctx, const jn_packed* p, const void* hidden, const jn_expert* ex,
                                    const jn_expert_io* io, int32_t G, void* ws, size_t ws_bytes);

/* ---------------------------------------------------- tenant optimizer --- */

/* One AdamW step for every tenant of a group: each tenant applies its own
 * optimizer step to its own parameters and nothing is shared (Sec. 5.2,
 * training-side group execution).  Tenant g owns n_tensors fp32 parameter
 * tensors with their gradients and first / second moments (device pointers,
 * same element counts, 16-byte aligned).  Per element, with t = step:
 *   m = b1 m + (1 - b1) g;   v = b2 v + (1 - b2) g^2;
 *   p = p (1 - lr wd) - (lr / (1 - b1^t)) m / (sqrt(v) / sqrt(1 - b2^t) + eps)
 * `step` is this update's 1-based index, i.e. the tenant's version after it;
 * the caller advances it only for the tenants it passes.  bf16_out (optional;
 * NULL, or host [n] whose non-NULL entries are device bf16 tensors) receives
 * the new parameters rounded to bf16, for tenants whose forward reads bf16
 * copies.  One launch for all tensors of all tenants; the descriptor table
 * goes to the caller's workspace. */
typedef struct jn_adamw_tenant {
  float lr, beta1, beta2, eps, weight_decay;
  int32_t n_tensors;
  int64_t step;
  float* const* params;        /* host [n] of device fp32, updated in place */
  const float* const* grads;   /* host [n] of device fp32 */
  float* const* m;             /* host [n] of device fp32, updated in place */
  float* const* v;             /* host [n] of device fp32, updated in place */
  const int64_t* numel;        /* host [n] */
  void* const* bf16_out;       /* NULL or host [n] of device bf16 (entries may be NULL) */
} jn_adamw_tenant;

jn_status jn_adamw_workspace_size(const jn_adamw_tenant* t, int32_t G, size_t* bytes);

/* Errors: JN_EINVAL for null or unaligned pointers, step < 1, lr < 0,
 * betas outside [0, 1), eps <= 0 or numel < 0; nothing is enqueued then. */
jn_status jn_tenant_adamw_step(jn_ctx* ctx, const jn_adamw_tenant* t, int32_t G, void* ws, size_t ws_bytes);

/* -------------------------------------------------------------- unpack --- */

/* Scatter packed rows back to the requests: for sample i of request r and
 * j < max_len_r, out[r][s][j] = rows[cu_seqlens[i] + j] if j < seqlens[i],
 * else zero.  `rows`: device [T][row_bytes]; `req_out`: host array [R] of
 * device buffers [n_r][max_len_r][row_bytes]; row_bytes a multiple of 4.
 * `req` must list the requests the batch was packed from, in the same order:
 * requests whose sample counts or max_len differ (even with the same total)
 * are JN_ESHAPE, and nothing is enqueued. */
jn_status jn_unpack(jn_ctx* ctx, const jn_packed* p, const jn_request* req, int32_t R,
                    const void* rows, size_t row_bytes, void* const* req_out);


/* ----------------------------------------- inference-side group batching --- */

/* Request collector of the inference queue (App. A.3 "Inference Queue
 * Composition": requests are examined in arrival order and the largest FIFO
 * prefix that is compatible at the shared frozen-prefix boundary is formed,
 * bounded by the batching timeout and the maximum batch size).  Host only;
 * no device work.  Times are caller-supplied microseconds (any monotonic
 * clock), so the collector is deterministic.
 *
 * The prefix starts at the oldest queued request and takes whole requests in
 * arrival order while (a) each has the oldest request's prefix signature and
 * feature width -- compatibility is decided by the interface, not by tenant
 * identity -- and (b) the total sample count stays <= max_batch_samples (the
 * oldest request is always taken, even if larger).  It is released when it
 * can no longer grow (it holds max_batch_samples samples, or the next queued
 * request is incompatible or would overflow it) or when the oldest request
 * has waited timeout_us.  An incompatible request is never skipped: it heads
 * a later batch. */
typedef struct jn_collector jn_collector;
/* max_batch_samples >= 1, timeout_us >= 0, else JN_EINVAL. */
jn_status jn_collector_create(jn_collector** out, int32_t max_batch_samples, int64_t timeout_us);
void jn_collector_destroy(jn_collector* c);
/* Queue one request (metadata only).  arrival_us must not precede the last
 * queued request's (JN_EINVAL); n_samples, d_model >= 1. */
jn_status jn_collector_submit(jn_collector* c, int64_t request_id, uint64_t prefix_sig, int32_t d_model,
                              int32_t n_samples, int64_t arrival_us);
/* If a batch is ready at now_us, move its request ids (arrival order) to
 * ids[0 .. *n) and remove them from the queue; otherwise *n = 0.  JN_ENOSPACE
 * (queue untouched) if the ready batch has more than `cap` requests. */
jn_status jn_collector_poll(jn_collector* c, int64_t now_us, int64_t* ids, int32_t cap, int32_t* n);
/* Queued request count, and the time at which the current prefix becomes
 * ready (-1 if the queue is empty; the oldest arrival if it is ready already). */
jn_status jn_collector_status(const jn_collector* c, int32_t* pending, int64_t* deadline_us);

/* Resident inference plan for one physical batch: canonicalize + pad, shared
 * encode, split, per-tenant decode (App. A.3), with MLP heads run forward
 * only.  Creation validates everything, carves `ws` (caller-owned device
 * memory, jn_infer_workspace_size bytes, 256-byte aligned) and uploads every
 * index map and head descriptor once.  A launch then enqueues kernels only --
 * pack, backbone, pool, head forward -- reading the requests' `embeds`
 * buffers as they are at that time and writing actions[g] (device fp32
 * [n_g][action_dim * chunk], rows in tenant g's arrival order).  Because a
 * launch allocates, copies and synchronizes nothing, it can be recorded into
 * a HIP graph (jn_infer_plan_capture) and replayed with new observations
 * written into the same `embeds` buffers.  The plan keeps the device
 * pointers it was given (embeds, weights, actions, ws): they must stay valid
 * until jn_infer_plan_destroy.  Error statuses enqueue nothing. */
typedef struct jn_infer_plan jn_infer_plan;
jn_status jn_infer_workspace_size(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                                  const jn_pack_opts* opts, const jn_backbone* bb, const jn_head* heads,
                                  size_t* bytes);
jn_status jn_infer_plan_create(jn_ctx* ctx, const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                               const jn_pack_opts* opts, const jn_backbone* bb, const jn_head* heads,
                               float* const* actions, void* ws, size_t ws_bytes, jn_infer_plan** out);
/* The plan's physical batch (device pointers into ws) and its hidden rows
 * (device bf16 [T][d]), e.g. for jn_unpack. */
jn_status jn_infer_plan_packed(const jn_infer_plan* plan, jn_packed* out, void** hidden);
/* Enqueue one inference step on the context stream (kernels only). */
jn_status jn_infer_plan_launch(jn_ctx* ctx, const jn_infer_plan* plan);
/* Record one launch into a HIP graph on the context stream, which must not
 * be the null stream and must not have the launch trace enabled
 * (JN_EUNSUPPORTED); replaces a previously captured graph. */
jn_status jn_infer_plan_capture(jn_ctx* ctx, jn_infer_plan* plan);
/* Launch the captured graph on the context stream (JN_EINVAL if none). */
jn_status jn_infer_plan_replay(jn_ctx* ctx, const jn_infer_plan* plan);
void jn_infer_plan_destroy(jn_infer_plan* plan);

#ifdef __cplusplus
}
#endif
#endif
