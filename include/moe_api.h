/*
 * moe_api.h -- C ABI of the MI355X (gfx950) streaming-MoE decode hot path.
 *
 * One MoE layer does the following:
 * - routes a token: router logits, softmax, top-k (App. A, Softmax-topk);
 * - predicts the next layer's routing one token ahead with the prerouter head,
 *   and that prediction is then used as the routing (Sec. 3.2, Motivation and
 *   Prediction-as-routing);
 * - runs the selected int4 group-64 SwiGLU experts (Sec. 3.1, Math contract),
 *   each with the unmerged LoRA delta (alpha/r) B A v (Sec. 3.3, Fig. 1);
 * - combines the expert outputs with the routing weights.
 * Expert ids reach their weights through a device-resident slot table, so a
 * decode step never stacks weights (Sec. 3.1, Executor paths, "staged").
 *
 * Conventions for every call below:
 * - Plain C. Device pointers point to device memory, host pointers to host
 *   memory. `stream` is a hipStream_t passed as void* (NULL means the null stream).
 * - The caller owns every buffer passed in: inputs, outputs and workspaces.
 *   Only the slot-table object and its device table belong to the library.
 * - The hot-path calls (moe_rmsnorm_f16 through moe_topk) only enqueue work
 *   on `stream`. They never allocate, never synchronise the host, and are
 *   safe to capture in a HIP graph.
 * - Return value: MOE_OK (0) or a negative MOE_E* code. A failed argument
 *   check enqueues nothing.
 * - Alignment: device pointers must be 16-byte aligned, except the small
 *   int32/fp32 arrays idx, w, pred_idx, pred_w and the status word, which
 *   need 4 bytes (MOE_EALIGN otherwise).
 * - A kernel that meets an expert id outside [0, E) or a non-resident expert
 *   ORs a MOE_STATUS_* bit into the caller's status word. That expert then
 *   contributes zeros. The caller reads the status word after the step.
 * - Not thread-safe for concurrent calls on one slot table.
 */
#ifndef MOE_API_H
#define MOE_API_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes -------------------------------------------------------- */
#define MOE_OK            0
#define MOE_EINVAL       (-1)  /* bad spec, shape, NULL pointer or index     */
#define MOE_EALIGN       (-2)  /* device pointer not 16-byte aligned         */
#define MOE_ENOTRESIDENT (-3)  /* host-visible lookup of an unbound expert   */
#define MOE_EHIP         (-4)  /* a HIP runtime call or kernel launch failed */
#define MOE_ENOMEM       (-5)  /* workspace too small / allocation failed    */

/* ---- device status bits (OR-ed into *status_dev by the kernels) ---------- */
#define MOE_STATUS_SLOT_MISS 1u  /* routed expert has no resident slot       */
#define MOE_STATUS_BAD_INDEX 2u  /* expert id outside [0, E)                  */
#define MOE_STATUS_ENGINE_ABORT 4u /* decode engine left a wait on its time limit,
                                      or ran on an unexpected CU/XCD layout     */

/* ---- layer description (the MoESpec of Sec. 3) --------------------------- */
#define MOE_ROUTING_SOFTMAX_TOPK 0   /* App. A, Softmax-topk                    */
#define MOE_ROUTING_SIGMOID_GROUP 1  /* App. A, Sigmoid-group (moe_topk, moe_route,
                                        moe_preroute, moe_preroute_mlp, and the
                                        two-half schedule of moe_engine_chain;
                                        the whole-chip engines take softmax-topk
                                        only)                                   */

typedef struct moe_layer_spec {
  int32_t d_model;     /* hidden size d; multiple of 64, <= 8192             */
  int32_t n_experts;   /* routed experts E; 1..1024                          */
  int32_t top_k;       /* K; 1..min(E, 32)                                   */
  int32_t n_shared;    /* always-on shared experts S (weight 1.0); 0..4      */
  int32_t d_expert;    /* expert intermediate size I; multiple of 64, <= 8192 */
  int32_t group_size;  /* int4 quantization group; must be 64                */
  int32_t lora_rank;   /* r; 0 (no adapters) or 1..64                        */
  float   lora_scale;  /* alpha / r, the LoRA delta multiplier (Sec. 3.3)    */
  int32_t routing;     /* MOE_ROUTING_*                                      */
  int32_t n_groups;    /* sigmoid-group: groups n, E % n == 0, E <= 256; else 0 */
  int32_t top_groups;  /* sigmoid-group: surviving groups G, 1..n, K <= G E / n;
                          else 0                                             */
  float   route_scale; /* sigmoid-group: weight scale s > 0; else 0           */
  int32_t reserved[4]; /* must be zero                                       */
} moe_layer_spec;

/*
 * One int4 group-64 projection W [out x in] of an expert, in device memory
 * (Sec. 2, Quantization; Sec. 3.1, Executor paths: the three quantized
 * projections, each with its scales and biases):
 *   q      uint8 [out][in/2]. Row-major packed codes; byte j of a row holds
 *          input 2j in the low nibble and input 2j+1 in the high nibble.
 *   sz     fp16 pairs [out][in/64][2] = (scale s, zero z) of each 64-input group.
 *          The weight is w = s * q + z.
 *   lora_a fp16 [r][in] or NULL  (LoRA down-projection A)
 *   lora_b fp16 [out][r] or NULL (LoRA up-projection B); the delta is
 *          lora_scale * B (A v), applied only when both are non-NULL.
 */
typedef struct moe_proj {
  const void* q;
  const void* sz;
  const void* lora_a;
  const void* lora_b;
} moe_proj;

/* One expert: gate and up are [I x d], down is [d x I]. */
typedef struct moe_bundle {
  moe_proj gate, up, down;
} moe_bundle;

/* Check a spec. Returns MOE_OK or MOE_EINVAL. Host only. */
int moe_spec_check(const moe_layer_spec* spec);

/* Human-readable text of an error code. Static storage. */
const char* moe_strerror(int code);

/* ---- slot table (Sec. 3.1, Executor paths, "staged": routing indices map
 *      through a slot table and never leave the device) -------------------- */
typedef struct moe_slot_table moe_slot_table;

/*
 * Create a table for n_layers layers. Each layer has n_ids expert ids
 * (E routed ids first, then the S shared ids E .. E+S-1) and n_slots slots.
 * Only host memory is allocated here. The device copy is allocated by the
 * first moe_slot_table_sync. Destroy the table with moe_slot_table_destroy.
 */
int moe_slot_table_create(int n_layers, int n_ids, int n_slots, moe_slot_table** out);
int moe_slot_table_destroy(moe_slot_table* t);

/*
 * Bind expert `expert` of `layer` to `slot`, whose weights are *bundle (the
 * table copies the pointers). If the slot held another expert, that expert
 * becomes unbound. If `expert` was in another slot, that slot becomes free.
 * Host mirror only: call moe_slot_table_sync to publish.
 */
int moe_slot_bind(moe_slot_table* t, int layer, int expert, int slot, const moe_bundle* bundle);
/* Mark `expert` of `layer` as not resident (host mirror). */
int moe_slot_unbind(moe_slot_table* t, int layer, int expert);
/* Slot of `expert` in `layer` from the host mirror, or MOE_ENOTRESIDENT. */
int moe_slot_lookup(const moe_slot_table* t, int layer, int expert);
/*
 * Push the host mirror to the device copy with async copies on `stream`
 * (the first call allocates the device copy). The mirror is staged in a
 * library-owned pinned buffer, so the host may change it right after return.
 */
int moe_slot_table_sync(moe_slot_table* t, void* stream);

/* ---- hot path ------------------------------------------------------------ */

/*
 * Layer input: x[t] = fp16(xi[t] / sqrt(mean(xi[t]^2) + 1e-6)) for T rows
 * of d fp32 values. The normalized value is computed in fp64 and rounded
 * once to fp16 (round-to-nearest-even).
 * xi: device fp32 [T][d]; x_f16: device fp16 [T][d].
 */
int moe_rmsnorm_f16(const float* xi, int T, int d, void* x_f16, void* stream);

/* Workspace bytes needed by moe_route / moe_preroute / moe_expert_ffn_int4_lora
 * for T tokens. The caller allocates it and zero-fills it once. The library
 * leaves its internal counters at zero after every call. Calls that share one
 * workspace must be ordered on one stream. */
size_t moe_workspace_bytes(const moe_layer_spec* spec, int T);

/*
 * Router (App. A, Softmax-topk): fp32 logits l = W x, then the K largest
 * logits in descending order (ties go to the lower expert id), with weights
 * w_i = exp(l_i - l_max) / sum over the selected j of exp(l_j - l_max).
 * x_f16: device fp16 [T][d]; w_router_f16: device fp16 [E][d].
 * logits_opt: device fp32 [T][E], or NULL if not needed.
 * idx: device int32 [T][K]; w: device fp32 [T][K].
 */
int moe_route(const moe_layer_spec* spec, const void* x_f16, const void* w_router_f16, int T,
              float* logits_opt, int32_t* idx, float* w, void* workspace, size_t workspace_bytes,
              void* stream);

/*
 * Prerouter (Sec. 3.2, Head and Prediction-as-routing): the head of layer N
 * runs on layer N's input at token t. Its output (same math as moe_route,
 * with the head weights [E_next][d]) is layer N+1's routing at token t+1.
 * `next` describes layer N+1.
 */
int moe_preroute(const moe_layer_spec* next, const void* x_f16, const void* w_head_f16, int T,
                 float* logits_opt, int32_t* pred_idx, float* pred_w, void* workspace,
                 size_t workspace_bytes, void* stream);

/*
 * Full prerouter head (Sec. 3.2, Head): fc1 -> erf-GELU -> fc2 plus a linear
 * residual path on the hidden state. The input feature of token t is
 *   f = [x_t (d), onehot(routed_t[t]) (E), onehot(routed_tm1[t]) (E)],
 * the experts this layer routed to at this token and at the previous one.
 *   hidden = fp16(gelu(W1 f + b1)),  gelu(z) = z (1 + erf(z / sqrt 2)) / 2
 *   l      = W2 hidden + b2 + W_l x_t          (fp32)
 * then the softmax-top-k of moe_route on l. The result is layer N+1's
 * routing at token t+1 (Prediction-as-routing). `next` describes layer N+1;
 * this layer's expert count and K are taken to be next's.
 * Layout (all fp16, device, 16-byte aligned):
 *   w1_x [H][d]   the columns of W1 that multiply x
 *   w1_r [2E][H]  the columns of W1 that multiply the one-hots, transposed:
 *                 row e for expert e at this token, row E + e at the previous
 *   b1 [H] (or NULL: zero), w2 [E][H], b2 [E] (or NULL), w_l [E][d] (or NULL)
 * H = `hidden`, a multiple of 8; d and E multiples of 8.
 * routed_t: device int32 [T][K]; routed_tm1: device int32 [T][K] or NULL (no
 * previous token: a zero one-hot). Ids outside [0, E) contribute nothing.
 * logits_opt: device fp32 [T][E] or NULL; pred_idx [T][K], pred_w [T][K].
 * workspace: moe_preroute_mlp_workspace_bytes(next, hidden, T) bytes of
 * device memory (no initial contents needed).
 */
typedef struct moe_head_mlp {
  int32_t hidden;
  const void* w1_x;
  const void* w1_r;
  const void* b1;
  const void* w2;
  const void* b2;
  const void* w_l;
} moe_head_mlp;
size_t moe_preroute_mlp_workspace_bytes(const moe_layer_spec* next, int hidden, int T);
int moe_preroute_mlp(const moe_layer_spec* next, const moe_head_mlp* head, const void* x_f16, int T,
                     const int32_t* routed_t, const int32_t* routed_tm1, float* logits_opt,
                     int32_t* pred_idx, float* pred_w, void* workspace, size_t workspace_bytes,
                     void* stream);

/*
 * Experts (Sec. 3.1, Math contract; Sec. 3.3): for every token t and every
 * list position k in [0, K+S):
 *   e = idx[t][k] for k < K, else E + (k - K)
 *   y_experts[t][k] = down(silu(g) * u), where
 *   g = W_gate x + s_L B_gate (A_gate x), u likewise, and down likewise on h.
 * Weights are found through `table` (layer `layer`). All arithmetic is fp32.
 * idx: device int32 [T][K], for example the prerouter's output.
 * y_experts: device fp32 [T][K+S][d]. status_dev: device uint32.
 */
int moe_expert_ffn_int4_lora(const moe_layer_spec* spec, const moe_slot_table* table, int layer,
                             const void* x_f16, int T, const int32_t* idx, float* y_experts,
                             uint32_t* status_dev, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * The same computation as moe_expert_ffn_int4_lora (same kernels, same
 * results bit for bit), for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation. There is no workspace argument: the intermediate values live in
 * a static device array of MOE_NOALLOC_SCRATCH_BYTES per GPU, which the library
 * holds until the process ends (its address on each device is looked up once,
 * at the first call on that device). The call allocates nothing and frees
 * nothing. A call whose workspace layout (moe_workspace_bytes(spec, T)) exceeds
 * the array returns MOE_ENOMEM before any work is enqueued. Every call on one
 * GPU shares that GPU's array: calls that overlap (other streams, other host
 * threads) race, so order them on one stream. Nothing in the array has to
 * start at zero: each call writes every value before it reads it.
 */
#define MOE_NOALLOC_SCRATCH_BYTES (4u << 20)
int moe_expert_ffn_int4_lora_noalloc(const moe_layer_spec* spec, const moe_slot_table* table,
                                     int layer, const void* x_f16, int T, const int32_t* idx,
                                     float* y_experts, uint32_t* status_dev, void* stream);

/*
 * Batched decode / prefill experts (Sec. 3.1, Executor paths: the whole-layer
 * path serves prefill; Math contract: every path gives the same outputs).
 * Same inputs, outputs and status behaviour as moe_expert_ffn_int4_lora, for
 * many tokens at once: the (token, expert) pairs are grouped by expert and
 * each group runs as a dense contraction on the matrix cores. The int4
 * weights are dequantized to fp16 (w = s q + z, rounded once), the token
 * activations are fp16, h = silu(g) u is rounded to fp16 between the two
 * contractions, and lora_scale * (A v) is rounded to fp16 for the LoRA-B
 * step; every sum accumulates in fp32.
 * Shapes: d and I multiples of 128, lora_rank <= 16, E + S <= 2048; other
 * specs give MOE_EINVAL. Uses the workspace of moe_workspace_bytes(spec, T).
 */
int moe_expert_ffn_grouped_int4_lora(const moe_layer_spec* spec, const moe_slot_table* table,
                                     int layer, const void* x_f16, int T, const int32_t* idx,
                                     float* y_experts, uint32_t* status_dev, void* workspace,
                                     size_t workspace_bytes, void* stream);

/*
 * Combine (Fig. 1 sum node): y[t] = sum_{k<K} w[t][k] y_experts[t][k]
 *                                  + sum_{s<S} y_experts[t][K+s].
 * y: device fp32 [T][d].
 */
int moe_combine(const moe_layer_spec* spec, const float* y_experts, const float* w, int T,
                float* y, void* stream);

/* As moe_combine, but adds into y_inout: y_inout[t] += (the combine of token t).
 * A decode chain uses it to add the layer output into the residual. */
int moe_combine_add(const moe_layer_spec* spec, const float* y_experts, const float* w, int T,
                    float* y_inout, void* stream);

/*
 * Top-k on given logits (App. A), by spec->routing: logits device fp32
 * [T][E] -> idx [T][K], w [T][K]. Same selection and weights as moe_route.
 * Softmax-topk: the K largest logits (descending, ties to the lower id),
 * w = softmax over the selected set. Sigmoid-group: sigma = sigmoid(l); a
 * group's score is the sum of its two largest sigma (groups are contiguous
 * runs of E / n ids); the G best groups survive (ties to the lower group);
 * the K largest sigma among the survivors are selected (descending, ties to
 * the lower id) and w = s sigma / (sum of the selected sigma + 1e-20).
 */
int moe_topk(const moe_layer_spec* spec, const float* logits, int T, int32_t* idx, float* w,
             void* stream);

/* Sigmoid-group top-k with a selection bias (App. A: selection uses the
 * biased score sigma + bias, the weights the raw sigma): bias device fp32 [E]
 * or NULL. MOE_EINVAL unless spec->routing is MOE_ROUTING_SIGMOID_GROUP. */
int moe_topk_biased(const moe_layer_spec* spec, const float* logits, const float* bias, int T,
                    int32_t* idx, float* w, void* stream);

/* ---- decode-chain stand-in for attention ---------------------------------
 * The paper's decoder runs attention before each MoE layer, and the head of
 * layer N reads layer N's post-attention norm output (Sec. 3.2, Motivation).
 * A multi-layer decode chain without attention uses these two O(d) steps on
 * an fp32 residual r [d] (one token), so that each layer's input depends on
 * every earlier layer and token:
 *   moe_chain_token_start: r = xi + rmsnorm(r)   (r = 0 before the first token)
 *   moe_chain_mix_rmsnorm: r = r + D * r[perm], then x = fp16(rmsnorm(r))
 * rmsnorm(v) = v / sqrt(mean(v^2) + 1e-6), computed in fp64. The residual
 * update of token_start is rounded once to fp32, and x is rounded once to
 * fp16. D: fp16 [d]. perm: int32 [d], a permutation of 0..d-1.
 * xi, r: fp32 [d]. x_f16: fp16 [d]. d <= 8192. */
int moe_chain_token_start(const float* xi, int d, float* r_inout, void* stream);
int moe_chain_mix_rmsnorm(const void* mix_d_f16, const int32_t* perm, int d, float* r_inout,
                          void* x_f16, void* stream);

/* ---- persistent decode engine -------------------------------------------
 * The same hot path (layer input, routing or prediction-as-routing, experts
 * with LoRA, combine, head prediction), but many single-token layer steps
 * run in ONE cooperative launch of 256 workgroups (one per CU; the work
 * split assumes 8 XCDs of 32 CUs). Workgroups exchange intermediate vectors
 * through the workspace, so no step pays a kernel launch. This amortises
 * the per-step graph and launch cost (the paper's engine spends 44 ms of
 * graph building per step, Sec. 6) down to device-side waits.
 *
 * Every wait is bounded. On a time limit the engine ORs
 * MOE_STATUS_ENGINE_ABORT into *status, sets a sticky abort word in the
 * workspace, and all workgroups return. After an abort, zero-fill the
 * workspace before the next call. Supported shapes: moe_engine_supported.
 * The workspace (moe_engine_workspace_bytes) must be zero-filled before its
 * first use. Consecutive calls on one workspace must be ordered on one stream.
 */
/* All four pointers are device addresses, 16-byte aligned (the engine stages
 * them into LDS with 16-byte loads). */
typedef struct moe_engine_layer {
  const void* router;      /* fp16 [E][d] (the layer's own router)              */
  const void* head;        /* fp16 [E][d] prerouter head, or NULL               */
  const void* mix_d;       /* chain only: fp16 [d] (see moe_chain_mix_rmsnorm)  */
  const int32_t* mix_perm; /* chain only: int32 [d]                             */
} moe_engine_layer;

/* MOE_OK if the engine handles this layer shape on this device, else MOE_EINVAL. */
int moe_engine_supported(const moe_layer_spec* spec);
/* Workspace bytes of the engine for chains of up to n_layers layers. */
size_t moe_engine_workspace_bytes(const moe_layer_spec* spec, int n_layers);

/*
 * Independent single-token steps. Step s reads table layer step_layer[s]
 * (a device int32 array). It computes x = fp16(rmsnorm(xi[s])), the layer's
 * own routing, the experts, the combine into y[s] (fp32 [d]), and the head's
 * prediction. layers: a device array indexed by table layer.
 * The *_rec arrays are optional device arrays [n_steps][K]: routing used and
 * head prediction.
 */
int moe_engine_layers(const moe_layer_spec* spec, const moe_slot_table* table,
                      const moe_engine_layer* layers, const int32_t* step_layer, int n_steps,
                      const float* xi, float* y, int32_t* idx_rec, float* w_rec,
                      int32_t* pidx_rec, float* pw_rec, uint32_t* status, void* workspace,
                      size_t workspace_bytes, void* stream);

/*
 * The same independent single-token steps and outputs as moe_engine_layers,
 * scheduled for throughput: the 256 workgroups form 16 teams of 16 (two per
 * XCD); team t runs its own steps s = t, t + 16, t + 32, ..., so sixteen
 * steps are in flight at once and the waits of one (exchanges, top-k, slot
 * lookups) overlap the weight streaming of the others. Every step is still one token through one layer
 * and reads its weights for that token alone; a step takes longer than under
 * moe_engine_layers, the sequence of steps less time. Results equal the
 * oracle's to the same tolerance as moe_engine_layers' (fp32 sums in another
 * order, so not bit-identical to it). Precision: h = silu(g) u is computed in
 * fp32 and rounded once to fp16 for the down projection (valid while
 * |h| < 65504; larger values become infinities), whose int4 codes meet it in
 * fp16 dot products with fp32 accumulation; moe_engine_layers keeps h in
 * fp32. Shapes: moe_engine_tokens_supported.
 * Same workspace (moe_engine_workspace_bytes) and ordering rules.
 */
int moe_engine_tokens_supported(const moe_layer_spec* spec);
int moe_engine_tokens(const moe_layer_spec* spec, const moe_slot_table* table,
                      const moe_engine_layer* layers, const int32_t* step_layer, int n_steps,
                      const float* xi, float* y, int32_t* idx_rec, float* w_rec,
                      int32_t* pidx_rec, float* pw_rec, uint32_t* status, void* workspace,
                      size_t workspace_bytes, void* stream);

/*
 * Decode chain (Sec. 3.2): n_tokens tokens, numbered first_token .. , each
 * through the n_layers layers held at table layers 0..n_layers-1, on the
 * residual r_state (device fp32 [d], in/out; zero before the first token):
 *   r = xi[t] + rmsnorm(r) at the start of each token, then per layer N:
 *   r = r + D_N * r[perm_N];  x = fp16(rmsnorm(r));  r = r + layer_N(x).
 * Layer 0 and every layer of token 0 route by their own router. Layer N >= 1
 * at token t >= 1 routes by the prediction that the head of layer N-1 made at
 * token t-1. The predictions persist in the workspace between calls.
 * Optional records (device, [n_tokens*n_layers] rows in token-major order):
 * x_rec fp16 [.][d] (the layer input), r_rec fp32 [.][d] (the residual after
 * the mixing, before the layer output is added), idx_rec / w_rec (the
 * routing used) and pidx_rec / pw_rec (the head's prediction) [.][K],
 * y_rec fp32 [.][d] (the layer output).
 * Schedule: on a 256-CU device, for the layer shapes the two-half schedule
 * is compiled for (d 2048 / I 512 / r 16 with K + S <= 9 and E <= 256;
 * d 512 / I 256 / r 8 with K + S <= 2 and E <= 16; d 4096 / I 1024 / r 16
 * with K + S <= 4 and E <= 64, the 8B tier's layer; the K + S experts' rows
 * splitting evenly over its 128 workgroups), layer steps alternate between
 * two halves of the chip (even and odd XCDs): one half computes a layer
 * while the other loads the experts of its next layer, known a token ahead
 * from the prediction. There h = silu(g) u is rounded once to fp16 (valid while
 * |h| < 65504) for the down projection and the down adapter's A product, and
 * both the own router and the head select by spec->routing (softmax-topk or
 * sigmoid-group). Other shapes run the whole-chip engine of moe_engine_layers
 * (h in fp32; softmax-topk only); moe_engine_chain_supported says whether
 * either takes a spec.
 */
/* MOE_OK if moe_engine_chain runs this layer shape on this device (on the
 * two-half schedule or on the whole-chip engine), else MOE_EINVAL. */
int moe_engine_chain_supported(const moe_layer_spec* spec);
int moe_engine_chain(const moe_layer_spec* spec, const moe_slot_table* table,
                     const moe_engine_layer* layers, int n_layers, int first_token, int n_tokens,
                     const float* xi, float* r_state, void* x_rec, float* r_rec, int32_t* idx_rec,
                     float* w_rec, int32_t* pidx_rec, float* pw_rec, float* y_rec, uint32_t* status,
                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * The decode chain of moe_engine_chain with the full prerouter head (Sec. 3.2,
 * Head, Feature drift) as every layer's head: head n (n < n_layers - 1) is
 * heads[n], a DEVICE array of n_layers moe_head_mlp (entry n_layers - 1 is not
 * read; layers[n].head is not read), every one with this hidden size. Its
 * features are x of layer n, the routing layer n used at this token and the
 * routing it used at the last token (none at token 0; from the previous call
 * at first_token > 0, so every call of one chain must use this entry): the
 * same as moe_preroute_mlp's, here fed the chain's own routing (which is the
 * head's earlier prediction from layer 1 on: the feature drift the paper
 * describes). fc1 is computed in fp32 from x and the gathered one-hot columns,
 * erf-GELU, rounded once to fp16; fc2, its bias and the linear path add up in
 * fp32. Runs on the two-half schedule only: softmax-topk routing, d <= 2048
 * (the 35B-class and tiny shapes; the fc1 and fc2 rows of a workgroup are held
 * in LDS), hidden a multiple of 64 in [64, 512]; MOE_EINVAL otherwise
 * (moe_engine_chain_mlp_supported). heads must be 16-byte aligned (MOE_EALIGN).
 * The workspace is moe_engine_workspace_bytes(spec, n_layers); the prediction
 * and routing words persist in it between the calls of a chain.
 */
int moe_engine_chain_mlp_supported(const moe_layer_spec* spec, int hidden);
int moe_engine_chain_mlp(const moe_layer_spec* spec, const moe_slot_table* table,
                         const moe_engine_layer* layers, const moe_head_mlp* heads, int hidden, int n_layers,
                         int first_token, int n_tokens, const float* xi, float* r_state, void* x_rec,
                         float* r_rec, int32_t* idx_rec, float* w_rec, int32_t* pidx_rec, float* pw_rec,
                         float* y_rec, uint32_t* status, void* workspace, size_t workspace_bytes, void* stream);

/* ---- host-tier staging -----------------------------------------------------
 * The staged executor keeps a fixed set of device slots per layer and rewrites
 * only the slots whose expert changed (Sec. 3.1, Executor paths); head N's
 * prediction for layer N+1 at token t+1 lets that rewrite start a token early
 * (Sec. 3.2, Motivation).  Reading of the slot policy (the paper leaves it
 * open): every layer keeps a FIFO of staged-but-unused expert sets and a FIFO
 * of sets in use.  Staging a set walks it in routing order; a resident expert
 * costs nothing; a missing one takes the lowest free slot, else the slot with
 * the oldest last use among the slots that are not pinned, ties to the lowest
 * slot id.  Pinned: the slots of the set being staged, of every set still
 * queued for the layer and of every set in use.  A clock that advances on
 * every copy and every use orders "last use".  Using a set (in FIFO order; it
 * must equal the oldest staged set) moves it to the in-use FIFO; releasing the
 * layer (its kernels on that set finished) unpins the oldest set in use.
 */
typedef struct moe_slot_policy moe_slot_policy;
int moe_slot_policy_create(int n_layers, int n_ids, int n_slots, moe_slot_policy** out);
int moe_slot_policy_destroy(moe_slot_policy* p);
/* experts: host int32 [n], distinct ids in [0, n_ids). copies: host int32
 * [n][2] or NULL, filled with (expert, slot) in issue order. Returns the
 * number of copies, MOE_EINVAL (bad set), or MOE_ENOMEM (not enough unpinned
 * slots; the policy is unchanged). */
int moe_slot_policy_stage(moe_slot_policy* p, int layer, const int32_t* experts, int n,
                          int32_t* copies);
/* Consumes the oldest staged set of `layer`, which must equal experts[0..n).
 * slots: host int32 [n] or NULL. MOE_EINVAL if the set is not the oldest. */
int moe_slot_policy_use(moe_slot_policy* p, int layer, const int32_t* experts, int n,
                        int32_t* slots);
/* The layer finished with its oldest set in use. MOE_EINVAL if none. */
int moe_slot_policy_release(moe_slot_policy* p, int layer);
/* Slot of (layer, expert), or MOE_ENOTRESIDENT. */
int moe_slot_policy_lookup(const moe_slot_policy* p, int layer, int expert);

/* Byte offsets of the tensors of one packed bundle (16-byte aligned), in the
 * order q, sz, lora_a, lora_b of gate, up and down; -1 for absent LoRA. */
typedef struct moe_bundle_layout {
  int64_t gate[4], up[4], down[4];
} moe_bundle_layout;

typedef struct moe_stager_stats {
  int64_t stages, uses, copies, bytes;
} moe_stager_stats;

/*
 * The policy above driving a slot table: the experts of every layer are packed
 * bundles of bundle_bytes bytes in caller-owned PINNED host memory
 * (host_bundles: [n_layers][n_ids] pointers), and the device slots are a
 * caller-owned pool [n_layers][n_slots] of slot_stride bytes (256-aligned).
 * The stager owns every binding of `table` (it starts empty; the table must
 * have been synced once so that its device copy exists).
 */
typedef struct moe_stager moe_stager;
int moe_stager_create(moe_slot_table* table, const moe_bundle_layout* layout, size_t bundle_bytes,
                      const void* const* host_bundles, void* slot_pool, size_t slot_stride,
                      moe_stager** out);
/*
 * The same stager with the bundles in a file instead of pinned memory (the
 * SSD tier of Sec. 3.1, SSD streaming: per-layer stacked weights read through
 * the OS page cache). The file at `path` holds [n_layers][n_ids] records of
 * file_stride bytes (>= bundle_bytes); record (layer, e) is the packed bundle
 * of expert e, in the same layout as a pinned host bundle. It is mapped
 * read-only for the stager's lifetime and must not change meanwhile. The
 * stager's own I/O thread takes the staged sets in order: each copy reads its
 * record into one of n_bounce (1..16) pinned bounce buffers, split over n_io
 * (1..16) host threads (page faults read the file, or hit the page cache),
 * then enqueues the host -> slot copy on the set's copy_stream; a bounce
 * buffer is reused after the copy from it has completed. moe_stager_stage
 * returns once the set is queued; moe_stager_use blocks the calling thread
 * until the set's copies are enqueued. The stager uses the device that was
 * current at creation. MOE_EINVAL: a bad argument, a file that cannot be
 * opened or is shorter than n_layers * n_ids * file_stride; MOE_ENOMEM: the
 * mapping, the bounce buffers or the thread failed.
 */
int moe_stager_create_file(moe_slot_table* table, const moe_bundle_layout* layout,
                           size_t bundle_bytes, const char* path, size_t file_stride, int n_bounce,
                           int n_io, void* slot_pool, size_t slot_stride, moe_stager** out);
int moe_stager_destroy(moe_stager* s);
/* Stages a set (policy stage), rewrites the layer's slot-table rows on the
 * device and copies each missing bundle host -> slot, all enqueued on
 * copy_stream (for the file tier, the copies by the I/O thread). Returns the
 * number of copies (copies as in the policy) or an error. A kernel may read a
 * slot only between the use and the release of a set that holds it, so
 * unpinned slots are free to overwrite. If a copy cannot be enqueued after the
 * policy took the set, the slots no longer hold what the table says: the
 * stager is then failed, and this and every later stage and use return
 * MOE_EHIP. */
int moe_stager_stage(moe_stager* s, int layer, const int32_t* experts, int n, void* copy_stream,
                     int32_t* copies);
/* Uses the oldest staged set of the layer: compute_stream waits for that
 * set's copies (no wait when it needed none). slots: host int32 [n] or NULL. */
int moe_stager_use(moe_stager* s, int layer, const int32_t* experts, int n, void* compute_stream,
                   int32_t* slots);
/* The kernels that read the layer's oldest set in use have finished (the host
 * knows it, e.g. from an event recorded after them): unpin that set. */
int moe_stager_release(moe_stager* s, int layer);
int moe_stager_stats_get(const moe_stager* s, moe_stager_stats* out);
/* File tier: host time spent reading records into bounce buffers (ns) and the
 * bytes read; both 0 for a pinned-memory stager. */
int moe_stager_io_stats(const moe_stager* s, int64_t* read_ns, int64_t* read_bytes);

/* ---- an adapter merged into the int4 weights (Sec. 3.3, Recovery LoRA:
 *      the merged alternative, kept to measure what merging loses) -------- */

/*
 * Fold the adapter of `src` into its weights and re-quantize to int4 g64,
 * the alternative to the unmerged delta that Sec. 3.3 rejects because most
 * of a small delta falls below the group step. Per 64-input group:
 *   w = s q + z and delta = lora_scale * (B A)[o][i] in float64,
 *   m = fp32(w + delta) (one rounding), lo / hi = the group's min / max of m,
 *   s' = fp16((hi - lo) / 15), z' = fp16(lo),
 *   q' = clamp(rint((m - z') / s'), 0, 15) in fp32 (0 when s' == 0);
 * the same quantizer as the format's (Sec. 2, Quantization).
 *   src       device projection [out_dim x in_dim] (moe_proj layout); with
 *             lora_a or lora_b NULL, delta = 0 (a plain re-quantization)
 *   rank      r of src's adapter (1..64), ignored without an adapter
 *   q_out     device uint8 [out_dim][in_dim/2], sz_out device fp16 pairs
 *             [out_dim][in_dim/64][2] (the moe_proj layout), caller-owned;
 *             must not overlap src
 *   stats     device double [out_dim][in_dim/64][2] or NULL: per group the sums
 *             of actual * delta and of delta^2, actual = (s' q' + z') - w; their
 *             totals give the weight-level retention sum(actual delta) / sum(delta^2)
 * Asynchronous on `stream`; nothing is allocated. MOE_EINVAL: NULL src, src->q,
 * src->sz, q_out or sz_out, out_dim < 1, in_dim < 64, in_dim % 64 != 0, or an
 * adapter with rank outside 1..64; MOE_EALIGN: sz, sz_out, lora_a, lora_b not
 * 2-byte aligned or stats not 8-byte aligned.
 */
int moe_merge_requantize(const moe_proj* src, int out_dim, int in_dim, int rank, float lora_scale,
                         void* q_out, void* sz_out, double* stats, void* stream);

/* ---- profiling (not part of the hot path) ------------------------------- */
#define MOE_PROF_FFN_MAIN 0  /* the expert kernel that streams the gate/up weights */
#define MOE_PROF_ENGINE_PHASES 1 /* the next decode-engine launch writes, for
                                    three workgroups of every step (0, 7 and 255
                                    of the launch; in the two-half decode chain
                                    0, 7 and 127 of the half that runs the step),
                                    the device wall clock (wall_clock64) at 24
                                    marks of the step into start_event, read as
                                    a device uint64 array [n_steps][3][24];
                                    stop_event is unused */

/*
 * Arm per-launch timing. For MOE_PROF_FFN_MAIN, the next launch of that
 * kernel on the calling host thread records `start_event` when the kernel
 * starts executing and `stop_event` when it ends (hipEvent_t values created
 * with timing enabled). For MOE_PROF_ENGINE_PHASES see above.
 * The hook then disarms itself. Do not arm it during graph capture.
 * Returns MOE_EINVAL for an unknown `which` or NULL events.
 */
int moe_profile_arm(int which, void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif
#endif /* MOE_API_H */
