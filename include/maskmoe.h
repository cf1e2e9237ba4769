/*
 * maskmoe.h -- C ABI of the masked co-adaptive MoE hot path on AMD Instinct MI355X (gfx950).
 *
 * The library computes, on one GPU, the masked-routing mixture-of-experts layer of
 * MaskCoFT (Masked Co-Adaptive Fine-Tuning): router logits and softmax, Top-K routing
 * under a hard binary expert mask (training, Section 3.2 Stage 1, Eq. 2) or a soft
 * re-ranking prior (inference, Section 3.2 "Evaluation and inference", Eq. 4), gate
 * values from the full softmax (Section 3.1, Eq. 1), the SwiGLU expert FFNs, the
 * gate-weighted combine with shared experts (Section 3.1), and the per-layer expert
 * cache simulation behind the paper's hit rate and fetches-per-token metrics
 * (Section 4.1, Eq. 5).
 *
 * Conventions shared by every entry point
 *  - Every pointer marked "device" must point to device memory of the current HIP device;
 *    pointers marked "host" are read synchronously during the call and not kept.
 *  - The caller owns every buffer. The library allocates no device memory, keeps no global
 *    state and is reentrant, with two exceptions: maskmoe_layer_forward_noalloc uses a device
 *    array of the library (one per device) and remembers its address per device, and
 *    maskmoe_layer_backward creates one extra stream per device on first use (kept until the
 *    process ends) for the zero gradients of unchosen experts, ordered with `stream` by
 *    events created and released per call. All work is enqueued asynchronously on `stream`
 *    (0 = the null stream); nothing is synchronised. Outputs are valid once the stream
 *    reaches that point.
 *  - Every argument is validated before anything is enqueued: a non-zero status means that
 *    nothing was written. MASKMOE_E_HIP reports a failed launch (work enqueued before the
 *    failing launch may still run).
 *  - Tensors are dense and row-major in the shapes given. bf16 tensors hold IEEE bfloat16
 *    bit patterns; arithmetic accumulates in fp32.
 *  - Results are deterministic: no atomics feed any output, so a repeated call on the same
 *    inputs gives bit-identical outputs.
 */
#ifndef MASKMOE_H_
#define MASKMOE_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes (returned, never thrown) ---- */
enum {
  MASKMOE_OK = 0,
  MASKMOE_E_INVAL = 1,        /* an argument is outside its documented range; nothing enqueued */
  MASKMOE_E_WORKSPACE = 2,    /* workspace NULL or smaller than maskmoe_layer_workspace_bytes() */
  MASKMOE_E_HIP = 3,          /* a HIP launch or runtime call failed */
  MASKMOE_E_UNSUPPORTED = 4   /* valid arguments outside what the kernels implement */
};

/* ---- routing rule (which keys Top-K ranks) ----
 * PLAIN:      A = Top-K(p)                      Section 3.1, Eq. 1
 * HARD_MASK:  A = Top-K(p * m), m binary        Section 3.2 Stage 1, Eq. 2 (training)
 * SOFT_PRIOR: A = Top-K(p * pi), pi > 0         Section 3.2 inference, Eq. 4
 * where p = softmax(W x) over all E routed experts. Ranking is done on log-domain keys
 * (z_i, or z_i + log pi_i; experts with m_i = 0 are never eligible), which order experts
 * exactly as the products do. Equal keys go to the lower expert index. */
enum { MASKMOE_ROUTE_PLAIN = 0, MASKMOE_ROUTE_HARD_MASK = 1, MASKMOE_ROUTE_SOFT_PRIOR = 2 };

/* ---- gate rule (Section 3.1); gates always come from the full softmax p, in every
 * routing mode (Eq. 2 gates equal those of p on the active set; Eq. 4 keeps p's gates) ----
 * GATE_P:      g_i = p_i                          (DeepSeek-V2-Lite)
 * GATE_RENORM: g_i = p_i / sum_{j in A} p_j       (Mixtral-8x7B)                     */
enum { MASKMOE_GATE_P = 0, MASKMOE_GATE_RENORM = 1 };

/* ---- element type of x, router weights, expert weights and y ---- */
enum { MASKMOE_BF16 = 0, MASKMOE_F32 = 1 };

/* ---- storage order of the expert weights (w_gate_up, w_down, ws_gate_up, ws_down) ----
 * LAYOUT_ROWS:   row-major, as documented at each entry point.
 * LAYOUT_PACKED: bf16 only, written by maskmoe_pack_expert_weights. Same size and the same
 *   values per expert, stored in 16 KiB blocks of 128 rows x 64 columns, so that the expert
 *   kernels read each weight block as one contiguous stream instead of 128-byte pieces of
 *   128 different rows (measured on MI355X: ~10% more HBM bandwidth for the few-token
 *   weight stream). The router weights are never packed.                              */
enum { MASKMOE_LAYOUT_ROWS = 0, MASKMOE_LAYOUT_PACKED = 1 };

/* ---- cache replacement policy of maskmoe_cache_fetches (Section 4.1, Table 2) ---- */
enum { MASKMOE_CACHE_LRU = 0, MASKMOE_CACHE_LFU = 1, MASKMOE_CACHE_FIFO = 2 };

/* One masked MoE layer.
 *  T          tokens (T >= 0; T = 0 is a no-op)
 *  d          hidden size; F expert FFN width
 *  E          routed experts, 1 <= E <= 256; K experts per token, 1 <= K <= E, K <= 16
 *  n_shared   shared experts (0..8): see every token, gate 1, never routed or masked
 *  dtype      MASKMOE_BF16 or MASKMOE_F32
 *  route_mode MASKMOE_ROUTE_*; gate_mode MASKMOE_GATE_*
 *  weight_layout MASKMOE_LAYOUT_*: order of the expert weights. LAYOUT_PACKED needs bf16,
 *             d % 128 == 0 and F % 64 == 0 (else E_UNSUPPORTED) and is taken by the inference
 *             entry points (maskmoe_layer_forward, _profiled, _lora, maskmoe_offload_decode_step);
 *             the training and backward entry points return E_UNSUPPORTED for it.
 *             maskmoe_route ignores it. */
typedef struct maskmoe_layer_desc {
  int32_t T, d, E, K, F, n_shared, dtype, route_mode, gate_mode, weight_layout;
} maskmoe_layer_desc;

/*
 * maskmoe_pack_expert_weights -- rewrites n experts' weights from LAYOUT_ROWS into
 * LAYOUT_PACKED (a one-time conversion of static parameters, like loading them):
 *   gate/up, expert e, group q = 0 .. F/64-1 (W_gate rows 64q .. 64q+63, then the matching
 *     W_up rows F+64q ..), chunk c = 0 .. d/64-1:
 *       packed[e][q][c][i][j] = w_gate_up[e][row_i][64c + j], i < 128, j < 64,
 *       row_i = 64q + i for i < 64, F + 64q + i - 64 otherwise;
 *   down, expert e, group q = 0 .. d/128-1, chunk c = 0 .. F/64-1:
 *       packed[e][q][c][i][j] = w_down[e][128q + i][64c + j].
 *  desc         d, F and dtype are used (dtype must be MASKMOE_BF16; d % 128 == 0,
 *               F % 64 == 0); the other fields are ignored.
 *  n            experts in each array (n >= 0; 0 is a no-op).
 *  w_gate_up    device [n, 2F, d] bf16 source, packed_gate_up device destination of the
 *               same size; both NULL to skip. w_down / packed_down likewise ([n, d, F]).
 *  The destinations must not overlap the sources. Asynchronous on `stream`.
 *  Errors: E_INVAL for d < 1, F < 1, n < 0, a source without its destination (or the
 *  reverse), a destination equal to its source, or pointers not 16-byte aligned;
 *  E_UNSUPPORTED for f32 or for d, F not multiples of 128 and 64.
 */
int maskmoe_pack_expert_weights(const maskmoe_layer_desc* desc, int32_t n, const void* w_gate_up,
                                const void* w_down, void* packed_gate_up, void* packed_down,
                                hipStream_t stream);

/*
 * maskmoe_route -- router logits, softmax, masked / prior-re-ranked Top-K and gates for
 * L independent layers that read the same tokens (Section 3.1 Eq. 1; Eq. 2; Eq. 4).
 *
 *  desc        T, d, E, K, dtype, route_mode, gate_mode are used (F, n_shared ignored).
 *  L           number of layers, L >= 1.
 *  x           device [T, d] tokens (dtype).
 *  w_router    device [L, E, d] router weights W_l (dtype), no bias.
 *  mask        host [L, E] uint8, HARD_MASK only (else ignored, may be NULL): 1 keeps the
 *              expert; each layer must keep at least K experts.
 *  prior       host [L, E] float, SOFT_PRIOR only (else ignored, may be NULL): every value
 *              finite and > 0 (the prior excludes no expert).
 *  topk_idx    device [L, T, K] int32: selected experts of token t at layer l, by decreasing
 *              key, ties by increasing index.
 *  topk_gate   device [L, T, K] float: gate of each selected expert (gate_mode).
 *  topk_margin device [L, T] float or NULL: gap in logit units between the K-th and the
 *              (K+1)-th largest log-domain key (+inf when fewer than K+1 experts are
 *              eligible). Index sets are unique wherever the margin is clearly positive.
 *  workspace   device buffer of at least maskmoe_route_workspace_bytes(desc, L) bytes,
 *              16-byte aligned, owned by the caller, or NULL. Given, many-token launches
 *              write the router logits there first and select in a second kernel (faster
 *              when the selection would otherwise run at the logit GEMM's occupancy); NULL
 *              selects inside the logit kernel. Both give bit-identical outputs. Its
 *              contents on entry are irrelevant; calls that may overlap must not share it.
 *  workspace_bytes  size of workspace in bytes (ignored when workspace is NULL).
 *  Errors: E_INVAL for T < 0, L < 1, d < 1, K/E outside their ranges, an unknown mode, a
 *  NULL required pointer, a mask row with fewer than K ones, a prior value that is not
 *  finite and > 0, or a workspace that is too small or misaligned; E_UNSUPPORTED for bf16
 *  with d % 32 != 0.
 */
int maskmoe_route(const maskmoe_layer_desc* desc, int32_t L, const void* x, const void* w_router,
                  const uint8_t* mask, const float* prior, int32_t* topk_idx, float* topk_gate,
                  float* topk_margin, void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * maskmoe_route_workspace_bytes -- workspace that maskmoe_route uses for `desc` and L layers
 * (fp32 [L, T, E] router logits when the launch splits logits and selection; 0 when it never
 * does, e.g. fp32 inputs, fewer than 512 tokens or more than 64 experts). Returns 0 for an
 * invalid desc or L < 1.
 */
size_t maskmoe_route_workspace_bytes(const maskmoe_layer_desc* desc, int32_t L);

/*
 * maskmoe_layer_workspace_bytes -- device workspace that maskmoe_layer_forward needs for
 * `desc` (routing outputs, the expert permutation, the SwiGLU activations and the
 * per-(token, expert) FFN outputs). Returns 0 for an invalid desc. Monotone in T.
 */
size_t maskmoe_layer_workspace_bytes(const maskmoe_layer_desc* desc);

/*
 * maskmoe_layer_forward -- one masked MoE layer:
 *     y_t = sum_{i in A_t} g_{t,i} F_i(x_t) + sum_s F_s(x_t)          (Section 3.1, Eq. 1)
 * with A_t and g from maskmoe_route's rule (L = 1) and the SwiGLU expert
 *     F(x) = W_down (SiLU(W_gate x) * (W_up x)),  SiLU(u) = u / (1 + e^-u).
 *
 *  x            device [T, d] (dtype).
 *  w_router     device [E, d] (dtype).   mask / prior: host [E], as in maskmoe_route.
 *  w_gate_up    device [E, 2F, d] (dtype): rows 0..F-1 = W_gate, rows F..2F-1 = W_up.
 *  w_down       device [E, d, F] (dtype).
 *  ws_gate_up   device [n_shared, 2F, d], ws_down device [n_shared, d, F]; NULL when
 *               n_shared == 0. All four in desc->weight_layout order (packed: as written
 *               by maskmoe_pack_expert_weights); the results do not depend on the layout.
 *  y            device [T, d] (dtype) output.
 *  topk_idx     device [T, K] int32 or NULL; topk_gate device [T, K] float or NULL:
 *               when given, the routing decision is also written there.
 *  workspace    device, at least maskmoe_layer_workspace_bytes(desc) bytes, 256-byte
 *               aligned; its contents on entry do not matter and are clobbered.
 *  Rounding (bf16): fp32 accumulation; the SwiGLU activation is rounded to bf16 before the
 *  down projection; each expert's output is rounded to bf16 (the layer's dtype); the combine
 *  sums the gate-weighted expert outputs in fp32 and rounds once to bf16. f32: no
 *  intermediate rounding beyond fp32 arithmetic.
 *  Errors: as maskmoe_route, plus E_INVAL for F < 1 or n_shared outside 0..8 or a NULL
 *  shared-weight pointer with n_shared > 0; E_WORKSPACE when the workspace is too small;
 *  E_UNSUPPORTED for bf16 with d % 64 != 0 or F % 64 != 0, or with T*d, T*(K+n_shared)*F or
 *  2*F*d at or above 2^31 elements. weight_layout: E_INVAL for a value other than
 *  MASKMOE_LAYOUT_*, E_UNSUPPORTED for LAYOUT_PACKED with f32, d % 128 != 0 or F % 64 != 0.
 */
int maskmoe_layer_forward(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                          const uint8_t* mask, const float* prior, const void* w_gate_up,
                          const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                          int32_t* topk_idx, float* topk_gate, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/* Stages of maskmoe_layer_forward, in launch order. */
enum {
  MASKMOE_STAGE_ROUTE = 0,       /* router logits + masked / prior Top-K + gates        */
  MASKMOE_STAGE_PERMUTE = 1,     /* grouping of (token, slot) pairs by expert           */
  MASKMOE_STAGE_GATE_UP = 2,     /* H = SiLU(X W_gate^T) * (X W_up^T) per expert        */
  MASKMOE_STAGE_DOWN = 3,        /* O = H W_down^T per expert (few tokens: with combine) */
  MASKMOE_STAGE_COMBINE = 4,     /* y = sum_k g O + shared experts                      */
  MASKMOE_NUM_STAGES = 5
};

/*
 * maskmoe_layer_forward_noalloc -- maskmoe_layer_forward without a caller workspace, for
 * callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation). The workspace is a file-scope device array of the
 * library, MASKMOE_NOALLOC_SCRATCH_BYTES (128 MiB) per device, created when the library's code
 * is loaded onto a device and held until the process ends; its device address is looked up
 * once per device, on the first call made with that device current. The call allocates
 * nothing (no hipMalloc / hipFree, no allocating library routine).
 *
 *  Arguments, outputs, rounding and determinism are those of maskmoe_layer_forward, whose
 *  kernels it runs; the results are bit-identical to it. 128 MiB covers every desc with
 *  maskmoe_layer_workspace_bytes(desc) <= MASKMOE_NOALLOC_SCRATCH_BYTES, e.g. the bf16
 *  Mixtral-shaped layer (d = 4096, F = 14336, E = 8, K = 2) up to 400 tokens, which includes
 *  the decode batches.
 *  Shared state: every call on one GPU uses that GPU's single array and leaves its last
 *  contents there (nothing in it needs to start at zero). Calls that overlap on one GPU (on
 *  different streams, or from different threads without ordering) race on it and give
 *  undefined results; calls on different GPUs do not interact.
 *  Errors: those of maskmoe_layer_forward, except that E_WORKSPACE means that
 *  maskmoe_layer_workspace_bytes(desc) exceeds MASKMOE_NOALLOC_SCRATCH_BYTES; E_HIP when the
 *  array's device address cannot be obtained (nothing is enqueued then); E_UNSUPPORTED for a
 *  device ordinal >= 64.
 */
#define MASKMOE_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int maskmoe_layer_forward_noalloc(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                  const uint8_t* mask, const float* prior, const void* w_gate_up,
                                  const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                                  int32_t* topk_idx, float* topk_gate, hipStream_t stream);

/*
 * maskmoe_layer_forward_profiled -- maskmoe_layer_forward that also records caller-owned
 * HIP events on `stream`, for measuring each stage on the device timeline: events[0]
 * before the first launch and events[s + 1] after stage s (MASKMOE_STAGE_*). A stage that
 * a path fuses into the previous one (the permutation of the few-token path, done by the
 * routing kernel) gets its event right after that one; the few-token path's SwiGLU pass
 * over split gate/up partial sums is timed with the DOWN stage. `events` holds
 * MASKMOE_NUM_STAGES + 1 entries; a NULL entry is skipped, so a caller can bracket one
 * stage without adding event records elsewhere. Same computation, outputs and errors as
 * maskmoe_layer_forward; E_INVAL when `events` is NULL.
 */
int maskmoe_layer_forward_profiled(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                   const uint8_t* mask, const float* prior, const void* w_gate_up,
                                   const void* w_down, const void* ws_gate_up, const void* ws_down,
                                   void* y, int32_t* topk_idx, float* topk_gate, void* workspace,
                                   size_t workspace_bytes, hipEvent_t* events, hipStream_t stream);

/*
 * maskmoe_cache_fetches -- replay expert-selection traces through per-layer expert caches
 * (Section 4.1 "Simulation", its LRU / LFU / FIFO policies; metrics of Eq. 5).
 *
 * Each (layer l, stream s) pair is an independent cache of B routed experts that sees the
 * steps n = 0..N-1 of trace[l, s]. At a step, h = number of selected experts already
 * cached, f = misses (= K - h for a trace of K distinct valid experts); every miss is one
 * fetch and, in a full cache, one eviction. The hits are handled first, in ascending expert
 * index, then the misses are inserted in ascending expert index; each miss evicts one cached
 * expert not selected at this step:
 *   LRU  the least recently used one;
 *   FIFO the one inserted earliest (hits do not refresh it);
 *   LFU  the one with the fewest accesses so far in this stream (every selection counts, and
 *        counts survive eviction), ties to the least recently used.
 * Eq. 5 then gives HR = sum h / (N L K) and Fetches/tok = sum f / N (per stream).
 *
 *  trace       device [L, S, N, K] int32 expert ids. An id outside [0, E) or repeating an
 *              earlier id of the same step is skipped (neither hit nor miss) and flags
 *              *dev_error.
 *  L, S, N, K  sizes, L, S, N >= 0, 1 <= K <= E; E experts, 1 <= E <= 64;
 *              B cache slots, K <= B (B >= E never evicts); N * K + B < 2^24.
 *  policy      MASKMOE_CACHE_LRU, MASKMOE_CACHE_LFU or MASKMOE_CACHE_FIFO.
 *  state       device [L, S, B] int32 in/out or NULL. In: initial cache, oldest first (least
 *              recently used first for LRU and LFU, first inserted first for FIFO), -1 = empty
 *              slot (entries must be distinct ids in [0, E) or -1; bad entries are dropped and
 *              flag *dev_error). Out: final cache in the same form. NULL: every cache starts
 *              empty and the final state is not kept.
 *  counts      device [L, S, E] int32 in/out or NULL: LFU access counts per expert (ignored
 *              by LRU and FIFO). NULL: counts start at zero and are not kept.
 *  fetches     device [L, S] int64: sum of f over the N steps.
 *  hits        device [L, S] int64: sum of h over the N steps.
 *  f_per_step  device [L, S, N] uint8 or NULL: f at every step.
 *  dev_error   device int32 or NULL: set to 1 (never cleared) when a trace or state entry
 *              was skipped.
 *  Errors: E_INVAL for negative sizes, K < 1, K > E, B < K, an unknown policy, NULL
 *  required pointers; E_UNSUPPORTED for E > 64 or N * K + B >= 2^24.
 */
int maskmoe_cache_fetches(const int32_t* trace, int32_t L, int32_t S, int32_t N, int32_t K,
                          int32_t E, int32_t B, int32_t policy, int32_t* state, int32_t* counts,
                          int64_t* fetches, int64_t* hits, uint8_t* f_per_step, int32_t* dev_error,
                          hipStream_t stream);

/* ---- Stage 1 of fine-tuning (Section 3.2, Stage 1 and Mask optimization) ---- */

/*
 * maskmoe_sample_mask -- the binary masks of Eq. 2: for each of L layers, e_keep = E'
 * distinct experts drawn without replacement from pi = softmax(m~). Draw s takes, among the
 * experts not yet drawn and in increasing index order, the first whose running sum of pi
 * exceeds uniforms[s] times their total (all in double precision). Host function; nothing is
 * enqueued.
 *
 *  mask_logits host [L, E] float m~ (finite).
 *  uniforms    host [L, e_keep] double in [0, 1): the random draws, supplied by the caller.
 *  mask        host [L, E] uint8 output: exactly e_keep ones per layer.
 *  Errors: E_INVAL for L < 1, E outside 1..256, e_keep outside 1..E, a NULL pointer, a
 *  non-finite logit or a uniform outside [0, 1).
 */
int maskmoe_sample_mask(const float* mask_logits, const double* uniforms, int32_t L, int32_t E,
                        int32_t e_keep, uint8_t* mask);

/*
 * maskmoe_layer_forward_train -- maskmoe_layer_forward that also returns what the Stage 1
 * backward reads: the routing decision, the fp32 router logits and every selected expert's
 * output before gating (Section 3.1, Eq. 1: y_t = sum_k g_{t,k} F_{A_t[k]}(x_t) + shared).
 *
 *  topk_idx      device [T, K] int32, required.   topk_gate device [T, K] float, required.
 *  router_logits device [T, E] float, required: z = W x in fp32.
 *  expert_out    device [T, K, d] float, required, 16-byte aligned: F_{A_t[k]}(x_t) as the
 *                combine used it (for bf16 layers: from the bf16-rounded SwiGLU activation,
 *                and itself rounded to bf16, as in y).
 *  workspace     at least maskmoe_layer_train_workspace_bytes(desc) bytes; for bf16 layers it
 *                keeps what maskmoe_layer_backward reads (the permutation, the SwiGLU
 *                activations and the gate / up pre-activations, bf16).
 *  Other arguments, rounding and errors as maskmoe_layer_forward (whatever T, bf16 layers take
 *  the grouped-GEMM path), plus E_INVAL for a NULL output above when T > 0 and E_UNSUPPORTED for
 *  packed weights (LAYOUT_PACKED).
 */
int maskmoe_layer_forward_train(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                const uint8_t* mask, const float* prior, const void* w_gate_up,
                                const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                                int32_t* topk_idx, float* topk_gate, float* router_logits,
                                float* expert_out, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * maskmoe_layer_train_workspace_bytes -- device workspace that maskmoe_layer_forward_train needs
 * for `desc`: that of maskmoe_layer_forward plus, for bf16 layers, the gate / up pre-activations
 * [T (K + n_shared), 2F] that maskmoe_layer_backward reads. Returns 0 for an invalid desc.
 */
size_t maskmoe_layer_train_workspace_bytes(const maskmoe_layer_desc* desc);

/*
 * maskmoe_offload_workspace_bytes -- device workspace of maskmoe_offload_decode_step for `desc`
 * (that of maskmoe_layer_forward plus the step's fetch list). Returns 0 for an invalid desc.
 */
size_t maskmoe_offload_workspace_bytes(const maskmoe_layer_desc* desc);

/*
 * maskmoe_offload_decode_step -- one decode step of one layer, batch 1, with the routed experts
 * offloaded to host memory (Section 1 and Section 3.1: a layer keeps B experts in GPU memory and
 * every selected expert that is not cached is fetched over PCIe; Section 4.1: a full cache
 * evicts one expert per fetch under LRU, LFU or FIFO, with the rules of maskmoe_cache_fetches).
 * In stream order and without a host round trip it routes the token (as maskmoe_layer_forward),
 * applies the cache step to its selected experts, copies each fetched expert's weights from
 * host memory into its slot of the device pool, and computes y from the pool (Eq. 1; shared
 * experts stay resident).
 *
 *  desc          T = 1, bf16, E <= 64; d and F multiples of 64.
 *  host_w_gate_up, host_w_down: pinned host memory (hipHostMalloc or an allocator built on it),
 *                [E, 2F, d] and [E, d, F] bf16, 16-byte aligned; read by a kernel through its
 *                device mapping, so it must stay allocated until the step has run.
 *  B             slots of the pool, K <= B <= E.   policy: MASKMOE_CACHE_LRU, _LFU or _FIFO.
 *  slots_gate_up, slots_down: device [B, 2F, d] and [B, d, F] bf16, the pool.
 *  cache_state   device int32 [B + 2E], kept by the caller across the steps of a sequence:
 *                [0, B) the cached experts, least recently used (LRU, LFU) or first inserted
 *                (FIFO) first, -1 for empty slots (the state layout of maskmoe_cache_fetches);
 *                [B, B + E) the LFU access counts; [B + E, B + 2E) the pool slot of each expert,
 *                -1 when it is not cached. An empty cache is -1, 0, -1. A state that is not
 *                self-consistent (an expert twice or out of range, slots that collide, are out
 *                of range or belong to an uncached expert) sets *dev_error and is replaced by an
 *                empty cache before the step.
 *  y, topk_idx, topk_gate: as maskmoe_layer_forward (T = 1).
 *  counters      device int64 [2] or NULL: the step's fetches and hits are added to [0] and [1]
 *                (a plain read-modify-write: calls that may overlap, e.g. on different streams,
 *                must not share counters, and none may share a cache_state or a pool).
 *  dev_error     device int32 or NULL: set to 1 (never cleared) on an inconsistent state.
 *  workspace     maskmoe_offload_workspace_bytes(desc) bytes, 256-byte aligned.
 *  events        NULL, or 2 caller-created HIP events (entries may be NULL) recorded on `stream`
 *                right before and right after the host-to-pool copy, to time the transfer.
 *  Rounding: as the few-token path of maskmoe_layer_forward (y is bit-identical to a forward
 *  with the same experts resident).
 *  Errors: E_INVAL for NULL or misaligned required pointers, host copies that are not pinned
 *  host memory, B outside [K, E], an unknown policy, or a bad mask / prior; E_UNSUPPORTED for
 *  T != 1, f32, E > 64 or d, F not multiples of 64. Packed weights (desc->weight_layout):
 *  the host copies, the shared experts and hence the pool are all in the packed layout.
 */
int maskmoe_offload_decode_step(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                const uint8_t* mask, const float* prior, const void* host_w_gate_up,
                                const void* host_w_down, const void* ws_gate_up, const void* ws_down, int32_t B,
                                int32_t policy, void* slots_gate_up, void* slots_down, int32_t* cache_state,
                                void* y, int32_t* topk_idx, float* topk_gate, int64_t* counters,
                                int32_t* dev_error, void* workspace, size_t workspace_bytes,
                                hipEvent_t* events, hipStream_t stream);

/*
 * maskmoe_lora -- low-rank adapters of every expert (Stage 2 of the fine-tuning, Section 3.2;
 * rank 8 and alpha 16 in Appendix B, routed and shared experts alike). An adapted projection
 * W [out, in] computes W v + (alpha / rank) B (A v) with A [rank, in] and B [out, rank].
 * All matrices are device bf16, row-major, owned by the caller:
 *  a_gate_up  [E, 2 rank, d]: rows 0..rank-1 A of W_gate, rows rank..2 rank-1 A of W_up
 *             (16-byte aligned).
 *  b_gate_up  [E, 2F, rank]: rows 0..F-1 B of W_gate, rows F..2F-1 B of W_up.
 *  a_down     [E, rank, F] (16-byte aligned).   b_down [E, d, rank].
 *  as_gate_up, bs_gate_up, as_down, bs_down: the same for the n_shared shared experts
 *             ([n_shared, ...]); NULL when n_shared == 0.
 */
typedef struct maskmoe_lora {
  int32_t rank;
  float alpha;
  const void *a_gate_up, *b_gate_up, *a_down, *b_down;
  const void *as_gate_up, *bs_gate_up, *as_down, *bs_down;
} maskmoe_lora;

/*
 * maskmoe_layer_lora_workspace_bytes -- device workspace that maskmoe_layer_forward_lora needs
 * for `desc`: that of maskmoe_layer_forward plus the adapters' rank projections of every expert
 * row ([T (K + n_shared), 64] bf16, twice) and the scaled B matrices ([E + n_shared, 2F + d, 64]
 * bf16). Returns 0 for an invalid desc.
 */
size_t maskmoe_layer_lora_workspace_bytes(const maskmoe_layer_desc* desc);

/*
 * maskmoe_layer_forward_lora -- maskmoe_layer_forward with adapted experts (Section 3.2,
 * Stage 2): every routed and shared expert computes
 *   F(x) = W'_down (SiLU(W'_gate x) * (W'_up x)),  W' v = W v + (alpha / rank) B (A v).
 * Routing, gating and the combine are those of maskmoe_layer_forward (the router carries no
 * adapter).
 *
 *  lora       host pointer to the adapters; 1 <= rank <= 16, alpha finite.
 *  Other arguments as maskmoe_layer_forward; bf16 layers only, whatever T (the grouped-GEMM
 *  path).
 *  Rounding: A x, A h (fp32 sums) and (alpha / rank) B are rounded to bf16; each adapted
 *  product is then accumulated with W v in one fp32 sum; the rest as maskmoe_layer_forward.
 *  Errors: as maskmoe_layer_forward; E_INVAL for a NULL or misaligned adapter, a rank outside
 *  1..16 or a non-finite alpha; E_UNSUPPORTED for f32 layers or T (K + n_shared) >= 2^25.
 */
int maskmoe_layer_forward_lora(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                               const uint8_t* mask, const float* prior, const void* w_gate_up,
                               const void* w_down, const void* ws_gate_up, const void* ws_down,
                               const maskmoe_lora* lora, void* y, int32_t* topk_idx, float* topk_gate,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * maskmoe_layer_backward_workspace_bytes -- device workspace of maskmoe_layer_backward for
 * `desc` (transposed weights and activations, dO, [da db], per-row dx). Returns 0 for an
 * invalid desc.
 */
size_t maskmoe_layer_backward_workspace_bytes(const maskmoe_layer_desc* desc);

/*
 * maskmoe_layer_backward -- the experts' side of the layer backward for a cotangent dy of y,
 * with the routing held fixed (the routers and experts update at every step: Section 3.2,
 * Stage 1; Stage 2 continues with them). By Eq. 1 routed expert i receives g dy on the tokens
 * that chose it, a shared expert dy on every token; through its SwiGLU
 * F(x) = W_down (SiLU(W_gate x) * (W_up x)), with a = W_gate x, b = W_up x, h = SiLU(a) b:
 *   dh = dO W_down,  da = dh * b * SiLU'(a),  db = dh * SiLU(a),
 *   dL/dx (experts' share) = sum over the token's rows of da W_gate + db W_up,
 *   dL/dW_down = dO^T h,  dL/dW_gate = da^T x,  dL/dW_up = db^T x.
 * The gates' own gradient and the router's share of dL/dx come from maskmoe_stage1_backward.
 *
 *  desc            as given to maskmoe_layer_forward_train; bf16 only.
 *  x, w_gate_up, w_down, ws_gate_up, ws_down: as given to the forward.
 *  topk_gate       device [T, K] float, the forward's gates.
 *  dy              device [T, d] bf16.
 *  train_workspace the workspace of the maskmoe_layer_forward_train call with the same
 *                  arguments, unchanged since (it holds the permutation, h and a, b), at least
 *                  maskmoe_layer_train_workspace_bytes(desc) bytes.
 *  d_x             device [T, d] float output: the experts' share of dL/dx.
 *  d_w_gate_up     device [E, 2F, d] float output (zero for experts no token chose).
 *  d_w_down        device [E, d, F] float output.
 *  d_ws_gate_up, d_ws_down: the shared experts' gradients, [n_shared, ...]; NULL when
 *                  n_shared == 0.
 *  workspace       device, maskmoe_layer_backward_workspace_bytes(desc) bytes, 256-byte aligned.
 *  Rounding: dO = g dy and [da db] are rounded to bf16 before their products, a and b are the
 *  forward's bf16-rounded pre-activations; accumulation and all outputs are fp32.
 *  Errors: as maskmoe_layer_forward; E_UNSUPPORTED for f32 layers, packed weights
 *  (LAYOUT_PACKED) or index ranges at or above 2^31 elements; E_WORKSPACE for a missing, small
 *  or misaligned workspace of either kind.
 *  T = 0 writes nothing.
 */
int maskmoe_layer_backward(const maskmoe_layer_desc* desc, const void* x, const void* w_gate_up,
                           const void* w_down, const void* ws_gate_up, const void* ws_down,
                           const float* topk_gate, const void* dy, const void* train_workspace,
                           size_t train_workspace_bytes, float* d_x, float* d_w_gate_up, float* d_w_down,
                           float* d_ws_gate_up, float* d_ws_down, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/*
 * maskmoe_stage1_backward_workspace_bytes -- device workspace of maskmoe_stage1_backward for
 * `desc` (T, d, E used). Returns 0 for an invalid desc.
 */
size_t maskmoe_stage1_backward_workspace_bytes(const maskmoe_layer_desc* desc);

/*
 * maskmoe_stage1_backward -- the gradients that reach the mask and the router through the
 * gate values of a hard-mask layer (Section 3.2, Eq. 2 and Eq. 3), for a cotangent dy of y:
 *   dg_{t,k} = <dy_t, F_{A_t[k]}(x_t)>                                      (from Eq. 1)
 *   gates from p * m, A fixed, m = 1 on A:
 *     GATE_P:      dL/dm_e = sum_t p_e dg_e [e in A_t];  dz = p (dp - <p, dp>), dp = dg on A
 *     GATE_RENORM: dL/dm_e = sum_t g_e (dg_e - gbar_t) [e in A_t] = sum_t dz_{t,e},
 *                  gbar_t = sum_{A_t} g dg
 *   dL/dm~ += (diag(pi) - pi pi^T) dL/dm, pi = softmax(m~)            (Eq. 3, straight-through)
 *   dL/dW = dz^T x,  router share of dL/dx = dz W                      (z = W x)
 * All tokens share the mask (Stage 1), so dL/dm sums over the batch. The expert FFN weights'
 * own gradients are not computed here.
 *
 *  desc          route_mode must be MASKMOE_ROUTE_HARD_MASK; T, d, E, K, dtype, gate_mode
 *                are used.
 *  x, w_router   device [T, d], [E, d] (dtype), as given to the forward.
 *  mask          host [E] uint8, the step's binary mask; must be 1 on every expert in
 *                topk_idx (as the forward's routing guarantees).
 *  mask_logits   host [E] float m~; required when d_mask_logits is given.
 *  topk_idx      device [T, K] int32 and router_logits device [T, E] float from
 *                maskmoe_layer_forward_train.
 *  dy            device [T, d] (dtype).  expert_out device [T, K, d] float from the forward.
 *  d_gate        device [T, K] float output (dg) or NULL.
 *  d_mask        device [E] float output (dL/dm) or NULL.
 *  d_mask_logits device [E] float, ACCUMULATED: dL/dm~ of this step is added to it, so a
 *                caller sums T steps before one update (Stage 1); or NULL.
 *  d_w_router    device [E, d] float output, required.
 *  d_x           device [T, d] float output (the router's share of dL/dx) or NULL.
 *  workspace     device, maskmoe_stage1_backward_workspace_bytes(desc) bytes, 256-byte aligned.
 *  Reductions run in a fixed order: results are deterministic. T = 0 writes nothing.
 *  Errors: E_INVAL for an invalid desc, a mode other than HARD_MASK, a mask row with fewer
 *  than K ones, a NULL required pointer, a misaligned pointer or a non-finite mask logit;
 *  E_UNSUPPORTED for T*E at or above 2^31; E_WORKSPACE when the workspace is too small.
 */
int maskmoe_stage1_backward(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                            const uint8_t* mask, const float* mask_logits, const int32_t* topk_idx,
                            const float* router_logits, const void* dy, const float* expert_out,
                            float* d_gate, float* d_mask, float* d_mask_logits, float* d_w_router,
                            float* d_x, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* maskmoe_status_string -- static, NUL-terminated description of a status code. */
const char* maskmoe_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* MASKMOE_H_ */
