// Internal launchers of the masked-MoE kernels. Every launcher enqueues on `stream` and
// returns hipSuccess or the launch error; arguments are validated by the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace maskmoe {

// Group the T*K routed (token, slot) entries by expert, stably in entry order, and append
// n_shared groups of all T tokens. Writes offsets/tile_off [G+1], active [G], n_active [1],
// perm/inv [T*K], row_tok [T*(K+n_shared)], with G = E + n_shared.
struct PermBuffers {
  int32_t* offsets;
  int32_t* tile_off;
  int32_t* active;
  int32_t* n_active;
  int32_t* perm;
  int32_t* inv;
  int32_t* row_tok;
};
// Router logits + softmax + mask/prior Top-K + gates for layers [0, L) of w_router
// ([L, E, d]); host `mask` [L, E] (HARD_MASK) or `prior` [L, E] (SOFT_PRIOR), unused for
// PLAIN. Outputs idx/gate [L, T, K], margin [L, T].
// logits (fp32 [L, T, E]) and margin ([L, T]) are optional outputs (null: not written).
// When route_splits(bf16, T, E) and a logits buffer is at hand (logits, else split_ws: fp32
// [L, T, E] workspace), the logits are written first and selected by a second kernel at full
// occupancy; otherwise the logit kernel selects itself. Both give the same bits.
constexpr int kRouteSplitMinT = 512;
constexpr int kRouteSplitMaxE = 64;
inline bool route_splits(bool bf16, int T, int E) { return bf16 && T >= kRouteSplitMinT && E <= kRouteSplitMaxE; }
hipError_t launch_route(bool bf16, const void* x, const void* w_router, int T, int d, int E, int K,
                        int L, int mode, int gate_mode, const uint8_t* mask, const float* prior,
                        int32_t* idx, float* gate, float* margin, float* logits, float* split_ws,
                        hipStream_t stream);

// Tokens at or below which one bf16 routing workgroup covers every token, so the routing
// kernel can also perform the permutation (launch_route_permute).
constexpr int kRouteOneBlockT = 16;
// Routing of one layer (L = 1, bf16, T <= kRouteOneBlockT) followed, in the same workgroup,
// by the permutation into `pb` (rows tiled by tile_rows, n_shared shared groups).
hipError_t launch_route_permute(const void* x, const void* w_router, int T, int d, int E, int K, int mode,
                                int gate_mode, const uint8_t* mask, const float* prior, int32_t* idx,
                                float* gate, float* logits, int n_shared, int tile_rows, const PermBuffers& pb,
                                hipStream_t stream);

// Many tokens: the same grouping over chunks of kPermChunk entries; chunk_counts is workspace
// int32 [permute_chunks(T, K), E].
constexpr int kPermChunk = 1024;
inline int permute_chunks(int T, int K) {
  return static_cast<int>((static_cast<int64_t>(T) * K + kPermChunk - 1) / kPermChunk);
}
hipError_t launch_permute(const int32_t* idx, int T, int K, int E, int n_shared, int tile_rows,
                          const PermBuffers& pb, int32_t* chunk_counts, hipStream_t stream);

// Row-tile size of the bf16 grouped GEMMs (the permutation counts tiles of this many rows).
constexpr int kGemmBM = 256;
// Tokens at or below which the bf16 layer uses the weight-streaming decode kernels.
constexpr int kDecodeMaxT = 16;

struct ExpertArgs {
  const void* x;           // [T, d]
  const void* w_gate_up;   // [E, 2F, d]
  const void* w_down;      // [E, d, F]
  const void* ws_gate_up;  // [n_shared, 2F, d]
  const void* ws_down;     // [n_shared, d, F]
  const float* gate;       // [T, K]
  float* expert_out;       // [T, K, d] fp32 output of each selected expert before gating, or null
  const int32_t* slot_of = nullptr;   // few-token path: routed expert -> block of w_gate_up / w_down
  int n_slots = 0;                    // blocks in w_gate_up / w_down when slot_of is given
  int T, d, F, E, K, n_shared;
  bool packed = false;                // weights in the packed layout (pack_weights_kernel)
};

// Packed expert weights (bf16): each matrix is cut into groups of kPackRows rows (gate/up:
// 64 W_gate rows and their 64 W_up rows) and kPackCols-column chunks; block (group q,
// chunk c) is [kPackRows][kPackCols] contiguous at (q * cols / kPackCols + c) * kPackBlock.
constexpr int kPackRows = 128, kPackCols = 64, kPackBlock = kPackRows * kPackCols;
hipError_t launch_pack_weights(const uint16_t* w_gate_up, const uint16_t* w_down, uint16_t* p_gate_up,
                               uint16_t* p_down, int n, int d, int F, hipStream_t stream);

// Optional stage markers: when `marks` is non-null, marks[i] is recorded on the stream after
// the i-th of the three expert stages (gate/up, down, combine); a stage that a path fuses
// away is marked right after the previous one.
inline void record_mark(hipEvent_t* marks, int i, hipStream_t stream) {
  if (marks && marks[i]) (void)hipEventRecord(marks[i], stream);
}

// Offloaded decode, batch 1 (offload.hip). state: int32 [B + 2E] (cached experts oldest first,
// LFU counts, slot of each expert); fetch: int32 [1 + 2K] workspace (count, experts, slots);
// counters: int64 [2] (fetches, hits) accumulated, or null. E <= 64, K <= B <= E.
constexpr int kOffloadMaxE = 64;
constexpr int kOffloadFetchBlocks = 512;   // workgroups per fetched expert
hipError_t launch_offload_cache(int policy, const int32_t* idx, int E, int K, int B, int32_t* state, int32_t* fetch,
                                int64_t* counters, int32_t* dev_error, hipStream_t stream);
// host_gu / host_dn: device-side addresses of the pinned host copies [E, 2F, d] and [E, d, F];
// slots_gu / slots_dn: the device pool [B, 2F, d] and [B, d, F].
hipError_t launch_offload_fetch(const int32_t* fetch, int K, int E, int B, int d, int F, const void* host_gu,
                                const void* host_dn, void* slots_gu, void* slots_dn, hipStream_t stream);

// Low-rank adapters of the experts (lora.hip). rank r <= kMaxLoraRank; adapters bf16:
// a_gate_up [E, 2r, d], b_gate_up [E, 2F, r], a_down [E, r, F], b_down [E, d, r] and the shared
// experts' as_* / bs_* [n_shared, ...]; u, v [rows, 64] and bp_gate_up [G, 2F, 64], bp_down
// [G, d, 64] are workspace.
constexpr int kMaxLoraRank = 16;
struct LoraArgs {
  int rank;
  float scale;   // alpha / rank
  const uint16_t *a_gate_up, *b_gate_up, *a_down, *b_down;
  const uint16_t *as_gate_up, *bs_gate_up, *as_down, *bs_down;
  uint16_t *u, *v, *bp_gate_up, *bp_down;
};
hipError_t launch_lora_pack(const LoraArgs& l, int G, int E, int F, int d, hipStream_t stream);
// out [rows, 64] = src rows (gathered through row_tok when given) times the rows' group adapter
// A [nq, K]^T, zero-padded; rows tiled as the permutation (kGemmBM rows per tile).
hipError_t launch_lora_down(const uint16_t* src, const int32_t* row_tok, int K, const uint16_t* a, const uint16_t* as,
                            int nq, int G, int E, const PermBuffers& pb, int max_tiles, uint16_t* out,
                            hipStream_t stream);

// Partial-tile slots of the grouped GEMMs' split tail tiles (fp32 256 x 256 each, 64 MiB).
// Workgroups one XCD of the current device runs at once (one 256 x 256 tile per CU, the CUs
// split evenly over the 8 XCDs): queried for the current device on every call, so devices with
// different CU counts each get their own figure.
int device_cus_per_xcd();

constexpr int kTailSlots = 256;
constexpr size_t kTailPartBytes = static_cast<size_t>(kTailSlots) * 256 * 256 * 4;

// bf16, T > kDecodeMaxT (any T when training or with adapters): H = SwiGLU(X_g W_gate,up^T)
// per group; O = H W_down^T; y = combine. ab (training): the gate and up pre-activations,
// bf16 [rows, 2F]. lora: the experts' low-rank adapters, added inside both GEMMs.
// part: kTailPartBytes of workspace for the split tail tiles.
hipError_t launch_experts_bf16(const ExpertArgs& a, const PermBuffers& pb, uint16_t* H, float* O, float* part,
                               void* y, int max_tiles, hipStream_t stream, hipEvent_t* marks,
                               uint16_t* ab = nullptr, const LoraArgs* lora = nullptr);
// bf16, T <= kDecodeMaxT: weight-streaming gate/up kernel (split-K into P [split_gu, rows, 2F]
// plus a SwiGLU pass when decode_split_gate_up() > 1), split-K down projection into
// O [split, rows, d] with split = decode_split(), then the combine.
constexpr int kDecodeMaxSplit = 16;
constexpr int kDecodeMaxSplitGateUp = 8;
int decode_split(int T, int d, int F, int E, int K, int n_shared);
int decode_split_gate_up(int T, int d, int F, int E, int K, int n_shared);
hipError_t launch_experts_bf16_decode(const ExpertArgs& a, const PermBuffers& pb, uint16_t* H, float* P, float* O,
                                      void* y, hipStream_t stream, hipEvent_t* marks);
// f32 path (no MFMA; fp32 end to end).
hipError_t launch_experts_f32(const ExpertArgs& a, const PermBuffers& pb, float* H, float* O,
                              void* y, hipStream_t stream, hipEvent_t* marks);

// Per-(layer, stream) expert cache replay (policy 0 LRU, 1 LFU, 2 FIFO), one wavefront per
// stream.
hipError_t launch_cache(int policy, const int32_t* trace, int L, int S, int N, int K, int E, int B,
                        int32_t* state, int32_t* counts, int64_t* fetches, int64_t* hits,
                        uint8_t* f_per_step, int32_t* dev_error, hipStream_t stream);

// ---- expert-side backward (backward.hip)
constexpr int kMaxGroupsBwd = 256 + 8;

struct BwdLayout {          // byte offsets into the backward workspace
  size_t dout, dab, dxr, xg, part, total;
};
BwdLayout backward_layout(int T, int d, int F, int E, int K, int S);

struct BwdArgs {
  const uint16_t* x;          // [T, d]
  const uint16_t* w_gate_up;  // [E, 2F, d]
  const uint16_t* w_down;     // [E, d, F]
  const uint16_t* ws_gate_up; // [S, 2F, d]
  const uint16_t* ws_down;    // [S, d, F]
  const float* gate;          // [T, K]
  const uint16_t* dy;         // [T, d]
  PermBuffers pb;             // the training forward's permutation
  const uint16_t* h;          // [rows, F] SwiGLU activations of the forward
  const uint16_t* ab;         // [rows, 2F] gate / up pre-activations of the forward
  float* d_x;                 // [T, d]
  float* d_w_gate_up;         // [E, 2F, d]
  float* d_w_down;            // [E, d, F]
  float* d_ws_gate_up;        // [S, 2F, d]
  float* d_ws_down;           // [S, d, F]
  void* workspace;
  BwdLayout lay;
  int T, d, F, E, K, S, max_tiles;
};
hipError_t launch_layer_backward(const BwdArgs& a, hipStream_t stream);

// ---- Stage 1 training: mask and router gradients (train.hip)
constexpr int kMaxKTrain = 16;
constexpr int kMaxETrain = 256;
constexpr int kMaxWgradSlices = 64;

struct Stage1Args {
  const void* x;              // [T, d] layer dtype
  const void* w_router;       // [E, d] layer dtype
  const void* dy;             // [T, d] layer dtype
  const float* expert_out;    // [T, K, d]
  const float* router_logits; // [T, E]
  const int32_t* idx;         // [T, K]
  const double* pi;           // host [E]: softmax of the mask logits
  float* d_gate;              // [T, K] or null
  float* d_mask;              // [E] or null
  float* d_mask_logits;       // [E] accumulated (+=), or null
  float* d_w_router;          // [E, d]
  float* d_x;                 // [T, d] or null
  float* dz;                  // workspace [T, E]
  float* dm_tok;              // workspace [T, E]
  float* dm;                  // workspace [E]: dL/dm before Eq. 3
  float* wgrad_partial;       // workspace [slices, E, d]
  int T, d, E, K, gate_mode;
  bool vec_rows;              // d % 4 == 0 and dy, expert_out rows allow 4-element vector loads
  bool vec_x;                 // rows of x are 16-byte aligned: 16-byte loads of x
};
size_t stage1_workspace_bytes(int T, int d, int E);
hipError_t launch_stage1_backward(const Stage1Args& a, bool bf16, hipStream_t stream);
// Host helpers: softmax in double precision; mask sampling without replacement (one uniform
// per draw, inverse CDF over the remaining experts in index order).
void softmax_f64(const float* logits, int E, double* pi);
void sample_mask_host(const float* mask_logits, const double* uniforms, int E, int e_keep, uint8_t* mask);

}  // namespace maskmoe
