// C-ABI entry points: argument validation, workspace layout and launch sequencing.
// Nothing here touches the device before every argument has been checked; the only
// device work is the kernel launches, enqueued on the caller's stream.

#include <math.h>
#include <stdint.h>

#include <atomic>

#include "kernels.hpp"
#include "maskmoe.h"

// Workspace of maskmoe_layer_forward_noalloc: one copy per device, held while the process
// runs. Host code reaches it only through the device address that hipGetSymbolAddress returns
// for the current device (noalloc_scratch below), never through this name.
static __device__ __align__(256) unsigned char scratch[MASKMOE_NOALLOC_SCRATCH_BYTES];

namespace {

using maskmoe::PermBuffers;

constexpr int kMaxE = 256;
constexpr int kMaxK = 16;
constexpr int kMaxShared = 8;
constexpr int kCacheMaxE = 64;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }
size_t round256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

// Checks shared by maskmoe_route and maskmoe_layer_forward (routing part of desc).
int check_route_desc(const maskmoe_layer_desc* d) {
  if (!d) return MASKMOE_E_INVAL;
  if (d->T < 0 || d->d < 1 || d->E < 1 || d->E > kMaxE || d->K < 1 || d->K > d->E || d->K > kMaxK)
    return MASKMOE_E_INVAL;
  if (d->dtype != MASKMOE_BF16 && d->dtype != MASKMOE_F32) return MASKMOE_E_INVAL;
  if (d->route_mode < MASKMOE_ROUTE_PLAIN || d->route_mode > MASKMOE_ROUTE_SOFT_PRIOR) return MASKMOE_E_INVAL;
  if (d->gate_mode != MASKMOE_GATE_P && d->gate_mode != MASKMOE_GATE_RENORM) return MASKMOE_E_INVAL;
  if (static_cast<int64_t>(d->T) * d->K >= (int64_t{1} << 31)) return MASKMOE_E_INVAL;
  return MASKMOE_OK;
}

// Mask rows need at least K ones (Eq. 2 draws E' >= K experts); prior values must be
// finite and positive (Eq. 4: the prior excludes no expert).
int check_mask_prior(int mode, int L, int E, int K, const uint8_t* mask, const float* prior) {
  if (mode == MASKMOE_ROUTE_HARD_MASK) {
    if (!mask) return MASKMOE_E_INVAL;
    for (int l = 0; l < L; ++l) {
      int ones = 0;
      for (int e = 0; e < E; ++e) ones += mask[static_cast<size_t>(l) * E + e] != 0;
      if (ones < K) return MASKMOE_E_INVAL;
    }
  } else if (mode == MASKMOE_ROUTE_SOFT_PRIOR) {
    if (!prior) return MASKMOE_E_INVAL;
    for (size_t i = 0; i < static_cast<size_t>(L) * E; ++i) {
      const float v = prior[i];
      if (!(v > 0.0f) || !isfinite(v)) return MASKMOE_E_INVAL;
    }
  }
  return MASKMOE_OK;
}

struct Layout {
  size_t idx, gate, offsets, tile_off, active, n_active, perm, inv, row_tok, pcount, Z, H, P, O, TP, total;
  size_t AB, train_total;   // training (bf16): gate / up pre-activations [rows, 2F] after `total`
  // adapters (bf16), after `total`: rank projections U, V [rows, 64], scaled B [G, 2F | d, 64]
  size_t LU, LV, LBGU, LBD, lora_total;
  // offloaded decode, after `total`: the step's fetch list int32 [1 + 2K]
  size_t FL, offload_total;
};

static_assert(maskmoe::kDecodeMaxT <= maskmoe::kRouteOneBlockT,
              "the few-token path routes and permutes in one workgroup");

bool uses_decode_path(const maskmoe_layer_desc& d) {
  return d.dtype == MASKMOE_BF16 && d.T <= maskmoe::kDecodeMaxT;
}

Layout layout(const maskmoe_layer_desc& d) {
  Layout w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += round256(bytes);
    return o;
  };
  const size_t TK = static_cast<size_t>(d.T) * d.K;
  const size_t G = static_cast<size_t>(d.E) + d.n_shared;
  const size_t rows = static_cast<size_t>(d.T) * (d.K + d.n_shared);
  const size_t hsz = d.dtype == MASKMOE_BF16 ? 2 : 4;
  w.idx = take(TK * 4);
  w.gate = take(TK * 4);
  w.offsets = take((G + 1) * 4);
  w.tile_off = take((G + 1) * 4);
  w.active = take(G * 4);
  w.n_active = take(4);
  w.perm = take(TK * 4);
  w.inv = take(TK * 4);
  w.row_tok = take(rows * 4);
  w.pcount = take(static_cast<size_t>(maskmoe::permute_chunks(d.T, d.K)) * d.E * 4);
  // router logits of split routing (fp32 [T, E]) when no logits output is requested
  w.Z = take(maskmoe::route_splits(d.dtype == MASKMOE_BF16, d.T, d.E) ? static_cast<size_t>(d.T) * d.E * 4 : 0);
  w.H = take(rows * d.F * hsz);
  // O holds the expert outputs: [rows, d], or [split, rows, d] on the few-token path; P the
  // few-token partial gate/up sums [split_gu, rows, 2F]. Both are sized for the largest
  // splits of up to kDecodeMaxT tokens so the total stays monotone in T.
  const size_t dec_T = static_cast<size_t>(d.T < maskmoe::kDecodeMaxT ? d.T : maskmoe::kDecodeMaxT);
  const size_t dec_rows = dec_T * (d.K + d.n_shared);
  w.P = take(maskmoe::kDecodeMaxSplitGateUp * dec_rows * 2 * d.F * 4);
  const size_t o_rows = maskmoe::kDecodeMaxSplit * dec_rows;
  w.O = take((rows > o_rows ? rows : o_rows) * d.d * 4);
  // partial tiles of the grouped GEMMs' split tail tiles (bf16 layers)
  w.TP = take(d.dtype == MASKMOE_BF16 ? maskmoe::kTailPartBytes : 0);
  w.total = off;
  w.AB = take(d.dtype == MASKMOE_BF16 ? rows * 2 * d.F * 2 : 0);
  w.train_total = off;
  off = w.total;
  w.LU = take(rows * 64 * 2);
  w.LV = take(rows * 64 * 2);
  w.LBGU = take(G * 2 * d.F * 64 * 2);
  w.LBD = take(G * d.d * 64 * 2);
  w.lora_total = off;
  off = w.total;
  w.FL = take((1 + 2 * static_cast<size_t>(d.K)) * 4);
  w.offload_total = off;
  return w;
}

// The packed weight layout: bf16, groups of 128 rows of W_down (d) and 64-column chunks.
bool packable(int dtype, int d, int F) {
  return dtype == MASKMOE_BF16 && d % maskmoe::kPackRows == 0 && F % maskmoe::kPackCols == 0;
}

int check_layer_desc(const maskmoe_layer_desc* d) {
  int st = check_route_desc(d);
  if (st != MASKMOE_OK) return st;
  if (d->F < 1 || d->n_shared < 0 || d->n_shared > kMaxShared) return MASKMOE_E_INVAL;
  if (static_cast<int64_t>(d->T) * (d->K + d->n_shared) >= (int64_t{1} << 31)) return MASKMOE_E_INVAL;
  if (d->weight_layout != MASKMOE_LAYOUT_ROWS && d->weight_layout != MASKMOE_LAYOUT_PACKED) return MASKMOE_E_INVAL;
  if (d->weight_layout == MASKMOE_LAYOUT_PACKED && !packable(d->dtype, d->d, d->F)) return MASKMOE_E_UNSUPPORTED;
  return MASKMOE_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? MASKMOE_OK : MASKMOE_E_HIP; }

// Device address of `scratch` on the current device, looked up once per device (with that
// device current) and kept; concurrent first calls store the same address.
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];

int noalloc_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MASKMOE_E_HIP;
  if (dev < 0 || dev >= kMaxDevices) return MASKMOE_E_UNSUPPORTED;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MASKMOE_E_HIP;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return MASKMOE_OK;
}

}  // namespace

extern "C" {

int maskmoe_pack_expert_weights(const maskmoe_layer_desc* desc, int32_t n, const void* w_gate_up,
                                const void* w_down, void* packed_gate_up, void* packed_down,
                                hipStream_t stream) {
  if (!desc || desc->d < 1 || desc->F < 1 || n < 0) return MASKMOE_E_INVAL;
  if ((w_gate_up == nullptr) != (packed_gate_up == nullptr) || (w_down == nullptr) != (packed_down == nullptr))
    return MASKMOE_E_INVAL;
  if ((w_gate_up && w_gate_up == packed_gate_up) || (w_down && w_down == packed_down)) return MASKMOE_E_INVAL;
  const void* ptrs[] = {w_gate_up, w_down, packed_gate_up, packed_down};
  for (const void* p : ptrs)
    if (p && !aligned(p, 16)) return MASKMOE_E_INVAL;
  if (desc->dtype != MASKMOE_BF16 && desc->dtype != MASKMOE_F32) return MASKMOE_E_INVAL;
  if (!packable(desc->dtype, desc->d, desc->F)) return MASKMOE_E_UNSUPPORTED;
  if (n == 0) return MASKMOE_OK;
  return hip_status(maskmoe::launch_pack_weights(static_cast<const uint16_t*>(w_gate_up),
                                                 static_cast<const uint16_t*>(w_down),
                                                 static_cast<uint16_t*>(packed_gate_up),
                                                 static_cast<uint16_t*>(packed_down), n, desc->d, desc->F, stream));
}

const char* maskmoe_status_string(int status) {
  switch (status) {
    case MASKMOE_OK: return "ok";
    case MASKMOE_E_INVAL: return "invalid argument";
    case MASKMOE_E_WORKSPACE: return "workspace missing or too small";
    case MASKMOE_E_HIP: return "HIP launch or runtime error";
    case MASKMOE_E_UNSUPPORTED: return "unsupported size or configuration";
    default: return "unknown status";
  }
}

size_t maskmoe_route_workspace_bytes(const maskmoe_layer_desc* desc, int32_t L) {
  if (check_route_desc(desc) != MASKMOE_OK || L < 1) return 0;
  if (!maskmoe::route_splits(desc->dtype == MASKMOE_BF16, desc->T, desc->E)) return 0;
  return static_cast<size_t>(L) * desc->T * desc->E * 4;
}

int maskmoe_route(const maskmoe_layer_desc* desc, int32_t L, const void* x, const void* w_router,
                  const uint8_t* mask, const float* prior, int32_t* topk_idx, float* topk_gate,
                  float* topk_margin, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = check_route_desc(desc);
  if (st != MASKMOE_OK) return st;
  if (L < 1 || static_cast<int64_t>(L) * desc->T * desc->K >= (int64_t{1} << 31)) return MASKMOE_E_INVAL;
  if (workspace && (workspace_bytes < maskmoe_route_workspace_bytes(desc, L) || !aligned(workspace, 16)))
    return MASKMOE_E_INVAL;
  st = check_mask_prior(desc->route_mode, L, desc->E, desc->K, mask, prior);
  if (st != MASKMOE_OK) return st;
  if (desc->T == 0) return MASKMOE_OK;
  if (!x || !w_router || !topk_idx || !topk_gate) return MASKMOE_E_INVAL;
  const bool bf16 = desc->dtype == MASKMOE_BF16;
  if (bf16 && desc->d % 32 != 0) return MASKMOE_E_UNSUPPORTED;
  if (!aligned(x, 16) || !aligned(w_router, 16) || !aligned(topk_idx, 4) || !aligned(topk_gate, 4) ||
      (topk_margin && !aligned(topk_margin, 4)))
    return MASKMOE_E_INVAL;
  return hip_status(maskmoe::launch_route(bf16, x, w_router, desc->T, desc->d, desc->E, desc->K, L,
                                         desc->route_mode, desc->gate_mode, mask, prior, topk_idx,
                                         topk_gate, topk_margin, nullptr, static_cast<float*>(workspace),
                                         stream));
}

size_t maskmoe_layer_workspace_bytes(const maskmoe_layer_desc* desc) {
  if (check_layer_desc(desc) != MASKMOE_OK) return 0;
  return layout(*desc).total;
}

size_t maskmoe_layer_train_workspace_bytes(const maskmoe_layer_desc* desc) {
  if (check_layer_desc(desc) != MASKMOE_OK) return 0;
  return layout(*desc).train_total;
}

size_t maskmoe_layer_lora_workspace_bytes(const maskmoe_layer_desc* desc) {
  if (check_layer_desc(desc) != MASKMOE_OK) return 0;
  return layout(*desc).lora_total;
}

static int layer_forward_impl(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                              const uint8_t* mask, const float* prior, const void* w_gate_up,
                              const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                              int32_t* topk_idx, float* topk_gate, float* router_logits, float* expert_out,
                              void* workspace, size_t workspace_bytes, hipStream_t stream, hipEvent_t* events,
                              const maskmoe_lora* lora = nullptr) {
  int st = check_layer_desc(desc);
  if (st != MASKMOE_OK) return st;
  const maskmoe_layer_desc& d = *desc;
  st = check_mask_prior(d.route_mode, 1, d.E, d.K, mask, prior);
  if (st != MASKMOE_OK) return st;
  if (d.T == 0) return MASKMOE_OK;
  if (!x || !w_router || !w_gate_up || !w_down || !y) return MASKMOE_E_INVAL;
  if (d.n_shared > 0 && (!ws_gate_up || !ws_down)) return MASKMOE_E_INVAL;
  const bool bf16 = d.dtype == MASKMOE_BF16;
  if (bf16 && (d.d % 64 != 0 || d.F % 64 != 0)) return MASKMOE_E_UNSUPPORTED;
  // the grouped GEMMs address x, H and one expert's matrices with 32-bit element offsets
  const int64_t rows64 = static_cast<int64_t>(d.T) * (d.K + d.n_shared);
  if (bf16 && (static_cast<int64_t>(d.T) * d.d >= (int64_t{1} << 31) || rows64 * d.F >= (int64_t{1} << 31) ||
               int64_t{2} * d.F * d.d >= (int64_t{1} << 31)))
    return MASKMOE_E_UNSUPPORTED;
  const void* ptrs[] = {x, w_router, w_gate_up, w_down, y};
  for (const void* p : ptrs)
    if (!aligned(p, 16)) return MASKMOE_E_INVAL;
  if (d.n_shared > 0 && (!aligned(ws_gate_up, 16) || !aligned(ws_down, 16))) return MASKMOE_E_INVAL;
  if ((topk_idx && !aligned(topk_idx, 4)) || (topk_gate && !aligned(topk_gate, 4))) return MASKMOE_E_INVAL;
  if ((router_logits && !aligned(router_logits, 4)) || (expert_out && !aligned(expert_out, 16))) return MASKMOE_E_INVAL;
  if (lora) {
    if (!bf16) return MASKMOE_E_UNSUPPORTED;
    if (rows64 >= (int64_t{1} << 25)) return MASKMOE_E_UNSUPPORTED;   // U, V rows * 64 in 32 bits
    if (lora->rank < 1 || lora->rank > maskmoe::kMaxLoraRank || !std::isfinite(lora->alpha)) return MASKMOE_E_INVAL;
    const void* mats[] = {lora->a_gate_up, lora->b_gate_up, lora->a_down, lora->b_down};
    const void* smats[] = {lora->as_gate_up, lora->bs_gate_up, lora->as_down, lora->bs_down};
    for (int i = 0; i < 4; ++i) {
      const size_t al = i % 2 == 0 ? 16 : 2;   // A rows are read 16 bytes at a time
      if (!mats[i] || !aligned(mats[i], al)) return MASKMOE_E_INVAL;
      if (d.n_shared > 0 && (!smats[i] || !aligned(smats[i], al))) return MASKMOE_E_INVAL;
    }
  }
  const bool train = expert_out != nullptr;   // the training forward also keeps what the backward reads
  const bool packed = d.weight_layout == MASKMOE_LAYOUT_PACKED;
  if (packed && train) return MASKMOE_E_UNSUPPORTED;
  const Layout w = layout(d);
  const size_t need = lora ? w.lora_total : train ? w.train_total : w.total;
  if (!workspace || workspace_bytes < need || !aligned(workspace, 256)) return MASKMOE_E_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  int32_t* idx = topk_idx ? topk_idx : reinterpret_cast<int32_t*>(ws + w.idx);
  float* gate = topk_gate ? topk_gate : reinterpret_cast<float*>(ws + w.gate);
  PermBuffers pb;
  pb.offsets = reinterpret_cast<int32_t*>(ws + w.offsets);
  pb.tile_off = reinterpret_cast<int32_t*>(ws + w.tile_off);
  pb.active = reinterpret_cast<int32_t*>(ws + w.active);
  pb.n_active = reinterpret_cast<int32_t*>(ws + w.n_active);
  pb.perm = reinterpret_cast<int32_t*>(ws + w.perm);
  pb.inv = reinterpret_cast<int32_t*>(ws + w.inv);
  pb.row_tok = reinterpret_cast<int32_t*>(ws + w.row_tok);

  maskmoe::record_mark(events, 0, stream);
  hipError_t e;
  // Training always takes the grouped-GEMM path, whose gate/up epilogue can keep the
  // pre-activations for the backward.
  const bool decode = uses_decode_path(d) && !train && !lora;
  if (decode) {  // one workgroup routes every token and then permutes them
    e = maskmoe::launch_route_permute(x, w_router, d.T, d.d, d.E, d.K, d.route_mode, d.gate_mode, mask, prior, idx,
                                      gate, router_logits, d.n_shared, maskmoe::kGemmBM, pb, stream);
    if (e != hipSuccess) return MASKMOE_E_HIP;
    maskmoe::record_mark(events, 1, stream);
  } else {
    e = maskmoe::launch_route(bf16, x, w_router, d.T, d.d, d.E, d.K, 1, d.route_mode, d.gate_mode, mask, prior,
                              idx, gate, nullptr, router_logits, reinterpret_cast<float*>(ws + w.Z), stream);
    if (e != hipSuccess) return MASKMOE_E_HIP;
    maskmoe::record_mark(events, 1, stream);
    e = maskmoe::launch_permute(idx, d.T, d.K, d.E, d.n_shared, maskmoe::kGemmBM, pb,
                                reinterpret_cast<int32_t*>(ws + w.pcount), stream);
    if (e != hipSuccess) return MASKMOE_E_HIP;
  }
  maskmoe::record_mark(events, 2, stream);
  hipEvent_t* expert_marks = events ? events + 3 : nullptr;

  maskmoe::ExpertArgs a;
  a.x = x;
  a.w_gate_up = w_gate_up;
  a.w_down = w_down;
  a.ws_gate_up = ws_gate_up;
  a.ws_down = ws_down;
  a.gate = gate;
  a.expert_out = expert_out;
  a.T = d.T; a.d = d.d; a.F = d.F; a.E = d.E; a.K = d.K; a.n_shared = d.n_shared;
  a.packed = packed;
  if (!bf16) {
    e = maskmoe::launch_experts_f32(a, pb, reinterpret_cast<float*>(ws + w.H), reinterpret_cast<float*>(ws + w.O),
                                    y, stream, expert_marks);
  } else if (decode) {
    e = maskmoe::launch_experts_bf16_decode(a, pb, reinterpret_cast<uint16_t*>(ws + w.H),
                                            reinterpret_cast<float*>(ws + w.P), reinterpret_cast<float*>(ws + w.O), y,
                                            stream, expert_marks);
  } else {
    const int64_t TK = static_cast<int64_t>(d.T) * d.K;
    const int64_t nonempty = TK < d.E ? TK : d.E;
    const int64_t max_tiles = TK / maskmoe::kGemmBM + nonempty +
                              static_cast<int64_t>(d.n_shared) * ((d.T + maskmoe::kGemmBM - 1) / maskmoe::kGemmBM);
    maskmoe::LoraArgs la{};
    if (lora) {
      la.rank = lora->rank;
      la.scale = lora->alpha / static_cast<float>(lora->rank);
      la.a_gate_up = static_cast<const uint16_t*>(lora->a_gate_up);
      la.b_gate_up = static_cast<const uint16_t*>(lora->b_gate_up);
      la.a_down = static_cast<const uint16_t*>(lora->a_down);
      la.b_down = static_cast<const uint16_t*>(lora->b_down);
      la.as_gate_up = static_cast<const uint16_t*>(lora->as_gate_up);
      la.bs_gate_up = static_cast<const uint16_t*>(lora->bs_gate_up);
      la.as_down = static_cast<const uint16_t*>(lora->as_down);
      la.bs_down = static_cast<const uint16_t*>(lora->bs_down);
      la.u = reinterpret_cast<uint16_t*>(ws + w.LU);
      la.v = reinterpret_cast<uint16_t*>(ws + w.LV);
      la.bp_gate_up = reinterpret_cast<uint16_t*>(ws + w.LBGU);
      la.bp_down = reinterpret_cast<uint16_t*>(ws + w.LBD);
    }
    e = maskmoe::launch_experts_bf16(a, pb, reinterpret_cast<uint16_t*>(ws + w.H),
                                     reinterpret_cast<float*>(ws + w.O), reinterpret_cast<float*>(ws + w.TP), y,
                                     static_cast<int>(max_tiles), stream,
                                     expert_marks, train ? reinterpret_cast<uint16_t*>(ws + w.AB) : nullptr,
                                     lora ? &la : nullptr);
  }
  return hip_status(e);
}

int maskmoe_layer_forward(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                          const uint8_t* mask, const float* prior, const void* w_gate_up,
                          const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                          int32_t* topk_idx, float* topk_gate, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  return layer_forward_impl(desc, x, w_router, mask, prior, w_gate_up, w_down, ws_gate_up, ws_down, y,
                            topk_idx, topk_gate, nullptr, nullptr, workspace, workspace_bytes, stream, nullptr);
}

int maskmoe_layer_forward_noalloc(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                  const uint8_t* mask, const float* prior, const void* w_gate_up,
                                  const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                                  int32_t* topk_idx, float* topk_gate, hipStream_t stream) {
  int st = check_layer_desc(desc);
  if (st != MASKMOE_OK) return st;
  if (layout(*desc).total > MASKMOE_NOALLOC_SCRATCH_BYTES) return MASKMOE_E_WORKSPACE;
  void* ws = nullptr;
  st = noalloc_scratch(&ws);
  if (st != MASKMOE_OK) return st;
  return layer_forward_impl(desc, x, w_router, mask, prior, w_gate_up, w_down, ws_gate_up, ws_down, y, topk_idx,
                            topk_gate, nullptr, nullptr, ws, MASKMOE_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

int maskmoe_layer_forward_train(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                const uint8_t* mask, const float* prior, const void* w_gate_up,
                                const void* w_down, const void* ws_gate_up, const void* ws_down, void* y,
                                int32_t* topk_idx, float* topk_gate, float* router_logits, float* expert_out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (desc && desc->T > 0 && (!topk_idx || !topk_gate || !router_logits || !expert_out)) return MASKMOE_E_INVAL;
  return layer_forward_impl(desc, x, w_router, mask, prior, w_gate_up, w_down, ws_gate_up, ws_down, y,
                            topk_idx, topk_gate, router_logits, expert_out, workspace, workspace_bytes, stream,
                            nullptr);
}

int maskmoe_layer_forward_lora(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                               const uint8_t* mask, const float* prior, const void* w_gate_up,
                               const void* w_down, const void* ws_gate_up, const void* ws_down,
                               const maskmoe_lora* lora, void* y, int32_t* topk_idx, float* topk_gate,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!lora) return MASKMOE_E_INVAL;
  return layer_forward_impl(desc, x, w_router, mask, prior, w_gate_up, w_down, ws_gate_up, ws_down, y,
                            topk_idx, topk_gate, nullptr, nullptr, workspace, workspace_bytes, stream, nullptr,
                            lora);
}

int maskmoe_layer_forward_profiled(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                   const uint8_t* mask, const float* prior, const void* w_gate_up,
                                   const void* w_down, const void* ws_gate_up, const void* ws_down,
                                   void* y, int32_t* topk_idx, float* topk_gate, void* workspace,
                                   size_t workspace_bytes, hipEvent_t* events, hipStream_t stream) {
  if (!events) return MASKMOE_E_INVAL;
  return layer_forward_impl(desc, x, w_router, mask, prior, w_gate_up, w_down, ws_gate_up, ws_down, y,
                            topk_idx, topk_gate, nullptr, nullptr, workspace, workspace_bytes, stream, events);
}

size_t maskmoe_layer_backward_workspace_bytes(const maskmoe_layer_desc* desc) {
  if (check_layer_desc(desc) != MASKMOE_OK) return 0;
  const maskmoe_layer_desc& d = *desc;
  return maskmoe::backward_layout(d.T, d.d, d.F, d.E, d.K, d.n_shared).total;
}

int maskmoe_layer_backward(const maskmoe_layer_desc* desc, const void* x, const void* w_gate_up,
                           const void* w_down, const void* ws_gate_up, const void* ws_down, const float* topk_gate,
                           const void* dy, const void* train_workspace, size_t train_workspace_bytes, float* d_x,
                           float* d_w_gate_up, float* d_w_down, float* d_ws_gate_up, float* d_ws_down,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = check_layer_desc(desc);
  if (st != MASKMOE_OK) return st;
  const maskmoe_layer_desc& d = *desc;
  if (d.dtype != MASKMOE_BF16 || d.weight_layout != MASKMOE_LAYOUT_ROWS) return MASKMOE_E_UNSUPPORTED;
  if (d.d % 64 != 0 || d.F % 64 != 0) return MASKMOE_E_UNSUPPORTED;
  if (d.T == 0) return MASKMOE_OK;
  if (!x || !w_gate_up || !w_down || !topk_gate || !dy || !d_x || !d_w_gate_up || !d_w_down) return MASKMOE_E_INVAL;
  if (d.n_shared > 0 && (!ws_gate_up || !ws_down || !d_ws_gate_up || !d_ws_down)) return MASKMOE_E_INVAL;
  const void* p16[] = {x, w_gate_up, w_down, dy, d_x};
  for (const void* p : p16)
    if (!aligned(p, 16)) return MASKMOE_E_INVAL;
  if (!aligned(topk_gate, 4) || !aligned(d_w_gate_up, 4) || !aligned(d_w_down, 4)) return MASKMOE_E_INVAL;
  if (d.n_shared > 0 && (!aligned(ws_gate_up, 16) || !aligned(ws_down, 16) || !aligned(d_ws_gate_up, 4) ||
                         !aligned(d_ws_down, 4)))
    return MASKMOE_E_INVAL;
  const maskmoe::BwdLayout bl = maskmoe::backward_layout(d.T, d.d, d.F, d.E, d.K, d.n_shared);
  // the GEMMs address rows with 32-bit element offsets
  const int64_t rows = static_cast<int64_t>(d.T) * (d.K + d.n_shared);
  if (rows * 2 * d.F >= (int64_t{1} << 31) || rows * d.d >= (int64_t{1} << 31) ||
      static_cast<int64_t>(d.T) * d.d >= (int64_t{1} << 31) || int64_t{2} * d.F * d.d >= (int64_t{1} << 31))
    return MASKMOE_E_UNSUPPORTED;
  const Layout w = layout(d);
  if (!train_workspace || train_workspace_bytes < w.train_total || !aligned(train_workspace, 256))
    return MASKMOE_E_WORKSPACE;
  if (!workspace || workspace_bytes < bl.total || !aligned(workspace, 256)) return MASKMOE_E_WORKSPACE;

  char* tw = static_cast<char*>(const_cast<void*>(train_workspace));
  maskmoe::BwdArgs a;
  a.x = static_cast<const uint16_t*>(x);
  a.w_gate_up = static_cast<const uint16_t*>(w_gate_up);
  a.w_down = static_cast<const uint16_t*>(w_down);
  a.ws_gate_up = static_cast<const uint16_t*>(ws_gate_up);
  a.ws_down = static_cast<const uint16_t*>(ws_down);
  a.gate = topk_gate;
  a.dy = static_cast<const uint16_t*>(dy);
  a.pb.offsets = reinterpret_cast<int32_t*>(tw + w.offsets);
  a.pb.tile_off = reinterpret_cast<int32_t*>(tw + w.tile_off);
  a.pb.active = reinterpret_cast<int32_t*>(tw + w.active);
  a.pb.n_active = reinterpret_cast<int32_t*>(tw + w.n_active);
  a.pb.perm = reinterpret_cast<int32_t*>(tw + w.perm);
  a.pb.inv = reinterpret_cast<int32_t*>(tw + w.inv);
  a.pb.row_tok = reinterpret_cast<int32_t*>(tw + w.row_tok);
  a.h = reinterpret_cast<const uint16_t*>(tw + w.H);
  a.ab = reinterpret_cast<const uint16_t*>(tw + w.AB);
  a.d_x = d_x;
  a.d_w_gate_up = d_w_gate_up;
  a.d_w_down = d_w_down;
  a.d_ws_gate_up = d_ws_gate_up;
  a.d_ws_down = d_ws_down;
  a.workspace = workspace;
  a.lay = bl;
  a.T = d.T; a.d = d.d; a.F = d.F; a.E = d.E; a.K = d.K; a.S = d.n_shared;
  const int64_t TK = static_cast<int64_t>(d.T) * d.K;
  const int64_t nonempty = TK < d.E ? TK : d.E;
  a.max_tiles = static_cast<int>(TK / maskmoe::kGemmBM + nonempty +
                                 static_cast<int64_t>(d.n_shared) * ((d.T + maskmoe::kGemmBM - 1) / maskmoe::kGemmBM));
  return hip_status(maskmoe::launch_layer_backward(a, stream));
}

size_t maskmoe_stage1_backward_workspace_bytes(const maskmoe_layer_desc* desc) {
  if (check_route_desc(desc) != MASKMOE_OK) return 0;
  return maskmoe::stage1_workspace_bytes(desc->T, desc->d, desc->E);
}

int maskmoe_stage1_backward(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                            const uint8_t* mask, const float* mask_logits, const int32_t* topk_idx,
                            const float* router_logits, const void* dy, const float* expert_out, float* d_gate,
                            float* d_mask, float* d_mask_logits, float* d_w_router, float* d_x, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  int st = check_route_desc(desc);
  if (st != MASKMOE_OK) return st;
  const maskmoe_layer_desc& d = *desc;
  if (d.route_mode != MASKMOE_ROUTE_HARD_MASK) return MASKMOE_E_INVAL;   // Stage 1 trains under the mask
  if (d.K > maskmoe::kMaxKTrain || d.E > maskmoe::kMaxETrain) return MASKMOE_E_UNSUPPORTED;
  st = check_mask_prior(d.route_mode, 1, d.E, d.K, mask, nullptr);
  if (st != MASKMOE_OK) return st;
  if (d_mask_logits) {
    if (!mask_logits) return MASKMOE_E_INVAL;
    for (int e = 0; e < d.E; ++e)
      if (!isfinite(mask_logits[e])) return MASKMOE_E_INVAL;
  }
  if (!d_w_router) return MASKMOE_E_INVAL;
  if (static_cast<int64_t>(d.T) * d.E >= (int64_t{1} << 31)) return MASKMOE_E_UNSUPPORTED;
  if (d.T == 0) return MASKMOE_OK;   // no token: no gradient is written or accumulated
  if (!x || !w_router || !topk_idx || !router_logits || !dy || !expert_out) return MASKMOE_E_INVAL;
  const size_t el = d.dtype == MASKMOE_BF16 ? 2 : 4;
  const void* in[] = {x, w_router, dy};
  for (const void* p : in)
    if (!aligned(p, el)) return MASKMOE_E_INVAL;
  const void* f4[] = {topk_idx, router_logits, expert_out, d_w_router};
  for (const void* p : f4)
    if (!aligned(p, 4)) return MASKMOE_E_INVAL;
  if ((d_gate && !aligned(d_gate, 4)) || (d_mask && !aligned(d_mask, 4)) ||
      (d_mask_logits && !aligned(d_mask_logits, 4)) || (d_x && !aligned(d_x, 4)))
    return MASKMOE_E_INVAL;
  const size_t need = maskmoe::stage1_workspace_bytes(d.T, d.d, d.E);
  if (!workspace || workspace_bytes < need || !aligned(workspace, 256)) return MASKMOE_E_WORKSPACE;

  double pi[maskmoe::kMaxETrain];
  if (mask_logits) maskmoe::softmax_f64(mask_logits, d.E, pi);
  else for (int e = 0; e < d.E; ++e) pi[e] = 0.0;
  char* ws = static_cast<char*>(workspace);
  const size_t tok = (static_cast<size_t>(d.T) * d.E * 4 + 255) / 256 * 256;
  maskmoe::Stage1Args a;
  a.x = x; a.w_router = w_router; a.dy = dy; a.expert_out = expert_out; a.router_logits = router_logits;
  a.idx = topk_idx; a.pi = pi; a.d_gate = d_gate; a.d_mask = d_mask; a.d_mask_logits = d_mask_logits;
  a.d_w_router = d_w_router; a.d_x = d_x;
  const size_t dmb = (static_cast<size_t>(d.E) * 4 + 255) / 256 * 256;
  a.dz = reinterpret_cast<float*>(ws);
  a.dm_tok = reinterpret_cast<float*>(ws + tok);
  a.dm = reinterpret_cast<float*>(ws + 2 * tok);
  a.wgrad_partial = reinterpret_cast<float*>(ws + 2 * tok + dmb);
  a.T = d.T; a.d = d.d; a.E = d.E; a.K = d.K; a.gate_mode = d.gate_mode;
  a.vec_rows = d.d % 4 == 0 && aligned(expert_out, 16) && aligned(dy, 4 * el);
  a.vec_x = (d.d * el) % 16 == 0 && aligned(x, 16);
  return hip_status(maskmoe::launch_stage1_backward(a, d.dtype == MASKMOE_BF16, stream));
}

int maskmoe_sample_mask(const float* mask_logits, const double* uniforms, int32_t L, int32_t E, int32_t e_keep,
                        uint8_t* mask) {
  if (L < 1 || E < 1 || E > maskmoe::kMaxETrain || e_keep < 1 || e_keep > E) return MASKMOE_E_INVAL;
  if (!mask_logits || !uniforms || !mask) return MASKMOE_E_INVAL;
  for (size_t i = 0; i < static_cast<size_t>(L) * E; ++i)
    if (!isfinite(mask_logits[i])) return MASKMOE_E_INVAL;
  for (size_t i = 0; i < static_cast<size_t>(L) * e_keep; ++i)
    if (!(uniforms[i] >= 0.0 && uniforms[i] < 1.0)) return MASKMOE_E_INVAL;
  for (int l = 0; l < L; ++l)
    maskmoe::sample_mask_host(mask_logits + static_cast<size_t>(l) * E, uniforms + static_cast<size_t>(l) * e_keep,
                              E, e_keep, mask + static_cast<size_t>(l) * E);
  return MASKMOE_OK;
}

int maskmoe_cache_fetches(const int32_t* trace, int32_t L, int32_t S, int32_t N, int32_t K, int32_t E,
                          int32_t B, int32_t policy, int32_t* state, int32_t* counts, int64_t* fetches,
                          int64_t* hits, uint8_t* f_per_step, int32_t* dev_error, hipStream_t stream) {
  if (L < 0 || S < 0 || N < 0 || K < 1 || E < 1 || K > E || B < K) return MASKMOE_E_INVAL;
  if (policy != MASKMOE_CACHE_LRU && policy != MASKMOE_CACHE_LFU && policy != MASKMOE_CACHE_FIFO)
    return MASKMOE_E_INVAL;
  if (E > kCacheMaxE) return MASKMOE_E_UNSUPPORTED;
  if (static_cast<int64_t>(N) * K + B >= (int64_t{1} << 24)) return MASKMOE_E_UNSUPPORTED;
  if (static_cast<int64_t>(L) * S >= (int64_t{1} << 31)) return MASKMOE_E_INVAL;
  if (static_cast<int64_t>(L) * S == 0) return MASKMOE_OK;
  if (!fetches || !hits || (N > 0 && !trace)) return MASKMOE_E_INVAL;
  if (!aligned(fetches, 8) || !aligned(hits, 8) || (trace && !aligned(trace, 4)) ||
      (state && !aligned(state, 4)) || (counts && !aligned(counts, 4)) || (dev_error && !aligned(dev_error, 4)))
    return MASKMOE_E_INVAL;
  return hip_status(maskmoe::launch_cache(policy, trace, L, S, N, K, E, B, state,
                                          policy == MASKMOE_CACHE_LFU ? counts : nullptr, fetches, hits,
                                          f_per_step, dev_error, stream));
}

size_t maskmoe_offload_workspace_bytes(const maskmoe_layer_desc* desc) {
  if (check_layer_desc(desc) != MASKMOE_OK) return 0;
  return layout(*desc).offload_total;
}

// Device-side address of pinned host memory; null when p is not pinned host memory.
static const void* host_device_address(const void* p) {
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
    (void)hipGetLastError();   // clear the error this query leaves for unknown pointers
    return nullptr;
  }
  if (attr.type != hipMemoryTypeHost) return nullptr;
  return attr.devicePointer;
}

int maskmoe_offload_decode_step(const maskmoe_layer_desc* desc, const void* x, const void* w_router,
                                const uint8_t* mask, const float* prior, const void* host_w_gate_up,
                                const void* host_w_down, const void* ws_gate_up, const void* ws_down, int32_t B,
                                int32_t policy, void* slots_gate_up, void* slots_down, int32_t* cache_state,
                                void* y, int32_t* topk_idx, float* topk_gate, int64_t* counters,
                                int32_t* dev_error, void* workspace, size_t workspace_bytes, hipEvent_t* events,
                                hipStream_t stream) {
  int st = check_layer_desc(desc);
  if (st != MASKMOE_OK) return st;
  const maskmoe_layer_desc& d = *desc;
  st = check_mask_prior(d.route_mode, 1, d.E, d.K, mask, prior);
  if (st != MASKMOE_OK) return st;
  if (policy != MASKMOE_CACHE_LRU && policy != MASKMOE_CACHE_LFU && policy != MASKMOE_CACHE_FIFO)
    return MASKMOE_E_INVAL;
  if (B < d.K || B > d.E) return MASKMOE_E_INVAL;
  if (d.T != 1 || d.dtype != MASKMOE_BF16 || d.E > maskmoe::kOffloadMaxE) return MASKMOE_E_UNSUPPORTED;
  if (d.d % 64 != 0 || d.F % 64 != 0 || int64_t{2} * d.F * d.d >= (int64_t{1} << 31)) return MASKMOE_E_UNSUPPORTED;
  if (!x || !w_router || !host_w_gate_up || !host_w_down || !slots_gate_up || !slots_down || !cache_state || !y)
    return MASKMOE_E_INVAL;
  if (d.n_shared > 0 && (!ws_gate_up || !ws_down)) return MASKMOE_E_INVAL;
  const void* p16[] = {x, w_router, host_w_gate_up, host_w_down, slots_gate_up, slots_down, y};
  for (const void* p : p16)
    if (!aligned(p, 16)) return MASKMOE_E_INVAL;
  if (d.n_shared > 0 && (!aligned(ws_gate_up, 16) || !aligned(ws_down, 16))) return MASKMOE_E_INVAL;
  if (!aligned(cache_state, 4) || (topk_idx && !aligned(topk_idx, 4)) || (topk_gate && !aligned(topk_gate, 4)) ||
      (counters && !aligned(counters, 8)) || (dev_error && !aligned(dev_error, 4)))
    return MASKMOE_E_INVAL;
  // the expert copies must be pinned host memory, which the fetch kernel reads through its
  // device mapping
  const void* host_gu = host_device_address(host_w_gate_up);
  const void* host_dn = host_device_address(host_w_down);
  if (!host_gu || !host_dn) return MASKMOE_E_INVAL;
  const Layout w = layout(d);
  if (!workspace || workspace_bytes < w.offload_total || !aligned(workspace, 256)) return MASKMOE_E_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  int32_t* idx = topk_idx ? topk_idx : reinterpret_cast<int32_t*>(ws + w.idx);
  float* gate = topk_gate ? topk_gate : reinterpret_cast<float*>(ws + w.gate);
  PermBuffers pb;
  pb.offsets = reinterpret_cast<int32_t*>(ws + w.offsets);
  pb.tile_off = reinterpret_cast<int32_t*>(ws + w.tile_off);
  pb.active = reinterpret_cast<int32_t*>(ws + w.active);
  pb.n_active = reinterpret_cast<int32_t*>(ws + w.n_active);
  pb.perm = reinterpret_cast<int32_t*>(ws + w.perm);
  pb.inv = reinterpret_cast<int32_t*>(ws + w.inv);
  pb.row_tok = reinterpret_cast<int32_t*>(ws + w.row_tok);
  int32_t* fetch = reinterpret_cast<int32_t*>(ws + w.FL);

  hipError_t e = maskmoe::launch_route_permute(x, w_router, d.T, d.d, d.E, d.K, d.route_mode, d.gate_mode, mask,
                                               prior, idx, gate, nullptr, d.n_shared, maskmoe::kGemmBM, pb, stream);
  if (e != hipSuccess) return MASKMOE_E_HIP;
  e = maskmoe::launch_offload_cache(policy, idx, d.E, d.K, B, cache_state, fetch, counters, dev_error, stream);
  if (e != hipSuccess) return MASKMOE_E_HIP;
  maskmoe::record_mark(events, 0, stream);
  e = maskmoe::launch_offload_fetch(fetch, d.K, d.E, B, d.d, d.F, host_gu, host_dn, slots_gate_up, slots_down,
                                    stream);
  if (e != hipSuccess) return MASKMOE_E_HIP;
  maskmoe::record_mark(events, 1, stream);
  maskmoe::ExpertArgs a;
  a.x = x;
  a.w_gate_up = slots_gate_up;
  a.w_down = slots_down;
  a.ws_gate_up = ws_gate_up;
  a.ws_down = ws_down;
  a.gate = gate;
  a.expert_out = nullptr;
  a.slot_of = cache_state + B + d.E;
  a.n_slots = B;
  a.packed = d.weight_layout == MASKMOE_LAYOUT_PACKED;   // the pool holds copies of the host experts
  a.T = d.T; a.d = d.d; a.F = d.F; a.E = d.E; a.K = d.K; a.n_shared = d.n_shared;
  e = maskmoe::launch_experts_bf16_decode(a, pb, reinterpret_cast<uint16_t*>(ws + w.H),
                                          reinterpret_cast<float*>(ws + w.P), reinterpret_cast<float*>(ws + w.O), y,
                                          stream, nullptr);
  return hip_status(e);
}

}  // extern "C"
