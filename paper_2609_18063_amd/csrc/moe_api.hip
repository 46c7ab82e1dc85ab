// C ABI of the MoE decode hot path (declarations and contracts in
// include/moe_api.h): argument checks, the slot table, the workspace layout
// and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "moe_engine.h"
#include "moe_grouped.h"
#include "moe_kernels.h"
#include "moe_table.h"

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

bool pow2_dim(int v) {
  return v == 256 || v == 512 || v == 1024 || v == 2048 || v == 4096 || v == 8192;
}

struct WsLayout {
  size_t counters, logits, gx, ux, h, ag, au, adpart;
  size_t g_perm, g_tiles, g_tok, g_ntiles, g_h, g_xp, g_ax, g_adp;  // grouped (batched) path
  int g_max_tiles;
  size_t total;
};

WsLayout ws_layout(const moe_layer_spec* s, int T) {
  WsLayout w{};
  const size_t n = (size_t)(s->top_k + s->n_shared);
  const size_t r = (size_t)(s->lora_rank > 0 ? s->lora_rank : 1);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = round_up(off + bytes, kAlign);
    return o;
  };
  w.counters = take((size_t)T * sizeof(uint32_t));
  w.logits = take((size_t)T * s->n_experts * sizeof(float));
  w.gx = take((size_t)T * n * s->d_expert * sizeof(float));
  w.ux = take((size_t)T * n * s->d_expert * sizeof(float));
  w.h = take((size_t)T * n * s->d_expert * sizeof(float));
  w.ag = take((size_t)T * n * r * sizeof(float));
  w.au = take((size_t)T * n * r * sizeof(float));
  w.adpart = take((size_t)T * n * (s->d_expert / 64) * r * sizeof(float));
  w.g_max_tiles = moe::grouped_max_tiles(T, (int)n, s->n_experts + s->n_shared);
  w.g_perm = take((size_t)T * n * sizeof(int32_t));
  w.g_tiles = take((size_t)w.g_max_tiles * sizeof(moe::GroupTile));
  w.g_tok = take((size_t)w.g_max_tiles * moe::kGroupRows * sizeof(int32_t));
  w.g_ntiles = take(sizeof(int32_t));
  w.g_h = take((size_t)T * n * s->d_expert * sizeof(__half));
  w.g_xp = take((size_t)T * s->d_model * sizeof(__half));
  w.g_ax = take((size_t)T * n * 4 * 2 * 16 * sizeof(float));
  w.g_adp = take((size_t)T * n * (s->d_expert / moe::kGroupSlab > 0 ? s->d_expert / moe::kGroupSlab : 1) * 16 * sizeof(float));
  w.total = off;
  return w;
}

int from_hip(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_EHIP; }

// Armed per-launch timing events (moe_profile_arm), per host thread.
struct ProfArm {
  hipEvent_t start = nullptr, stop = nullptr;
};
thread_local ProfArm g_prof_ffn;
thread_local void* g_prof_engine_ts = nullptr;

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

// Scratch of moe_expert_ffn_int4_lora_noalloc: one array per device, resident
// until the process ends. Host code never passes `scratch` itself (on the host
// it names a stand-in, not device memory): it passes the device address that
// hipGetSymbolAddress returns for the current device, looked up once per device.
__device__ __align__(256) char scratch[MOE_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_of_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return MOE_EINVAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MOE_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MOE_OK;
}

}  // namespace

extern "C" {

int moe_spec_check(const moe_layer_spec* s) {
  if (!s) return MOE_EINVAL;
  if (!pow2_dim(s->d_model) || s->d_model < 512) return MOE_EINVAL;
  if (!pow2_dim(s->d_expert)) return MOE_EINVAL;
  if (s->n_experts < 1 || s->n_experts > 1024) return MOE_EINVAL;
  if (s->top_k < 1 || s->top_k > 32 || s->top_k > s->n_experts) return MOE_EINVAL;
  if (s->n_shared < 0 || s->n_shared > 4) return MOE_EINVAL;
  if (s->group_size != 64) return MOE_EINVAL;
  if (s->lora_rank < 0 || s->lora_rank > 64) return MOE_EINVAL;
  if (!(s->lora_scale == s->lora_scale)) return MOE_EINVAL;
  if (s->routing == MOE_ROUTING_SOFTMAX_TOPK) {
    if (s->n_groups != 0 || s->top_groups != 0 || s->route_scale != 0.f) return MOE_EINVAL;
  } else if (s->routing == MOE_ROUTING_SIGMOID_GROUP) {
    const int n = s->n_groups, E = s->n_experts;
    if (n < 1 || E > 256 || E % n) return MOE_EINVAL;
    if (s->top_groups < 1 || s->top_groups > n || s->top_k > s->top_groups * (E / n)) return MOE_EINVAL;
    if (!(s->route_scale > 0.f) || s->route_scale > 1e30f) return MOE_EINVAL;
  } else {
    return MOE_EINVAL;
  }
  for (int i = 0; i < 4; ++i)
    if (s->reserved[i] != 0) return MOE_EINVAL;
  return MOE_OK;
}

const char* moe_strerror(int code) {
  switch (code) {
    case MOE_OK: return "ok";
    case MOE_EINVAL: return "invalid argument (spec, shape, null pointer or index)";
    case MOE_EALIGN: return "device pointer not 16-byte aligned";
    case MOE_ENOTRESIDENT: return "expert not resident in the slot table";
    case MOE_EHIP: return "HIP runtime or kernel launch error";
    case MOE_ENOMEM: return "workspace too small or allocation failed";
  }
  return "unknown error";
}

// ---- slot table ------------------------------------------------------------

int moe_slot_table_create(int n_layers, int n_ids, int n_slots, moe_slot_table** out) {
  if (!out || n_layers < 1 || n_ids < 1 || n_slots < 1) return MOE_EINVAL;
  if ((long long)n_layers * n_ids > (1LL << 28) || (long long)n_layers * n_slots > (1LL << 24))
    return MOE_EINVAL;
  moe_slot_table* t = new (std::nothrow) moe_slot_table;
  if (!t) return MOE_ENOMEM;
  t->n_layers = n_layers;
  t->n_ids = n_ids;
  t->n_slots = n_slots;
  t->slot_of.assign((size_t)n_layers * n_ids, -1);
  t->expert_in.assign((size_t)n_layers * n_slots, -1);
  t->bundles.assign((size_t)n_layers * n_slots, moe_bundle{});
  *out = t;
  return MOE_OK;
}

int moe_slot_table_destroy(moe_slot_table* t) {
  if (!t) return MOE_EINVAL;
  int rc = MOE_OK;
  if (t->copied) {
    if (t->copy_pending && hipEventSynchronize(t->copied) != hipSuccess) rc = MOE_EHIP;
    (void)hipEventDestroy(t->copied);
  }
  if (t->pinned) (void)hipHostFree(t->pinned);
  if (t->dev) (void)hipFree(t->dev);
  delete t;
  return rc;
}

int moe_slot_bind(moe_slot_table* t, int layer, int expert, int slot, const moe_bundle* b) {
  if (!t || !b || layer < 0 || layer >= t->n_layers || expert < 0 || expert >= t->n_ids ||
      slot < 0 || slot >= t->n_slots)
    return MOE_EINVAL;
  const moe_proj* ps[3] = {&b->gate, &b->up, &b->down};
  for (const moe_proj* p : ps) {
    if (!p->q || !p->sz) return MOE_EINVAL;
    if (!aligned16(p->q) || !aligned16(p->sz)) return MOE_EALIGN;
    if ((p->lora_a && !aligned16(p->lora_a)) || (p->lora_b && !aligned16(p->lora_b)))
      return MOE_EALIGN;
  }
  int32_t* so = &t->slot_of[(size_t)layer * t->n_ids];
  int32_t* ei = &t->expert_in[(size_t)layer * t->n_slots];
  const int old = ei[slot];
  if (old >= 0) so[old] = -1;
  const int prev = so[expert];
  if (prev >= 0) ei[prev] = -1;
  so[expert] = slot;
  ei[slot] = expert;
  t->bundles[(size_t)layer * t->n_slots + slot] = *b;
  return MOE_OK;
}

int moe_slot_unbind(moe_slot_table* t, int layer, int expert) {
  if (!t || layer < 0 || layer >= t->n_layers || expert < 0 || expert >= t->n_ids)
    return MOE_EINVAL;
  int32_t* so = &t->slot_of[(size_t)layer * t->n_ids];
  const int s = so[expert];
  if (s >= 0) t->expert_in[(size_t)layer * t->n_slots + s] = -1;
  so[expert] = -1;
  return MOE_OK;
}

int moe_slot_lookup(const moe_slot_table* t, int layer, int expert) {
  if (!t || layer < 0 || layer >= t->n_layers || expert < 0 || expert >= t->n_ids)
    return MOE_EINVAL;
  const int s = t->slot_of[(size_t)layer * t->n_ids + expert];
  return s >= 0 ? s : MOE_ENOTRESIDENT;
}

int moe_slot_table_sync(moe_slot_table* t, void* stream) {
  if (!t) return MOE_EINVAL;
  const size_t so_bytes = t->slot_of.size() * sizeof(int32_t);
  const size_t b_off = round_up(so_bytes, kAlign);
  const size_t total = b_off + t->bundles.size() * sizeof(moe_bundle);
  if (!t->dev) {
    if (hipMalloc(&t->dev, total) != hipSuccess) {
      t->dev = nullptr;
      return MOE_ENOMEM;
    }
    if (hipHostMalloc(&t->pinned, total, hipHostMallocDefault) != hipSuccess) {
      t->pinned = nullptr;
      return MOE_ENOMEM;
    }
    if (hipEventCreateWithFlags(&t->copied, hipEventDisableTiming) != hipSuccess) return MOE_EHIP;
    t->dev_bytes = total;
    t->bundles_off = b_off;
  }
  // the staging buffer may still be read by the previous copy
  if (t->copy_pending && hipEventSynchronize(t->copied) != hipSuccess) return MOE_EHIP;
  std::memcpy(t->pinned, t->slot_of.data(), so_bytes);
  std::memcpy(static_cast<char*>(t->pinned) + b_off, t->bundles.data(),
              t->bundles.size() * sizeof(moe_bundle));
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipMemcpyAsync(t->dev, t->pinned, total, hipMemcpyHostToDevice, st) != hipSuccess)
    return MOE_EHIP;
  if (hipEventRecord(t->copied, st) != hipSuccess) return MOE_EHIP;
  t->copy_pending = true;
  return MOE_OK;
}

// ---- hot path ----------------------------------------------------------------

int moe_rmsnorm_f16(const float* xi, int T, int d, void* x_f16, void* stream) {
  if (T < 0 || d < 1) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!xi || !x_f16) return MOE_EINVAL;
  if (!aligned16(xi) || !aligned16(x_f16)) return MOE_EALIGN;
  return from_hip(moe::launch_rmsnorm(xi, T, d, static_cast<__half*>(x_f16),
                                      static_cast<hipStream_t>(stream)));
}

size_t moe_workspace_bytes(const moe_layer_spec* spec, int T) {
  if (moe_spec_check(spec) != MOE_OK || T < 0) return 0;
  return ws_layout(spec, T < 1 ? 1 : T).total;
}

static int route_common(const moe_layer_spec* s, const void* x, const void* W, int T,
                        float* logits_opt, int32_t* idx, float* w, void* ws, size_t ws_bytes,
                        void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (T < 0) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!x || !W || !idx || !w || !ws) return MOE_EINVAL;
  if (!aligned16(x) || !aligned16(W) || !aligned16(ws) || !aligned4(idx) || !aligned4(w) ||
      (logits_opt && !aligned16(logits_opt)))
    return MOE_EALIGN;
  const WsLayout L = ws_layout(s, T);
  if (ws_bytes < L.total) return MOE_ENOMEM;
  float* logits = logits_opt ? logits_opt : at<float>(ws, L.logits);
  const bool sg = s->routing == MOE_ROUTING_SIGMOID_GROUP;
  hipError_t e = moe::launch_route(static_cast<const __half*>(x), static_cast<const __half*>(W), T,
                                   s->n_experts, s->d_model, s->top_k, logits, sg ? nullptr : idx, w,
                                   at<uint32_t>(ws, L.counters), static_cast<hipStream_t>(stream));
  if (e == hipSuccess && sg)
    e = moe::launch_topk_sigmoid_group(logits, nullptr, T, s->n_experts, s->top_k, s->n_groups,
                                       s->top_groups, s->route_scale, idx, w,
                                       static_cast<hipStream_t>(stream));
  return from_hip(e);
}

int moe_route(const moe_layer_spec* spec, const void* x_f16, const void* w_router_f16, int T,
              float* logits_opt, int32_t* idx, float* w, void* workspace, size_t workspace_bytes,
              void* stream) {
  return route_common(spec, x_f16, w_router_f16, T, logits_opt, idx, w, workspace,
                      workspace_bytes, stream);
}

int moe_preroute(const moe_layer_spec* next, const void* x_f16, const void* w_head_f16, int T,
                 float* logits_opt, int32_t* pred_idx, float* pred_w, void* workspace,
                 size_t workspace_bytes, void* stream) {
  return route_common(next, x_f16, w_head_f16, T, logits_opt, pred_idx, pred_w, workspace,
                      workspace_bytes, stream);
}

size_t moe_preroute_mlp_workspace_bytes(const moe_layer_spec* next, int hidden, int T) {
  if (moe_spec_check(next) != MOE_OK || hidden <= 0 || T < 0) return 0;
  const size_t t = (size_t)(T < 1 ? 1 : T);
  return (t * hidden * 2 + 255) / 256 * 256 + t * next->n_experts * 4;
}

int moe_preroute_mlp(const moe_layer_spec* next, const moe_head_mlp* head, const void* x_f16, int T,
                     const int32_t* routed_t, const int32_t* routed_tm1, float* logits_opt,
                     int32_t* pred_idx, float* pred_w, void* ws, size_t ws_bytes, void* stream) {
  int rc = moe_spec_check(next);
  if (rc != MOE_OK) return rc;
  if (!head || T < 0) return MOE_EINVAL;
  const int H = head->hidden, d = next->d_model, E = next->n_experts, K = next->top_k;
  if (H <= 0 || H % 8 || d % 8 || E % 8 || K > 32) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!x_f16 || !head->w1_x || !head->w1_r || !head->w2 || !routed_t || !pred_idx || !pred_w || !ws)
    return MOE_EINVAL;
  if (!aligned16(x_f16) || !aligned16(head->w1_x) || !aligned16(head->w1_r) || !aligned16(head->w2) ||
      (head->b1 && !aligned16(head->b1)) || (head->b2 && !aligned16(head->b2)) ||
      (head->w_l && !aligned16(head->w_l)) || !aligned4(routed_t) || (routed_tm1 && !aligned4(routed_tm1)) ||
      !aligned4(pred_idx) || !aligned4(pred_w) || !aligned16(ws) || (logits_opt && !aligned16(logits_opt)))
    return MOE_EALIGN;
  if (ws_bytes < moe_preroute_mlp_workspace_bytes(next, H, T)) return MOE_ENOMEM;
  moe::HeadMlpArgs a{};
  a.T = T;
  a.d = d;
  a.E = E;
  a.K = K;
  a.H = H;
  a.x = static_cast<const __half*>(x_f16);
  a.w1x = static_cast<const __half*>(head->w1_x);
  a.w1r = static_cast<const __half*>(head->w1_r);
  a.b1 = static_cast<const __half*>(head->b1);
  a.w2 = static_cast<const __half*>(head->w2);
  a.b2 = static_cast<const __half*>(head->b2);
  a.wl = static_cast<const __half*>(head->w_l);
  a.routed_t = routed_t;
  a.routed_tm1 = routed_tm1;
  a.hidden = static_cast<__half*>(ws);
  a.logits = logits_opt ? logits_opt
                        : reinterpret_cast<float*>(static_cast<char*>(ws) + ((size_t)T * H * 2 + 255) / 256 * 256);
  a.idx = pred_idx;
  a.w = pred_w;
  a.n_groups = next->routing == MOE_ROUTING_SIGMOID_GROUP ? next->n_groups : 0;
  a.top_groups = next->top_groups;
  a.route_scale = next->route_scale;
  return from_hip(moe::launch_head_mlp(a, static_cast<hipStream_t>(stream)));
}

int moe_expert_ffn_int4_lora(const moe_layer_spec* s, const moe_slot_table* t, int layer,
                             const void* x_f16, int T, const int32_t* idx, float* y_experts,
                             uint32_t* status_dev, void* ws, size_t ws_bytes, void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (!t || T < 0) return MOE_EINVAL;
  if (layer < 0 || layer >= t->n_layers || t->n_ids < s->n_experts + s->n_shared)
    return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!x_f16 || !idx || !y_experts || !ws) return MOE_EINVAL;
  if (!t->dev) return MOE_EINVAL;  // never synced to the device
  if (!aligned16(x_f16) || !aligned16(y_experts) || !aligned16(ws) || !aligned4(idx) ||
      (status_dev && !aligned4(status_dev)))
    return MOE_EALIGN;
  const WsLayout L = ws_layout(s, T);
  if (ws_bytes < L.total) return MOE_ENOMEM;
  moe::FfnArgs a{};
  a.d = s->d_model;
  a.I = s->d_expert;
  a.E = s->n_experts;
  a.K = s->top_k;
  a.S = s->n_shared;
  a.r = s->lora_rank;
  a.n_list = a.K + a.S;
  a.lora_scale = s->lora_scale;
  a.x = static_cast<const __half*>(x_f16);
  a.idx = idx;
  a.slot_of = reinterpret_cast<const int32_t*>(t->dev) + (size_t)layer * t->n_ids;
  a.bundles = reinterpret_cast<const moe_bundle*>(static_cast<const char*>(t->dev) + t->bundles_off) +
              (size_t)layer * t->n_slots;
  a.status = status_dev;
  a.gx = at<float>(ws, L.gx);
  a.ux = at<float>(ws, L.ux);
  a.h = at<float>(ws, L.h);
  a.ag = at<float>(ws, L.ag);
  a.au = at<float>(ws, L.au);
  a.adpart = at<float>(ws, L.adpart);
  a.y_experts = y_experts;
  ProfArm arm = g_prof_ffn;
  g_prof_ffn = ProfArm{};
  return from_hip(moe::launch_ffn(a, T, static_cast<hipStream_t>(stream), arm.start, arm.stop));
}

int moe_expert_ffn_int4_lora_noalloc(const moe_layer_spec* s, const moe_slot_table* t, int layer,
                                     const void* x_f16, int T, const int32_t* idx, float* y_experts,
                                     uint32_t* status_dev, void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (T < 0) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (ws_layout(s, T).total > MOE_NOALLOC_SCRATCH_BYTES) return MOE_ENOMEM;
  void* ws = nullptr;
  rc = scratch_of_current_device(&ws);
  if (rc != MOE_OK) return rc;
  return moe_expert_ffn_int4_lora(s, t, layer, x_f16, T, idx, y_experts, status_dev, ws,
                                  MOE_NOALLOC_SCRATCH_BYTES, stream);
}

int moe_expert_ffn_grouped_int4_lora(const moe_layer_spec* s, const moe_slot_table* t, int layer,
                                     const void* x_f16, int T, const int32_t* idx, float* y_experts,
                                     uint32_t* status_dev, void* ws, size_t ws_bytes, void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (!t || T < 0) return MOE_EINVAL;
  if (layer < 0 || layer >= t->n_layers || t->n_ids < s->n_experts + s->n_shared)
    return MOE_EINVAL;
  if (!moe::grouped_shape_supported(s->d_model, s->d_expert, s->lora_rank,
                                    s->n_experts + s->n_shared))
    return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!x_f16 || !idx || !y_experts || !ws) return MOE_EINVAL;
  if (!t->dev) return MOE_EINVAL;  // never synced to the device
  if (!aligned16(x_f16) || !aligned16(y_experts) || !aligned16(ws) || !aligned4(idx) ||
      (status_dev && !aligned4(status_dev)))
    return MOE_EALIGN;
  const WsLayout L = ws_layout(s, T);
  if (ws_bytes < L.total) return MOE_ENOMEM;
  moe::GroupedArgs a{};
  a.T = T;
  a.d = s->d_model;
  a.I = s->d_expert;
  a.E = s->n_experts;
  a.K = s->top_k;
  a.S = s->n_shared;
  a.r = s->lora_rank;
  a.n_list = a.K + a.S;
  a.n_ids = t->n_ids;
  a.lora_scale = s->lora_scale;
  a.x = static_cast<const __half*>(x_f16);
  a.idx = idx;
  a.slot_of = reinterpret_cast<const int32_t*>(t->dev) + (size_t)layer * t->n_ids;
  a.bundles = reinterpret_cast<const moe_bundle*>(static_cast<const char*>(t->dev) + t->bundles_off) +
              (size_t)layer * t->n_slots;
  a.status = status_dev;
  a.perm = at<int32_t>(ws, L.g_perm);
  a.tiles = at<moe::GroupTile>(ws, L.g_tiles);
  a.tile_tok = at<int32_t>(ws, L.g_tok);
  a.n_tiles = at<int32_t>(ws, L.g_ntiles);
  a.max_tiles = L.g_max_tiles;
  a.h = at<__half>(ws, L.g_h);
  a.xp = at<__half>(ws, L.g_xp);
  a.ax = at<float>(ws, L.g_ax);
  a.adp = at<float>(ws, L.g_adp);
  a.y_experts = y_experts;
  return from_hip(moe::launch_grouped_ffn(a, static_cast<hipStream_t>(stream)));
}

static int combine_common(const moe_layer_spec* s, const float* y_experts, const float* w, int T,
                          float* y, int accumulate, void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (T < 0) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!y_experts || !w || !y) return MOE_EINVAL;
  if (!aligned16(y_experts) || !aligned4(w) || !aligned16(y)) return MOE_EALIGN;
  return from_hip(moe::launch_combine(y_experts, w, T, s->top_k, s->n_shared, s->d_model, y,
                                      accumulate, static_cast<hipStream_t>(stream)));
}

int moe_merge_requantize(const moe_proj* src, int out_dim, int in_dim, int rank, float lora_scale,
                         void* q_out, void* sz_out, double* stats, void* stream) {
  if (!src || !src->q || !src->sz || !q_out || !sz_out) return MOE_EINVAL;
  if (out_dim < 1 || in_dim < 64 || in_dim % 64) return MOE_EINVAL;
  const bool adapter = src->lora_a && src->lora_b;
  if (adapter && (rank < 1 || rank > 64)) return MOE_EINVAL;
  if ((long long)out_dim * (in_dim / 64) > (1ll << 31) - 4) return MOE_EINVAL;
  auto a2 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 1) == 0; };
  if (!a2(src->sz) || !a2(sz_out) || (adapter && (!a2(src->lora_a) || !a2(src->lora_b))) ||
      (stats && (reinterpret_cast<uintptr_t>(stats) & 7)))
    return MOE_EALIGN;
  return from_hip(moe::launch_merge_requantize(
      static_cast<const uint8_t*>(src->q), static_cast<const __half*>(src->sz),
      adapter ? static_cast<const __half*>(src->lora_a) : nullptr,
      adapter ? static_cast<const __half*>(src->lora_b) : nullptr, out_dim, in_dim,
      adapter ? rank : 0, lora_scale, static_cast<uint8_t*>(q_out), static_cast<__half*>(sz_out),
      stats, static_cast<hipStream_t>(stream)));
}

int moe_combine(const moe_layer_spec* s, const float* y_experts, const float* w, int T, float* y,
                void* stream) {
  return combine_common(s, y_experts, w, T, y, 0, stream);
}

int moe_combine_add(const moe_layer_spec* s, const float* y_experts, const float* w, int T,
                    float* y_inout, void* stream) {
  return combine_common(s, y_experts, w, T, y_inout, 1, stream);
}

int moe_chain_token_start(const float* xi, int d, float* r_inout, void* stream) {
  if (!xi || !r_inout || d < 1 || d > 8192) return MOE_EINVAL;
  if (!aligned16(xi) || !aligned16(r_inout)) return MOE_EALIGN;
  return from_hip(moe::launch_chain_token_start(xi, d, r_inout, static_cast<hipStream_t>(stream)));
}

int moe_chain_mix_rmsnorm(const void* mix_d_f16, const int32_t* perm, int d, float* r_inout,
                          void* x_f16, void* stream) {
  if (!mix_d_f16 || !perm || !r_inout || !x_f16 || d < 1 || d > 8192) return MOE_EINVAL;
  if (!aligned16(mix_d_f16) || !aligned16(perm) || !aligned16(r_inout) || !aligned16(x_f16))
    return MOE_EALIGN;
  return from_hip(moe::launch_chain_mix_rmsnorm(static_cast<const __half*>(mix_d_f16), perm, d,
                                                r_inout, static_cast<__half*>(x_f16),
                                                static_cast<hipStream_t>(stream)));
}

int moe_topk(const moe_layer_spec* s, const float* logits, int T, int32_t* idx, float* w,
             void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (T < 0) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!logits || !idx || !w) return MOE_EINVAL;
  if (!aligned16(logits) || !aligned4(idx) || !aligned4(w)) return MOE_EALIGN;
  if (s->routing == MOE_ROUTING_SIGMOID_GROUP)
    return from_hip(moe::launch_topk_sigmoid_group(logits, nullptr, T, s->n_experts, s->top_k, s->n_groups,
                                                   s->top_groups, s->route_scale, idx, w,
                                                   static_cast<hipStream_t>(stream)));
  return from_hip(moe::launch_topk(logits, T, s->n_experts, s->top_k, idx, w,
                                   static_cast<hipStream_t>(stream)));
}

int moe_topk_biased(const moe_layer_spec* s, const float* logits, const float* bias, int T, int32_t* idx,
                    float* w, void* stream) {
  int rc = moe_spec_check(s);
  if (rc != MOE_OK) return rc;
  if (s->routing != MOE_ROUTING_SIGMOID_GROUP || T < 0) return MOE_EINVAL;
  if (T == 0) return MOE_OK;
  if (!logits || !idx || !w) return MOE_EINVAL;
  if (!aligned16(logits) || !aligned4(idx) || !aligned4(w) || (bias && !aligned4(bias))) return MOE_EALIGN;
  return from_hip(moe::launch_topk_sigmoid_group(logits, bias, T, s->n_experts, s->top_k, s->n_groups,
                                                 s->top_groups, s->route_scale, idx, w,
                                                 static_cast<hipStream_t>(stream)));
}

// ---- persistent decode engine ----------------------------------------------

int moe_engine_supported(const moe_layer_spec* s) {
  if (moe_spec_check(s) != MOE_OK || s->routing != MOE_ROUTING_SOFTMAX_TOPK) return MOE_EINVAL;
  if (!moe::engine_shape_supported(s->d_model, s->d_expert, s->lora_rank, s->top_k, s->n_shared,
                                   s->n_experts))
    return MOE_EINVAL;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_EHIP;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return MOE_EHIP;
  return cus == 256 ? MOE_OK : MOE_EINVAL;
}

static constexpr size_t kEngineCtlBytes = 256;

// the chain on two alternating halves of the chip (same device rule as
// moe_engine_supported); softmax-top-k or sigmoid-group routing
static int engine_pipe_supported(const moe_layer_spec* s) {
  if (moe_spec_check(s) != MOE_OK) return MOE_EINVAL;
  if (s->routing != MOE_ROUTING_SOFTMAX_TOPK && s->routing != MOE_ROUTING_SIGMOID_GROUP) return MOE_EINVAL;
  if (!moe::engine_pipe_supported(s->d_model, s->d_expert, s->lora_rank, s->top_k, s->n_shared,
                                  s->n_experts))
    return MOE_EINVAL;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_EHIP;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return MOE_EHIP;
  return cus == 256 ? MOE_OK : MOE_EINVAL;
}

// exchange words of the engine's schedule for a.mode (fills a's offsets)
static size_t engine_words(const moe_layer_spec* s, int n_layers, moe::EngineArgs* a) {
  if (a->mode == 3)
    return moe::engine_pipe_workspace_words(s->n_experts, s->d_model, s->d_expert, s->lora_rank,
                                            s->top_k + s->n_shared, n_layers, a);
  if (a->mode == 2)
    return moe::engine_tokens_workspace_words(s->n_experts, s->d_model, s->d_expert, s->lora_rank,
                                              s->top_k + s->n_shared, a);
  return moe::engine_workspace_words(s->n_experts, s->d_model, n_layers, a);
}

size_t moe_engine_workspace_bytes(const moe_layer_spec* s, int n_layers) {
  if (moe_spec_check(s) != MOE_OK || n_layers < 0) return 0;
  moe::EngineArgs a{};
  const size_t w0 = engine_words(s, n_layers, &a);
  a.mode = 2;
  const size_t w2 = engine_words(s, n_layers, &a);
  a.mode = 3;
  const size_t w3 = engine_words(s, n_layers, &a);
  return kEngineCtlBytes + std::max(w0, std::max(w2, w3)) * 8;
}

int moe_engine_tokens_supported(const moe_layer_spec* s) {
  if (moe_spec_check(s) != MOE_OK || s->routing != MOE_ROUTING_SOFTMAX_TOPK) return MOE_EINVAL;
  if (!moe::engine_tokens_supported(s->d_model, s->d_expert, s->lora_rank, s->top_k, s->n_shared,
                                    s->n_experts))
    return MOE_EINVAL;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return MOE_EHIP;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return MOE_EHIP;
  return cus == 256 ? MOE_OK : MOE_EINVAL;
}

static int engine_common(const moe_layer_spec* s, const moe_slot_table* t, int n_table_layers,
                         moe::EngineArgs& a, void* ws, size_t ws_bytes, void* stream) {
  int rc = a.mode == 2 ? moe_engine_tokens_supported(s)
                       : (a.mode == 3 ? engine_pipe_supported(s) : moe_engine_supported(s));
  if (rc != MOE_OK) return rc;
  if (!t || !ws || !a.layers || !a.xi) return MOE_EINVAL;
  if (!t->dev) return MOE_EINVAL;
  if (n_table_layers > t->n_layers || t->n_ids < s->n_experts + s->n_shared) return MOE_EINVAL;
  if (!aligned16(ws) || !aligned16(a.xi) || (a.y && !aligned16(a.y)) ||
      (a.r_state && !aligned16(a.r_state)) || (a.x_rec && !aligned16(a.x_rec)) ||
      (a.r_rec && !aligned4(a.r_rec)) ||
      (a.idx_rec && !aligned4(a.idx_rec)) || (a.w_rec && !aligned4(a.w_rec)) ||
      (a.pidx_rec && !aligned4(a.pidx_rec)) || (a.pw_rec && !aligned4(a.pw_rec)) ||
      (a.status && !aligned4(a.status)))
    return MOE_EALIGN;
  const size_t words = engine_words(s, a.L, &a);
  if (ws_bytes < kEngineCtlBytes + words * 8) return MOE_ENOMEM;
  a.E = s->n_experts;
  a.K = s->top_k;
  a.S = s->n_shared;
  a.r = s->lora_rank;
  a.lora_scale = s->lora_scale;
  a.n_groups = s->routing == MOE_ROUTING_SIGMOID_GROUP ? s->n_groups : 0;
  a.top_groups = s->top_groups;
  a.route_scale = s->route_scale;
  a.n_ids = t->n_ids;
  a.n_slots = t->n_slots;
  a.n_table_layers = t->n_layers;
  a.slot_of = reinterpret_cast<const int32_t*>(t->dev);
  a.bundles = reinterpret_cast<const moe_bundle*>(static_cast<const char*>(t->dev) + t->bundles_off);
  a.phase_ts = static_cast<uint64_t*>(g_prof_engine_ts);
  g_prof_engine_ts = nullptr;
  a.ctl = static_cast<uint32_t*>(ws);
  a.xw = reinterpret_cast<uint64_t*>(static_cast<char*>(ws) + kEngineCtlBytes);
  if (a.mode == 2)
    return from_hip(moe::launch_engine_tokens(a, s->d_model, s->d_expert, s->lora_rank,
                                              static_cast<hipStream_t>(stream)));
  if (a.mode == 3)
    return from_hip(moe::launch_engine_pipe(a, s->d_model, s->d_expert, s->lora_rank,
                                            static_cast<hipStream_t>(stream)));
  return from_hip(moe::launch_engine(a, s->d_model, s->d_expert, s->lora_rank,
                                     static_cast<hipStream_t>(stream)));
}

static int engine_steps(int mode, const moe_layer_spec* s, const moe_slot_table* t,
                        const moe_engine_layer* layers, const int32_t* step_layer, int n_steps,
                        const float* xi, float* y, int32_t* idx_rec, float* w_rec, int32_t* pidx_rec,
                        float* pw_rec, uint32_t* status, void* ws, size_t ws_bytes, void* stream) {
  if (n_steps < 0 || !step_layer || !y) return MOE_EINVAL;
  if (n_steps == 0) return MOE_OK;
  moe::EngineArgs a{};
  a.mode = mode;
  a.n_steps = n_steps;
  a.L = 0;
  a.layers = layers;
  a.step_layer = step_layer;
  a.xi = xi;
  a.y = y;
  a.idx_rec = idx_rec;
  a.w_rec = w_rec;
  a.pidx_rec = pidx_rec;
  a.pw_rec = pw_rec;
  a.status = status;
  return engine_common(s, t, t ? t->n_layers : 0, a, ws, ws_bytes, stream);
}

int moe_engine_layers(const moe_layer_spec* s, const moe_slot_table* t,
                      const moe_engine_layer* layers, const int32_t* step_layer, int n_steps,
                      const float* xi, float* y, int32_t* idx_rec, float* w_rec, int32_t* pidx_rec,
                      float* pw_rec, uint32_t* status, void* ws, size_t ws_bytes, void* stream) {
  return engine_steps(0, s, t, layers, step_layer, n_steps, xi, y, idx_rec, w_rec, pidx_rec, pw_rec,
                      status, ws, ws_bytes, stream);
}

int moe_engine_tokens(const moe_layer_spec* s, const moe_slot_table* t,
                      const moe_engine_layer* layers, const int32_t* step_layer, int n_steps,
                      const float* xi, float* y, int32_t* idx_rec, float* w_rec, int32_t* pidx_rec,
                      float* pw_rec, uint32_t* status, void* ws, size_t ws_bytes, void* stream) {
  return engine_steps(2, s, t, layers, step_layer, n_steps, xi, y, idx_rec, w_rec, pidx_rec, pw_rec,
                      status, ws, ws_bytes, stream);
}

int moe_engine_chain_supported(const moe_layer_spec* s) {
  const int rc = engine_pipe_supported(s);
  return rc == MOE_OK ? MOE_OK : moe_engine_supported(s);
}

int moe_engine_chain(const moe_layer_spec* s, const moe_slot_table* t,
                     const moe_engine_layer* layers, int n_layers, int first_token, int n_tokens,
                     const float* xi, float* r_state, void* x_rec, float* r_rec, int32_t* idx_rec,
                     float* w_rec, int32_t* pidx_rec, float* pw_rec, float* y_rec, uint32_t* status,
                     void* ws, size_t ws_bytes, void* stream) {
  if (n_layers < 1 || n_tokens < 0 || first_token < 0 || !r_state) return MOE_EINVAL;
  if ((long long)n_tokens * n_layers > (1LL << 30)) return MOE_EINVAL;
  if (n_tokens == 0) return MOE_OK;
  moe::EngineArgs a{};
  // the two-half pipeline where the shape allows it, else the whole-chip chain
  a.mode = engine_pipe_supported(s) == MOE_OK ? 3 : 1;
  a.n_steps = n_tokens * n_layers;
  a.L = n_layers;
  a.first_token = first_token;
  a.consumer_lo = 1;
  a.consumer_hi = n_layers - 1;
  a.layers = layers;
  a.xi = xi;
  a.r_state = r_state;
  a.x_rec = static_cast<__half*>(x_rec);
  a.r_rec = r_rec;
  a.idx_rec = idx_rec;
  a.w_rec = w_rec;
  a.pidx_rec = pidx_rec;
  a.pw_rec = pw_rec;
  a.y = y_rec;
  a.status = status;
  return engine_common(s, t, n_layers, a, ws, ws_bytes, stream);
}

int moe_engine_chain_mlp_supported(const moe_layer_spec* s, int hidden) {
  const int rc = engine_pipe_supported(s);
  if (rc != MOE_OK) return rc;
  if (s->routing != MOE_ROUTING_SOFTMAX_TOPK || s->d_model > 2048) return MOE_EINVAL;
  if (hidden < 64 || hidden > moe::kHidMax || hidden % 64) return MOE_EINVAL;
  return MOE_OK;
}

int moe_engine_chain_mlp(const moe_layer_spec* s, const moe_slot_table* t, const moe_engine_layer* layers,
                         const moe_head_mlp* heads, int hidden, int n_layers, int first_token, int n_tokens,
                         const float* xi, float* r_state, void* x_rec, float* r_rec, int32_t* idx_rec,
                         float* w_rec, int32_t* pidx_rec, float* pw_rec, float* y_rec, uint32_t* status,
                         void* ws, size_t ws_bytes, void* stream) {
  int rc = moe_engine_chain_mlp_supported(s, hidden);
  if (rc != MOE_OK) return rc;
  if (!heads || !aligned16(heads)) return heads ? MOE_EALIGN : MOE_EINVAL;
  if (n_layers < 1 || n_tokens < 0 || first_token < 0 || !r_state) return MOE_EINVAL;
  if ((long long)n_tokens * n_layers > (1LL << 30)) return MOE_EINVAL;
  if (n_tokens == 0) return MOE_OK;
  moe::EngineArgs a{};
  a.mode = 3;
  a.n_steps = n_tokens * n_layers;
  a.L = n_layers;
  a.first_token = first_token;
  a.consumer_lo = 1;
  a.consumer_hi = n_layers - 1;
  a.layers = layers;
  a.heads = heads;
  a.hidden = hidden;
  a.xi = xi;
  a.r_state = r_state;
  a.x_rec = static_cast<__half*>(x_rec);
  a.r_rec = r_rec;
  a.idx_rec = idx_rec;
  a.w_rec = w_rec;
  a.pidx_rec = pidx_rec;
  a.pw_rec = pw_rec;
  a.y = y_rec;
  a.status = status;
  return engine_common(s, t, n_layers, a, ws, ws_bytes, stream);
}

int moe_profile_arm(int which, void* start_event, void* stop_event) {
  if (which == MOE_PROF_ENGINE_PHASES) {
    if (!start_event || !aligned16(start_event)) return MOE_EINVAL;
    g_prof_engine_ts = start_event;
    return MOE_OK;
  }
  if (which != MOE_PROF_FFN_MAIN || !start_event || !stop_event) return MOE_EINVAL;
  g_prof_ffn.start = static_cast<hipEvent_t>(start_event);
  g_prof_ffn.stop = static_cast<hipEvent_t>(stop_event);
  return MOE_OK;
}

}  // extern "C"
