// Kernel launch interface used by the C ABI (host side of moe_kernels.hip).
#pragma once

#include "moe_device.h"

namespace moe {

// Everything the expert kernels need for one layer call.
struct FfnArgs {
  int d, I, E, K, S, r, n_list;   // n_list = K + S experts per token
  float lora_scale;
  const __half* x;                // [T][d]
  const int32_t* idx;             // [T][K]
  const int32_t* slot_of;         // [E + S] of this layer
  const moe_bundle* bundles;      // [n_slots] of this layer
  uint32_t* status;               // may be null
  // workspace
  float* gx;                      // [T][n][I]
  float* ux;                      // [T][n][I]
  float* h;                       // [T][n][I]
  float* ag;                      // [T][n][r]
  float* au;                      // [T][n][r]
  float* adpart;                  // [T][n][I/64][r]
  float* y_experts;               // [T][n][d]
};

hipError_t launch_rmsnorm(const float* xi, int T, int d, __half* x, hipStream_t st);
hipError_t launch_route(const __half* x, const __half* W, int T, int E, int d, int K,
                        float* logits, int32_t* idx, float* w, uint32_t* counters,
                        hipStream_t st);
hipError_t launch_topk(const float* logits, int T, int E, int K, int32_t* idx, float* w,
                       hipStream_t st);
// Sigmoid-group top-k (App. A), E <= 256; bias [E] or null.
hipError_t launch_topk_sigmoid_group(const float* logits, const float* bias, int T, int E, int K,
                                     int n_groups, int top_groups, float scale, int32_t* idx, float* w,
                                     hipStream_t st);

// Full prerouter head (moe_head.hip): fc1 + erf-GELU into `hidden`, fc2 + b2 +
// the residual path into `logits`, then softmax-top-k into idx / w.
struct HeadMlpArgs {
  int T, d, E, K, H;
  const __half* x;                // [T][d]
  const __half* w1x;              // [H][d]
  const __half* w1r;              // [2E][H]
  const __half* b1;               // [H] or null
  const __half* w2;               // [E][H]
  const __half* b2;               // [E] or null
  const __half* wl;               // [E][d] or null
  const int32_t* routed_t;        // [T][K]
  const int32_t* routed_tm1;      // [T][K] or null
  __half* hidden;                 // [T][H]
  float* logits;                  // [T][E]
  int32_t* idx;                   // [T][K]
  float* w;                       // [T][K]
  int n_groups, top_groups;       // sigmoid-group selection when n_groups > 0
  float route_scale;
};
hipError_t launch_head_mlp(const HeadMlpArgs& a, hipStream_t st);
// Adapter merged into one int4 g64 projection and re-quantized (moe_merge.hip).
hipError_t launch_merge_requantize(const uint8_t* q, const __half* sz, const __half* A,
                                   const __half* B, int out_dim, int in_dim, int rank,
                                   float lora_scale, uint8_t* q_out, __half* sz_out, double* stats,
                                   hipStream_t st);
// prof_start / prof_stop: if non-null, the gate/up kernel is launched with
// hipExtLaunchKernelGGL and records them around its execution.
hipError_t launch_ffn(const FfnArgs& a, int T, hipStream_t st, hipEvent_t prof_start,
                      hipEvent_t prof_stop);
hipError_t launch_combine(const float* ye, const float* w, int T, int K, int S, int d, float* y,
                          int accumulate, hipStream_t st);
hipError_t launch_chain_token_start(const float* xi, int d, float* r, hipStream_t st);
hipError_t launch_chain_mix_rmsnorm(const __half* mix_d, const int32_t* perm, int d, float* r,
                                    __half* x, hipStream_t st);

}  // namespace moe
