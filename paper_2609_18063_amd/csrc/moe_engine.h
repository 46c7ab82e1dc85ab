// Persistent decode engine (moe_engine.hip): launch interface.
#pragma once

#include "moe_device.h"

namespace moe {

struct EngineArgs {
  int mode;          // 0: independent single-token steps; 1: decode chain;
                     // 2: independent steps, one per team in flight;
                     // 3: decode chain on two alternating halves of the chip
  int n_steps;
  int L;             // chain: layers per token
  int first_token;   // chain: token index of the first step
  int consumer_lo, consumer_hi;  // chain: layers that route by the prediction (after token 0)
  int E, K, S, r;
  float lora_scale;
  int n_ids, n_slots, n_table_layers;
  const int32_t* slot_of;        // slot-table device copy
  const moe_bundle* bundles;
  const moe_engine_layer* layers;
  const int32_t* step_layer;     // mode 0: [n_steps] table layer of each step
  const float* xi;               // mode 0: [n_steps][d]; mode 1: [n_tokens][d]
  float* y;                      // mode 0: [n_steps][d] output; mode 1: optional record
  float* r_state;                // mode 1: [d] residual, in/out
  __half* x_rec;                 // optional [n_steps][d]
  float* r_rec;                  // optional [n_steps][d]: chain residual after the mixing
  int32_t* idx_rec;              // optional [n_steps][K]
  float* w_rec;
  int32_t* pidx_rec;
  float* pw_rec;
  uint32_t* status;
  uint64_t* phase_ts;            // profiling: [n_steps][3][24] wall-clock marks, or null
  uint32_t* ctl;                 // workspace control words
  uint64_t* xw;                  // workspace exchange words
  // exchange-area offsets and per-parity strides (in 64-bit words)
  size_t xo_logr, xs_logr, xo_loghm, xo_av, xs_av, xo_hv, xs_hv, xo_adp, xs_adp, xo_part, xs_part,
      xo_rv, xs_rv, xo_logh, xs_logh_layer, xo_pred, xs_pred;
  int n_groups, top_groups;  // sigmoid-group selection (App. A) when n_groups > 0, else softmax-top-k
  float route_scale;
  // two-half chain with the full prerouter head: heads[n] of every layer n < L - 1
  // (device array), hidden size `hidden`; null: the linear head of layers[n]
  const moe_head_mlp* heads;
  int hidden;
  size_t xo_hid, xo_rtm1;    // hidden words [2 halves][4][kHidMax], routing words [2][L][32]
};

constexpr int kHidMax = 512;  // largest hidden size of the full head in the two-half chain

bool engine_shape_supported(int d, int I, int r, int K, int S, int E);
// Fills the exchange offsets of `a`; returns the exchange area size in words.
size_t engine_workspace_words(int E, int d, int L, EngineArgs* a);
hipError_t launch_engine(EngineArgs& a, int d, int I, int r, hipStream_t st);

// Throughput schedule of independent steps (moe_engine_tokens.hip): one step
// per team of 16 workgroups in flight (16 teams). Uses the exchange offsets
// xo/xs of logr (router logits), loghm (head logits), av, hv and adp, each
// strided per team.
bool engine_tokens_supported(int d, int I, int r, int K, int S, int E);
size_t engine_tokens_workspace_words(int E, int d, int I, int r, int n_list, EngineArgs* a);
hipError_t launch_engine_tokens(EngineArgs& a, int d, int I, int r, hipStream_t st);

// Decode chain on two alternating halves of the chip (moe_engine_pipe.hip):
// one half computes a layer while the other loads its next layer's experts.
// Uses the offsets xo/xs of logr, av, hv, part, rv, logh and pred.
bool engine_pipe_supported(int d, int I, int r, int K, int S, int E);
size_t engine_pipe_workspace_words(int E, int d, int I, int r, int n_list, int L, EngineArgs* a);
hipError_t launch_engine_pipe(EngineArgs& a, int d, int I, int r, hipStream_t st);

}  // namespace moe
