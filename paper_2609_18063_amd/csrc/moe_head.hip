// Full prerouter head for gfx950 (Sec. 3.2, Head): per layer fc1 -> erf-GELU
// -> fc2 plus a linear residual path on the hidden state; the input feature is
// the hidden state followed by the one-hots of the experts this layer routed
// to at this token and at the previous one (d + 2E features).
//
//   fc1   hidden row j: the fp16 dot product of fc1's hidden-state columns
//         with x (fp32 accumulation, one wave per row), plus the fc1 columns
//         of the 2K set members (a one-hot times a matrix is a sum of
//         columns: the transposed one-hot block is read one row per member),
//         plus b1; erf-GELU in fp32; stored as fp16 (fc2's fp16 input).
//   fc2   logit e: fc2 row e against the hidden activation, plus b2, plus the
//         residual path's row e against x; fp32.
// The selection is the router's softmax-top-k (launch_topk).
#include <hip/hip_runtime.h>

#include "moe_kernels.h"

namespace moe {
namespace {

// One row per wave, two waves per workgroup: at batch 1 the rows of fc1
// (512) and fc2 (256) spread over the whole chip, each wave's row loads
// issued at once.
constexpr int kHeadRows = 2;

__global__ void __launch_bounds__(128) head_fc1_kernel(const __half* __restrict__ x, int d, int E, int K,
                                                       int H, const __half* __restrict__ w1x,
                                                       const __half* __restrict__ w1r,
                                                       const __half* __restrict__ b1,
                                                       const int32_t* __restrict__ rt,
                                                       const int32_t* __restrict__ rtm1,
                                                       __half* __restrict__ hid) {
  const int t = blockIdx.y, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const __half* xr = x + (size_t)t * d;
  {
    const int row = blockIdx.x * kHeadRows + wave;  // H % 8 == 0: always < H
    // The set members' fc1 columns, requested before the row's dot product
    // (lane k < K: member k at t; lane K + k: member k at t - 1), so that
    // their two dependent loads overlap it; added below in member order.
    const bool lanes = 2 * K <= kWave;
    float mv = 0.f;
    int mok = 0;
    if (lanes && lane < 2 * K) {
      const bool prev = lane >= K;
      const int k = prev ? lane - K : lane;
      const int e = prev ? (rtm1 ? rtm1[(size_t)t * K + k] : -1) : rt[(size_t)t * K + k];
      mok = e >= 0 && e < E;
      if (mok) mv = __half2float(w1r[(size_t)(prev ? E + e : e) * H + row]);
    }
    const float bv = b1 ? __half2float(b1[row]) : 0.f;
    const __half* wr = w1x + (size_t)row * d;
    float acc = 0.f;
#pragma unroll 4
    for (int c = lane; c < d / 8; c += kWave) acc = dot8_h(ld16(wr + (size_t)c * 8), ld16(xr + (size_t)c * 8), acc);
    acc = wave_sum(acc);
    if (lanes) {
      for (int k = 0; k < 2 * K; ++k)
        if (__builtin_amdgcn_readlane(mok, k)) acc += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mv), k));
    }
    if (lane == 0) {
      if (!lanes) {
        for (int k = 0; k < K; ++k) {
          const int e = rt[(size_t)t * K + k];
          if (e >= 0 && e < E) acc += __half2float(w1r[(size_t)e * H + row]);
        }
        if (rtm1) {
          for (int k = 0; k < K; ++k) {
            const int e = rtm1[(size_t)t * K + k];
            if (e >= 0 && e < E) acc += __half2float(w1r[(size_t)(E + e) * H + row]);
          }
        }
      }
      if (b1) acc += bv;
      const float g = 0.5f * acc * (1.0f + erff(acc * 0.70710678118654752f));
      hid[(size_t)t * H + row] = __float2half(g);
    }
  }
}

__global__ void __launch_bounds__(128) head_fc2_kernel(const __half* __restrict__ hid, int H,
                                                       const __half* __restrict__ x, int d, int E,
                                                       const __half* __restrict__ w2,
                                                       const __half* __restrict__ b2,
                                                       const __half* __restrict__ wl,
                                                       float* __restrict__ logits) {
  const int t = blockIdx.y, wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const __half* hr = hid + (size_t)t * H;
  const __half* xr = x + (size_t)t * d;
  {
    const int e = blockIdx.x * kHeadRows + wave;  // E % 8 == 0: always < E
    const float b2v = b2 ? __half2float(b2[e]) : 0.f;  // requested with the rows
    float acc = 0.f, res = 0.f;
    const __half* w2r = w2 + (size_t)e * H;
    for (int c = lane; c < H / 8; c += kWave) acc = dot8_h(ld16(w2r + (size_t)c * 8), ld16(hr + (size_t)c * 8), acc);
    if (wl) {
      const __half* wlr = wl + (size_t)e * d;
#pragma unroll 4
      for (int c = lane; c < d / 8; c += kWave) res = dot8_h(ld16(wlr + (size_t)c * 8), ld16(xr + (size_t)c * 8), res);
    }
    acc = wave_sum(acc);
    res = wave_sum(res);
    if (lane == 0) logits[(size_t)t * E + e] = acc + b2v + res;
  }
}

}  // namespace

hipError_t launch_head_mlp(const HeadMlpArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(head_fc1_kernel, dim3(a.H / kHeadRows, a.T), dim3(64 * kHeadRows), 0, st, a.x, a.d, a.E, a.K, a.H,
                     a.w1x, a.w1r, a.b1, a.routed_t, a.routed_tm1, a.hidden);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_fc2_kernel, dim3(a.E / kHeadRows, a.T), dim3(64 * kHeadRows), 0, st, a.hidden, a.H, a.x, a.d,
                     a.E, a.w2, a.b2, a.wl, a.logits);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.n_groups > 0)
    return launch_topk_sigmoid_group(a.logits, nullptr, a.T, a.E, a.K, a.n_groups, a.top_groups,
                                     a.route_scale, a.idx, a.w, st);
  return launch_topk(a.logits, a.T, a.E, a.K, a.idx, a.w, st);
}

}  // namespace moe
