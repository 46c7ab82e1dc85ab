// Device-side helpers shared by the gfx950 kernels of the MoE decode path.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

#include "../../include/moe_api.h"

namespace moe {

constexpr int kWave = 64;

// 16-byte vector load / store through the vector memory path.
struct alignas(16) U4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ U4 ld16(const void* p) {
  return *reinterpret_cast<const U4*>(p);
}

// Cross-workgroup data (written by one workgroup and read by another in the
// same launch) goes through agent-scope atomics so that it is coherent
// across the XCDs' L2 caches.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// DPP lane moves (gfx9 data-parallel primitives): a few cycles each, against
// an LDS round trip for a shuffle.  Controls used: quad_perm [1,0,3,2] (0xB1)
// and [2,3,0,1] (0x4E), row_half_mirror (0x141), row_mirror (0x140),
// row_bcast15 (0x142), row_bcast31 (0x143).  `old` is the value a lane keeps
// when its row is masked off.
template <int CTRL, int ROWMASK = 0xf>
__device__ __forceinline__ float dpp_f(float old, float v) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), CTRL, ROWMASK, 0xf, false));
}
template <int CTRL, int ROWMASK = 0xf>
__device__ __forceinline__ int dpp_i(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROWMASK, 0xf, false);
}

// Sum over each row of 16 lanes; every lane of the row receives the sum.
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<0xB1>(0.f, v);
  v += dpp_f<0x4E>(0.f, v);
  v += dpp_f<0x141>(0.f, v);
  v += dpp_f<0x140>(0.f, v);
  return v;
}

// Sum over the 64 lanes of a wave, returned to every lane.
__device__ __forceinline__ float wave_sum(float v) {
  v = row16_sum(v);
  v += dpp_f<0x142, 0xa>(0.f, v);
  v += dpp_f<0x143, 0xc>(0.f, v);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Sum over groups of `width` consecutive lanes (width a power of two <= 64);
// every lane of a group receives its group's sum.
__device__ __forceinline__ float group_sum(float v, int width) {
  if (width >= 64) return wave_sum(v);
  if (width >= 2) v += dpp_f<0xB1>(0.f, v);
  if (width >= 4) v += dpp_f<0x4E>(0.f, v);
  if (width >= 8) v += dpp_f<0x141>(0.f, v);
  if (width >= 16) v += dpp_f<0x140>(0.f, v);
  if (width >= 32) v += __shfl_xor(v, 16, kWave);
  return v;
}

// (value, index) arg-max over the wave: larger value wins, equal values go
// to the lower index; the winner is returned to every lane.
__device__ __forceinline__ void argmax_step(float& v, int& i, float ov, int oi) {
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
  argmax_step(v, i, dpp_f<0xB1>(v, v), dpp_i<0xB1>(i, i));
  argmax_step(v, i, dpp_f<0x4E>(v, v), dpp_i<0x4E>(i, i));
  argmax_step(v, i, dpp_f<0x141>(v, v), dpp_i<0x141>(i, i));
  argmax_step(v, i, dpp_f<0x140>(v, v), dpp_i<0x140>(i, i));
  argmax_step(v, i, dpp_f<0x142, 0xa>(v, v), dpp_i<0x142, 0xa>(i, i));
  argmax_step(v, i, dpp_f<0x143, 0xc>(v, v), dpp_i<0x143, 0xc>(i, i));
  v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
  i = __builtin_amdgcn_readlane(i, 63);
}

// Dot product of 32 int4 codes (16 bytes, even input in the low nibble) with
// 32 fp32 activations.  Codes are exact small integers in fp32.
__device__ __forceinline__ float dot32_q4(const U4& q, const float* x) {
  const uint32_t w[4] = {q.x, q.y, q.z, q.w};
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = w[i] & 0x0F0F0F0Fu;
    const uint32_t hi = (w[i] >> 4) & 0x0F0F0F0Fu;
    const float* xv = x + 8 * i;
    a0 = fmaf((float)(lo & 0xFFu), xv[0], a0);
    a1 = fmaf((float)(hi & 0xFFu), xv[1], a1);
    a0 = fmaf((float)((lo >> 8) & 0xFFu), xv[2], a0);
    a1 = fmaf((float)((hi >> 8) & 0xFFu), xv[3], a1);
    a0 = fmaf((float)((lo >> 16) & 0xFFu), xv[4], a0);
    a1 = fmaf((float)((hi >> 16) & 0xFFu), xv[5], a1);
    a0 = fmaf((float)(lo >> 24), xv[6], a0);
    a1 = fmaf((float)(hi >> 24), xv[7], a1);
  }
  return a0 + a1;
}

// Dot product of 8 fp16 weights with 8 fp16 activations, fp32 accumulate.
__device__ __forceinline__ float dot8_h(const U4& a, const U4& b, float acc) {
  const uint32_t wa[4] = {a.x, a.y, a.z, a.w};
  const uint32_t wb[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    __half2 ha = *reinterpret_cast<const __half2*>(&wa[i]);
    __half2 hb = *reinterpret_cast<const __half2*>(&wb[i]);
    float2 fa = __half22float2(ha);
    float2 fb = __half22float2(hb);
    acc = fmaf(fa.x, fb.x, acc);
    acc = fmaf(fa.y, fb.y, acc);
  }
  return acc;
}

__device__ __forceinline__ float2 h2f2(uint32_t bits) {
  return __half22float2(*reinterpret_cast<const __half2*>(&bits));
}

// Resolve list position k of token t to a bundle, or nullptr (status set).
__device__ __forceinline__ const moe_bundle* resolve_expert(int k, int K, int E, const int32_t* idx_t,
                                                            const int32_t* slot_of,
                                                            const moe_bundle* bundles,
                                                            uint32_t* status, bool report) {
  int e = (k < K) ? idx_t[k] : E + (k - K);
  if (k < K && (e < 0 || e >= E)) {
    if (report && status) atomicOr(status, MOE_STATUS_BAD_INDEX);
    return nullptr;
  }
  int s = slot_of[e];
  if (s < 0) {
    if (report && status) atomicOr(status, MOE_STATUS_SLOT_MISS);
    return nullptr;
  }
  return bundles + s;
}

// Softmax-top-k of one token's logits by one wave.  Selection is on the fp32
// logits (the softmax is increasing), descending, ties to the lower index;
// weights are the softmax renormalized over the selected set.
constexpr int kTopkVals = 16;  // E <= 64 * 16

// Branch-free: every lane keeps its values with a taken mask; each of the K
// rounds takes the lane-local best with selects and one DPP arg-max.
template <bool kAgent, int NV = kTopkVals>
__device__ void wave_topk(const float* l, int E, int K, int32_t* idx_out, float* w_out) {
  const int lane = threadIdx.x & 63;
  const int nv = (E + 63) >> 6;  // values per lane actually used (<= NV)
  float v[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int e = lane + 64 * j;
    float a = -INFINITY;
    if (j < nv && e < E) a = kAgent ? ld_agent(l + e) : l[e];
    v[j] = (a != a) ? -INFINITY : a;
  }
  uint32_t taken = 0;
  float mine = -INFINITY;
  for (int k = 0; k < K; ++k) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int e = lane + 64 * j;
      const bool cand = (j < nv) & (e < E) & !((taken >> j) & 1u);
      const bool better = cand & ((v[j] > bv) | ((v[j] == bv) & (e < bi)));
      bv = better ? v[j] : bv;
      bi = better ? e : bi;
    }
    wave_argmax(bv, bi);
    taken |= ((bi & 63) == lane) ? (1u << ((bi >> 6) & 31)) : 0u;
    mine = (lane == k) ? bv : mine;
    if (lane == 0) idx_out[k] = bi;
  }
  const float m = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mine), 0));
  const float ex = (lane < K) ? expf(mine - m) : 0.f;
  const float s = wave_sum(ex);
  if (lane < K) w_out[lane] = ex / s;
}

}  // namespace moe
