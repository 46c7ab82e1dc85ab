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
//
// Each logit becomes a 32-bit order key (NaN as -inf, -0 as +0).  The K-th
// largest key T is found bit by bit from the top: a candidate stays if at
// least K keys reach it (one ballot and a scalar popcount per key register).
// The selected set is every key above T plus the lowest-index keys equal to
// T; its K members are compacted to LDS and ranked against each other.
constexpr int kTopkVals = 16;  // E <= 64 * 16

__device__ __forceinline__ uint32_t topk_key(float v) {
  if (v != v) v = -INFINITY;
  if (v == 0.f) v = 0.f;
  const uint32_t b = __float_as_uint(v);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float topk_key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// scratch: LDS, at least 2 * 32 words, private to the calling wave.
template <bool kAgent, int NV = kTopkVals>
__device__ void wave_topk(const float* l, int E, int K, int32_t* idx_out, float* w_out,
                          uint32_t* scratch) {
  const int lane = threadIdx.x & 63;
  uint32_t key[NV];
  bool valid[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int e = lane + 64 * j;
    valid[j] = e < E;
    key[j] = valid[j] ? topk_key(kAgent ? ld_agent(l + e) : l[e]) : 0u;
  }
  // T: the largest value with at least K keys >= T (invalid positions count as
  // key 0, which no real key equals: -inf is 0x007FFFFF)
  uint32_t T = 0;
  for (int b = 31; b >= 0; --b) {
    const uint32_t cand = T | (1u << b);
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < NV; ++j) cnt += __popcll(__ballot(valid[j] && key[j] >= cand));
    if (cnt >= K) T = cand;
  }
  // keys above T are in; keys equal to T fill the rest, lowest index first
  int n_gt = 0;
#pragma unroll
  for (int j = 0; j < NV; ++j) n_gt += __popcll(__ballot(valid[j] && key[j] > T));
  const int need = K - n_gt;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  int eq_before = 0, sel_before = 0;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const bool eq = valid[j] && key[j] == T;
    const uint64_t meq = __ballot(eq);
    const int eq_rank = eq_before + __popcll(meq & below);
    const bool sel = (valid[j] && key[j] > T) || (eq && eq_rank < need);
    const uint64_t msel = __ballot(sel);
    if (sel) {
      const int ci = sel_before + __popcll(msel & below);
      scratch[2 * ci] = key[j];
      scratch[2 * ci + 1] = (uint32_t)(lane + 64 * j);
    }
    eq_before += __popcll(meq);
    sel_before += __popcll(msel);
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  // rank of member `lane` among the K: larger key first, then lower index
  uint32_t mk = 0, mi = 0;
  int rank = 0;
  if (lane < K) {
    mk = scratch[2 * lane];
    mi = scratch[2 * lane + 1];
    for (int q = 0; q < K; ++q) {
      const uint32_t ok = scratch[2 * q], oi = scratch[2 * q + 1];
      rank += (ok > mk) || (ok == mk && oi < mi);
    }
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  if (lane < K) {
    scratch[2 * rank] = mk;
    scratch[2 * rank + 1] = mi;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  // lane r holds the r-th selected logit; weights as a softmax over the set
  const float v = lane < K ? topk_key_value(scratch[2 * lane]) : 0.f;
  const int id = lane < K ? (int)scratch[2 * lane + 1] : 0;
  const float m = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float ex = (lane < K) ? expf(v - m) : 0.f;
  const float s = wave_sum(ex);
  if (lane < K) {
    idx_out[lane] = id;
    w_out[lane] = ex / s;
  }
}

}  // namespace moe
