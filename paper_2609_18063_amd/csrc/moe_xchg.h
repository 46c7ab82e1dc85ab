// Helpers of the persistent engines (moe_engine.hip, moe_engine_tokens.hip):
// tagged exchange words between workgroups, the XCD id, fp64 sums and the
// single-rounding fp64 -> fp16 conversion of the layer input.
#pragma once

#include "moe_device.h"

namespace moe {
namespace eng {

constexpr long kSpinMax = 1L << 20;   // polls of about a microsecond each

// Tagged exchange words {tag, fp32 value}, written and polled with agent-scope
// relaxed atomics (coherent across the XCDs' L2 caches).
__device__ __forceinline__ void st_tag(uint64_t* p, uint32_t tag, float v) {
  const uint64_t w = ((uint64_t)tag << 32) | (uint64_t)__float_as_uint(v);
  __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_tag(const uint64_t* p) {
  return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_u32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ unsigned xcc_id() {
  unsigned v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v;
}

__device__ __forceinline__ float silu(float z) { return z / (1.f + expf(-z)); }

// fp64 sum over the wave (DPP on the two 32-bit halves of each step's operand)
template <int CTRL, int ROWMASK = 0xf>
__device__ __forceinline__ double dpp_d(double v) {
  const uint64_t b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROWMASK, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, ROWMASK, 0xf, false);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}
__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_d<0xB1>(v);
  v += dpp_d<0x4E>(v);
  v += dpp_d<0x141>(v);
  v += dpp_d<0x140>(v);
  v += dpp_d<0x142, 0xa>(v);
  v += dpp_d<0x143, 0xc>(v);
  const uint64_t b = __double_as_longlong(v);
  const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)b, 63);
  const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), 63);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// 1 / sqrt(m) in fp64 for m > 0: the fp32 estimate refined by two Newton
// steps, within a few fp64 ulps (x is rounded to fp16 afterwards).
__device__ __forceinline__ double rsqrt_f64(double m) {
  double y = (double)rsqrtf((float)m);
  y = y * (1.5 - 0.5 * m * y * y);
  y = y * (1.5 - 0.5 * m * y * y);
  return y;
}

// fp64 -> fp16 rounded once to nearest even: the value is first narrowed to
// fp32 rounding to odd (truncated, last bit set when bits were dropped), and
// an odd-rounded value with 13 spare bits rounds to fp16 as the exact one does.
__device__ __forceinline__ __half f64_to_h(double d) {
  float f = (float)d;
  const double back = (double)f;
  if (back != d) {
    uint32_t u = __float_as_uint(f);
    if (fabs(back) > fabs(d)) u -= 1u;  // rounded away from zero: step back
    f = __uint_as_float(u | 1u);
  }
  return __float2half_rn(f);
}

// Position of input j in the pair order of x: inside each group of 8 the
// halves run x0,x4,x1,x5,x2,x6,x3,x7, the order in which the nibbles of one
// code dword pair up under a 0x000F000F mask at shifts 0, 4, 8, 12.
__device__ __forceinline__ int pair_pos(int j) {
  const int r = j & 7;
  return (j & ~7) + (r < 4 ? 2 * r : 2 * (r - 4) + 1);
}

}  // namespace eng
}  // namespace moe
