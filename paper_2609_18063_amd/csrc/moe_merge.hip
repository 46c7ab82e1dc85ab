// Merging an adapter into int4 group-64 weights and re-quantizing them
// (Sec. 3.3, Recovery LoRA: the merged alternative the paper rejects; it is
// here so that what the merge loses can be measured on the device).
//
// One wave per 64-weight group, one weight per lane:
//   w      = s q + z                       (float64, exact)
//   delta  = lora_scale * sum_k B[o][k] A[k][i]   (float64)
//   m      = fp32(w + delta)               (one rounding)
//   lo, hi = group min / max of m; s' = fp16((hi - lo) / 15), z' = fp16(lo)
//   q'     = clamp(rint((m - z') / s'), 0, 15) in fp32; 0 when s' == 0
// The code is an integer decided by floating point, so every step that
// decides it runs in the precision stated above (fp32 division correctly
// rounded, round-half-to-even). Per group the kernel also writes
// sum(actual * delta) and sum(delta^2), actual = s' q' + z' - w, the two
// sums of the weight-level retention.
#include <hip/hip_runtime.h>

#include "moe_kernels.h"

namespace moe {
namespace {

constexpr int kMergeWaves = 4;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ void __launch_bounds__(64 * kMergeWaves)
    merge_requant_kernel(const uint8_t* __restrict__ q, const __half* __restrict__ sz,
                         const __half* __restrict__ A, const __half* __restrict__ B, int out_dim,
                         int in_dim, int rank, float lora_scale, uint8_t* __restrict__ q_out,
                         __half* __restrict__ sz_out, double* __restrict__ stats) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int ng = in_dim / 64;
  const long long gid = (long long)blockIdx.x * kMergeWaves + wave;
  if (gid >= (long long)out_dim * ng) return;  // whole wave
  const int row = (int)(gid / ng), grp = (int)(gid % ng), col = grp * 64 + lane;
  const uint8_t byte = q[(size_t)row * (in_dim / 2) + col / 2];
  const int code = (col & 1) ? (byte >> 4) : (byte & 15);
  const double s = (double)__half2float(sz[(size_t)gid * 2]);
  const double z = (double)__half2float(sz[(size_t)gid * 2 + 1]);
  const double w = s * (double)code + z;
  double delta = 0.0;
  if (A && B) {
    double acc = 0.0;
    for (int k = 0; k < rank; ++k)
      acc += (double)__half2float(B[(size_t)row * rank + k]) *
             (double)__half2float(A[(size_t)k * in_dim + col]);
    delta = (double)lora_scale * acc;
  }
  const float m = (float)(w + delta);
  float lo = m, hi = m;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, o, 64));
    hi = fmaxf(hi, __shfl_xor(hi, o, 64));
  }
  const __half s2h = __float2half((hi - lo) / 15.0f);
  const __half z2h = __float2half(lo);
  const float s2 = __half2float(s2h), z2 = __half2float(z2h);
  int c2 = 0;
  if (s2 != 0.0f) c2 = (int)fminf(fmaxf(rintf((m - z2) / s2), 0.0f), 15.0f);
  const int next = __shfl_down(c2, 1, 64);
  if ((lane & 1) == 0) q_out[(size_t)row * (in_dim / 2) + col / 2] = (uint8_t)(c2 | (next << 4));
  if (lane == 0) {
    sz_out[(size_t)gid * 2] = s2h;
    sz_out[(size_t)gid * 2 + 1] = z2h;
  }
  if (stats) {
    const double actual = ((double)s2 * (double)c2 + (double)z2) - w;
    const double sa = wave_sum_f64(actual * delta), sd = wave_sum_f64(delta * delta);
    if (lane == 0) {
      stats[(size_t)gid * 2] = sa;
      stats[(size_t)gid * 2 + 1] = sd;
    }
  }
}

}  // namespace

hipError_t launch_merge_requantize(const uint8_t* q, const __half* sz, const __half* A,
                                   const __half* B, int out_dim, int in_dim, int rank,
                                   float lora_scale, uint8_t* q_out, __half* sz_out, double* stats,
                                   hipStream_t st) {
  const long long groups = (long long)out_dim * (in_dim / 64);
  const unsigned blocks = (unsigned)((groups + kMergeWaves - 1) / kMergeWaves);
  hipLaunchKernelGGL(merge_requant_kernel, dim3(blocks), dim3(64 * kMergeWaves), 0, st, q, sz, A, B,
                     out_dim, in_dim, rank, lora_scale, q_out, sz_out, stats);
  return hipGetLastError();
}

}  // namespace moe
