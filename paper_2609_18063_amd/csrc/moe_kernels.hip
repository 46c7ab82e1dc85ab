// gfx950 kernels of the MoE decode hot path: layer input, routing / prerouting,
// int4 group-64 SwiGLU experts with the unmerged LoRA delta, combine.
//
// Data layout (all row-major, see include/moe_api.h): int4 codes [out][in/2]
// with the even input in the low nibble, (scale, zero) fp16 pairs
// [out][in/64], LoRA A [r][in] and B [out][r] fp16.
//
// Lane mapping of the int4 matvecs: a row of `in` inputs is split into 16-byte
// chunks of 32 codes; LPR = min(64, in/32) lanes share one row and each lane
// owns CPL = max(1, in/2048) chunks, so one wave instruction covers 64/LPR
// rows with fully coalesced 16-byte loads.  A lane's chunks are the same for
// every row it visits, so the 32*CPL activations it needs stay in registers.
#include "moe_kernels.h"
#include "moe_xchg.h"

namespace moe {

// ------------------------------------------------------------------------
// Layer input: RMS normalization to fp16.  The sum of squares, the scale and
// the product are fp64 and the product is rounded once to fp16, so the fp16
// rounding of every element does not depend on the order of the reduction.
// ------------------------------------------------------------------------
__global__ void __launch_bounds__(256) rmsnorm_f16_kernel(const float* __restrict__ xi, int d,
                                                          __half* __restrict__ x) {
  const int t = blockIdx.x;
  const float* row = xi + (size_t)t * d;
  double acc = 0.0;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    const double v = row[j];
    acc += v * v;
  }
  __shared__ double red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  const double r = 1.0 / sqrt(red[0] / (double)d + 1e-6);
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    x[(size_t)t * d + j] = __half(static_cast<_Float16>((double)row[j] * r));
}

// Router / prerouter logits for one token per grid row, then (if idx is
// given) softmax-top-k by the last workgroup of that token to finish (a
// counter in the workspace, left at zero afterwards).
template <int RPW>
__global__ void __launch_bounds__(256) route_kernel(const __half* __restrict__ x,
                                                    const __half* __restrict__ W, int E, int d,
                                                    int K, float* __restrict__ logits,
                                                    int32_t* __restrict__ idx,
                                                    float* __restrict__ wout,
                                                    uint32_t* __restrict__ counters) {
  const int t = blockIdx.y;
  const int nch = d >> 3;
  // x is read by every wave from the cache, in the same loads as the rows (a
  // copy into LDS first would put a barrier and one more memory round trip
  // ahead of the row loads)
  const U4* xrow = reinterpret_cast<const U4*>(x + (size_t)t * d);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int row0 = (blockIdx.x * 4 + wave) * RPW;
  float acc[RPW];
#pragma unroll
  for (int r = 0; r < RPW; ++r) acc[r] = 0.f;
  for (int c = lane; c < nch; c += kWave) {
    const U4 xv = xrow[c];
    U4 wv[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int e = row0 + r;
      wv[r] = (e < E) ? ld16(W + (size_t)e * d + (size_t)c * 8) : U4{0, 0, 0, 0};
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r) acc[r] = dot8_h(wv[r], xv, acc[r]);
  }
  float* lt = logits + (size_t)t * E;
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const float s = wave_sum(acc[r]);
    if (lane == 0 && row0 + r < E) st_agent(lt + row0 + r, s);
  }
  __threadfence();
  __syncthreads();
  __shared__ int last;
  __shared__ uint32_t tk_scratch[64];
  if (threadIdx.x == 0) {
    const uint32_t prev = atomicAdd(&counters[t], 1u);
    last = (prev == gridDim.x - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  if (wave == 0 && idx) wave_topk<true>(lt, E, K, idx + (size_t)t * K, wout + (size_t)t * K, tk_scratch);
  if (threadIdx.x == 0)
    __hip_atomic_store(&counters[t], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The same selection and weights by one 512-thread workgroup per token
// (E <= 256, K <= 32): two-stage ranking of the keys (moe_xchg.h), a few
// barriers instead of one wave's 32 ballot rounds.
__global__ void __launch_bounds__(512) topk_block_kernel(const float* __restrict__ logits, int E, int K,
                                                         int32_t* __restrict__ idx,
                                                         float* __restrict__ w) {
  __shared__ float lg[256];
  __shared__ uint64_t keys[256];
  __shared__ int part[256];
  __shared__ uint64_t cand[128];
  __shared__ uint64_t sorted[32];
  const int t = blockIdx.x;
  if ((int)threadIdx.x < E) lg[threadIdx.x] = logits[(size_t)t * E + threadIdx.x];
  __syncthreads();
  eng::block_topk(lg, E, K, idx + (size_t)t * K, w + (size_t)t * K, keys, part, cand, sorted);
}

// Sigmoid-group selection (App. A), one 512-thread workgroup per token
// (E <= 256): sigma = sigmoid(l) in fp32, the selection score sigma + bias;
// a group's score is the sum of its two largest selection scores (its one
// score if it has one member); the top_groups best groups survive (ties to
// the lower group); the K largest surviving scores are selected with the
// engines' two-stage ranking (descending, ties to the lower id); the weights
// use the raw sigma: w = scale sigma / (sum of the selected sigma + 1e-20).
__global__ void __launch_bounds__(512) topk_sigmoid_group_kernel(const float* __restrict__ logits,
                                                                 const float* __restrict__ bias, int E,
                                                                 int K, int n_groups, int top_groups,
                                                                 float scale, int32_t* __restrict__ idx,
                                                                 float* __restrict__ w) {
  __shared__ float lg[256];
  __shared__ eng::SigmoidScratch sc;
  __shared__ uint64_t keys[256];
  __shared__ int part[256];
  __shared__ uint64_t cand[128];
  __shared__ uint64_t sorted[32];
  const int t = blockIdx.x;
  if ((int)threadIdx.x < E) lg[threadIdx.x] = logits[(size_t)t * E + threadIdx.x];
  __syncthreads();
  eng::block_topk_sigmoid_group(lg, bias, E, K, n_groups, top_groups, scale, idx + (size_t)t * K,
                                w + (size_t)t * K, sc, keys, part, cand, sorted);
}

__global__ void __launch_bounds__(64) topk_kernel(const float* __restrict__ logits, int E, int K,
                                                  int32_t* __restrict__ idx,
                                                  float* __restrict__ w) {
  __shared__ uint32_t tk_scratch[64];
  const int t = blockIdx.x;
  wave_topk<false>(logits + (size_t)t * E, E, K, idx + (size_t)t * K, w + (size_t)t * K, tk_scratch);
}

// ------------------------------------------------------------------------
// Expert stage 1: raw int4 matvecs W_gate x, W_up x (row pairs) and the LoRA
// projections A_gate x, A_up x.
// ------------------------------------------------------------------------
template <int CPL>
__device__ __forceinline__ void load_x_lane(const __half* x, int c0, int lpr, float (&xf)[CPL][32],
                                            float (&xs)[CPL]) {
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int c = c0 + lpr * cc;
    const U4* p = reinterpret_cast<const U4*>(x + (size_t)c * 32);
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const U4 v = p[q];
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 f = h2f2(w[i]);
        xf[cc][q * 8 + 2 * i] = f.x;
        xf[cc][q * 8 + 2 * i + 1] = f.y;
        s += f.x + f.y;
      }
    }
    xs[cc] = s;
  }
}

template <int LPR, int CPL, int RP>
__global__ void __launch_bounds__(256) ffn_gateup_kernel(FfnArgs a) {
  constexpr int RPI = kWave / LPR;               // rows per wave instruction
  constexpr int PAIRS_PER_WG = 4 * RP * RPI;
  const int t = blockIdx.y;
  const int nblk_w = (a.I + PAIRS_PER_WG - 1) / PAIRS_PER_WG;
  const int nblk_a = (2 * a.r + 3) / 4;
  const int nblk = nblk_w + nblk_a;
  const int k = blockIdx.x / nblk, b = blockIdx.x % nblk;
  const int n = a.n_list;
  const moe_bundle* bd = resolve_expert(k, a.K, a.E, a.idx + (size_t)t * a.K, a.slot_of,
                                        a.bundles, a.status, b == 0 && threadIdx.x == 0);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const __half* x = a.x + (size_t)t * a.d;
  const size_t tk = (size_t)t * n + k;

  if (b >= nblk_w) {
    // LoRA A rows: wave handles row rr = 4 * (b - nblk_w) + wave of [A_gate; A_up].
    const int rr = 4 * (b - nblk_w) + wave;
    if (rr >= 2 * a.r) return;
    const int p = rr / a.r, kk = rr % a.r;
    float* dst = (p == 0 ? a.ag : a.au) + tk * a.r + kk;
    const moe_proj* pr = bd ? (p == 0 ? &bd->gate : &bd->up) : nullptr;
    if (!pr || !pr->lora_a || !pr->lora_b) {
      if (lane == 0) *dst = 0.f;
      return;
    }
    const __half* arow = reinterpret_cast<const __half*>(pr->lora_a) + (size_t)kk * a.d;
    float acc = 0.f;
    for (int c = lane; c < (a.d >> 3); c += kWave)
      acc = dot8_h(ld16(arow + (size_t)c * 8), ld16(x + (size_t)c * 8), acc);
    acc = wave_sum(acc);
    if (lane == 0) *dst = acc;
    return;
  }

  const int c0 = lane % LPR;
  const int sub = lane / LPR;
  const int pair0 = b * PAIRS_PER_WG + wave * RP * RPI;
  if (!bd) {
#pragma unroll
    for (int rp = 0; rp < RP; ++rp) {
      const int i = pair0 + rp * RPI + sub;
      if (c0 == 0 && i < a.I) {
        a.gx[tk * a.I + i] = 0.f;
        a.ux[tk * a.I + i] = 0.f;
      }
    }
    return;
  }
  float xf[CPL][32], xsum[CPL];
  load_x_lane<CPL>(x, c0, LPR, xf, xsum);

  const int in_bytes = a.d >> 1;
  const int ngroups = a.d >> 6;
  const uint8_t* qg = reinterpret_cast<const uint8_t*>(bd->gate.q);
  const uint8_t* qu = reinterpret_cast<const uint8_t*>(bd->up.q);
  const uint32_t* szg = reinterpret_cast<const uint32_t*>(bd->gate.sz);
  const uint32_t* szu = reinterpret_cast<const uint32_t*>(bd->up.sz);

  U4 wq[RP][2][CPL];
  uint32_t wsz[RP][2][CPL];
#pragma unroll
  for (int rp = 0; rp < RP; ++rp) {
    int i = pair0 + rp * RPI + sub;
    i = i < a.I ? i : a.I - 1;
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int c = c0 + LPR * cc;
      wq[rp][0][cc] = ld16(qg + (size_t)i * in_bytes + (size_t)c * 16);
      wq[rp][1][cc] = ld16(qu + (size_t)i * in_bytes + (size_t)c * 16);
      wsz[rp][0][cc] = szg[(size_t)i * ngroups + (c >> 1)];
      wsz[rp][1][cc] = szu[(size_t)i * ngroups + (c >> 1)];
    }
  }
#pragma unroll
  for (int rp = 0; rp < RP; ++rp) {
    const int i = pair0 + rp * RPI + sub;
    float res[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      float acc = 0.f;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const float2 sz = h2f2(wsz[rp][p][cc]);
        acc += sz.x * dot32_q4(wq[rp][p][cc], xf[cc]) + sz.y * xsum[cc];
      }
      res[p] = group_sum(acc, LPR);
    }
    if (c0 == 0 && i < a.I) {
      a.gx[tk * a.I + i] = res[0];
      a.ux[tk * a.I + i] = res[1];
    }
  }
}

// ------------------------------------------------------------------------
// Expert stage 2: LoRA-B of gate / up, SwiGLU, and the slice-partial LoRA-A
// projection of down.  One wave per 64 intermediate units.
// ------------------------------------------------------------------------
__global__ void __launch_bounds__(64) ffn_h_kernel(FfnArgs a) {
  const int t = blockIdx.y;
  const int nsl = a.I >> 6;
  const int k = blockIdx.x / nsl, sl = blockIdx.x % nsl;
  const int lane = threadIdx.x;
  const int i = sl * 64 + lane;
  const int n = a.n_list;
  const size_t tk = (size_t)t * n + k;
  const moe_bundle* bd = resolve_expert(k, a.K, a.E, a.idx + (size_t)t * a.K, a.slot_of,
                                        a.bundles, a.status, false);
  float* adp = a.adpart + (tk * nsl + sl) * a.r;
  if (!bd) {
    a.h[tk * a.I + i] = 0.f;
    if (lane < a.r) adp[lane] = 0.f;
    return;
  }
  float g = a.gx[tk * a.I + i];
  float u = a.ux[tk * a.I + i];
  if (a.r > 0) {
    if (bd->gate.lora_a && bd->gate.lora_b) {
      const __half* brow = reinterpret_cast<const __half*>(bd->gate.lora_b) + (size_t)i * a.r;
      const float* av = a.ag + tk * a.r;
      float acc = 0.f;
      for (int kk = 0; kk < a.r; ++kk) acc = fmaf(__half2float(brow[kk]), av[kk], acc);
      g = fmaf(a.lora_scale, acc, g);
    }
    if (bd->up.lora_a && bd->up.lora_b) {
      const __half* brow = reinterpret_cast<const __half*>(bd->up.lora_b) + (size_t)i * a.r;
      const float* av = a.au + tk * a.r;
      float acc = 0.f;
      for (int kk = 0; kk < a.r; ++kk) acc = fmaf(__half2float(brow[kk]), av[kk], acc);
      u = fmaf(a.lora_scale, acc, u);
    }
  }
  const float hv = g / (1.f + expf(-g)) * u;
  a.h[tk * a.I + i] = hv;
  const bool has_down = a.r > 0 && bd->down.lora_a && bd->down.lora_b;
  for (int kk = 0; kk < a.r; ++kk) {
    const float p =
        has_down ? __half2float(reinterpret_cast<const __half*>(bd->down.lora_a)[(size_t)kk * a.I + i]) * hv
                 : 0.f;
    const float s = wave_sum(p);
    if (lane == 0) adp[kk] = s;
  }
}

// ------------------------------------------------------------------------
// Expert stage 3: down int4 matvec on h plus the LoRA-B of down, folded into
// the same cross-lane reduction.
// ------------------------------------------------------------------------
template <int LPR, int CPL, int RIT>
__global__ void __launch_bounds__(256) ffn_down_kernel(FfnArgs a) {
  constexpr int RPI = kWave / LPR;
  constexpr int ROWS_PER_WG = 4 * RIT * RPI;
  const int t = blockIdx.y;
  const int nblk = (a.d + ROWS_PER_WG - 1) / ROWS_PER_WG;
  const int k = blockIdx.x / nblk, b = blockIdx.x % nblk;
  const int n = a.n_list;
  const size_t tk = (size_t)t * n + k;
  const moe_bundle* bd = resolve_expert(k, a.K, a.E, a.idx + (size_t)t * a.K, a.slot_of,
                                        a.bundles, a.status, false);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c0 = lane % LPR, sub = lane / LPR;
  const int row0 = b * ROWS_PER_WG + wave * RIT * RPI;
  float* ye = a.y_experts + tk * a.d;
  if (!bd) {
#pragma unroll
    for (int it = 0; it < RIT; ++it) {
      const int j = row0 + it * RPI + sub;
      if (c0 == 0 && j < a.d) ye[j] = 0.f;
    }
    return;
  }
  // h for this lane's chunks
  float hf[CPL][32], hsum[CPL];
  const float* hrow = a.h + tk * a.I;
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int c = c0 + LPR * cc;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 v = reinterpret_cast<const float4*>(hrow + (size_t)c * 32)[q];
      hf[cc][4 * q] = v.x;
      hf[cc][4 * q + 1] = v.y;
      hf[cc][4 * q + 2] = v.z;
      hf[cc][4 * q + 3] = v.w;
      s += (v.x + v.y) + (v.z + v.w);
    }
    hsum[cc] = s;
  }
  // LoRA: lane c0 owns rank components c0, c0 + LPR, ... < r
  const bool has_lora = a.r > 0 && bd->down.lora_a && bd->down.lora_b;
  constexpr int KMAX = 64 / LPR > 0 ? (64 + LPR - 1) / LPR : 1;
  float adv[KMAX];
  const int nsl = a.I >> 6;
#pragma unroll
  for (int m = 0; m < KMAX; ++m) {
    const int kk = c0 + LPR * m;
    float s = 0.f;
    if (has_lora && kk < a.r)
      for (int sl = 0; sl < nsl; ++sl) s += a.adpart[(tk * nsl + sl) * a.r + kk];
    adv[m] = s;
  }
  const int in_bytes = a.I >> 1;
  const int ngroups = a.I >> 6;
  const uint8_t* qd = reinterpret_cast<const uint8_t*>(bd->down.q);
  const uint32_t* szd = reinterpret_cast<const uint32_t*>(bd->down.sz);
  const __half* bl = has_lora ? reinterpret_cast<const __half*>(bd->down.lora_b) : nullptr;

  U4 wq[RIT][CPL];
  uint32_t wsz[RIT][CPL];
#pragma unroll
  for (int it = 0; it < RIT; ++it) {
    int j = row0 + it * RPI + sub;
    j = j < a.d ? j : a.d - 1;
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int c = c0 + LPR * cc;
      wq[it][cc] = ld16(qd + (size_t)j * in_bytes + (size_t)c * 16);
      wsz[it][cc] = szd[(size_t)j * ngroups + (c >> 1)];
    }
  }
#pragma unroll
  for (int it = 0; it < RIT; ++it) {
    const int j = row0 + it * RPI + sub;
    const int jc = j < a.d ? j : a.d - 1;
    float acc = 0.f;
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const float2 sz = h2f2(wsz[it][cc]);
      acc += sz.x * dot32_q4(wq[it][cc], hf[cc]) + sz.y * hsum[cc];
    }
    if (has_lora) {
      float la = 0.f;
#pragma unroll
      for (int m = 0; m < KMAX; ++m) {
        const int kk = c0 + LPR * m;
        if (kk < a.r) la = fmaf(__half2float(bl[(size_t)jc * a.r + kk]), adv[m], la);
      }
      acc = fmaf(a.lora_scale, la, acc);
    }
    acc = group_sum(acc, LPR);
    if (c0 == 0 && j < a.d) ye[j] = acc;
  }
}

// ------------------------------------------------------------------------
// Combine: y = sum_k w_k y_k + sum_s y_shared_s.
// ------------------------------------------------------------------------
__global__ void __launch_bounds__(256) combine_kernel(const float* __restrict__ ye,
                                                      const float* __restrict__ w, int K, int S,
                                                      int d, float* __restrict__ y, int accumulate) {
  const int t = blockIdx.y;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= d) return;
  const int n = K + S;
  const float* base = ye + (size_t)t * n * d + j;
  float acc = 0.f;
  for (int k = 0; k < K; ++k) acc = fmaf(w[(size_t)t * K + k], base[(size_t)k * d], acc);
  for (int s = 0; s < S; ++s) acc += base[(size_t)(K + s) * d];
  float* out = y + (size_t)t * d + j;
  *out = accumulate ? *out + acc : acc;
}

// ------------------------------------------------------------------------
// Decode-chain stand-in for attention (one workgroup per call):
//   token start:  r = xi + rmsnorm(r)         (norm in fp64, r kept fp32)
//   layer input:  r = r + D * r[perm];  x = fp16(rmsnorm(r))
// ------------------------------------------------------------------------
__device__ double block_sum_sq(const float* v, int d, double* red) {
  double acc = 0.0;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    const double a = v[j];
    acc += a * a;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = blockDim.x >> 1; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__global__ void __launch_bounds__(256) chain_token_start_kernel(const float* __restrict__ xi, int d,
                                                                float* __restrict__ r) {
  __shared__ double red[256];
  const double inv = 1.0 / sqrt(block_sum_sq(r, d, red) / (double)d + 1e-6);
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    r[j] = (float)((double)xi[j] + (double)r[j] * inv);
}

__global__ void __launch_bounds__(256) chain_mix_rmsnorm_kernel(const __half* __restrict__ mix_d,
                                                                const int32_t* __restrict__ perm,
                                                                int d, float* __restrict__ r,
                                                                __half* __restrict__ x) {
  extern __shared__ float rs[];
  __shared__ double red[256];
  for (int j = threadIdx.x; j < d; j += blockDim.x) rs[j] = r[j];
  __syncthreads();
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    const int p = perm[j];
    const float v = (p >= 0 && p < d) ? rs[p] : 0.f;
    r[j] = fmaf(__half2float(mix_d[j]), v, rs[j]);
  }
  __syncthreads();
  const double inv = 1.0 / sqrt(block_sum_sq(r, d, red) / (double)d + 1e-6);
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    x[j] = __half(static_cast<_Float16>((double)r[j] * inv));
}

// ------------------------------------------------------------------------
// Launchers
// ------------------------------------------------------------------------
hipError_t launch_rmsnorm(const float* xi, int T, int d, __half* x, hipStream_t st) {
  hipLaunchKernelGGL(rmsnorm_f16_kernel, dim3(T), dim3(256), 0, st, xi, d, x);
  return hipGetLastError();
}

hipError_t launch_route(const __half* x, const __half* W, int T, int E, int d, int K,
                        float* logits, int32_t* idx, float* w, uint32_t* counters,
                        hipStream_t st) {
  constexpr int RPW = 2;
  const int rows_per_wg = 4 * RPW;
  dim3 grid((E + rows_per_wg - 1) / rows_per_wg, T);
  hipLaunchKernelGGL(route_kernel<RPW>, grid, dim3(256), 0, st, x, W, E, d, K, logits,
                     idx, w, counters);
  return hipGetLastError();
}

hipError_t launch_topk_sigmoid_group(const float* logits, const float* bias, int T, int E, int K,
                                     int n_groups, int top_groups, float scale, int32_t* idx, float* w,
                                     hipStream_t st) {
  if (E > 256 || K > 32 || n_groups < 1 || E % n_groups) return hipErrorInvalidValue;
  hipLaunchKernelGGL(topk_sigmoid_group_kernel, dim3(T), dim3(512), 0, st, logits, bias, E, K, n_groups,
                     top_groups, scale, idx, w);
  return hipGetLastError();
}

hipError_t launch_topk(const float* logits, int T, int E, int K, int32_t* idx, float* w,
                       hipStream_t st) {
  if (E <= 256 && K <= 32)
    hipLaunchKernelGGL(topk_block_kernel, dim3(T), dim3(512), 0, st, logits, E, K, idx, w);
  else
    hipLaunchKernelGGL(topk_kernel, dim3(T), dim3(64), 0, st, logits, E, K, idx, w);
  return hipGetLastError();
}

template <int LPR, int CPL>
static void gateup(const FfnArgs& a, int T, hipStream_t st, hipEvent_t ps, hipEvent_t pe) {
  constexpr int RP = 4;
  constexpr int PAIRS = 4 * RP * (kWave / LPR);
  const int nblk = (a.I + PAIRS - 1) / PAIRS + (2 * a.r + 3) / 4;
  if (ps && pe)
    hipExtLaunchKernelGGL((ffn_gateup_kernel<LPR, CPL, RP>), dim3(nblk * a.n_list, T), dim3(256),
                          0, st, ps, pe, 0, a);
  else
    hipLaunchKernelGGL((ffn_gateup_kernel<LPR, CPL, RP>), dim3(nblk * a.n_list, T), dim3(256), 0,
                       st, a);
}

template <int LPR, int CPL>
static void down(const FfnArgs& a, int T, hipStream_t st) {
  constexpr int RIT = 4;
  constexpr int ROWS = 4 * RIT * (kWave / LPR);
  const int nblk = (a.d + ROWS - 1) / ROWS;
  hipLaunchKernelGGL((ffn_down_kernel<LPR, CPL, RIT>), dim3(nblk * a.n_list, T), dim3(256), 0, st,
                     a);
}

static bool dispatch_gateup(const FfnArgs& a, int T, hipStream_t st, hipEvent_t ps,
                            hipEvent_t pe) {
  switch (a.d) {
    case 256: gateup<8, 1>(a, T, st, ps, pe); return true;
    case 512: gateup<16, 1>(a, T, st, ps, pe); return true;
    case 1024: gateup<32, 1>(a, T, st, ps, pe); return true;
    case 2048: gateup<64, 1>(a, T, st, ps, pe); return true;
    case 4096: gateup<64, 2>(a, T, st, ps, pe); return true;
    case 8192: gateup<64, 4>(a, T, st, ps, pe); return true;
  }
  return false;
}

static bool dispatch_down(const FfnArgs& a, int T, hipStream_t st) {
  switch (a.I) {
    case 256: down<8, 1>(a, T, st); return true;
    case 512: down<16, 1>(a, T, st); return true;
    case 1024: down<32, 1>(a, T, st); return true;
    case 2048: down<64, 1>(a, T, st); return true;
    case 4096: down<64, 2>(a, T, st); return true;
    case 8192: down<64, 4>(a, T, st); return true;
  }
  return false;
}

hipError_t launch_ffn(const FfnArgs& a, int T, hipStream_t st, hipEvent_t prof_start,
                      hipEvent_t prof_stop) {
  if (!dispatch_gateup(a, T, st, prof_start, prof_stop)) return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ffn_h_kernel, dim3((a.I >> 6) * a.n_list, T), dim3(64), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (!dispatch_down(a, T, st)) return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_combine(const float* ye, const float* w, int T, int K, int S, int d, float* y,
                          int accumulate, hipStream_t st) {
  hipLaunchKernelGGL(combine_kernel, dim3((d + 255) / 256, T), dim3(256), 0, st, ye, w, K, S, d, y,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_chain_token_start(const float* xi, int d, float* r, hipStream_t st) {
  hipLaunchKernelGGL(chain_token_start_kernel, dim3(1), dim3(256), 0, st, xi, d, r);
  return hipGetLastError();
}

hipError_t launch_chain_mix_rmsnorm(const __half* mix_d, const int32_t* perm, int d, float* r,
                                    __half* x, hipStream_t st) {
  hipLaunchKernelGGL(chain_mix_rmsnorm_kernel, dim3(1), dim3(256), (size_t)d * 4, st, mix_d, perm, d,
                     r, x);
  return hipGetLastError();
}

}  // namespace moe
