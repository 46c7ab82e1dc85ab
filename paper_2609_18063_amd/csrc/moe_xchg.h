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

// The workgroup's place in a launch of nx * nm workgroups, one per CU: its
// XCD from the hardware register and its member index = its arrival order
// among the workgroups of that XCD (per-XCD counters ctl[8 + x]; the last
// workgroup to finish the launch clears them with release_places). Each XCD
// holds exactly nm of them, but which blockIdx lands on which XCD depends on
// the dispatcher's state (its round robin need not start at XCD 0). Thread 0
// calls it; false if the counts do not fit.
constexpr int kPlaceWord = 8;
__device__ __forceinline__ bool claim_place(uint32_t* ctl, int nx, int nm, int* x_out, int* m_out) {
  const unsigned x = xcc_id();
  if ((int)x >= nx) return false;
  const uint32_t m = atomicAdd(&ctl[kPlaceWord + x], 1u);
  *x_out = (int)x;
  *m_out = (int)m;
  return (int)m < nm;
}
__device__ __forceinline__ void release_places(uint32_t* ctl, int nx) {
  for (int i = 0; i < nx; ++i)
    __hip_atomic_store(&ctl[kPlaceWord + i], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

// One 16-byte direct global->LDS load per lane (lane l writes lds_wave +
// 16 l), from inline assembly: the compiler does not track it, so a prefetch
// stays in flight across later barriers and polls.  The issuing wave waits
// for it with dma_wait() before the barrier that hands the data over.
// M0 (the LDS destination) is saved and restored around the load, since the
// compiler reserves it; one wait state separates the M0 write from its use.
__device__ __forceinline__ void dma16(const void* g, void* lds_wave) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_wave;
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off nt\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(g)
      : "memory");
}
// The compiler does not see the copies above as memory instructions, so the
// builtin wait follows: it tells the compiler that nothing of its own is
// outstanding either. Otherwise a wait it places for one of its own loads or
// stores (a register reused right after a store, say) can land inside a copy
// loop, where it drains every copy issued so far on each iteration.
// simm16 0x0F70: vmcnt 0, expcnt and lgkmcnt unconstrained.
__device__ __forceinline__ void dma_wait() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);
}
// The same for 4 bytes per lane (lane l writes lds_wave + 4 l).
__device__ __forceinline__ void dma4(const void* g, void* lds_wave) {
  const uint32_t lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_wave;
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %2, off nt\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(g)
      : "memory");
}

// Softmax-top-k of the E <= 256 logits in l (512 threads; K <= 32 <= E), ties
// to the lower index: key = order(l) << 32 | ~index, largest keys first.
// Stage 1 ranks each group of 64 keys within its group (two waves per group,
// 32 comparisons a lane); a group's K best become candidates. Stage 2 ranks
// the 4K candidates among themselves: every key larger than one of the
// overall top K is itself in its group's top K, so for those keys the rank
// among the candidates is the overall rank, and every other key has at least
// K larger candidates. Scratch: keys [256], part [256], cand [128], sorted [32].
__device__ void block_topk(const float* l, int E, int K, int32_t* idx_out, float* w_out,
                           uint64_t* keys, int* part, uint64_t* cand, uint64_t* sorted) {
  const int tid = threadIdx.x;
  const int i = tid & 255, half = tid >> 8;
  const int NC = 4 * K;
  if (tid < 256)
    keys[tid] = tid < E ? ((uint64_t)topk_key(l[tid]) << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)tid)
                        : 0ull;  // below every real key
  else if (tid - 256 < NC)
    cand[tid - 256] = 0ull;
  __syncthreads();
  const uint64_t mine = keys[i];
  {
    const int j0 = (i & ~63) + half * 32;  // uniform across the wave
    int rank = 0;
#pragma unroll
    for (int j = j0; j < j0 + 32; j += 8) {
      const uint64_t k0 = keys[j], k1 = keys[j + 1], k2 = keys[j + 2], k3 = keys[j + 3];
      const uint64_t k4 = keys[j + 4], k5 = keys[j + 5], k6 = keys[j + 6], k7 = keys[j + 7];
      rank += (k0 > mine) + (k1 > mine) + (k2 > mine) + (k3 > mine) + (k4 > mine) + (k5 > mine) +
              (k6 > mine) + (k7 > mine);
    }
    if (half) part[i] = rank;
    __syncthreads();
    if (!half) {
      rank += part[i];
      if (rank < K) cand[(i >> 6) * K + rank] = mine;  // padding keys of a group share one slot
    }
  }
  __syncthreads();
  if (tid < NC) {
    const uint64_t me = cand[tid];
    int rank = 0;
    for (int j = 0; j < NC; j += 4)
      rank += (cand[j] > me) + (cand[j + 1] > me) + (cand[j + 2] > me) + (cand[j + 3] > me);
    if (rank < K) sorted[rank] = me;
  }
  __syncthreads();
  if (tid < 64) {
    const int lane = tid;
    const uint64_t k = lane < K ? sorted[lane] : 0;
    const float v = lane < K ? topk_key_value((uint32_t)(k >> 32)) : 0.f;
    const float m = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float ex = (lane < K) ? expf(v - m) : 0.f;
    const float sum = wave_sum(ex);
    if (lane < K) {
      idx_out[lane] = (int)(0xFFFFFFFFu - (uint32_t)k);
      w_out[lane] = ex / sum;
    }
  }
}

// Sigmoid-group selection (App. A) of one token's logits by a 512-thread
// block (E <= 256, K <= 32): sigma = sigmoid(l) in fp32, selection score
// sigma + bias (bias may be null: zero); a group's score is the sum of its two
// largest selection scores (its one score if it has one member); the
// top_groups best groups survive (ties to the lower group); the K largest
// surviving scores are selected with block_topk (descending, ties to the lower
// id); the weights use the raw sigma: w = scale sigma / (sum of the selected
// sigma + 1e-20). Every thread of the block calls it. Scratch (LDS): sig,
// masked, gsc [256] fp32, keep [256] int, tidx [32], tw [32], and
// block_topk's. idx_out / w_out: K entries (LDS or global).
struct SigmoidScratch {
  float sig[256], masked[256], gsc[256];
  int keep[256];
  int32_t tidx[32];
  float tw[32];
};

__device__ inline void block_topk_sigmoid_group(const float* l, const float* bias, int E, int K, int n_groups,
                                                int top_groups, float scale, int32_t* idx_out, float* w_out,
                                                SigmoidScratch& sc, uint64_t* keys, int* part, uint64_t* cand,
                                                uint64_t* sorted) {
  const int tid = threadIdx.x;
  if (tid < E) {
    const float s = 1.0f / (1.0f + expf(-l[tid]));
    sc.sig[tid] = s;
    sc.masked[tid] = bias ? s + bias[tid] : s;   // the selection score, masked below
  }
  __syncthreads();
  const int per = E / n_groups;
  if (tid < n_groups) {
    float m1 = -INFINITY, m2 = -INFINITY;
    for (int j = 0; j < per; ++j) {
      const float v = sc.masked[tid * per + j];
      if (v > m1) {
        m2 = m1;
        m1 = v;
      } else if (v > m2) {
        m2 = v;
      }
    }
    sc.gsc[tid] = per >= 2 ? m1 + m2 : m1;
  }
  __syncthreads();
  if (tid < n_groups) {
    const float me = sc.gsc[tid];
    int rank = 0;
    for (int g = 0; g < n_groups; ++g) rank += (sc.gsc[g] > me) || (sc.gsc[g] == me && g < tid);
    sc.keep[tid] = rank < top_groups;
  }
  __syncthreads();
  if (tid < E && !sc.keep[tid / per]) sc.masked[tid] = -INFINITY;
  __syncthreads();
  block_topk(sc.masked, E, K, sc.tidx, sc.tw, keys, part, cand, sorted);
  __syncthreads();
  if (tid < 64) {
    const float s = tid < K ? sc.sig[sc.tidx[tid]] : 0.f;
    const float sum = wave_sum(s);
    if (tid < K) {
      idx_out[tid] = sc.tidx[tid];
      w_out[tid] = scale * s / (sum + 1e-20f);
    }
  }
  __syncthreads();
}

}  // namespace eng
}  // namespace moe
