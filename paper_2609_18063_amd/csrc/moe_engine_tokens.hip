// Throughput schedule of independent single-token layer steps for gfx950.
//
// One cooperative launch of 256 workgroups (one per CU), split into 16 teams
// of 16 workgroups, two teams per XCD. Team t runs the steps s = t, t + 16,
// t + 32, ... so sixteen steps are in flight at once: while one team waits on
// an exchange, a top-k or a slot lookup, the others stream weights. Each step
// is still one token through one layer, and every weight byte a step reads
// serves that token only. Exchanges never leave the XCD.
//
// Work split of one step on team t, member m (NM = 16 members):
//   routing  member m computes router and head rows e = m + NM (w + 8 q) on
//            wave w; the team exchanges the logits; every member runs the
//            softmax-top-k (Appendix A) and resolves the K + S bundles
//            through the slot table.
//   gate/up  the K + S experts' intermediate rows lie end to end (n_list I
//            row pairs); member m owns rows [m RP, (m + 1) RP), RP =
//            n_list I / NM, at most two experts (segments). It streams their
//            gate and up rows through registers, plus one of every NM LoRA-A
//            rows of the step (published first, so that their exchange
//            overlaps the streaming).
//   h        with the LoRA-A products of its segments: h = silu(g) u for its
//            rows (Sec. 3.1 Math contract; unmerged LoRA, Sec. 3.3),
//            published, and its partial A_down h per segment.
//   down     member m owns output rows [m d/NM, (m + 1) d/NM) over all
//            n_list I columns. Its first down rows are loaded before it polls
//            h; it then writes its rows of y = sum_k w_k y_k + y_shared
//            directly, so no partial sums cross workgroups.
//
// The streaming loops are runtime loops over batches of four wave
// instructions held in three register buffers (two batches in flight while
// one is computed), so the code of a step stays small.
//
// Exchange words are {tag, fp32} (moe_xchg.h): the tag is the step's index
// on a device counter that persists across launches. Every exchange area is
// used once per step and is rewritten only after every member has read it
// (each rewrite of step s + 16 depends on an exchange that every member joins
// after finishing step s), so no area is double-buffered.
#include <hip/hip_runtime.h>

#include "moe_engine.h"
#include "moe_xchg.h"

namespace moe {
namespace tok {

using eng::kSpinMax;
using eng::ld_tag;
using eng::ld_u32;
using eng::st_tag;

constexpr int NX = 8, NPX = 32, NWG = NX * NPX, NT = 512, NWV = NT / 64;  // XCDs, workgroups per XCD
// A team is NM workgroups of one XCD that run one step at a time; NTM teams
// (NPX / NM per XCD) keep NTM steps in flight.
constexpr int NM = 16, NTM = NWG / NM;
static_assert(NPX % NM == 0, "whole teams per XCD");

typedef _Float16 hv2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Loads through the global address space (the pointers come from LDS, where
// the compiler cannot tell them from LDS addresses and would emit flat loads).
// Weights are streamed once: non-temporal.
__device__ __forceinline__ U4 ldw16(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(
      (const __attribute__((address_space(1))) u32x4*)(p));
  return U4{v.x, v.y, v.z, v.w};
}
__device__ __forceinline__ uint32_t ldw4(const void* p) {
  return __builtin_nontemporal_load((const __attribute__((address_space(1))) uint32_t*)(p));
}
__device__ __forceinline__ U4 ldg16(const void* p) {
  const u32x4 v = *(const __attribute__((address_space(1))) u32x4*)(p);
  return U4{v.x, v.y, v.z, v.w};
}
__device__ __forceinline__ uint16_t ldg2(const void* p) {
  return *(const __attribute__((address_space(1))) uint16_t*)(p);
}

// The routing of one step, resolved: list position k (k < K routed, then
// the shared experts) -> expert, weight, bundle and which adapters apply.
template <int NLX>
struct Route {
  int idx[32];
  float w[32];
  int ok[NLX];      // resolved to a resident bundle
  float wl[NLX];    // combine weight (0 when not resolved)
  float dsc[NLX];   // wl * lora_scale where the down adapter applies, else 0
  int lg[NLX], lu[NLX], ld[NLX];  // gate / up / down adapter applies
  moe_bundle bd[NLX];
};

// D: hidden size, IE: expert intermediate size, R: LoRA rank, NLX: most
// experts per token (K + S), EX: most routed experts (<= 256).
template <int D_, int IE_, int R_, int NLX_, int EX_>
struct TShape {
  static constexpr int D = D_, IE = IE_, R = R_, NLX = NLX_, EX = EX_;
  static constexpr int RPX = NLX * IE / NM;                   // most row pairs per workgroup
  static constexpr int LPR = D / 32 < 64 ? D / 32 : 64;       // lanes per gate/up row
  static constexpr int RPI = 64 / LPR;                        // gate/up rows per wave instruction
  static constexpr int CPL = D / 32 / LPR;                    // 16-byte code chunks per lane
  static constexpr int NGW = (2 * RPX / RPI + NWV - 1) / NWV; // most gate/up instructions per wave
  static constexpr int NB = NGW < 4 ? NGW : 4;                // gate/up instructions per batch
  static constexpr int CH = IE / 32;                          // lanes per down (row, expert) unit
  static constexpr int UPI = 64 / CH;                         // units per wave instruction
  static constexpr int DR = D / NM;                           // down rows per workgroup
  static constexpr int NDH = DR / UPI < 4 ? DR / UPI : 4;     // down instructions per batch (one expert)
  static constexpr int DRP = (DR * 8 + NT - 1) / NT;          // output-sum passes (eight lanes per row)
  static constexpr int NRW = (EX + NM * NWV - 1) / (NM * NWV); // router (and head) rows per wave
  static constexpr int NAX = (NLX * 2 * R + NM - 1) / NM;     // most LoRA-A rows per workgroup
  static constexpr int NPA = (RPX + 15) / 16;                 // rows per lane of an A_down term
  static constexpr int NEF = (NLX + 7) / 8;                   // experts per lane of the output sum
  static constexpr int NH = NLX * IE;                         // h entries of a step (most)
  static constexpr int MAXI_L = (EX + NT - 1) / NT;           // polled logits per thread
  static constexpr int MAXI_H = (NH + NM * 2 * R + NT - 1) / NT;  // polled h + A_down partials
  static constexpr int MAXI_A = (2 * 2 * R + NT - 1) / NT;    // polled LoRA-A products
  static_assert(D % 512 == 0 && IE % 64 == 0 && D % NM == 0, "shape");
  static_assert(RPX <= IE, "a workgroup's rows span at most two experts");
  static_assert(DR % (UPI * NDH) == 0, "a down batch stays inside one expert");
  static_assert(2 * R * 16 <= NT && R % 8 == 0, "one 16-lane group per A_down term");
  static_assert(DR * 8 <= NT || DR * 8 % NT == 0, "eight lanes per output row");
  static_assert(EX <= 256 && NRW <= 2, "at most two router rows per wave");
  static_assert(LPR != 64 || NB % 4 == 0, "whole-wave rows are summed four at a time");
  // LDS layout (bytes)
  static constexpr int NBAT = (NGW + NB - 1) / NB;            // gate/up batches per wave
  static constexpr int O_XH = 0;                          // [2][D] fp16, natural order, by step parity
  static constexpr int O_XQ = O_XH + 2 * D * 2;           // [2][D] fp16, pair order, by step parity
  static constexpr int O_LG = O_XQ + 2 * D * 2;           // [EX] router logits
  static constexpr int O_LH = O_LG + EX * 4;              // [EX] head logits
  static constexpr int O_TK = O_LH + EX * 4;              // top-k scratch: keys, ranks, candidates, result
  static constexpr int O_RT = O_TK + 256 * 8 + 256 * 4 + 128 * 8 + 32 * 8;  // [2] Route<NLX>, by step parity
  static constexpr int O_GXU = O_RT + 2 * (int)sizeof(Route<NLX>);  // [2 RPX] raw g, u
  static constexpr int O_AV = O_GXU + 2 * RPX * 4;        // [2][2R] LoRA-A products of the segments
  static constexpr int O_HL = O_AV + 2 * 2 * R * 4;       // [RPX] own h
  static constexpr int O_HX = O_HL + RPX * 4;             // h of the step, 32-entry chunks at stride 36
  static constexpr int O_ADP = O_HX + NH / 32 * 36 * 4;   // [NM][2][R] A_down partials
  static constexpr int O_ADV = O_ADP + NM * 2 * R * 4;    // [NLX][R] A_down h
  static constexpr int O_YP = O_ADV + NLX * R * 4;        // [DR][NLX] weighted down rows
  static constexpr int O_GUT = (O_YP + DR * NLX * 4 + 15) / 16 * 16;  // [2][2][2 RPX] gate/up row addresses
  static constexpr int NDX = NLX * DR / UPI;              // most down instructions per workgroup
  static constexpr int O_DNT = O_GUT + 2 * 2 * 2 * RPX * 8;  // [2][2][NDX] down row addresses
  static constexpr int O_AR = O_DNT + 2 * 2 * NDX * 8;    // [NAX][D] fp16 LoRA-A rows of the next step
  static constexpr int SOX = (EX + 32 + 63) / 64 * 64;    // slot-map entries staged (routed + shared ids)
  static constexpr int O_SO = O_AR + NAX * D * 2;         // [SOX] int32 slot map of the next step's layer
  static constexpr int O_SB = O_SO + SOX * 4;             // [SLX] bundles of the next step's layer
  // most slots per layer whose bundles are staged (none when they do not fit)
  static constexpr int SLX = O_SB + 320 * 96 + NWV * 8 + 1024 <= 160 * 1024 ? 320 : 0;
  static constexpr int O_RED = O_SB + SLX * 96;           // [NWV] fp64
  static constexpr int O_MISC = O_RED + NWV * 8;          // Misc
  static constexpr int LDS_USED = O_MISC + 1024;
  // More than half of the CU's LDS, so that no two workgroups share a CU.
  static constexpr int LDS_BYTES = LDS_USED > 82 * 1024 ? LDS_USED : 82 * 1024;
};

struct Misc {
  int abort;
  int x, m;  // this workgroup's XCD and member index
  int pidx[32];
  float pw[32];
};

struct Ctl {
  uint32_t* ctl;
  uint32_t* status;
};

// Abort: status bit and the sticky abort word; the first abort also leaves
// its cause in control words 4..7 (reason: 1 the workgroups do not spread 32
// per XCD, 2 wait time limit; blockIdx << 16 | wait site; then two details).
__device__ __forceinline__ void raise_abort(const Ctl& c, uint32_t reason = 2, uint32_t site = 0,
                                            uint32_t d0 = 0, uint32_t d1 = 0) {
  if (c.status) atomicOr(c.status, MOE_STATUS_ENGINE_ABORT);
  if (atomicCAS(&c.ctl[4], 0u, reason) == 0u) {
    __hip_atomic_store(&c.ctl[5], ((uint32_t)blockIdx.x << 16) | site, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&c.ctl[6], d0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&c.ctl[7], d1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __hip_atomic_store(&c.ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every thread polls items tid + q NT (q < MAXI) of `count` tagged words until
// each carries `tag`, storing the values; two barriers. Items are polled G at
// a time (G < MAXI holds fewer registers across the wait, at one memory round
// trip per group). False if a wait ran out or another workgroup raised the
// abort word.
template <int MAXI, int G = 4, typename AddrF, typename StoreF>
__device__ bool poll_all(int tid, int count, uint32_t tag, AddrF addr, StoreF store, const Ctl& c,
                         int* sh_abort, uint32_t site = 0) {
  long spin = 0;
  bool fail = false;
#pragma unroll
  for (int q0 = 0; q0 < MAXI; q0 += G) {
    uint32_t pending = 0;
#pragma unroll
    for (int q = 0; q < G; ++q)
      if (q0 + q < MAXI && tid + (q0 + q) * NT < count) pending |= 1u << q;
    while (pending && !fail) {
      uint64_t v[G];
#pragma unroll
      for (int q = 0; q < G; ++q)
        if ((pending >> q) & 1u) v[q] = ld_tag(addr(tid + (q0 + q) * NT));
#pragma unroll
      for (int q = 0; q < G; ++q)
        if (((pending >> q) & 1u) && (uint32_t)(v[q] >> 32) == tag) {
          store(tid + (q0 + q) * NT, __uint_as_float((uint32_t)v[q]));
          pending &= ~(1u << q);
        }
      if (!pending) break;
      if (++spin > kSpinMax) {
        raise_abort(c, 2, site, tag, (uint32_t)(tid + q0 * NT));
        fail = true;
      } else if ((spin & 63) == 0 && ld_u32(&c.ctl[2])) {
        fail = true;
      } else {
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  if (fail) *sh_abort = 1;
  __syncthreads();
  const bool ok = *sh_abort == 0;
  __syncthreads();
  return ok;
}

// fp16 row (global, D halves) held as this lane's D/512 16-byte chunks
// (chunk lane + 64 j) dotted with x (LDS, natural order); fp32 accumulate,
// summed over the wave.
template <int D>
__device__ __forceinline__ float row_dot(const U4 (&r)[D / 512], const __half* xh, int lane) {
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < D / 512; ++j)
    acc = dot8_h(r[j], *reinterpret_cast<const U4*>(xh + (lane + 64 * j) * 8), acc);
  return wave_sum(acc);
}
template <int D>
__device__ __forceinline__ void row_load(U4 (&r)[D / 512], const __half* row, int lane) {
#pragma unroll
  for (int j = 0; j < D / 512; ++j) r[j] = ldw16(row + (lane + 64 * j) * 8);
}

// Sum of 32 int4 codes (16 bytes, even input in the low nibble) times 32
// fp16 activations held in pair order (xp[4 i + mm] = inputs 8 i + mm and
// 8 i + mm + 4), in units of 2^-24: a code pair masked out of a dword is a
// pair of exact fp16 subnormals for v_dot2_f32_f16. Nibbles 1 and 3 of each
// byte pair are masked in place (16 times their value, still subnormal), so
// one shift per dword serves all four pairs; their sum is scaled back by 1/16
// (exact).
__device__ __forceinline__ float dot32_codes(const U4& q, const hv2 (&xp)[16]) {
  const uint32_t wd[4] = {q.x, q.y, q.z, q.w};
  float d0 = 0.f, d1 = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t w = wd[i], w8 = wd[i] >> 8;
    d0 = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w & 0x000F000Fu), xp[4 * i + 0], d0, false);
    d1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w & 0x00F000F0u), xp[4 * i + 1], d1, false);
    d0 = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w8 & 0x000F000Fu), xp[4 * i + 2], d0, false);
    d1 = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w8 & 0x00F000F0u), xp[4 * i + 3], d1, false);
  }
  return fmaf(d1, 0.0625f, d0);
}
// Sums over the wave of four values per lane at once: lane l returns the
// total of value (l & 3). Two exchange stages leave each lane one value
// summed over its lane pair and quad; rotations within the 16-lane row and
// two cross-row exchanges finish the sum.
__device__ __forceinline__ float rows4_sum(float v0, float v1, float v2, float v3, int lane) {
  const bool o1 = lane & 1, o2 = lane & 2;
  float a = o1 ? v1 : v0, b = o1 ? v0 : v1;
  float c = o1 ? v3 : v2, d = o1 ? v2 : v3;
  a += dpp_f<0xB1>(0.f, b);   // partner lane ^ 1
  c += dpp_f<0xB1>(0.f, d);
  float e = o2 ? c : a, f = o2 ? a : c;
  e += dpp_f<0x4E>(0.f, f);   // partner lane ^ 2
  e += dpp_f<0x124>(0.f, e);  // row_ror:4
  e += dpp_f<0x128>(0.f, e);  // row_ror:8
  e += __shfl_xor(e, 16, kWave);
  e += __shfl_xor(e, 32, kWave);
  return e;
}

// A value every lane holds alike, moved to scalar registers.
__device__ __forceinline__ const uint8_t* uniform_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ int uniform_int(int v) { return __builtin_amdgcn_readfirstlane(v); }

// fp64 sum of one value per thread over the workgroup (two barriers)
__device__ double block_sum_f64(double v, double* red) {
  v = eng::wave_sum_f64(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double tot = 0.0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) tot += red[w];
  __syncthreads();
  return tot;
}

// Phase timestamps for the profiling hook: thread 0 of members 0, 1 and 31 of
// XCD 0 writes the constant-rate wall clock at the marks of its steps.
constexpr int kProfMarks = 24;
__device__ __forceinline__ void mark(const EngineArgs& a, int g, int s, int k) {
  if (!a.phase_ts || threadIdx.x != 0) return;
  const int slot = g == 0 ? 0 : (g == NTM ? 1 : (g == NWG - NTM ? 2 : -1));
  if (slot < 0) return;
  a.phase_ts[((size_t)s * 3 + slot) * kProfMarks + k] = wall_clock64();
}

template <class SH>
__global__ void __launch_bounds__(NT) tokens_kernel(EngineArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int D = SH::D, IE = SH::IE, R = SH::R, NLX = SH::NLX;
  __half* const xh2 = reinterpret_cast<__half*>(smem + SH::O_XH);
  __half* const xq2 = reinterpret_cast<__half*>(smem + SH::O_XQ);
  float* lg = reinterpret_cast<float*>(smem + SH::O_LG);
  float* lh = reinterpret_cast<float*>(smem + SH::O_LH);
  uint64_t* const tk_keys = reinterpret_cast<uint64_t*>(smem + SH::O_TK);  // [256]
  int* const tk_part = reinterpret_cast<int*>(tk_keys + 256);               // [256]
  uint64_t* const tk_cand = reinterpret_cast<uint64_t*>(tk_part + 256);     // [128]
  uint64_t* const tk_sorted = tk_cand + 128;                                 // [32]
  Route<NLX>* routes = reinterpret_cast<Route<NLX>*>(smem + SH::O_RT);
  float* gxu = reinterpret_cast<float*>(smem + SH::O_GXU);
  float* av = reinterpret_cast<float*>(smem + SH::O_AV);
  float* hl = reinterpret_cast<float*>(smem + SH::O_HL);
  float* hx = reinterpret_cast<float*>(smem + SH::O_HX);
  float* adp = reinterpret_cast<float*>(smem + SH::O_ADP);
  float* adv = reinterpret_cast<float*>(smem + SH::O_ADV);
  float* yp = reinterpret_cast<float*>(smem + SH::O_YP);
  double* red = reinterpret_cast<double*>(smem + SH::O_RED);
  Misc* mi = reinterpret_cast<Misc*>(smem + SH::O_MISC);
  static_assert(sizeof(Misc) <= 1024, "misc block");
  // per-step address tables, by step parity: gate/up item t (gate rows, then
  // up rows) -> its code row and (scale, zero) row; down instruction n -> the
  // code and (scale, zero) rows of its first output row
  const uint8_t** const gu_q2 = reinterpret_cast<const uint8_t**>(smem + SH::O_GUT);
  const uint8_t** const dn_q2 = reinterpret_cast<const uint8_t**>(smem + SH::O_DNT);
  __half* const arow = reinterpret_cast<__half*>(smem + SH::O_AR);
  int32_t* const slot_lds = reinterpret_cast<int32_t*>(smem + SH::O_SO);
  char* const bund_lds = smem + SH::O_SB;
  const bool stage_bund = a.n_slots <= SH::SLX;  // else the bundles are read from the table

  const int tid0 = threadIdx.x;
  if (tid0 == 0) {
    mi->abort = 0;
    int px = 0, pm = 0;
    if (!eng::claim_place(a.ctl, NX, NPX, &px, &pm)) {
      raise_abort(Ctl{a.ctl, a.status}, 1, 0, eng::xcc_id(), (uint32_t)pm);
      mi->abort = 1;
    }
    mi->x = px + NX * (pm / NM);  // team
    mi->m = pm % NM;             // member of the team
    if (ld_u32(&a.ctl[2])) mi->abort = 1;
  }
  __syncthreads();
  // XCD and member index (uniform)
  const int x = __builtin_amdgcn_readfirstlane(mi->abort ? 0 : mi->x);
  const int m = __builtin_amdgcn_readfirstlane(mi->abort ? 0 : mi->m);
  int wave = __builtin_amdgcn_readfirstlane(tid0 >> 6);  // passed through an empty asm each step
  const int lane0 = tid0 & 63;
  const Ctl c{a.ctl, a.status};
  const int K = a.K, E = a.E, n_list = K + a.S;
  const int RP = n_list * IE / NM;           // row pairs of this workgroup
  const int row0 = m * RP;                   // first list row
  const int k0 = row0 / IE;                  // list position of segment 0
  const int split = min(RP, (k0 + 1) * IE - row0);  // local rows of segment 0
  const int nseg = split < RP ? 2 : 1;
  const int NG = 2 * RP / SH::RPI;           // gate/up wave instructions
  const int DI = SH::DR / SH::UPI;           // down instructions per expert
  const int NDI = n_list * DI;               // down instructions
  const int NA = n_list * 2 * R;             // LoRA-A rows of a step
  const int NHS = n_list * IE;               // h entries of a step

  // router and head logits by step parity; the other areas once per step
  uint64_t* const LG0 = a.xw + a.xo_logr + (size_t)x * 2 * a.xs_logr;
  uint64_t* const LH0 = a.xw + a.xo_loghm + (size_t)x * 2 * a.xs_logr;
  uint64_t* const AV = a.xw + a.xo_av + (size_t)x * a.xs_av;
  uint64_t* const HV = a.xw + a.xo_hv + (size_t)x * a.xs_hv;
  uint64_t* const ADP = a.xw + a.xo_adp + (size_t)x * a.xs_adp;

  const uint32_t base = ld_u32(&a.ctl[0]);

  // ---- a step's inputs, fetched a step ahead --------------------------------
  // step_layer early, the layer's pointers later, the draws and the router
  // rows at the end of the step before: each load is consumed long after it
  // is issued, so no wait lands in the middle of a step. The head rows are
  // loaded when the step's routing starts and consumed after the LoRA-A
  // products.
  constexpr int XPT = D / NT;
  float xin[XPT];
  U4 rrow[SH::NRW][D / 512];
  typedef U4 HRows[SH::NRW][D / 512];
  // this wave's router and head rows e = m + NM (wave + NWV q)
  auto e_row = [&](int q) { return m + NM * (wave + NWV * q); };
  int lay_f = -1, lay_n = -1;       // the layer of the fetched inputs; of the next fetch
  bool head_f = false;
  const __half *rt_n = nullptr, *hd_n = nullptr, *hd_f = nullptr;
  auto layer_ok = [&](int l) { return l >= 0 && l < a.n_table_layers; };
  auto fetch_layer = [&]() {
    rt_n = hd_n = nullptr;
    if (layer_ok(lay_n)) {
      rt_n = reinterpret_cast<const __half*>(a.layers[lay_n].router);
      hd_n = reinterpret_cast<const __half*>(a.layers[lay_n].head);
    }
  };
  // every register it writes is written on every path (no value lives
  // through a whole step)
  auto fetch_rows = [&](int s1) {
#pragma unroll
    for (int q = 0; q < XPT; ++q) xin[q] = a.xi[(size_t)s1 * D + tid0 + q * NT];
    lay_f = lay_n;
    head_f = layer_ok(lay_f) && hd_n != nullptr;
    hd_f = hd_n;
#pragma unroll
    for (int q = 0; q < SH::NRW; ++q) {
      const bool rows = layer_ok(lay_f) && e_row(q) < E;
      const __half* rsrc = rows ? rt_n + (size_t)e_row(q) * D : reinterpret_cast<const __half*>(a.xi);
      row_load<D>(rrow[q], rsrc, lane0);
    }
  };

  // ---- routing of step s1, in two halves -----------------------------------
  // the head rows of the fetched step (on = it is routed here); every
  // register of hr is written on every path
  auto head_load = [&](bool on, HRows& hr, int lane) {
#pragma unroll
    for (int q = 0; q < SH::NRW; ++q) {
      const bool rows = on && head_f && e_row(q) < E;
      row_load<D>(hr[q], rows ? hd_f + (size_t)e_row(q) * D : reinterpret_cast<const __half*>(a.xi), lane);
    }
  };
  // publish: x = fp16(rmsnorm(xi)) (single rounding from fp64) and this
  // workgroup's router logits. Uses the fetched inputs.
  auto route_publish = [&](int s1, int tid, int lane) {
    const uint32_t tag1 = base + (uint32_t)s1 + 1u;
    const int par1 = (s1 / NTM) & 1;
    __half* const xh = xh2 + par1 * D;
    __half* const xq = xq2 + par1 * D;
    double acc = 0.0;
#pragma unroll
    for (int q = 0; q < XPT; ++q) acc += (double)xin[q] * (double)xin[q];
    const double inv = eng::rsqrt_f64(block_sum_f64(acc, red) / (double)D + 1e-6);
#pragma unroll
    for (int q = 0; q < XPT; ++q) {
      const int j = tid + q * NT;
      const __half h = eng::f64_to_h((double)xin[q] * inv);
      xh[j] = h;
      xq[eng::pair_pos(j)] = h;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < SH::NRW; ++q) {
      const int e = e_row(q);
      if (e >= E) continue;
      const float v = row_dot<D>(rrow[q], xh, lane);
      if (lane == 0) st_tag(LG0 + (size_t)par1 * a.xs_logr + e, tag1, v);
    }
  };
  // the head logits of step s1 (after route_publish, whose barrier made x
  // visible)
  auto head_publish = [&](int s1, const HRows& hr, int lane) {
    if (!head_f) return;
    const uint32_t tag1 = base + (uint32_t)s1 + 1u;
    const int par1 = (s1 / NTM) & 1;
    const __half* const xh = xh2 + par1 * D;
#pragma unroll
    for (int q = 0; q < SH::NRW; ++q) {
      const int e = e_row(q);
      if (e >= E) continue;
      const float vh = row_dot<D>(hr[q], xh, lane);
      if (lane == 0) st_tag(LH0 + (size_t)par1 * a.xs_logr + e, tag1, vh);
    }
  };
  // poll: the step's router logits into lg (every thread). False on abort.
  auto route_poll = [&](int s1, int tid) -> bool {
    const uint32_t tag1 = base + (uint32_t)s1 + 1u;
    uint64_t* const LG = LG0 + (size_t)((s1 / NTM) & 1) * a.xs_logr;
    return poll_all<SH::MAXI_L>(tid, E, tag1, [&](int i) { return LG + i; }, [&](int i, float v) { lg[i] = v; },
                                c, &mi->abort, 1);
  };
  // select: softmax-top-k of lg (every thread, two barriers) into
  // routes[parity]; then wave 0 resolves the slots and bundles (staged slot
  // map and bundles, waited for before an earlier barrier) and, when
  // predictions are recorded, the
  // workgroup polls the head's logits and records their top-k. Returns false
  // on abort. The caller's next barrier publishes routes[parity].
  auto route_select = [&](int s1, int lay1, bool head1, int tid, int lane) -> bool {
    const uint32_t tag1 = base + (uint32_t)s1 + 1u;
    const int par1 = (s1 / NTM) & 1;
    uint64_t* const LH = LH0 + (size_t)par1 * a.xs_logr;
    Route<NLX>& rt = routes[par1];
    eng::block_topk(lg, E, K, rt.idx, rt.w, tk_keys, tk_part, tk_cand, tk_sorted);
    __syncthreads();
    if (wave == 0) {
      if (lane < n_list) {  // list position k = lane
        const int k = lane;
        const int e = k < K ? rt.idx[k] : E + (k - K);
        const bool bad = k < K && (e < 0 || e >= E);
        const int slot = bad ? -1 : slot_lds[e];
        const bool ok = slot >= 0;
        // the bundle's 12 pointers as six 16-byte words (gate, up, down: q,
        // sz, lora_a, lora_b each), copied to LDS
        static_assert(sizeof(moe_bundle) == 96, "bundle layout");
        U4 bw[6];
        if (stage_bund) {
          const U4* bl = reinterpret_cast<const U4*>(bund_lds + (size_t)(ok ? slot : 0) * 96);
#pragma unroll
          for (int i = 0; i < 6; ++i) bw[i] = ok ? bl[i] : U4{0u, 0u, 0u, 0u};
        } else {
          const char* bsrc = reinterpret_cast<const char*>(a.bundles + (size_t)lay1 * a.n_slots + (ok ? slot : 0));
#pragma unroll
          for (int i = 0; i < 6; ++i) bw[i] = ok ? ldg16(bsrc + 16 * i) : U4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int i = 0; i < 6; ++i) reinterpret_cast<U4*>(&rt.bd[k])[i] = bw[i];
        // lora_a, lora_b of projection j are the words 2j + 1 (both halves)
        auto both = [](const U4& v) { return (v.x | v.y) != 0u && (v.z | v.w) != 0u; };
        const float wk = ok ? (k < K ? rt.w[k] : 1.f) : 0.f;
        const bool lora = ok && a.r > 0;
        rt.ok[k] = ok;
        rt.wl[k] = wk;
        rt.lg[k] = lora && both(bw[1]);
        rt.lu[k] = lora && both(bw[3]);
        rt.ld[k] = lora && both(bw[5]);
        rt.dsc[k] = rt.ld[k] ? wk * a.lora_scale : 0.f;
        if (m == 0 && a.status) {
          if (bad) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
          else if (slot < 0) atomicOr(a.status, MOE_STATUS_SLOT_MISS);
        }
      }
      if (m == 0 && lane < K) {
        if (a.idx_rec) a.idx_rec[(size_t)s1 * K + lane] = rt.idx[lane];
        if (a.w_rec) a.w_rec[(size_t)s1 * K + lane] = rt.w[lane];
      }
    }
    if (m == 0 && head1 && (a.pidx_rec || a.pw_rec)) {  // the head's prediction, recorded
      if (!poll_all<SH::MAXI_L>(tid, E, tag1, [&](int i) { return LH + i; }, [&](int i, float v) { lh[i] = v; },
                                c, &mi->abort, 4))
        return false;
      eng::block_topk(lh, E, K, mi->pidx, mi->pw, tk_keys, tk_part, tk_cand, tk_sorted);
      if (tid < K) {
        if (a.pidx_rec) a.pidx_rec[(size_t)s1 * K + tid] = mi->pidx[tid];
        if (a.pw_rec) a.pw_rec[(size_t)s1 * K + tid] = mi->pw[tid];
      }
    }
    return true;
  };

  // The slot map row and the bundle row of a layer, staged into LDS by every
  // wave (64-entry blocks dealt round-robin). Each wave waits for its own
  // copies (dma_wait) before a barrier that precedes their reader. Slot-map
  // entries past n_ids repeat the last one.
  auto stage_slots = [&](int lay1, int lane) {
    const int32_t* row = a.slot_of + (size_t)lay1 * a.n_ids;
    for (int i0 = 64 * wave; i0 < a.n_ids && i0 < SH::SOX; i0 += 64 * NWV) {
      const int i = min(i0 + lane, a.n_ids - 1);
      eng::dma4(row + i, slot_lds + i0);
    }
    if (stage_bund) {  // the layer's bundle row, 16-byte chunks
      const char* brow = reinterpret_cast<const char*>(a.bundles + (size_t)lay1 * a.n_slots);
      const int nch = a.n_slots * 6;
      for (int c0 = 64 * wave; c0 < nch; c0 += 64 * NWV) {
        const int ch = min(c0 + lane, nch - 1);
        eng::dma16(brow + (size_t)ch * 16, bund_lds + (size_t)c0 * 16);
      }
    }
  };
  // This wave's LoRA-A rows of a resolved step (rows ar = m + NM qa, qa =
  // wave, wave + 8, ...), staged into arow[qa]; the wave reads them after its
  // own dma_wait.
  auto stage_arows = [&](const Route<NLX>& r1, int lane) {
    for (int qa = wave; qa < SH::NAX; qa += NWV) {
      const int ar = m + NM * qa;
      if (ar >= NA) break;
      const int k = ar / (2 * R), proj = (ar / R) & 1, kk = ar % R;
      if (!(proj ? r1.lu[k] : r1.lg[k])) continue;
      const __half* A = reinterpret_cast<const __half*>(proj ? r1.bd[k].up.lora_a : r1.bd[k].gate.lora_a) +
                        (size_t)kk * D;
#pragma unroll
      for (int c8 = 0; c8 < D / 512; ++c8) eng::dma16(A + (c8 * 64 + lane) * 8, arow + (size_t)qa * D + c8 * 512);
    }
  };

  // The address tables of a resolved step (rows of an expert that is not
  // resident read row 0 of the draws instead; their results are discarded).
  auto fill_tables = [&](const Route<NLX>& r1, int par1, int tid) {
    const uint8_t* const dummy = reinterpret_cast<const uint8_t*>(a.xi);
    const uint8_t** const gq = gu_q2 + par1 * 4 * SH::RPX;
    const uint8_t** const gs = gq + 2 * SH::RPX;
    const uint8_t** const dq = dn_q2 + par1 * 2 * SH::NDX;
    const uint8_t** const ds = dq + SH::NDX;
    for (int t = tid; t < 2 * RP; t += NT) {
      const bool up = t >= RP;
      const int p = up ? t - RP : t;
      const int k = k0 + (p >= split ? 1 : 0);
      const int er = row0 + p - k * IE;
      const moe_proj& pj = up ? r1.bd[k].up : r1.bd[k].gate;
      const bool ok = r1.ok[k];
      gq[t] = ok ? reinterpret_cast<const uint8_t*>(pj.q) + (size_t)er * (D / 2) : dummy;
      gs[t] = ok ? reinterpret_cast<const uint8_t*>(pj.sz) + (size_t)er * (D / 16) : dummy;
    }
    for (int n = tid; n < NDI; n += NT) {
      const int k = n / DI, jj0 = (n % DI) * SH::UPI;
      const bool ok = r1.ok[k];
      const size_t row = (size_t)m * SH::DR + jj0;
      dq[n] = ok ? reinterpret_cast<const uint8_t*>(r1.bd[k].down.q) + row * (IE / 2) : dummy;
      ds[n] = ok ? reinterpret_cast<const uint8_t*>(r1.bd[k].down.sz) + row * (IE / 16) : dummy;
    }
  };

  // ---- first step of this team: routed before the loop -----------------------
  int lay = -1;      // layer of the current step
  bool cur_ok = false;
  if (x < a.n_steps && !mi->abort) {
    lay_n = a.step_layer[x];
    fetch_layer();
    fetch_rows(x);
    lay = lay_f;
    cur_ok = layer_ok(lay);
    if (cur_ok) {
      const bool head0 = head_f;
      {
        HRows hr;
        head_load(true, hr, lane0);
        route_publish(x, tid0, lane0);
        head_publish(x, hr, lane0);
      }
      lay_n = a.step_layer[x + NTM < a.n_steps ? x + NTM : x];
      fetch_layer();
      stage_slots(lay, lane0);
      eng::dma_wait();
      if (route_poll(x, tid0) && route_select(x, lay, head0, tid0, lane0)) {
        __syncthreads();
        if (!mi->abort) {
          fill_tables(routes[(x / NTM) & 1], (x / NTM) & 1, tid0);
          stage_arows(routes[(x / NTM) & 1], lane0);
          fetch_rows(x + NTM < a.n_steps ? x + NTM : x);
        }
      }
    }
  }

  for (int s = x; s < a.n_steps && !mi->abort; s += NTM) {
    // The thread's index passes through an empty asm each step, so that the
    // compiler recomputes the addresses derived from it inside the step
    // rather than keeping all of them in registers across the loop.
    int tid = tid0, lane = lane0;
    asm volatile("" : "+v"(tid), "+v"(lane), "+s"(wave));
    const uint32_t tag = base + (uint32_t)s + 1u;
    mark(a, x + NTM * m, s, 0);
    if (!cur_ok) {  // the same for every member of the team
      if (m == 0 && tid == 0 && a.status) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      break;
    }
    const int par = (s / NTM) & 1;
    const Route<NLX>& rt = routes[par];
    const __half* const xh = xh2 + par * D;
    const __half* const xq = xq2 + par * D;
    // the next step of this team, routed during this one (its inputs are in
    // xin / rrow / hrow, its layer in lay_f)
    const int s1 = s + NTM;
    const bool has_next = s1 < a.n_steps;
    const int lay1 = lay_f;
    const bool next_ok = has_next && layer_ok(lay1);
    const bool head1 = head_f;
    const int s2 = s1 + NTM < a.n_steps ? s1 + NTM : (has_next ? s1 : s);
    lay_n = a.step_layer[s2];
    const uint8_t* const* const gu_q = gu_q2 + par * 4 * SH::RPX;
    const uint8_t* const* const gu_s = gu_q + 2 * SH::RPX;
    const uint8_t* const* const dn_q = dn_q2 + par * 2 * SH::NDX;
    const uint8_t* const* const dn_s = dn_q + SH::NDX;
    // ---- gate/up rows (raw int4 matvecs), set up and first two batches issued
    eng::dma_wait();  // this wave's LoRA-A rows, staged during the previous step
    // Item t < RP is the gate row of local row t, item RP + t its up row.
    // Codes become fp16 pairs q 2^-24 (exact subnormals) under one mask and
    // meet x in its pair order in v_dot2_f32_f16; 2^24 goes into the scale.
    // Batches of NB wave instructions in three register buffers: two batches
    // are in flight while one is computed. The first two are issued at the
    // start of the step, ahead of the routing work.
    const int c0 = lane % SH::LPR, gsub = SH::RPI == 1 ? 0 : lane / SH::LPR;
    hv2 xp[SH::CPL][16];
    float xs[SH::CPL];
    const hv2 one2 = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
    for (int cc = 0; cc < SH::CPL; ++cc) {
      const int ch = c0 + SH::LPR * cc;
      const U4* src = reinterpret_cast<const U4*>(xq + ch * 32);
      float sacc = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const U4 v = src[i];
        xp[cc][4 * i + 0] = __builtin_bit_cast(hv2, v.x);
        xp[cc][4 * i + 1] = __builtin_bit_cast(hv2, v.y);
        xp[cc][4 * i + 2] = __builtin_bit_cast(hv2, v.z);
        xp[cc][4 * i + 3] = __builtin_bit_cast(hv2, v.w);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc = __builtin_amdgcn_fdot2(xp[cc][i], one2, sacc, false);
      xs[cc] = sacc;
    }
    typedef U4 QB[SH::NB][SH::CPL];
    typedef uint32_t SB[SH::NB][SH::CPL];
    // rows come from the step's address table (the compiler keeps no
    // per-row address in registers across the batches)
    const int nbat = ((NG + NWV - 1) / NWV + SH::NB - 1) / SH::NB;  // batches per wave (most)
    // (loads past the last batch read the first bytes of the draws, which
    // the caches hold: a load skipped on some paths would keep its registers
    // live across the whole step)
    const uint8_t* const hot = reinterpret_cast<const uint8_t*>(a.xi);
    auto gu_load = [&](int b, QB& qv, SB& szw) {
      const uint8_t* pq[SH::NB];
      const uint8_t* ps[SH::NB];
#pragma unroll
      for (int j = 0; j < SH::NB; ++j) {
        int n = wave + NWV * (b * SH::NB + j);  // wave-uniform
        const bool in = b < nbat;
        if (n >= NG) n = NG - 1;                // loaded again, not stored
        const int t = n * SH::RPI + gsub;
        pq[j] = in ? gu_q[t] : hot;
        ps[j] = in ? gu_s[t] : hot;
      }
#pragma unroll
      for (int j = 0; j < SH::NB; ++j) {
#pragma unroll
        for (int cc = 0; cc < SH::CPL; ++cc) {
          const int ch = c0 + SH::LPR * cc;
          qv[j][cc] = ldw16(pq[j] + ch * 16);
          szw[j][cc] = ldw4(ps[j] + (ch >> 1) * 4);
        }
      }
    };
    auto gu_row = [&](const U4 (&qv)[SH::CPL], const uint32_t (&szw)[SH::CPL]) {
      float acc = 0.f;
#pragma unroll
      for (int cc = 0; cc < SH::CPL; ++cc) {
        const float2 sz = h2f2(szw[cc]);
        acc += (sz.x * 16777216.f) * dot32_codes(qv[cc], xp[cc]) + sz.y * xs[cc];
      }
      return acc;
    };
    auto gu_compute = [&](int b, const QB& qv, const SB& szw) {
      if constexpr (SH::LPR == 64) {  // one row per instruction: sum four rows at once
#pragma unroll
        for (int j = 0; j < SH::NB; j += 4) {
          const int n0 = wave + NWV * (b * SH::NB + j);
          if (n0 >= NG) continue;
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = n0 + NWV * r < NG ? gu_row(qv[j + r], szw[j + r]) : 0.f;
          const float tot = rows4_sum(v[0], v[1], v[2], v[3], lane);
          const int nr = n0 + NWV * (lane & 3);
          if (lane < 4 && nr < NG) gxu[nr] = tot;
        }
      } else {
#pragma unroll
        for (int j = 0; j < SH::NB; ++j) {
          const int n = wave + NWV * (b * SH::NB + j);
          if (n >= NG) continue;
          const float acc = group_sum(gu_row(qv[j], szw[j]), SH::LPR);
          if (c0 == 0) gxu[n * SH::RPI + gsub] = acc;
        }
      }
    };
    QB q0, q1, q2;
    SB z0, z1, z2;
    gu_load(0, q0, z0);
    gu_load(1, q1, z1);
    if (next_ok) stage_slots(lay1, lane);
    mark(a, x + NTM * m, s, 10);
    // ---- the next step's routing, first half: its x and router rows -----------
    // (into the other parity's x buffer; the fetched inputs die here); the
    // head rows are loaded meanwhile and dotted after the LoRA-A products
    HRows hr;
    head_load(next_ok, hr, lane);
    if (next_ok) route_publish(s1, tid, lane);
    mark(a, x + NTM * m, s, 11);

    // ---- LoRA-A rows of the step: row ar = m + NM qa of the list's
    // (position, projection, rank) rows, published first ----------------------
    for (int qa = wave; qa < SH::NAX; qa += NWV) {
      const int ar = m + NM * qa;
      if (ar >= NA) break;
      const int k = ar / (2 * R), proj = (ar / R) & 1;
      const bool on = proj ? rt.lu[k] : rt.lg[k];
      float v = 0.f;
      if (on) {
        U4 ra[D / 512];
#pragma unroll
        for (int c8 = 0; c8 < D / 512; ++c8)
          ra[c8] = *reinterpret_cast<const U4*>(arow + (size_t)qa * D + (c8 * 64 + lane) * 8);
        v = row_dot<D>(ra, xh, lane);
      }
      if (lane == 0) st_tag(AV + ar, tag, v);
    }
    if (next_ok) head_publish(s1, hr, lane);
    mark(a, x + NTM * m, s, 1);

    // ---- LoRA-B rows of gate and up (thread t < RP: local row t), loaded
    // before the gate/up rows so that they arrive during the streaming
    constexpr int BV = R / 8;
    U4 bg[BV], bu[BV];
    int kt = k0, ert = 0;
    if (tid < RP) {
      kt = k0 + (tid >= split ? 1 : 0);
      ert = row0 + tid - kt * IE;
#pragma unroll
      for (int v = 0; v < BV; ++v) {
        bg[v] = rt.lg[kt] ? ldw16(reinterpret_cast<const __half*>(rt.bd[kt].gate.lora_b) + (size_t)ert * R + 8 * v)
                          : U4{0u, 0u, 0u, 0u};
        bu[v] = rt.lu[kt] ? ldw16(reinterpret_cast<const __half*>(rt.bd[kt].up.lora_b) + (size_t)ert * R + 8 * v)
                          : U4{0u, 0u, 0u, 0u};
      }
    }
    // A_down at this workgroup's rows, also loaded ahead of the gate/up rows
    // (term (q, kk) = tid / 16, rows sub + 16 j)
    const int term = tid >> 4, sub = tid & 15;
    const int qd = term / R, kkd = term % R;
    const int kd = k0 + qd;
    const bool dterm = term < 2 * R && qd < nseg && rt.ld[kd];
    const int plo = qd ? split : 0, phi = qd ? RP : split;
    float ad[SH::NPA];
#pragma unroll
    for (int j = 0; j < SH::NPA; ++j) {
      const int p = plo + sub + 16 * j;
      ad[j] = 0.f;
      if (dterm && p < phi)
        ad[j] = __half2float(__ushort_as_half(
            ldg2(reinterpret_cast<const __half*>(rt.bd[kd].down.lora_a) + (size_t)kkd * IE + row0 + p - kd * IE)));
    }

    // ---- gate/up rows: the batch loop ----------------------------------------
    for (int b = 0; b < nbat; b += 3) {
      gu_load(b + 2, q2, z2);
      gu_compute(b, q0, z0);
      gu_load(b + 3, q0, z0);
      gu_compute(b + 1, q1, z1);
      gu_load(b + 4, q1, z1);
      gu_compute(b + 2, q2, z2);
    }
    mark(a, x + NTM * m, s, 2);

    // ---- the next step's routing, second half: its logits (published by every
    // member at the start of this step) -> top-k, slots, bundles; then its
    // address tables ------------------------------------------------------------
    eng::dma_wait();  // this wave's copies of the slot map and bundles
    if (next_ok) {
      if (!route_poll(s1, tid)) break;
      if (!route_select(s1, lay1, head1, tid, lane)) break;
    }
    __syncthreads();
    if (mi->abort) break;
    if (next_ok) fill_tables(routes[par ^ 1], par ^ 1, tid);
    mark(a, x + NTM * m, s, 3);

    // ---- LoRA-A products of the segments -> h of this workgroup's rows ---------
    {
      if (!poll_all<SH::MAXI_A>(tid, nseg * 2 * R, tag, [&](int i) { return AV + (size_t)k0 * 2 * R + i; },
                                [&](int i, float v) { av[i] = v; }, c, &mi->abort, 2))
        break;
      mark(a, x + NTM * m, s, 4);
      if (tid < RP) {
        const int q = kt - k0;
        float sg = 0.f, su = 0.f;
#pragma unroll
        for (int v = 0; v < BV; ++v) {
          const uint32_t wg[4] = {bg[v].x, bg[v].y, bg[v].z, bg[v].w};
          const uint32_t wu[4] = {bu[v].x, bu[v].y, bu[v].z, bu[v].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 fg = h2f2(wg[i]), fu = h2f2(wu[i]);
            const int kk = 8 * v + 2 * i;
            sg = fmaf(fg.x, av[q * 2 * R + kk], sg);
            sg = fmaf(fg.y, av[q * 2 * R + kk + 1], sg);
            su = fmaf(fu.x, av[q * 2 * R + R + kk], su);
            su = fmaf(fu.y, av[q * 2 * R + R + kk + 1], su);
          }
        }
        float hv = 0.f;
        if (rt.ok[kt]) {
          const float gg = rt.lg[kt] ? fmaf(a.lora_scale, sg, gxu[tid]) : gxu[tid];
          const float uu = rt.lu[kt] ? fmaf(a.lora_scale, su, gxu[RP + tid]) : gxu[RP + tid];
          hv = eng::silu(gg) * uu;
        }
        st_tag(HV + row0 + tid, tag, hv);
        hl[tid] = hv;
      }
      __syncthreads();
      // partial A_down h of segment qd over this workgroup's rows
      if (term < 2 * R) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < SH::NPA; ++j) {
          const int p = plo + sub + 16 * j;
          if (dterm && p < phi) acc = fmaf(ad[j], hl[p], acc);
        }
        acc = group_sum(acc, 16);
        if (sub == 0) st_tag(ADP + ((size_t)m * 2 + qd) * R + kkd, tag, acc);
      }
    }
    mark(a, x + NTM * m, s, 5);

    // ---- down rows of this workgroup over every expert of the step -------------
    {
      // Batches of NDH consecutive instructions n, all of one list position
      // k = n / DI (rows (n % DI) UPI + lane / CH, 32-column chunk lane % CH);
      // wave w takes batches [w nbw, (w + 1) nbw). Three register buffers:
      // the first two batches are loaded before the waits of this phase, each
      // later one while the batch two before it is computed.
      const int cl = lane % SH::CH, su = lane / SH::CH;
      constexpr int NDH = SH::NDH;
      const int nbt = NDI / NDH;                  // batches of the step
      const int nbw = (nbt + NWV - 1) / NWV;      // per wave (most)
      const int nbe = max(0, min(nbw, nbt - wave * nbw));  // this wave's
      typedef U4 DQ[NDH];
      typedef uint32_t DS[NDH];
      auto dn_load = [&](int i, DQ& dq, DS& dsz) {  // past the end: the draws' first bytes
        const bool in = i < nbe;
        const int n0 = min(wave * nbw + min(i, nbe - 1), nbt - 1) * NDH;
        const uint8_t* pq[NDH];
        const uint8_t* ps[NDH];
#pragma unroll
        for (int jh = 0; jh < NDH; ++jh) {
          pq[jh] = in ? dn_q[n0 + jh] : hot;
          ps[jh] = in ? dn_s[n0 + jh] : hot;
        }
#pragma unroll
        for (int jh = 0; jh < NDH; ++jh) {
          dq[jh] = ldw16(pq[jh] + su * (IE / 2) + cl * 16);
          dsz[jh] = ldw4(ps[jh] + su * (IE / 16) + (cl >> 1) * 4);
        }
      };
      DQ dq0, dq1, dq2;
      DS ds0, ds1, ds2;
      dn_load(0, dq0, ds0);
      dn_load(1, dq1, ds1);
      if (next_ok) fetch_layer();
      // LoRA-B rows of down for the output sum: lane (j, part) = (tid / 8 +
      // NT / 8 p, tid % 8) in pass p; loaded after the waits of this phase
      constexpr int BV = R / 8;
      const int part = tid & 7;
      auto jo_of = [&](int p) { return (tid >> 3) + (NT / 8) * p; };
      U4 bd[SH::DRP][SH::NEF][BV];
      auto bd_load = [&]() {
#pragma unroll
        for (int p = 0; p < SH::DRP; ++p) {
          const int jo = jo_of(p);
#pragma unroll
          for (int i = 0; i < SH::NEF; ++i) {
            const int k = part + 8 * i;
#pragma unroll
            for (int v = 0; v < BV; ++v) {
              bd[p][i][v] = U4{0u, 0u, 0u, 0u};
              if (jo < SH::DR && k < n_list && rt.ld[k])
                bd[p][i][v] = ldw16(reinterpret_cast<const __half*>(rt.bd[k].down.lora_b) +
                                    ((size_t)m * SH::DR + jo) * R + 8 * v);
            }
          }
        }
      };
      // the next step's LoRA-A rows (the current step's were read at its start)
      if (next_ok) stage_arows(routes[par ^ 1], lane);
      mark(a, x + NTM * m, s, 6);
      // h of the step and the A_down partials of the team
      if (!poll_all<SH::MAXI_H, (SH::MAXI_H + 1) / 2>(
              tid, NHS + NM * 2 * R, tag,
              [&](int i) { return i < NHS ? HV + i : ADP + (i - NHS); },
              [&](int i, float v) {
                if (i < NHS) hx[(i >> 5) * 36 + (i & 31)] = v;
                else adp[i - NHS] = v;
              },
              c, &mi->abort, 3))
        break;
      mark(a, x + NTM * m, s, 7);
      // A_down h of list position k: the partials of the workgroups whose rows
      // meet expert k, in workgroup order
      if (tid < n_list * R) {
        const int k = tid / R, kk = tid % R;
        const int mlo = k * IE / RP, mhi = ((k + 1) * IE - 1) / RP;
        float acc = 0.f;
        for (int mm = mlo; mm <= mhi; ++mm) {
          const int q = k == mm * RP / IE ? 0 : 1;
          acc += adp[(mm * 2 + q) * R + kk];
        }
        adv[tid] = acc;
      }
      bd_load();
      // down dot products: h of the batch's expert is reloaded when the
      // expert changes. The lane's 32 h values (fp32) are rounded once to
      // fp16 (|h| < 65504), in pair order, so the codes meet them in
      // v_dot2_f32_f16 with fp32 accumulation; the zero-point term takes the
      // fp32 sum of h.
      hv2 hh[16];
      float hsum = 0.f;
      int kc = -1;
      auto dn_compute = [&](int i, const DQ& dq, const DS& dsz) {
        if (i >= nbe) return;
        const int n0 = (wave * nbw + i) * NDH;
        const int k = n0 / DI;
        if (k != kc) {
          kc = k;
          const float4* hp = reinterpret_cast<const float4*>(hx + ((k * IE) / 32 + cl) * 36);
          float hv[32];
          hsum = 0.f;
#pragma unroll
          for (int e4 = 0; e4 < 8; ++e4) {
            const float4 v4 = hp[e4];
            hv[4 * e4] = v4.x;
            hv[4 * e4 + 1] = v4.y;
            hv[4 * e4 + 2] = v4.z;
            hv[4 * e4 + 3] = v4.w;
            hsum += (v4.x + v4.y) + (v4.z + v4.w);
          }
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
#pragma unroll
            for (int mm = 0; mm < 4; ++mm) {
              const float a0 = hv[8 * q4 + mm], a1 = hv[8 * q4 + mm + 4];
              hh[4 * q4 + mm] = hv2{(_Float16)a0, (_Float16)a1};
            }
          }
        }
#pragma unroll
        for (int jh = 0; jh < NDH; ++jh) {
          const int jj = ((n0 + jh) % DI) * SH::UPI + su;
          const float2 sz = h2f2(dsz[jh]);
          float v = (sz.x * 16777216.f) * dot32_codes(dq[jh], hh) + sz.y * hsum;
          v = group_sum(v, SH::CH);
          if (cl == 0) yp[jj * NLX + k] = rt.wl[k] * v;
        }
      };
      for (int i = 0; i < nbw; i += 3) {
        dn_load(i + 2, dq2, ds2);
        dn_compute(i, dq0, ds0);
        dn_load(i + 3, dq0, ds0);
        dn_compute(i + 1, dq1, ds1);
        dn_load(i + 4, dq1, ds1);
        dn_compute(i + 2, dq2, ds2);
      }
      __syncthreads();
      mark(a, x + NTM * m, s, 8);
      // the inputs of the step after next arrive while y is summed
      fetch_rows(s2);
      // y = sum over list positions of the weighted down rows and LoRA terms
#pragma unroll
      for (int p = 0; p < SH::DRP; ++p) {
        const int jo = jo_of(p);
        if (jo >= SH::DR) continue;
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < SH::NEF; ++i) {
          const int k = part + 8 * i;
          if (k >= n_list) continue;
          acc += yp[jo * NLX + k];
          const float sc = rt.dsc[k];
          if (sc != 0.f) {
            float t = 0.f;
#pragma unroll
            for (int v = 0; v < BV; ++v) {
              const uint32_t wb[4] = {bd[p][i][v].x, bd[p][i][v].y, bd[p][i][v].z, bd[p][i][v].w};
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const float2 fb = h2f2(wb[q]);
                t = fmaf(fb.x, adv[k * R + 8 * v + 2 * q], t);
                t = fmaf(fb.y, adv[k * R + 8 * v + 2 * q + 1], t);
              }
            }
            acc = fmaf(sc, t, acc);
          }
        }
        acc = group_sum(acc, 8);
        if (part == 0) a.y[(size_t)s * D + (size_t)m * SH::DR + jo] = acc;
      }
      __syncthreads();
      mark(a, x + NTM * m, s, 9);
    }
    cur_ok = next_ok;
    if (has_next && !next_ok) {  // the next step's layer is outside the table
      if (m == 0 && tid == 0 && a.status) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      break;
    }
  }

  // ---- finish: the last workgroup moves the tag base past this launch --------
  __syncthreads();
  if (tid0 == 0) {
    const uint32_t old = atomicAdd(&a.ctl[1], 1u);
    if (old == NWG - 1) {
      eng::release_places(a.ctl, NX);
      __hip_atomic_store(&a.ctl[1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctl[0], base + (uint32_t)a.n_steps, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

using TShapeMoe35b = TShape<2048, 512, 16, 9, 256>;
using TShapeTiny = TShape<512, 256, 8, 16, 16>;

template <class SH>
static hipError_t launch(EngineArgs& a, hipStream_t st) {
  static_assert(SH::LDS_BYTES <= 160 * 1024, "LDS budget");
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)tokens_kernel<SH>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, SH::LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  void* args[] = {&a};
  return hipLaunchCooperativeKernel((const void*)tokens_kernel<SH>, dim3(NWG), dim3(NT), args,
                                    SH::LDS_BYTES, st);
}

template <class SH>
static bool fits(int d, int I, int r, int n_list, int E) {
  return d == SH::D && I == SH::IE && r == SH::R && n_list <= SH::NLX && E <= SH::EX &&
         (n_list * I) % NM == 0 && n_list * I / NM <= I;
}

}  // namespace tok

bool engine_tokens_supported(int d, int I, int r, int K, int S, int E) {
  const int n = K + S;
  if (K < 1 || K > 32 || K > E || n > 32) return false;
  return tok::fits<tok::TShapeMoe35b>(d, I, r, n, E) || tok::fits<tok::TShapeTiny>(d, I, r, n, E);
}

size_t engine_tokens_workspace_words(int E, int d, int I, int r, int n_list, EngineArgs* a) {
  (void)d;
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t o = off;
    off += (n + 31) / 32 * 32;
    return o;
  };
  const size_t rr = (size_t)(r > 0 ? r : 1);
  a->xs_logr = (size_t)(E + 31) / 32 * 32;  // one parity of one XCD
  a->xo_logr = take(tok::NTM * 2 * a->xs_logr);
  a->xo_loghm = take(tok::NTM * 2 * a->xs_logr);
  a->xs_av = (size_t)n_list * 2 * rr;
  a->xo_av = take(tok::NTM * a->xs_av);
  a->xs_hv = (size_t)n_list * I;
  a->xo_hv = take(tok::NTM * a->xs_hv);
  a->xs_adp = (size_t)tok::NM * 2 * rr;
  a->xo_adp = take(tok::NTM * a->xs_adp);
  return off;
}

hipError_t launch_engine_tokens(EngineArgs& a, int d, int I, int r, hipStream_t st) {
  if (d == 2048 && I == 512 && r == 16) return tok::launch<tok::TShapeMoe35b>(a, st);
  if (d == 512 && I == 256 && r == 8) return tok::launch<tok::TShapeTiny>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace moe
