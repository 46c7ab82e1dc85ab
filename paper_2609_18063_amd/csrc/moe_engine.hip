// Persistent decode engine for gfx950: a sequence of single-token MoE layer
// steps in one cooperative launch (256 workgroups = one per CU, 8 XCDs of 32).
//
// Work split of one step (one token through one layer), per XCD x:
//   The K routed + S shared experts of the token are laid end to end along
//   their intermediate dimension (n_list * I rows). XCD x owns the rows
//   [x*GX, (x+1)*GX), GX = n_list*I/8, as at most three segments of experts.
//   Its 32 workgroups split the segments' gate/up rows and LoRA-A rows,
//   compute h = silu(g)*u for their rows, and then split the d rows of the
//   down projection restricted to the XCD's columns. That is the XCD's
//   weighted partial of the layer output: the down projection and its LoRA
//   term are linear in h, so partials over intermediate rows add up.
//   Reducer workgroups sum the 8 XCD partials for 8 rows each.
//
// Cross-workgroup data travels as 8-byte words {tag, fp32 value}, written
// and polled with agent-scope relaxed atomics. The tag is the step number
// of a device-side counter that persists across launches, so a reader never
// takes a stale value for a fresh one. Every wait is bounded. A timeout sets
// MOE_STATUS_ENGINE_ABORT and a sticky abort word, and every workgroup
// leaves the kernel.
//
// Weights are staged into LDS with direct global->LDS loads
// (global_load_lds_dwordx4) issued by waves 4-7 only; waves 0-3 make every
// other global access. The vector-memory counter of a wave is in order, so
// this split lets a prefetch stay in flight while waves 0-3 poll. Each LDS
// region is refilled for step s+1 as soon as step s has read it: router and
// head rows always (a layer's weights are known ahead), the expert weights
// when step s+1 is routed by a prediction made at the previous token
// (Sec. 3.2, Prediction-as-routing: the next layer's experts are known
// before the current layer finishes), in which case its routing is computed
// during step s as well.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "moe_engine.h"
#include "moe_xchg.h"

namespace moe {
namespace eng {

constexpr int NX = 8, NM = 32, NWG = NX * NM, NT = 512, NWV = NT / 64;
// Waves 0 .. kStageW0-1 make every global access of a step except the weight
// staging (polls, exchange stores, inputs, records); waves kStageW0 .. issue
// the staging loads and nothing that would make them wait for those loads.
constexpr int kStageW0 = 4;
constexpr int NPT = kStageW0 * 64;    // polling threads

struct Ctl {
  uint32_t* ctl;      // [0] tag base, [1] finish counter, [2] abort
  uint32_t* status;
};

// Poll `count` tagged words (addr(i) for i < count) until all carry `tag`;
// store(i, value) each. The polling threads (threadIdx.x < NPT) take items
// threadIdx.x + q*NPT; every thread meets the two barriers. Returns false
// (after the barrier) if any thread timed out or saw the abort word.
template <int MAXI, typename AddrF, typename StoreF>
__device__ bool poll_all(int count, uint32_t tag, AddrF addr, StoreF store, const Ctl& c,
                         int* sh_abort) {
  uint32_t pending = 0;
  if ((int)threadIdx.x < NPT) {
#pragma unroll
    for (int q = 0; q < MAXI; ++q)
      if ((int)threadIdx.x + q * NPT < count) pending |= 1u << q;
  }
  long spin = 0;
  while (pending) {
    uint64_t v[MAXI];
#pragma unroll
    for (int q = 0; q < MAXI; ++q)
      if ((pending >> q) & 1u) v[q] = ld_tag(addr(threadIdx.x + q * NPT));
#pragma unroll
    for (int q = 0; q < MAXI; ++q)
      if (((pending >> q) & 1u) && (uint32_t)(v[q] >> 32) == tag) {
        store(threadIdx.x + q * NPT, __uint_as_float((uint32_t)v[q]));
        pending &= ~(1u << q);
      }
    if (!pending) break;
    if (++spin > kSpinMax) {
      if (c.status) atomicOr(c.status, MOE_STATUS_ENGINE_ABORT);
      __hip_atomic_store(&c.ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *sh_abort = 1;
      break;
    }
    if ((spin & 63) == 0 && ld_u32(&c.ctl[2])) {
      *sh_abort = 1;
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  __syncthreads();
  const bool ok = *sh_abort == 0;
  __syncthreads();
  return ok;
}

// ---------------------------------------------------------------------------
// per-shape constants
// ---------------------------------------------------------------------------
template <int D_, int IE_, int R_, int RMX_, int GXX_, int HRX_, int NSEGX_>
struct Shape {
  static constexpr int D = D_;        // hidden size
  static constexpr int IE = IE_;      // expert intermediate size
  static constexpr int R = R_;        // LoRA rank
  static constexpr int RMX = RMX_;    // max gate/up row pairs per workgroup
  static constexpr int GXX = GXX_;    // max intermediate rows per XCD
  static constexpr int HRX = HRX_;    // max router (and head) rows per workgroup
  static constexpr int NSEGX = NSEGX_;  // max expert segments per XCD
  static constexpr int LPR = D / 32 < 64 ? D / 32 : 64;   // lanes per gate/up row
  static constexpr int CPL = D / 32 / LPR;                 // 16-byte chunks per lane
  static constexpr int RPI = 64 / LPR;                     // gate/up rows per wave instruction
  static constexpr int NAX = (NSEGX * 2 * R + NM - 1) / NM; // max LoRA-A rows per workgroup
  static constexpr int DR = D / NM;   // down rows per workgroup
  static constexpr int RR = D / NWG;  // reducer rows per workgroup
  static constexpr int MAXI_P = (D + NPT - 1) / NPT;  // per polling thread: D items
  static constexpr int MAXI_E = 1;                      // E <= NPT logits
  // LDS layout (bytes); staged regions are rounded up to 1 KiB (one wave copy)
  static constexpr int kb(int b) { return (b + 1023) / 1024 * 1024; }
  static constexpr int O_GUQ = 0;                                   // [2*RMX][D/2]
  static constexpr int O_GUS = O_GUQ + kb(2 * RMX * D / 2);         // [2*RMX][D/16]
  static constexpr int O_AR = O_GUS + kb(2 * RMX * D / 16);         // [NAX][D] fp16
  static constexpr int O_RT = O_AR + kb(NAX * D * 2);               // [HRX][D] router rows
  static constexpr int O_HD = O_RT + kb(HRX * D * 2);               // [HRX][D] head rows
  static constexpr int O_BGU = O_HD + kb(HRX * D * 2);              // [2*RMX][R] fp16
  static constexpr int O_DQ = O_BGU + kb(2 * RMX * R * 2);          // [DR][GXX/2]
  static constexpr int O_DS = O_DQ + kb(DR * GXX / 2);              // [DR][NSEGX][IE/16]
  static constexpr int O_BD = O_DS + kb(DR * NSEGX * IE / 16);      // [DR][NSEGX][R] fp16
  static constexpr int O_ADM = O_BD + kb(DR * NSEGX * R * 2);       // [R][NSEGX][32] fp16
  static constexpr int O_XQ = O_ADM + kb(R * NSEGX * 32 * 2);       // [D] f16, pair order
  static constexpr int O_XH = O_XQ + D * 2;                         // [D] f16
  static constexpr int O_R0 = O_XH + D * 2;                         // [D] f32
  static constexpr int O_R1 = O_R0 + D * 4;                         // [D] f32
  static constexpr int O_LG = O_R1 + D * 4;                         // [1024] f32 logits
  static constexpr int O_HX = O_LG + 1024 * 4;                      // [GXX/32][36] f32 h of the XCD
  static constexpr int O_HL = O_HX + GXX / 32 * 36 * 4;             // [RMX] f32 own h
  static constexpr int O_GXU = O_HL + RMX * 4;                      // [2*RMX] f32
  static constexpr int O_DP = O_GXU + 2 * RMX * 4;                  // [DR][32] f32 down partials
  static constexpr int O_AV = O_DP + DR * 32 * 4;                   // [NSEGX][2R] f32
  static constexpr int O_ADV = O_AV + NSEGX * 2 * R * 4;            // [NSEGX][R] f32
  static constexpr int O_YL = O_ADV + NSEGX * R * 4;                // [RR][NX] f32
  static constexpr int O_RED = (O_YL + RR * NX * 4 + 63) / 64 * 64; // [NT] f64 reduction
  static constexpr int O_MISC = O_RED + NT * 8;                     // small ints / floats
  static constexpr int O_MD = O_MISC + 2048;                        // [D] f16 mixing scales
  static constexpr int O_MP = O_MD + kb(D * 2);                     // [D] i32 mixing permutation
  static constexpr int O_SRC = O_MP + kb(D * 4);                    // [2] Src tables (per parity)
  static constexpr int SRC_BYTES = (2 * RMX * 3 + NAX + GXX / 32) * 8; // one Src table
  static constexpr int LDS_BYTES = O_SRC + kb(2 * SRC_BYTES);
};

struct Seg {
  int k;       // list position (k < K routed, else shared E + k - K)
  int i0;      // first intermediate row of the expert in this segment
  int len;     // rows
  int col0;    // first column of the segment in the XCD's concatenation
};

// The routing of one step and the bundles of the XCD's segments under it.
struct Route {
  int step;              // the step this routing belongs to (-1: none)
  int idx[32];
  float w[32];
  int segok[4];
  float segw[4];
  int lg_gate[4], lg_up[4], lg_down[4];  // the segment's adapter on that projection is applied
  float dsc[4];          // segw * lora_scale where the down adapter is applied, else 0
  moe_bundle segbd[4];   // the segments' bundles, copied from the slot table
  int src_ok;            // the staging source table of this routing is filled
};

// Source addresses of one step's staged weights for this workgroup,
// resolved with the routing, so that the copy loops only add a chunk offset
// (null: the row is not used; its chunks are read from any valid address).
template <class SH>
struct Src {
  const uint8_t* gu[2 * SH::RMX];   // gate (rows < RM) then up codes, one row each
  const uint8_t* gus[2 * SH::RMX];  // their (scale, zero) rows
  const uint8_t* bgu[2 * SH::RMX];  // their LoRA-B rows
  const uint8_t* ar[SH::NAX];       // LoRA-A rows (gate, up) staged by this workgroup
  const uint8_t* dq[SH::GXX / 32];  // down codes at 32-column chunk ch of down row 0
};

struct Misc {
  int nseg;
  int abort;
  int px, pm;            // this workgroup's XCD and member index
  int rt_step, hd_step, mix_step;  // the step whose data each LDS region holds
  int pidx[32];
  float pw[32];
  Seg seg[4];
  Route rt[2];           // by step parity: this step and the next one
};

typedef _Float16 hv2 __attribute__((ext_vector_type(2)));

// LDS index of element i of a vector that lanes read in 32-element chunks
// (lane l reading chunk l): one pad word per chunk puts the 64 lanes' reads of
// the same element in 64 different banks.
// Position of h entry i in LDS: each 32-entry chunk (one down lane's
// columns) starts 36 floats after the previous, so that lanes of different
// chunks read it with 16-byte loads on disjoint banks.
__device__ __forceinline__ int hx_pos(int i) { return (i >> 5) * 36 + (i & 31); }

// Sum of one fp64 value per thread over the workgroup (two barriers).
__device__ double block_sum_f64(double acc, double* red) {
  acc = wave_sum_f64(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  double tot = 0.0;
#pragma unroll
  for (int w = 0; w < NWV; ++w) tot += red[w];
  __syncthreads();
  return tot;
}

// Sum of squares of v[0..D) in fp64 over the workgroup (two barriers).
template <class SH>
__device__ double block_sumsq(const float* v, double* red) {
  static_assert(SH::D % NT == 0, "D is a multiple of the workgroup size");
  double acc = 0.0;
#pragma unroll
  for (int q = 0; q < SH::D / NT; ++q) {
    const double a = v[threadIdx.x + q * NT];
    acc += a * a;
  }
  return block_sum_f64(acc, red);
}

// x = fp16(v * rms(v)^-1) of the D values in vv (this thread's: v[tid + q NT]),
// written to xh (natural order) and xq (pair order).
template <class SH>
__device__ __forceinline__ void rmsnorm_regs_to_x(const float (&vv)[SH::D / NT], double acc,
                                                  __half* xq, __half* xh, double* red) {
  const double inv = rsqrt_f64(block_sum_f64(acc, red) / (double)SH::D + 1e-6);
#pragma unroll
  for (int q = 0; q < SH::D / NT; ++q) {
    const int j = threadIdx.x + q * NT;
    const __half h = f64_to_h((double)vv[q] * inv);
    xh[j] = h;
    xq[pair_pos(j)] = h;
  }
}

template <class SH>
__device__ void block_rmsnorm_to_x(const float* v, __half* xq, __half* xh, double* red) {
  float vv[SH::D / NT];
  double acc = 0.0;
#pragma unroll
  for (int q = 0; q < SH::D / NT; ++q) {
    vv[q] = v[threadIdx.x + q * NT];
    acc += (double)vv[q] * (double)vv[q];
  }
  rmsnorm_regs_to_x<SH>(vv, acc, xq, xh, red);
}

// fp16 row (D halves in LDS) . x (fp16 in LDS) by one wave; fp32 accumulate.
template <class SH>
__device__ __forceinline__ float wave_dot_h(const __half* row, const __half* xh) {
  const int lane = threadIdx.x & 63;
  float acc = 0.f;
#pragma unroll
  for (int q = 0; q < SH::D / 512; ++q) {
    const int c = lane + 64 * q;
    acc = dot8_h(*reinterpret_cast<const U4*>(row + c * 8), *reinterpret_cast<const U4*>(xh + c * 8),
                 acc);
  }
  return wave_sum(acc);
}

// Stage `nchunks` 16-byte chunks into LDS region `dst` (1 KiB-padded);
// src(i) gives chunk i's global address (i < nchunks). Waves w0 .. w0+nw-1
// issue the loads, in 64-chunk blocks round-robin; lanes past the end re-read
// chunk 0 into the padding. The loads stay in flight until those waves call
// dma_wait().
struct Waves {
  int w0, nw;
};
constexpr Waves kAll{0, NWV}, kPollW{0, kStageW0}, kStageW{kStageW0, NWV - kStageW0};
template <typename SrcF>
__device__ __forceinline__ void stage(char* dst, int nchunks, Waves ws, SrcF src) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (wave < ws.w0 || wave >= ws.w0 + ws.nw) return;
  for (int b = wave - ws.w0; b * 64 < nchunks; b += ws.nw) {
    const int i = b * 64 + lane;
    dma16(src(i < nchunks ? i : 0), dst + b * 1024);
  }
}

// Phase timestamps for the profiling hook: thread 0 of workgroups 0, 7 and
// 255 writes the constant-rate wall clock at up to 24 marks of every step (mark 23 by the first thread of wave 4).
constexpr int kProfMarks = 24;
__device__ __forceinline__ void mark(const EngineArgs& a, int g, int s, int k, int tid = 0) {
  if (!a.phase_ts || threadIdx.x != tid) return;
  const int slot = g == 0 ? 0 : (g == 7 ? 1 : (g == NWG - 1 ? 2 : -1));
  if (slot < 0) return;
  a.phase_ts[((size_t)s * 3 + slot) * kProfMarks + k] = wall_clock64();
}

// Where step s runs: token, layer, routing source, head.
struct StepInfo {
  int t, N, lay;
  bool own;   // routed by the layer's own router (else by the previous token's head)
  bool head;  // the layer's head runs (prediction for the next layer)
  bool ok;    // the layer index is valid
};

template <int MODE>
__device__ __forceinline__ StepInfo step_info(const EngineArgs& a, int s) {
  StepInfo f;
  f.t = 0;
  f.N = 0;
  if (MODE == 0) {
    f.lay = a.step_layer[s];
    f.own = true;
  } else {
    f.t = a.first_token + s / a.L;
    f.N = s % a.L;
    f.lay = f.N;
    f.own = f.t == 0 || f.N < a.consumer_lo || f.N > a.consumer_hi;
  }
  f.ok = f.lay >= 0 && f.lay < a.n_table_layers;
  f.head = f.ok && a.layers[f.lay].head != nullptr && (MODE == 0 || f.N + 1 < a.L);
  return f;
}

// MODE 0: independent single-token steps; MODE 1: the decode chain. One
// kernel per mode keeps each loop body small enough for the instruction cache.
template <class SH, int MODE>
__global__ void __launch_bounds__(NT) engine_kernel(EngineArgs a) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  constexpr int D = SH::D, IE = SH::IE, R = SH::R;
  uint8_t* guq = reinterpret_cast<uint8_t*>(smem + SH::O_GUQ);
  uint8_t* gus = reinterpret_cast<uint8_t*>(smem + SH::O_GUS);
  __half* arow = reinterpret_cast<__half*>(smem + SH::O_AR);
  __half* rtrow = reinterpret_cast<__half*>(smem + SH::O_RT);
  __half* hdrow = reinterpret_cast<__half*>(smem + SH::O_HD);
  __half* bgu = reinterpret_cast<__half*>(smem + SH::O_BGU);
  uint8_t* dq = reinterpret_cast<uint8_t*>(smem + SH::O_DQ);
  uint8_t* ds = reinterpret_cast<uint8_t*>(smem + SH::O_DS);
  __half* bd = reinterpret_cast<__half*>(smem + SH::O_BD);
  __half* adm = reinterpret_cast<__half*>(smem + SH::O_ADM);
  __half* xq = reinterpret_cast<__half*>(smem + SH::O_XQ);
  __half* xh = reinterpret_cast<__half*>(smem + SH::O_XH);
  float* r0 = reinterpret_cast<float*>(smem + SH::O_R0);
  float* r1 = reinterpret_cast<float*>(smem + SH::O_R1);
  float* lg = reinterpret_cast<float*>(smem + SH::O_LG);
  float* hx = reinterpret_cast<float*>(smem + SH::O_HX);
  float* gxu = reinterpret_cast<float*>(smem + SH::O_GXU);
  float* hl = reinterpret_cast<float*>(smem + SH::O_HL);
  float* dp = reinterpret_cast<float*>(smem + SH::O_DP);
  float* av = reinterpret_cast<float*>(smem + SH::O_AV);
  float* adv = reinterpret_cast<float*>(smem + SH::O_ADV);
  float* yl = reinterpret_cast<float*>(smem + SH::O_YL);
  double* red = reinterpret_cast<double*>(smem + SH::O_RED);
  Misc* mi = reinterpret_cast<Misc*>(smem + SH::O_MISC);
  static_assert(sizeof(Src<SH>) <= SH::SRC_BYTES, "source table size");
  Src<SH>* const srcs = reinterpret_cast<Src<SH>*>(smem + SH::O_SRC);

  if (threadIdx.x == 0) {
    mi->abort = 0;
    int px = 0, pm = 0;
    if (!claim_place(a.ctl, NX, NM, &px, &pm)) {  // not 32 workgroups per XCD
      if (a.status) atomicOr(a.status, MOE_STATUS_ENGINE_ABORT);
      __hip_atomic_store(&a.ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      mi->abort = 1;
    }
    mi->px = px;
    mi->pm = pm;
  }
  __syncthreads();
  // XCD, member index and the logical workgroup id x + 8 m (uniform)
  const int x = __builtin_amdgcn_readfirstlane(mi->abort ? 0 : mi->px);
  const int m = __builtin_amdgcn_readfirstlane(mi->abort ? 0 : mi->pm);
  const int g = x + NX * m;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const bool poller = (int)threadIdx.x < NPT;
  const Ctl c{a.ctl, a.status};
  const int K = a.K, E = a.E;
  const int n_list = K + a.S;
  const int GX = n_list * IE / NX;    // rows of this XCD
  const int RM = GX / NM;             // gate/up row pairs of this workgroup
  const int LPRD = GX / 32;           // lanes per down row (one 32-column chunk each)
  const int RPID = 64 / LPRD;         // down rows per wave instruction

  if (threadIdx.x == 0) {
    mi->rt_step = mi->hd_step = mi->mix_step = -1;
    mi->rt[0].step = mi->rt[1].step = -1;
    mi->rt[0].src_ok = mi->rt[1].src_ok = 1;
    if (ld_u32(&a.ctl[2])) mi->abort = 1;
  }
  const uint32_t base = ld_u32(&a.ctl[0]);
  __syncthreads();

  // segments of this XCD (fixed for the launch)
  if (threadIdx.x == 0) {
    int row = x * GX, end = (x + 1) * GX, n = 0, col = 0;
    while (row < end && n < SH::NSEGX) {
      const int k = row / IE, i0 = row % IE;
      const int len = min(IE - i0, end - row);
      mi->seg[n] = Seg{k, i0, len, col};
      ++n;
      row += len;
      col += len;
    }
    mi->nseg = n;
  }
  __syncthreads();
  const int nseg = mi->nseg;
  auto row_seg = [&](int lr) {  // XCD-local row -> segment index
    int q = 0;
    while (q + 1 < nseg && lr >= mi->seg[q + 1].col0) ++q;
    return q;
  };
  // the source table that goes with routing Rt (one per step parity)
  auto src_of = [&](const Route& Rt) -> Src<SH>& { return srcs[&Rt == &mi->rt[0] ? 0 : 1]; };
  // Source table entries k = tid, tid + nthr, ... of a resolved routing Rt.
  // (entries part * ... of one kind only when part >= 0: 0 gate/up rows, 1 LoRA-A
  // rows, 2 down column chunks; a wave then runs one branch)
  auto fill_src = [&](const Route& Rt, int tid, int nthr, int part = -1) {
    Src<SH>& S = src_of(Rt);
    const int nrow = 2 * RM, nar = SH::NAX, ncol = GX / 32;
    const int k0 = part <= 0 ? 0 : (part == 1 ? nrow : nrow + nar);
    const int k1 = part < 0 ? nrow + nar + ncol : (part == 0 ? nrow : (part == 1 ? nrow + nar : nrow + nar + ncol));
    for (int k = k0 + tid; k < k1; k += nthr) {
      if (k < nrow) {  // gate / up row k
        const int lr = m * RM + (k < RM ? k : k - RM);
        const int q = row_seg(lr);
        const uint8_t *cq = nullptr, *cs = nullptr, *cb = nullptr;
        if (Rt.segok[q]) {
          const moe_proj& pj = k < RM ? Rt.segbd[q].gate : Rt.segbd[q].up;
          const int er = mi->seg[q].i0 + (lr - mi->seg[q].col0);
          cq = reinterpret_cast<const uint8_t*>(pj.q) + (size_t)er * (D / 2);
          cs = reinterpret_cast<const uint8_t*>(pj.sz) + (size_t)er * (D / 16);
          if (pj.lora_b) cb = reinterpret_cast<const uint8_t*>(pj.lora_b) + (size_t)er * R * 2;
        }
        S.gu[k] = cq;
        S.gus[k] = cs;
        S.bgu[k] = cb;
      } else if (k < nrow + nar) {  // LoRA-A row m + NM * qa of the XCD's list
        const int qa = k - nrow, ar = m + NM * qa;
        const uint8_t* p = nullptr;
        if (ar < nseg * 2 * R) {
          const int q = ar / (2 * R), rr = ar % (2 * R);
          if (Rt.segok[q]) {
            const void* A = rr < R ? Rt.segbd[q].gate.lora_a : Rt.segbd[q].up.lora_a;
            if (A) p = reinterpret_cast<const uint8_t*>(A) + (size_t)(rr % R) * D * 2;
          }
        }
        S.ar[qa] = p;
      } else {  // down codes, column chunk ch
        const int ch = k - nrow - nar, col = ch * 32;
        const int q = row_seg(col);
        const uint8_t* p = nullptr;
        if (Rt.segok[q])
          p = reinterpret_cast<const uint8_t*>(Rt.segbd[q].down.q) +
              (mi->seg[q].i0 + (col - mi->seg[q].col0)) / 2;
        S.dq[ch] = p;
      }
    }
  };

  // ---- staging of a step's weights (issued by the staging waves) ----------
  // gate/up codes, their (scale, zero), the XCD's LoRA-A rows of gate/up
  // (a chunk of an unused row is read from a.xi, any valid address)
  auto stage_gu = [&](const Route& Rt, Waves ws) {
    const Src<SH>& S = src_of(Rt);
    constexpr int QCH = D / 32;   // 16-byte code chunks per gate/up row
    stage(smem + SH::O_GUQ, 2 * RM * QCH, ws, [&](int i) -> const void* {
      const uint8_t* p = S.gu[i / QCH];
      return p ? p + (i % QCH) * 16 : reinterpret_cast<const uint8_t*>(a.xi);
    });
    constexpr int SCH = D / 256;  // 16-byte (scale, zero) chunks per row
    stage(smem + SH::O_GUS, 2 * RM * SCH, ws, [&](int i) -> const void* {
      const uint8_t* p = S.gus[i / SCH];
      return p ? p + (i % SCH) * 16 : reinterpret_cast<const uint8_t*>(a.xi);
    });
    stage(smem + SH::O_AR, SH::NAX * (D / 8), ws, [&](int i) -> const void* {
      const uint8_t* p = S.ar[i / (D / 8)];
      return p ? p + (i % (D / 8)) * 16 : reinterpret_cast<const uint8_t*>(a.xi);
    });
  };
  // LoRA-B of gate/up (read while h is formed), the down rows restricted to
  // the XCD's columns, their (scale, zero), LoRA-B and LoRA-A of down
  auto stage_dn = [&](const Route& Rt, Waves ws) {
    const Src<SH>& S = src_of(Rt);
    constexpr int BCH = R * 2 / 16;
    stage(smem + SH::O_BGU, 2 * RM * BCH, ws, [&](int i) -> const void* {
      const uint8_t* p = S.bgu[i / BCH];
      return p ? p + (i % BCH) * 16 : reinterpret_cast<const uint8_t*>(a.xi);
    });
    // i = jj * dqch + ch: jj = (i * magic) >> 20 is exact while i * dqch < 2^20
    // (magic * dqch - 2^20 <= dqch); here i < DR * dqch and dqch <= 32
    const int dqch = GX / 32;  // 16-byte chunks per staged down row
    const uint32_t magic = (1u << 20) / (uint32_t)dqch + 1u;
    stage(smem + SH::O_DQ, SH::DR * dqch, ws, [&](int i) -> const void* {
      const int jj = (int)(((uint32_t)i * magic) >> 20), ch = i - jj * dqch;
      const uint8_t* p = S.dq[ch];
      return p ? p + (size_t)(m * SH::DR + jj) * (IE / 2) : reinterpret_cast<const uint8_t*>(a.xi);
    });
    constexpr int DSCH = IE / 256;  // 16-byte chunks per (scale, zero) row
    stage(smem + SH::O_DS, SH::DR * SH::NSEGX * DSCH, ws, [&](int i) -> const void* {
      const int jq = i / DSCH, ch = i % DSCH;
      const int jj = jq / SH::NSEGX, q = jq % SH::NSEGX;
      if (q >= nseg || !Rt.segok[q]) return a.xi;
      const moe_bundle* b = &Rt.segbd[q];
      return reinterpret_cast<const uint8_t*>(b->down.sz) + (size_t)(m * SH::DR + jj) * (IE / 16) +
             ch * 16;
    });
    stage(smem + SH::O_BD, SH::DR * SH::NSEGX * BCH, ws, [&](int i) -> const void* {
      const int jq = i / BCH, ch = i % BCH;
      const int jj = jq / SH::NSEGX, q = jq % SH::NSEGX;
      if (q >= nseg || !Rt.segok[q]) return a.xi;
      const void* B = Rt.segbd[q].down.lora_b;
      if (!B) return a.xi;
      return reinterpret_cast<const __half*>(B) + (size_t)(m * SH::DR + jj) * R + ch * 8;
    });
    // LoRA-A of down at this workgroup's rows: [kk][q][4 chunks of 8 halves]
    // covering expert rows [e_lo(q) & ~7, e_hi(q)) of each segment q
    stage(smem + SH::O_ADM, R * SH::NSEGX * 4, ws, [&](int i) -> const void* {
      const int kk = i / (SH::NSEGX * 4), q = (i / 4) % SH::NSEGX, cch = i % 4;
      if (q >= nseg || !Rt.segok[q]) return a.xi;
      const int lo = max(m * RM, mi->seg[q].col0);
      const int hi = min(m * RM + RM, mi->seg[q].col0 + mi->seg[q].len);
      const void* A = Rt.segbd[q].down.lora_a;
      if (!A || lo >= hi) return a.xi;
      const int e0 = (mi->seg[q].i0 + (lo - mi->seg[q].col0)) & ~7;
      int ec = e0 + 8 * cch;
      if (ec > IE - 8) ec = IE - 8;
      return reinterpret_cast<const __half*>(A) + (size_t)kk * IE + ec;
    });
  };
  auto stage_mix = [&](const moe_engine_layer& L, Waves ws) {  // mixing scales and permutation
    const char* md = reinterpret_cast<const char*>(L.mix_d);
    const char* mp = reinterpret_cast<const char*>(L.mix_perm);
    stage(smem + SH::O_MD, D * 2 / 16, ws, [&](int i) { return md + (size_t)i * 16; });
    stage(smem + SH::O_MP, D * 4 / 16, ws, [&](int i) { return mp + (size_t)i * 16; });
  };
  auto stage_rows = [&](int off, const void* W, Waves ws) {  // router or head rows of this workgroup
    const __half* Wh = reinterpret_cast<const __half*>(W);
    stage(smem + off, SH::HRX * (D / 8), ws, [&](int i) {
      const int e = g + NWG * (i / (D / 8));
      return Wh + (size_t)(e < E ? e : 0) * D + (i % (D / 8)) * 8;
    });
  };
  // The slots of the XCD's segments under routing Rt.idx/w (threads < nseg,
  // wave 0); one barrier.
  // Segment q of routing Rt: expert e (routed: id idx[k]; shared: E + k - K)
  // with weight wk, resolved to its slot and bundle.
  // slot_pre >= -1: the slot, looked up earlier (-2: look it up now)
  auto resolve_seg = [&](Route& Rt, int lay, int q, int e, float wk, int slot_pre = -2) {
    const int k = mi->seg[q].k;
    const bool bad = k < K && (e < 0 || e >= E);
    const int slot = bad ? -1 : (slot_pre >= -1 ? slot_pre : a.slot_of[(size_t)lay * a.n_ids + e]);
    Rt.segok[q] = slot >= 0;
    moe_bundle b{};
    if (slot >= 0) b = a.bundles[(size_t)lay * a.n_slots + slot];
    Rt.segbd[q] = b;
    Rt.segw[q] = k < K ? wk : 1.f;
    const bool lora = slot >= 0 && a.r > 0;
    Rt.lg_gate[q] = lora && b.gate.lora_a && b.gate.lora_b;
    Rt.lg_up[q] = lora && b.up.lora_a && b.up.lora_b;
    Rt.lg_down[q] = lora && b.down.lora_a && b.down.lora_b;
    Rt.dsc[q] = Rt.lg_down[q] ? Rt.segw[q] * a.lora_scale : 0.f;
    if (m == 0 && a.status) {
      if (bad) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      else if (slot < 0) atomicOr(a.status, MOE_STATUS_SLOT_MISS);
    }
  };
  auto resolve_route = [&](Route& Rt, int lay, int step) {
    if ((int)threadIdx.x < nseg) {
      const int q = threadIdx.x;
      const int k = mi->seg[q].k;
      resolve_seg(Rt, lay, q, k < K ? Rt.idx[k] : E + (k - K), k < K ? Rt.w[k] : 1.f);
    }
    if (threadIdx.x == 0) {
      Rt.step = step;
      Rt.src_ok = 1;
    }
    __syncthreads();
    fill_src(Rt, threadIdx.x, NT);
    __syncthreads();
  };
  // Softmax-top-k of the logits in lg (wave 0), then resolve_route.
  uint64_t* tk_keys = reinterpret_cast<uint64_t*>(lg + 256);          // [256] after the logits
  int* tk_part = reinterpret_cast<int*>(lg + 768);                    // [256]
  uint64_t* tk_cand = reinterpret_cast<uint64_t*>(red);               // [128]; red is free here
  uint64_t* tk_sorted = tk_cand + 128;                                 // [32]
  auto compute_route = [&](Route& Rt, int lay, int step) {
    block_topk(lg, E, K, Rt.idx, Rt.w, tk_keys, tk_part, tk_cand, tk_sorted);
    __syncthreads();
    mark(a, g, step, 15);
    resolve_route(Rt, lay, step);
  };
  // The published prediction (ids and weights) that routes layer N at token t.
  auto pred_of = [&](int t, int N) {
    return a.xw + a.xo_pred + ((size_t)(t & 1) * a.L + N) * a.xs_pred;
  };
  // Route a consumer step from its published prediction; false on abort.
  auto route_from_pred = [&](Route& Rt, int t, int N, int lay, int step) {
    uint64_t* pw = pred_of(t, N);
    if (!poll_all<1>(2 * K, (uint32_t)t + 1u, [&](int i) { return pw + i; },
                     [&](int i, float v) {
                       if (i < K) Rt.idx[i] = __float_as_int(v);
                       else Rt.w[i - K] = v;
                     },
                     c, &mi->abort))
      return false;
    resolve_route(Rt, lay, step);
    return true;
  };
  // The same by one wave alone (no workgroup barrier): lane u < 2K polls word
  // u of the prediction (ids, then weights), lanes q < nseg resolve segment q.
  // The caller's next barrier hands Rt to the workgroup. On a timeout or an
  // abort it raises the abort flag the next poll_all reports.
  // `have`: lane u's word `pre` was loaded a step earlier (used if its tag is
  // already the expected one, else the word is polled as usual).
  auto route_from_pred_wave = [&](Route& Rt, int t, int N, int lay, int step, bool have,
                                  uint64_t pre, bool have_slot, int pre_slot) {
    const uint64_t* pw = pred_of(t, N);
    uint64_t v = 0;
    bool ok = true;
    if (lane < 2 * K) {
      long spin = 0;
      for (bool first = true;; first = false) {
        v = (first && have) ? pre : ld_tag(pw + lane);
        if ((uint32_t)(v >> 32) == (uint32_t)t + 1u) break;
        if (++spin > kSpinMax) {
          if (c.status) atomicOr(c.status, MOE_STATUS_ENGINE_ABORT);
          __hip_atomic_store(&c.ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ok = false;
          break;
        }
        if ((spin & 63) == 0 && ld_u32(&c.ctl[2])) {
          ok = false;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
    if (__any(!ok)) {
      if (lane == 0) mi->abort = 1;
      return;
    }
    const int word = (int)(uint32_t)v;
    if (lane < K) Rt.idx[lane] = word;
    else if (lane < 2 * K) Rt.w[lane - K] = __int_as_float(word);
    const int kq = lane < nseg ? mi->seg[lane].k : 0;
    const int ek = __shfl(word, kq < K ? kq : 0, kWave);
    const float wk = __int_as_float(__shfl(word, kq < K ? K + kq : 0, kWave));
    // the slots looked up from the same words a step earlier, if the words
    // used are those (their tag was already right then)
    const bool use_slot = have_slot && have && (uint32_t)(pre >> 32) == (uint32_t)t + 1u;
    if (lane < nseg) resolve_seg(Rt, lay, lane, kq < K ? ek : E + (kq - K), wk, use_slot ? pre_slot : -2);
    // the segments written by other lanes of this wave are read next
    // the source table is filled later (src_ok = 0): by this wave while the
    // polling waves wait in S4, else when the step starts staging
    if (lane == 0) {
      Rt.src_ok = 0;
      Rt.step = step;
    }
  };
  // the head logits that route layer N at token t (written at token t - 1)
  auto logh_of = [&](int t, int N) {
    return a.xw + a.xo_logh + ((size_t)(t & 1) * a.L + N) * a.xs_logh_layer;
  };

  uint64_t* const X = a.xw;
  float xi_next[SH::MAXI_P];
  if (MODE == 0 && poller)
#pragma unroll
    for (int q = 0; q < SH::MAXI_P; ++q) {
      const int j = threadIdx.x + q * NPT;
      xi_next[q] = j < D ? a.xi[j] : 0.f;
    }
  // The predicted routing of a step with a head is formed by one workgroup
  // (g == step % NWG) one step later, between publishing its share of the
  // next exchange and polling it, so that the top-k stays off the path every
  // workgroup waits on. Pending: the step (or -1), its head logits and tag.
  int pend_s = -1, pend_t = 0, pend_N = 0;
  const uint64_t* pend_lh = nullptr;
  uint32_t pend_htag = 0;
  auto flush_pred = [&]() -> bool {
    if (pend_s < 0) return true;
    const int ps = pend_s;
    pend_s = -1;
    if (!poll_all<SH::MAXI_E>(E, pend_htag, [&](int i) { return pend_lh + i; },
                              [&](int i, float v) { lg[i] = v; }, c, &mi->abort))
      return false;
    block_topk(lg, E, K, mi->pidx, mi->pw, tk_keys, tk_part, tk_cand, tk_sorted);
    if ((int)threadIdx.x < K) {  // the lanes that wrote pidx / pw
      const int i = threadIdx.x;
      if (MODE == 1) {
        uint64_t* pw = pred_of(pend_t + 1, pend_N + 1);
        st_tag(pw + i, pend_htag, __int_as_float(mi->pidx[i]));
        st_tag(pw + K + i, pend_htag, mi->pw[i]);
      }
      if (a.pidx_rec) a.pidx_rec[(size_t)ps * K + i] = mi->pidx[i];
      if (a.pw_rec) a.pw_rec[(size_t)ps * K + i] = mi->pw[i];
    }
    __syncthreads();
    return true;
  };
  // Wave 4 (chain): the prediction words of step s + 2, loaded during step s so
  // that routing step s + 1 ahead starts from them (pf_step: the step they are for).
  uint64_t pf_word = 0;
  int pf_step = -1;
  // ... and the slots of that step's segments, looked up during step s's S4
  int pf_slot = -1, pf_slot_step = -1;
  for (int s = 0; s < a.n_steps && !mi->abort; ++s) {
    const uint32_t tag = base + (uint32_t)s + 1u;
    const int par = s & 1;
    const StepInfo f = step_info<MODE>(a, s);
    if (!f.ok) {  // uniform across the grid: every workgroup stops
      if (g == 0 && threadIdx.x == 0 && a.status) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      break;
    }
    const int t = f.t, N = f.N, lay = f.lay;
    const bool has_head = f.head;
    const moe_engine_layer LY = a.layers[lay];
    Route& Rt = mi->rt[par];

    mark(a, g, s, 0);
    // ---- S0: layer input (global reads by the polling waves only) --------
    if (MODE == 0) {
      if (poller) {
#pragma unroll
        for (int q = 0; q < SH::MAXI_P; ++q) {
          const int j = threadIdx.x + q * NPT;
          if (j < D) r0[j] = xi_next[q];
        }
        if (s + 1 < a.n_steps) {  // the next step's draws arrive while this step runs
          const float* xn = a.xi + (size_t)(s + 1) * D;
#pragma unroll
          for (int q = 0; q < SH::MAXI_P; ++q) {
            const int j = threadIdx.x + q * NPT;
            xi_next[q] = j < D ? xn[j] : 0.f;
          }
        }
      }
      __syncthreads();
      block_rmsnorm_to_x<SH>(r0, xq, xh, red);
    } else {
      // the layer's mixing data: staged ahead by waves 4-7, else now
      if (wave >= kStageW0) dma_wait();
      if (mi->mix_step != s) {
        stage_mix(LY, kAll);
        dma_wait();
      }
      // a pending prediction; then wave 4 routes the next step where a
      // prediction gives it (published at least a step ago) while waves 0-3
      // poll the residual
      if (!flush_pred()) break;
      mark(a, g, s, 16);
      if (wave == kStageW0 && s + 1 < a.n_steps) {
        const StepInfo f1 = step_info<MODE>(a, s + 1);
        if (f1.ok && !f1.own)
          route_from_pred_wave(mi->rt[par ^ 1], f1.t, f1.N, f1.lay, s + 1, pf_step == s + 1, pf_word,
                               pf_slot_step == s + 1, pf_slot);
        pf_slot_step = -1;
        pf_step = -1;
        if (s + 2 < a.n_steps) {  // published at least a token ago: in flight until the next step
          const StepInfo f2 = step_info<MODE>(a, s + 2);
          if (f2.ok && !f2.own) {
            if (lane < 2 * K) pf_word = ld_tag(pred_of(f2.t, f2.N) + lane);
            pf_step = s + 2;
          }
        }
        mark(a, g, s, 23, kStageW0 * 64);
      }
      if (s == 0) {
        if (poller)
          for (int j = threadIdx.x; j < D; j += NPT) r0[j] = a.r_state[j];
        __syncthreads();
      } else {
        uint64_t* rv = X + a.xo_rv + (size_t)(par ^ 1) * a.xs_rv;
        if (!poll_all<SH::MAXI_P>(D, tag - 1u, [&](int i) { return rv + i; },
                                  [&](int i, float v) { r0[i] = v; }, c, &mi->abort))
          break;
      }
      mark(a, g, s, 17);
      if (N == 0) {  // token start: r = xi + rmsnorm(r)
        const double inv = rsqrt_f64(block_sumsq<SH>(r0, red) / (double)D + 1e-6);
        const float* xi = a.xi + (size_t)(s / a.L) * D;
        if (poller)
          for (int j = threadIdx.x; j < D; j += NPT) r0[j] = (float)((double)xi[j] + (double)r0[j] * inv);
        __syncthreads();
      }
      {  // r1 = r + d * r[perm] (kept in registers too), then x = rmsnorm(r1)
        const __half* md = reinterpret_cast<const __half*>(smem + SH::O_MD);
        const int* mp = reinterpret_cast<const int*>(smem + SH::O_MP);
        float vv[SH::D / NT];
        double acc = 0.0;
#pragma unroll
        for (int q = 0; q < SH::D / NT; ++q) {
          const int j = threadIdx.x + q * NT;
          const int p = mp[j];
          const float v = (p >= 0 && p < D) ? r0[p] : 0.f;
          vv[q] = fmaf(__half2float(md[j]), v, r0[j]);
          r1[j] = vv[q];
          acc += (double)vv[q] * (double)vv[q];
        }
        mark(a, g, s, 18);
        rmsnorm_regs_to_x<SH>(vv, acc, xq, xh, red);
      }
    }
    __syncthreads();
    if (g == 0 && a.x_rec && poller)
      for (int j = threadIdx.x; j < D; j += NPT) a.x_rec[(size_t)s * D + j] = xh[j];
    if (MODE == 1 && g == 1 && a.r_rec && poller)
      for (int j = threadIdx.x; j < D; j += NPT) a.r_rec[(size_t)s * D + j] = r1[j];

    mark(a, g, s, 1);
    // ---- S1: routing ----------------------------------------------------
    if (f.own) {
      uint64_t* lr = X + a.xo_logr + (size_t)par * a.xs_logr;
      if (mi->rt_step != s) stage_rows(SH::O_RT, LY.router, kAll);
      dma_wait();
      __syncthreads();
      for (int q = wave; q < SH::HRX; q += NWV) {
        const int e = g + NWG * q;
        const float v = wave_dot_h<SH>(rtrow + (size_t)q * D, xh);
        if (lane == 0 && e < E) st_tag(lr + e, tag, v);
      }
      if (!flush_pred()) break;
      mark(a, g, s, 12);
      if (!poll_all<SH::MAXI_E>(E, tag, [&](int i) { return lr + i; },
                                [&](int i, float v) { lg[i] = v; }, c, &mi->abort))
        break;
      mark(a, g, s, 10);
      compute_route(Rt, lay, s);
    } else if (Rt.step != s) {  // not routed ahead (first step of a launch)
      if (!route_from_pred(Rt, t, N, lay, s)) break;
    }
    mark(a, g, s, 11);
    if (g == 0 && threadIdx.x < K) {
      if (a.idx_rec) a.idx_rec[(size_t)s * K + threadIdx.x] = Rt.idx[threadIdx.x];
      if (a.w_rec) a.w_rec[(size_t)s * K + threadIdx.x] = Rt.w[threadIdx.x];
    }

    mark(a, g, s, 2);
    // ---- S2: expert weights of this step, then compute ------------------
    // Gate/up rows (and head rows, unless staged ahead) by waves 0-3, needed
    // at once; down rows by waves 4-7, needed from S3 on.
    {
      if (!Rt.src_ok) {  // routed ahead by one wave: this step's source table
        fill_src(Rt, threadIdx.x, NT);
        __syncthreads();
      }
      dma_wait();  // nothing outstanding here: keeps the copy loops free of waits
      stage_gu(Rt, kPollW);
      if (has_head && mi->hd_step != s) stage_rows(SH::O_HD, LY.head, kPollW);
      stage_dn(Rt, kStageW);
      if (wave < kStageW0) dma_wait();
      __syncthreads();
    }

    mark(a, g, s, 3);
    // LoRA-A rows first, so that their exchange overlaps the gate/up rows
    {
      uint64_t* AV = X + a.xo_av + (size_t)par * a.xs_av + (size_t)x * SH::NSEGX * 2 * R;
      for (int qa = wave; qa < SH::NAX; qa += NWV) {
        const int ar = m + NM * qa;
        if (ar >= nseg * 2 * R) continue;
        const int q = ar / (2 * R), rr = ar % (2 * R);
        const bool has = rr < R ? Rt.lg_gate[q] : Rt.lg_up[q];
        const float v = has ? wave_dot_h<SH>(arow + (size_t)qa * D, xh) : 0.f;
        if (lane == 0) st_tag(AV + q * 2 * R + rr, tag, v);
      }
    }
    // head rows -> tagged logits for the next layer at the next token
    if (has_head) {
      uint64_t* lh;
      uint32_t htag;
      if (MODE == 0) {
        lh = X + a.xo_loghm + (size_t)par * a.xs_logr;
        htag = tag;
      } else {
        lh = logh_of(t + 1, N + 1);
        htag = (uint32_t)t + 2u;
      }
      for (int q = (wave + NWV - 2) % NWV; q < SH::HRX; q += NWV) {  // from wave 2 on
        const int e = g + NWG * q;
        const float v = wave_dot_h<SH>(hdrow + (size_t)q * D, xh);
        if (lane == 0 && e < E) st_tag(lh + e, htag, v);
      }
    }
    // gate/up matvecs (raw): rows r of [gate RM | up RM], LPR lanes per row.
    // Codes become fp16 pairs q * 2^-24 (exact subnormals) under one mask and
    // meet x in its pair order in v_dot2_f32_f16; the 2^24 goes into the
    // scale. Rows are dealt from wave 7 down, so the waves that carry the
    // LoRA-A and head rows get fewer of them.
    {
      const int c0 = lane % SH::LPR, sub = lane / SH::LPR;
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
      for (int rg = NWV - 1 - wave; rg * SH::RPI < 2 * RM; rg += NWV) {
        const int rr = rg * SH::RPI + sub;
        const int rrc = rr < 2 * RM ? rr : 0;
        float acc = 0.f;
#pragma unroll
        for (int cc = 0; cc < SH::CPL; ++cc) {
          const int ch = c0 + SH::LPR * cc;
          const U4 qv = *reinterpret_cast<const U4*>(guq + (size_t)rrc * (D / 2) + ch * 16);
          const float2 sz = h2f2(*reinterpret_cast<const uint32_t*>(gus + (size_t)rrc * (D / 16) +
                                                                     (ch >> 1) * 4));
          const uint32_t wd[4] = {qv.x, qv.y, qv.z, qv.w};
          float d = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int mm = 0; mm < 4; ++mm) {
              const uint32_t p = (wd[i] >> (4 * mm)) & 0x000F000Fu;
              d = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, p), xp[cc][4 * i + mm], d, false);
            }
          }
          acc += (sz.x * 16777216.f) * d + sz.y * xs[cc];
        }
        acc = group_sum(acc, SH::LPR);
        if (c0 == 0 && rr < 2 * RM) gxu[rr] = acc;
      }
    }
    __syncthreads();

    mark(a, g, s, 4);
    // ---- ahead: the next step's router / head rows and mixing data --------
    // (expert weights are staged in their own step: staging them here delays
    // the exchanges queued behind the copies)
    if (wave >= kStageW0) dma_wait();  // this step's down weights (read from S3 on)
    if (s + 1 < a.n_steps) {
      const StepInfo f1 = step_info<MODE>(a, s + 1);
      if (f1.ok) {
        const moe_engine_layer L1 = a.layers[f1.lay];
        // every pointer arrives before the first copy is issued (a wait for a
        // later one would also drain the copies issued before it)
        asm volatile("" ::"v"(L1.router), "v"(L1.head), "v"(L1.mix_d), "v"(L1.mix_perm));
        if (f1.own) stage_rows(SH::O_RT, L1.router, kStageW);
        if (f1.head) stage_rows(SH::O_HD, L1.head, kStageW);
        if (MODE == 1) stage_mix(L1, kStageW);
        if (threadIdx.x == 0) {
          if (f1.own) mi->rt_step = s + 1;
          if (f1.head) mi->hd_step = s + 1;
          if (MODE == 1) mi->mix_step = s + 1;
        }
      }
    }

    mark(a, g, s, 13);
    // ---- S3: a-vectors of the XCD -> h of this workgroup's rows ---------
    {
      uint64_t* AV = X + a.xo_av + (size_t)par * a.xs_av + (size_t)x * SH::NSEGX * 2 * R;
      if (!poll_all<(SH::NSEGX * 2 * R + NPT - 1) / NPT>(
              nseg * 2 * R, tag, [&](int i) { return AV + i; }, [&](int i, float v) { av[i] = v; }, c,
              &mi->abort))
        break;
      mark(a, g, s, 19);
      uint64_t* HV = X + a.xo_hv + (size_t)par * a.xs_hv + (size_t)x * SH::GXX;
      // 16 lanes per row: the LoRA-B terms of gate and up, then a DPP sum
      static_assert(SH::RMX * 16 <= NT, "one 16-lane group per gate/up row");
      if ((int)threadIdx.x < RM * 16) {
        const int i = threadIdx.x >> 4, kl = threadIdx.x & 15;
        const int lr = m * RM + i;
        const int q = row_seg(lr);
        const bool ok = Rt.segok[q], lgg = ok && Rt.lg_gate[q], lgu = ok && Rt.lg_up[q];
        float sg = 0.f, su = 0.f;
        for (int kk = kl; kk < R; kk += 16) {
          if (lgg) sg = fmaf(__half2float(bgu[(size_t)i * R + kk]), av[q * 2 * R + kk], sg);
          if (lgu) su = fmaf(__half2float(bgu[(size_t)(RM + i) * R + kk]), av[q * 2 * R + R + kk], su);
        }
        sg = group_sum(sg, 16);
        su = group_sum(su, 16);
        if (kl == 0) {
          float hv = 0.f;
          if (ok) {
            const float gg = lgg ? fmaf(a.lora_scale, sg, gxu[i]) : gxu[i];
            const float uu = lgu ? fmaf(a.lora_scale, su, gxu[RM + i]) : gxu[RM + i];
            hv = silu(gg) * uu;
          }
          st_tag(HV + lr, tag, hv);
          hl[i] = hv;
        }
      }
      __syncthreads();
      mark(a, g, s, 20);
      // partial a_d[q][kk] over this workgroup's rows of segment q -> ADP
      uint64_t* ADP = X + a.xo_adp + (size_t)par * a.xs_adp +
                      ((size_t)x * NM + m) * SH::NSEGX * R;
      // 16 lanes per term (q, kk), rows dealt over the lanes, then a DPP sum
      static_assert(SH::NSEGX * SH::R * 16 <= NT, "one 16-lane group per down-LoRA term");
      {
        const int p = threadIdx.x >> 4, sub = threadIdx.x & 15;
        if (p < SH::NSEGX * R) {  // whole 16-lane groups
          float acc = 0.f;
          if (p < nseg * R) {
            const int q = p / R, kk = p % R;
            const int lo = max(m * RM, mi->seg[q].col0);
            const int hi = min(m * RM + RM, mi->seg[q].col0 + mi->seg[q].len);
            if (Rt.lg_down[q] && lo < hi) {
              const int e0 = (mi->seg[q].i0 + (lo - mi->seg[q].col0)) & ~7;
              for (int lr2 = lo + sub; lr2 < hi; lr2 += 16) {
                const int ec = mi->seg[q].i0 + (lr2 - mi->seg[q].col0);
                acc = fmaf(__half2float(adm[((size_t)kk * SH::NSEGX + q) * 32 + (ec - e0)]),
                           hl[lr2 - m * RM], acc);
              }
            }
          }
          acc = group_sum(acc, 16);
          if (sub == 0 && p < nseg * R) st_tag(ADP + p, tag, acc);
        }
      }
    }

    mark(a, g, s, 5);
    // ---- S4: h of the XCD -> down rows -> tagged partial of the output ---
    {
      uint64_t* HV = X + a.xo_hv + (size_t)par * a.xs_hv + (size_t)x * SH::GXX;
      if (MODE == 1 && wave >= kStageW0 && wave < kStageW0 + 3) {
        // the next step's source table (LDS only) while waves 0-3 poll: one
        // kind of entry per wave; marked filled after the poll's barriers
        Route& Rn = mi->rt[par ^ 1];
        if (Rn.step == s + 1 && !Rn.src_ok)
          fill_src(Rn, lane, kWave, wave - kStageW0);
        if (wave == kStageW0 && pf_step == s + 2) {  // the slots of step s + 2's segments
          const StepInfo f2 = step_info<MODE>(a, s + 2);
          const bool tag_ok = (uint32_t)(pf_word >> 32) == (uint32_t)f2.t + 1u;
          const int kq = lane < nseg ? mi->seg[lane].k : 0;
          const int ek = __shfl((int)(uint32_t)pf_word, kq < K ? kq : 0, kWave);
          const int e = kq < K ? ek : E + (kq - K);
          pf_slot = -1;
          if (lane < nseg && e >= 0 && e < a.n_ids) pf_slot = a.slot_of[(size_t)f2.lay * a.n_ids + e];
          pf_slot_step = __all(lane >= 2 * K || tag_ok) ? s + 2 : -1;
        }
      }
      if (!poll_all<(SH::GXX + NPT - 1) / NPT>(GX, tag, [&](int i) { return HV + i; },
                                              [&](int i, float v) { hx[hx_pos(i)] = v; }, c, &mi->abort))
        break;
      // every wave has passed the poll's barriers: the three parts are written
      if (MODE == 1 && threadIdx.x == 0 && mi->rt[par ^ 1].step == s + 1) mi->rt[par ^ 1].src_ok = 1;
      // a_d[q][kk] = sum of the 32 members' partials
      {
        uint64_t* ADP = X + a.xo_adp + (size_t)par * a.xs_adp + (size_t)x * NM * SH::NSEGX * R;
        const int per = nseg * R;
        if (!poll_all<(NM * SH::NSEGX * R + NPT - 1) / NPT>(
                NM * per, tag,
                [&](int i) { return ADP + (size_t)(i / per) * SH::NSEGX * R + (i % per); },
                [&](int i, float v) { dp[i] = v; }, c, &mi->abort))
          break;
        for (int p = threadIdx.x; p < per; p += NT) {
          float acc = 0.f;
          for (int mm = 0; mm < NM; ++mm) acc += dp[mm * per + p];
          adv[p] = acc;
        }
        __syncthreads();
      }
      mark(a, g, s, 6);
      // down matvec: lane -> 32-column chunk ch (fixed), RPID rows per wave instruction
      const int ch = lane % LPRD, sub = lane / LPRD;
      const bool active = sub < RPID;
      float hv[32], hsum = 0.f, wseg = 0.f;
      int qseg = 0, egrp = 0;
      if (active) {
        qseg = row_seg(ch * 32);
        wseg = Rt.segok[qseg] ? Rt.segw[qseg] : 0.f;
        egrp = (mi->seg[qseg].i0 + (ch * 32 - mi->seg[qseg].col0)) / 64;
        const float4* hp = reinterpret_cast<const float4*>(hx + ch * 36);
#pragma unroll
        for (int e4 = 0; e4 < 8; ++e4) {
          const float4 v4 = hp[e4];
          hv[4 * e4] = v4.x;
          hv[4 * e4 + 1] = v4.y;
          hv[4 * e4 + 2] = v4.z;
          hv[4 * e4 + 3] = v4.w;
          hsum += (v4.x + v4.y) + (v4.z + v4.w);
        }
      }
      mark(a, g, s, 21);
      for (int rg = wave; rg * RPID < SH::DR; rg += NWV) {
        const int jj = rg * RPID + sub;
        if (active && jj < SH::DR) {
          const U4 qv = *reinterpret_cast<const U4*>(dq + (size_t)jj * (GX / 2) + ch * 16);
          // (scale, zero) of the expert group holding XCD-local columns 32*ch ..
          const float2 sz = h2f2(*reinterpret_cast<const uint32_t*>(
              ds + ((size_t)jj * SH::NSEGX + qseg) * (IE / 16) + egrp * 4));
          const float p = wseg * (sz.x * dot32_q4(qv, hv) + sz.y * hsum);
          dp[jj * 32 + ch] = p;
        }
      }
      __syncthreads();
      mark(a, g, s, 22);
      uint64_t* PART = X + a.xo_part + (size_t)par * a.xs_part + (size_t)x * D;
      // 8 threads per row: chunk partials and LoRA-B terms, then a DPP sum
      for (int b0 = 0; b0 < SH::DR * 8; b0 += NT) {
        const int tt = b0 + (int)threadIdx.x;
        const int jj = tt >> 3, part = tt & 7;
        float acc = 0.f;
        if (jj < SH::DR) {
          for (int cc = part; cc < LPRD; cc += 8) acc += dp[jj * 32 + cc];
          for (int term = part; term < nseg * R; term += 8) {
            const int q = term / R, kk = term % R;
            const float sc = Rt.dsc[q];
            if (sc != 0.f)
              acc = fmaf(sc * __half2float(bd[((size_t)jj * SH::NSEGX + q) * R + kk]), adv[q * R + kk],
                         acc);
          }
        }
        acc = group_sum(acc, 8);
        if (part == 0 && jj < SH::DR) st_tag(PART + m * SH::DR + jj, tag, acc);
      }
    }
    __syncthreads();

    mark(a, g, s, 7);

    mark(a, g, s, 14);
    // ---- S5: reduce the 8 XCD partials of this workgroup's rows ---------
    {
      if (has_head && g == s % NWG && (MODE == 1 || a.pidx_rec || a.pw_rec)) {
        pend_s = s;
        pend_t = t;
        pend_N = N;
        if (MODE == 0) {
          pend_lh = X + a.xo_loghm + (size_t)par * a.xs_logr;
          pend_htag = tag;
        } else {
          pend_lh = logh_of(t + 1, N + 1);
          pend_htag = (uint32_t)t + 2u;
        }
      }
      uint64_t* PART = X + a.xo_part + (size_t)par * a.xs_part;
      if (!poll_all<(SH::RR * NX + NPT - 1) / NPT>(
              SH::RR * NX, tag, [&](int i) { return PART + (size_t)(i % NX) * D + g * SH::RR + i / NX; },
              [&](int i, float v) { yl[i] = v; }, c, &mi->abort))
        break;
      mark(a, g, s, 8);
      if ((int)threadIdx.x < SH::RR) {
        const int jr = threadIdx.x, j = g * SH::RR + jr;
        float y = 0.f;
        for (int xx = 0; xx < NX; ++xx) y += yl[jr * NX + xx];
        if (MODE == 0) {
          a.y[(size_t)s * D + j] = y;
        } else {
          const float rn = r1[j] + y;
          st_tag(X + a.xo_rv + (size_t)par * a.xs_rv + j, tag, rn);
          if (a.y) a.y[(size_t)s * D + j] = y;
          if (s + 1 == a.n_steps) a.r_state[j] = rn;
        }
      }
      __syncthreads();
      mark(a, g, s, 9);
    }
  }

  if (!mi->abort) flush_pred();  // the last step's prediction

  // ---- finish: wait for any staging still in flight; the last workgroup
  // moves the tag base past this launch ------------------------------------
  if (wave >= kStageW0) dma_wait();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t old = atomicAdd(&a.ctl[1], 1u);
    if (old == NWG - 1) {
      release_places(a.ctl, NX);
      __hip_atomic_store(&a.ctl[1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctl[0], base + (uint32_t)a.n_steps, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// shapes: (D, I, R, max row pairs per workgroup, max rows per XCD, router rows per workgroup)
using ShapeMoe35b = Shape<2048, 512, 16, 18, 576, 1, 2>;
using ShapeTiny = Shape<512, 256, 8, 2, 64, 1, 1>;

template <class SH, int MODE>
static hipError_t launch_mode(EngineArgs& a, hipStream_t st) {
  static_assert(SH::LDS_BYTES <= 160 * 1024, "engine LDS budget");
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)engine_kernel<SH, MODE>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, SH::LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  void* args[] = {&a};
  return hipLaunchCooperativeKernel((const void*)engine_kernel<SH, MODE>, dim3(NWG), dim3(NT), args,
                                    SH::LDS_BYTES, st);
}

template <class SH>
static hipError_t launch(EngineArgs& a, hipStream_t st) {
  return a.mode == 0 ? launch_mode<SH, 0>(a, st) : launch_mode<SH, 1>(a, st);
}

}  // namespace eng

// number of expert segments of the XCD with the most of them
static int max_segments(int n_list, int I) {
  const int GX = n_list * I / eng::NX;
  int most = 0;
  for (int x = 0; x < eng::NX; ++x) {
    int row = x * GX, end = (x + 1) * GX, n = 0;
    while (row < end) {
      row += std::min(I - row % I, end - row);
      ++n;
    }
    most = std::max(most, n);
  }
  return most;
}

template <class SH>
static bool fits(int GX, int n_list, int I) {
  return GX <= SH::GXX && GX / eng::NM <= SH::RMX && GX / 32 <= 32 &&
         max_segments(n_list, I) <= SH::NSEGX;
}

bool engine_shape_supported(int d, int I, int r, int K, int S, int E) {
  const int n = K + S;
  if (E > 256 || K > 32) return false;
  if ((n * I) % (eng::NX * 64) != 0) return false;
  const int GX = n * I / eng::NX;
  if (GX % eng::NM != 0 || GX % 64 != 0) return false;
  if (d == 2048 && I == 512 && r == 16) return fits<eng::ShapeMoe35b>(GX, n, I);
  if (d == 512 && I == 256 && r == 8) return fits<eng::ShapeTiny>(GX, n, I);
  return false;
}

size_t engine_workspace_words(int E, int d, int L, EngineArgs* a) {
  // offsets in 64-bit words; every area doubled by step parity
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t o = off;
    off += (n + 31) / 32 * 32;
    return o;
  };
  const int GXX = 576, NSEGX = 2, R = 64;
  a->xs_logr = (E + 31) / 32 * 32;
  a->xo_logr = take(2 * (size_t)a->xs_logr);
  a->xo_loghm = take(2 * (size_t)a->xs_logr);
  a->xs_av = (size_t)eng::NX * NSEGX * 2 * R;
  a->xo_av = take(2 * a->xs_av);
  a->xs_hv = (size_t)eng::NX * GXX;
  a->xo_hv = take(2 * a->xs_hv);
  a->xs_adp = (size_t)eng::NX * eng::NM * NSEGX * R;
  a->xo_adp = take(2 * a->xs_adp);
  a->xs_part = (size_t)eng::NX * d;
  a->xo_part = take(2 * a->xs_part);
  a->xs_rv = (size_t)d;
  a->xo_rv = take(2 * a->xs_rv);
  a->xs_logh_layer = (size_t)(E + 31) / 32 * 32;
  a->xo_logh = take(2 * (size_t)(L > 0 ? L : 1) * a->xs_logh_layer);
  a->xs_pred = 64;  // K ids + K weights, K <= 32
  a->xo_pred = take(2 * (size_t)(L > 0 ? L : 1) * a->xs_pred);
  return off;
}

hipError_t launch_engine(EngineArgs& a, int d, int I, int r, hipStream_t st) {
  if (d == 2048 && I == 512 && r == 16) return eng::launch<eng::ShapeMoe35b>(a, st);
  if (d == 512 && I == 256 && r == 8) return eng::launch<eng::ShapeTiny>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace moe
