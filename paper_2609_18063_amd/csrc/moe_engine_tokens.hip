// Throughput schedule of independent single-token layer steps for gfx950.
//
// One cooperative launch of 256 workgroups (one per CU). XCD x runs the steps
// s = x, x + 8, x + 16, ... on its own 32 workgroups, so eight steps are in
// flight at once: while one XCD waits on an exchange, a top-k or a slot
// lookup, the other seven stream weights. Each step is still one token
// through one layer, and every weight byte a step reads serves that token
// only. Exchanges never leave the XCD.
//
// Work split of one step on XCD x, member m (workgroup g = x + 8 m):
//   routing  member m computes router and head rows e = m + 32 q (one per
//            wave); the XCD exchanges the logits; every member runs the
//            softmax-top-k (Appendix A) and resolves the K + S bundles
//            through the slot table.
//   gate/up  the K + S experts' intermediate rows lie end to end (n_list I
//            row pairs); member m owns rows [m RP, (m + 1) RP), RP =
//            n_list I / 32, at most two experts (segments). It streams their
//            gate and up rows through registers, plus one of every 32 LoRA-A
//            rows of the step (published first, so that their exchange
//            overlaps the streaming).
//   h        with the LoRA-A products of its segments: h = silu(g) u for its
//            rows (Sec. 3.1 Math contract; unmerged LoRA, Sec. 3.3),
//            published, and its partial A_down h per segment.
//   down     member m owns output rows [m d/32, (m + 1) d/32) over all
//            n_list I columns. Its down rows are loaded before it polls h;
//            it then writes its rows of y = sum_k w_k y_k + y_shared
//            directly, so no partial sums cross workgroups.
//
// Exchange words are {tag, fp32} (moe_xchg.h): the tag is the step's index
// on a device counter that persists across launches. Every exchange area is
// used once per step and is rewritten only after every member has read it
// (each rewrite of step s + 8 depends on an exchange that every member joins
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

constexpr int NX = 8, NM = 32, NWG = NX * NM, NT = 512, NWV = NT / 64;

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
  static constexpr int NB = NGW < 9 ? NGW : 9;                // gate/up instructions in flight
  static constexpr int CH = IE / 32;                          // lanes per down (row, expert) unit
  static constexpr int UPI = 64 / CH;                         // units per wave instruction
  static constexpr int DR = D / NM;                           // down rows per workgroup
  static constexpr int NDW = (NLX * DR / UPI + NWV - 1) / NWV; // most down instructions per wave
  static constexpr int NAX = (NLX * 2 * R + NM - 1) / NM;     // most LoRA-A rows per workgroup
  static constexpr int NPA = (RPX + 15) / 16;                 // rows per lane of an A_down term
  static constexpr int NEF = (NLX + 7) / 8;                   // experts per lane of the output sum
  static constexpr int NH = NLX * IE;                         // h entries of a step (most)
  static constexpr int MAXI_L = (EX + NT - 1) / NT;           // polled logits per thread
  static constexpr int MAXI_H = (NH + NM * 2 * R + NT - 1) / NT;  // polled h + A_down partials
  static constexpr int MAXI_A = (2 * 2 * R + NT - 1) / NT;    // polled LoRA-A products
  static_assert(D % 512 == 0 && IE % 64 == 0 && D % NM == 0, "shape");
  static_assert(RPX <= IE, "a workgroup's rows span at most two experts");
  static_assert(DR % UPI == 0, "a down instruction stays inside one expert");
  static_assert(2 * R * 16 <= NT && R % 8 == 0, "one 16-lane group per A_down term");
  static_assert(DR * 8 <= NT, "eight lanes per output row");
  static_assert(EX <= 256 && (EX + NM - 1) / NM <= NWV, "one router row per wave");
  // LDS layout (bytes)
  static constexpr int O_XH = 0;                          // [D] fp16, natural order
  static constexpr int O_XQ = O_XH + D * 2;               // [D] fp16, pair order
  static constexpr int O_LG = O_XQ + D * 2;               // [EX] router logits
  static constexpr int O_LH = O_LG + EX * 4;              // [EX] head logits
  static constexpr int O_TK = O_LH + EX * 4;              // top-k scratch: 64 words per wave, two waves
  static constexpr int O_BD = O_TK + 2 * 64 * 4;          // [NLX] bundles
  static constexpr int O_GXU = O_BD + NLX * (int)sizeof(moe_bundle);  // [2 RPX] raw g, u
  static constexpr int O_AV = O_GXU + 2 * RPX * 4;        // [2][2R] LoRA-A products of the segments
  static constexpr int O_HL = O_AV + 2 * 2 * R * 4;       // [RPX] own h
  static constexpr int O_HX = O_HL + RPX * 4;             // h of the step, 32-entry chunks at stride 36
  static constexpr int O_ADP = O_HX + NH / 32 * 36 * 4;   // [NM][2][R] A_down partials
  static constexpr int O_ADV = O_ADP + NM * 2 * R * 4;    // [NLX][R] A_down h
  static constexpr int O_YP = O_ADV + NLX * R * 4;        // [DR][NLX] weighted down rows
  static constexpr int O_RED = (O_YP + DR * NLX * 4 + 15) / 16 * 16;  // [NWV] fp64
  static constexpr int O_MISC = O_RED + NWV * 8;          // Misc
  static constexpr int LDS_USED = O_MISC + 2048;
  // More than half of the CU's LDS, so that no two workgroups share a CU.
  static constexpr int LDS_BYTES = LDS_USED > 82 * 1024 ? LDS_USED : 82 * 1024;
};

struct Misc {
  int abort;
  int idx[32];
  float w[32];
  int pidx[32];
  float pw[32];
  int ok[32];      // list position k: resolved to a resident bundle
  float wl[32];    // its combine weight (0 when not resolved)
  float dsc[32];   // wl * lora_scale where its down adapter applies, else 0
  int lg[32];      // gate adapter applies
  int lu[32];      // up adapter applies
  int ld[32];      // down adapter applies
};

struct Ctl {
  uint32_t* ctl;
  uint32_t* status;
};

__device__ __forceinline__ void raise_abort(const Ctl& c) {
  if (c.status) atomicOr(c.status, MOE_STATUS_ENGINE_ABORT);
  __hip_atomic_store(&c.ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Every thread polls items tid + q NT (q < MAXI) of `count` tagged words until
// each carries `tag`, storing the values; two barriers. Items are polled four
// at a time (fewer registers held across the wait). False if a wait ran out
// or another workgroup raised the abort word.
template <int MAXI, typename AddrF, typename StoreF>
__device__ bool poll_all(int tid, int count, uint32_t tag, AddrF addr, StoreF store, const Ctl& c,
                         int* sh_abort) {
  constexpr int G = 4;
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
        raise_abort(c);
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

// The same by one wave: lane l polls items l + 64 q. No barrier; false on a
// time limit or an abort (the caller raises sh_abort for its workgroup).
template <typename AddrF, typename StoreF>
__device__ bool wave_poll(int count, uint32_t tag, AddrF addr, StoreF store, const Ctl& c) {
  const int lane = threadIdx.x & 63;
  long spin = 0;
  for (int i0 = 0; i0 < count; i0 += 64) {
    const int i = i0 + lane;
    bool done = i >= count;
    while (!__all(done)) {
      if (!done) {
        const uint64_t v = ld_tag(addr(i));
        if ((uint32_t)(v >> 32) == tag) {
          store(i, __uint_as_float((uint32_t)v));
          done = true;
        }
      }
      if (__all(done)) break;
      if (++spin > kSpinMax) {
        if (lane == 0) raise_abort(c);
        return false;
      }
      if ((spin & 63) == 0 && ld_u32(&c.ctl[2])) return false;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return true;
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

template <class SH>
__global__ void __launch_bounds__(NT) tokens_kernel(EngineArgs a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int D = SH::D, IE = SH::IE, R = SH::R, NLX = SH::NLX;
  __half* xh = reinterpret_cast<__half*>(smem + SH::O_XH);
  __half* xq = reinterpret_cast<__half*>(smem + SH::O_XQ);
  float* lg = reinterpret_cast<float*>(smem + SH::O_LG);
  float* lh = reinterpret_cast<float*>(smem + SH::O_LH);
  uint32_t* tks = reinterpret_cast<uint32_t*>(smem + SH::O_TK);
  moe_bundle* bund = reinterpret_cast<moe_bundle*>(smem + SH::O_BD);
  float* gxu = reinterpret_cast<float*>(smem + SH::O_GXU);
  float* av = reinterpret_cast<float*>(smem + SH::O_AV);
  float* hl = reinterpret_cast<float*>(smem + SH::O_HL);
  float* hx = reinterpret_cast<float*>(smem + SH::O_HX);
  float* adp = reinterpret_cast<float*>(smem + SH::O_ADP);
  float* adv = reinterpret_cast<float*>(smem + SH::O_ADV);
  float* yp = reinterpret_cast<float*>(smem + SH::O_YP);
  double* red = reinterpret_cast<double*>(smem + SH::O_RED);
  Misc* mi = reinterpret_cast<Misc*>(smem + SH::O_MISC);
  static_assert(sizeof(Misc) <= 2048, "misc block");

  const int g = blockIdx.x;
  const int x = g % NX, m = g / NX;
  const int tid0 = threadIdx.x, tid = tid0;
  const int wave = __builtin_amdgcn_readfirstlane(tid0 >> 6), lane0 = tid0 & 63;
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
  const int ndw = (NDI + NWV - 1) / NWV;     // per wave, contiguous
  const int NA = n_list * 2 * R;             // LoRA-A rows of a step
  const int NHS = n_list * IE;               // h entries of a step

  uint64_t* const LG = a.xw + a.xo_logr + (size_t)x * a.xs_logr;
  uint64_t* const LH = a.xw + a.xo_loghm + (size_t)x * a.xs_logr;
  uint64_t* const AV = a.xw + a.xo_av + (size_t)x * a.xs_av;
  uint64_t* const HV = a.xw + a.xo_hv + (size_t)x * a.xs_hv;
  uint64_t* const ADP = a.xw + a.xo_adp + (size_t)x * a.xs_adp;

  if (tid == 0) {
    mi->abort = 0;
    if ((int)eng::xcc_id() != x) {  // the work split relies on blockIdx % 8 == XCD
      raise_abort(c);
      mi->abort = 1;
    }
    if (ld_u32(&a.ctl[2])) mi->abort = 1;
  }
  const uint32_t base = ld_u32(&a.ctl[0]);
  __syncthreads();

  // ---- a step's inputs, fetched during the previous step of the XCD --------
  // step_layer early, the layer's pointers after the routing, the draws and
  // the router and head rows after the down rows: each load is consumed long
  // after it is issued, so no wait lands in the middle of a step.
  constexpr int XPT = D / NT;
  float xin[XPT];
  U4 rrow[D / 512], hrow[D / 512];
  const int e_row = m + NM * wave;  // this wave's router and head row
  int lay = -1, lay_n = -1;         // the step's layer; the next step's layer
  bool has_head = false;
  const __half *rt_n = nullptr, *hd_n = nullptr;  // the next step's router and head
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
    for (int q = 0; q < XPT; ++q) xin[q] = a.xi[(size_t)s1 * D + tid + q * NT];
    lay = lay_n;
    has_head = layer_ok(lay) && hd_n != nullptr;
    const bool rows = layer_ok(lay) && e_row < E;
    const __half* rsrc = rows ? rt_n + (size_t)e_row * D : reinterpret_cast<const __half*>(a.xi);
    const __half* hsrc = rows && has_head ? hd_n + (size_t)e_row * D : rsrc;
    row_load<D>(rrow, rsrc, lane0);
    row_load<D>(hrow, hsrc, lane0);
  };
  if (x < a.n_steps && !mi->abort) {
    lay_n = a.step_layer[x];
    fetch_layer();
    fetch_rows(x);
  }

  for (int s = x; s < a.n_steps && !mi->abort; s += NX) {
    // The thread's index passes through an empty asm each step, so that the
    // compiler recomputes the addresses derived from it inside the step
    // rather than keeping all of them in registers across the loop.
    int tid = tid0, lane = lane0;
    asm volatile("" : "+v"(tid), "+v"(lane));
    const uint32_t tag = base + (uint32_t)s + 1u;
    if (lay < 0 || lay >= a.n_table_layers) {  // the same for every member of the XCD
      if (m == 0 && tid == 0 && a.status) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      break;
    }
    const int cur_lay = lay;
    const bool cur_head = has_head;
    // the next step of this XCD (the last step fetches its own inputs again)
    const int s_next = s + NX < a.n_steps ? s + NX : s;
    lay_n = a.step_layer[s_next];

    // ---- layer input: x = fp16(rmsnorm(xi)), single rounding from fp64 ----
    {
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
    }
    __syncthreads();

    // ---- routing ------------------------------------------------------------
    if (e_row < E) {
      const float v = row_dot<D>(rrow, xh, lane);
      if (lane == 0) st_tag(LG + e_row, tag, v);
      if (cur_head) {
        const float vh = row_dot<D>(hrow, xh, lane);
        if (lane == 0) st_tag(LH + e_row, tag, vh);
      }
    }
    if (!poll_all<SH::MAXI_L>(tid, E, tag, [&](int i) { return LG + i; }, [&](int i, float v) { lg[i] = v; }, c,
                              &mi->abort))
      break;
    const bool rec_pred = m == 0 && cur_head && (a.pidx_rec || a.pw_rec);
    if (wave == 0) {
      wave_topk<false, 4>(lg, E, K, mi->idx, mi->w, tks);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // resolve list position k (lane k): slot, bundle, adapter flags
      if (lane < n_list) {
        const int k = lane;
        const int e = k < K ? mi->idx[k] : E + (k - K);
        const bool bad = k < K && (e < 0 || e >= E);
        const int slot = bad ? -1 : a.slot_of[(size_t)cur_lay * a.n_ids + e];
        moe_bundle b{};
        if (slot >= 0) b = a.bundles[(size_t)cur_lay * a.n_slots + slot];
        bund[k] = b;
        const bool ok = slot >= 0;
        const float wk = ok ? (k < K ? mi->w[k] : 1.f) : 0.f;
        const bool lora = ok && a.r > 0;
        mi->ok[k] = ok;
        mi->wl[k] = wk;
        mi->lg[k] = lora && b.gate.lora_a && b.gate.lora_b;
        mi->lu[k] = lora && b.up.lora_a && b.up.lora_b;
        mi->ld[k] = lora && b.down.lora_a && b.down.lora_b;
        mi->dsc[k] = mi->ld[k] ? wk * a.lora_scale : 0.f;
        if (m == 0 && a.status) {
          if (bad) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
          else if (slot < 0) atomicOr(a.status, MOE_STATUS_SLOT_MISS);
        }
      }
      if (m == 0 && lane < K) {
        if (a.idx_rec) a.idx_rec[(size_t)s * K + lane] = mi->idx[lane];
        if (a.w_rec) a.w_rec[(size_t)s * K + lane] = mi->w[lane];
      }
    } else if (wave == 1 && rec_pred) {  // the head's prediction, recorded
      if (!wave_poll(E, tag, [&](int i) { return LH + i; }, [&](int i, float v) { lh[i] = v; }, c)) {
        if (lane == 0) mi->abort = 1;
      } else {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        wave_topk<false, 4>(lh, E, K, mi->pidx, mi->pw, tks + 64);
        if (lane < K) {
          if (a.pidx_rec) a.pidx_rec[(size_t)s * K + lane] = mi->pidx[lane];
          if (a.pw_rec) a.pw_rec[(size_t)s * K + lane] = mi->pw[lane];
        }
      }
    }
    fetch_layer();
    __syncthreads();
    if (mi->abort) break;

    // ---- LoRA-A rows of the step: row ar = m + 32 qa of the list's
    // (position, projection, rank) rows, published first ----------------------
    for (int qa = wave; qa < SH::NAX; qa += NWV) {
      const int ar = m + NM * qa;
      if (ar >= NA) break;
      const int k = ar / (2 * R), proj = (ar / R) & 1, kk = ar % R;
      const bool on = proj ? mi->lu[k] : mi->lg[k];
      float v = 0.f;
      if (on) {
        U4 ra[D / 512];
        const __half* A = reinterpret_cast<const __half*>(proj ? bund[k].up.lora_a : bund[k].gate.lora_a);
        row_load<D>(ra, A + (size_t)kk * D, lane);
        v = row_dot<D>(ra, xh, lane);
      }
      if (lane == 0) st_tag(AV + ar, tag, v);
    }

    // ---- gate/up rows (raw int4 matvecs) ------------------------------------
    // Item t < RP is the gate row of local row t, item RP + t its up row.
    // Codes become fp16 pairs q 2^-24 (exact subnormals) under one mask and
    // meet x in its pair order in v_dot2_f32_f16; 2^24 goes into the scale.
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
      for (int b = 0; b < SH::NGW; b += SH::NB) {
        U4 qv[SH::NB][SH::CPL];
        uint32_t szw[SH::NB][SH::CPL];
#pragma unroll
        for (int j = 0; j < SH::NB; ++j) {
          const int n = wave + NWV * (b + j);  // wave-uniform
          const int t = n * SH::RPI + sub;
          bool live = n < NG;
          const uint8_t *pq = nullptr, *ps = nullptr;
          if (live) {
            const bool up = t >= RP;
            const int p = up ? t - RP : t;
            const int k = k0 + (p >= split ? 1 : 0);
            const int er = row0 + p - k * IE;
            live = mi->ok[k];
            const moe_proj& pj = up ? bund[k].up : bund[k].gate;
            pq = reinterpret_cast<const uint8_t*>(pj.q) + (size_t)er * (D / 2);
            ps = reinterpret_cast<const uint8_t*>(pj.sz) + (size_t)er * (D / 16);
          }
#pragma unroll
          for (int cc = 0; cc < SH::CPL; ++cc) {
            const int ch = c0 + SH::LPR * cc;
            if (live) {
              qv[j][cc] = ldw16(pq + ch * 16);
              szw[j][cc] = ldw4(ps + (ch >> 1) * 4);
            } else {
              qv[j][cc] = U4{0u, 0u, 0u, 0u};
              szw[j][cc] = 0u;
            }
          }
        }
#pragma unroll
        for (int j = 0; j < SH::NB; ++j) {
          const int n = wave + NWV * (b + j);
          if (n >= NG) continue;
          float acc = 0.f;
#pragma unroll
          for (int cc = 0; cc < SH::CPL; ++cc) {
            const uint32_t wd[4] = {qv[j][cc].x, qv[j][cc].y, qv[j][cc].z, qv[j][cc].w};
            float d = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma unroll
              for (int mm = 0; mm < 4; ++mm) {
                const uint32_t p = (wd[i] >> (4 * mm)) & 0x000F000Fu;
                d = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, p), xp[cc][4 * i + mm], d, false);
              }
            }
            const float2 sz = h2f2(szw[j][cc]);
            acc += (sz.x * 16777216.f) * d + sz.y * xs[cc];
          }
          acc = group_sum(acc, SH::LPR);
          if (c0 == 0) gxu[n * SH::RPI + sub] = acc;
        }
      }
    }

    // ---- LoRA-A products of the segments -> h of this workgroup's rows ---------
    {
      // LoRA-B rows of gate and up (thread t < RP: local row t)
      constexpr int BV = R / 8;
      U4 bg[BV], bu[BV];
      int kt = k0, ert = 0;
      if (tid < RP) {
        kt = k0 + (tid >= split ? 1 : 0);
        ert = row0 + tid - kt * IE;
#pragma unroll
        for (int v = 0; v < BV; ++v) {
          bg[v] = mi->lg[kt] ? ldw16(reinterpret_cast<const __half*>(bund[kt].gate.lora_b) + (size_t)ert * R + 8 * v)
                             : U4{0u, 0u, 0u, 0u};
          bu[v] = mi->lu[kt] ? ldw16(reinterpret_cast<const __half*>(bund[kt].up.lora_b) + (size_t)ert * R + 8 * v)
                             : U4{0u, 0u, 0u, 0u};
        }
      }
      // A_down at this workgroup's rows: term (q, kk) = tid / 16, rows sub + 16 j
      const int term = tid >> 4, sub = tid & 15;
      const int qd = term / R, kkd = term % R;
      const int kd = k0 + qd;
      const bool dterm = term < 2 * R && qd < nseg && mi->ld[kd];
      const int plo = qd ? split : 0, phi = qd ? RP : split;
      float ad[SH::NPA];
#pragma unroll
      for (int j = 0; j < SH::NPA; ++j) {
        const int p = plo + sub + 16 * j;
        ad[j] = 0.f;
        if (dterm && p < phi)
          ad[j] = __half2float(__ushort_as_half(
              ldg2(reinterpret_cast<const __half*>(bund[kd].down.lora_a) + (size_t)kkd * IE + row0 + p - kd * IE)));
      }
      if (!poll_all<SH::MAXI_A>(tid, nseg * 2 * R, tag, [&](int i) { return AV + (size_t)k0 * 2 * R + i; },
                                [&](int i, float v) { av[i] = v; }, c, &mi->abort))
        break;
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
        if (mi->ok[kt]) {
          const float gg = mi->lg[kt] ? fmaf(a.lora_scale, sg, gxu[tid]) : gxu[tid];
          const float uu = mi->lu[kt] ? fmaf(a.lora_scale, su, gxu[RP + tid]) : gxu[RP + tid];
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

    // ---- down rows of this workgroup over every expert of the step -------------
    {
      // this wave's instructions n = wave ndw + j: list position n / DI, rows
      // (n % DI) UPI + lane / CH, 32-column chunk lane % CH
      const int cl = lane % SH::CH, su = lane / SH::CH;
      U4 dq[SH::NDW];
      uint32_t dsz[SH::NDW];
#pragma unroll
      for (int j = 0; j < SH::NDW; ++j) {
        const int n = wave * ndw + j;
        dq[j] = U4{0u, 0u, 0u, 0u};
        dsz[j] = 0u;
        if (j < ndw && n < NDI) {
          const int k = n / DI, jj = (n % DI) * SH::UPI + su;
          if (mi->ok[k]) {
            const size_t row = (size_t)m * SH::DR + jj;
            dq[j] = ldw16(reinterpret_cast<const uint8_t*>(bund[k].down.q) + row * (IE / 2) + cl * 16);
            dsz[j] = ldw4(reinterpret_cast<const uint8_t*>(bund[k].down.sz) + row * (IE / 16) + (cl >> 1) * 4);
          }
        }
      }
      // LoRA-B rows of down for the output sum: lane (j, part) = (tid / 8, tid % 8)
      constexpr int BV = R / 8;
      const int jo = tid >> 3, part = tid & 7;
      U4 bd[SH::NEF][BV];
#pragma unroll
      for (int i = 0; i < SH::NEF; ++i) {
        const int k = part + 8 * i;
#pragma unroll
        for (int v = 0; v < BV; ++v) {
          bd[i][v] = U4{0u, 0u, 0u, 0u};
          if (jo < SH::DR && k < n_list && mi->ld[k])
            bd[i][v] = ldw16(reinterpret_cast<const __half*>(bund[k].down.lora_b) +
                             ((size_t)m * SH::DR + jo) * R + 8 * v);
        }
      }
      // h of the step and the A_down partials of the XCD
      if (!poll_all<SH::MAXI_H>(
              tid, NHS + NM * 2 * R, tag,
              [&](int i) { return i < NHS ? HV + i : ADP + (i - NHS); },
              [&](int i, float v) {
                if (i < NHS) hx[(i >> 5) * 36 + (i & 31)] = v;
                else adp[i - NHS] = v;
              },
              c, &mi->abort))
        break;
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
      // down dot products: reload the h chunk when the expert changes
      float hc[32], hsum = 0.f;
      int kc = -1;
#pragma unroll
      for (int j = 0; j < SH::NDW; ++j) {
        const int n = wave * ndw + j;
        if (j >= ndw || n >= NDI) continue;
        const int k = n / DI, jj = (n % DI) * SH::UPI + su;
        if (k != kc) {
          kc = k;
          const float4* hp = reinterpret_cast<const float4*>(hx + ((k * IE) / 32 + cl) * 36);
          hsum = 0.f;
#pragma unroll
          for (int e4 = 0; e4 < 8; ++e4) {
            const float4 v4 = hp[e4];
            hc[4 * e4] = v4.x;
            hc[4 * e4 + 1] = v4.y;
            hc[4 * e4 + 2] = v4.z;
            hc[4 * e4 + 3] = v4.w;
            hsum += (v4.x + v4.y) + (v4.z + v4.w);
          }
        }
        const float2 sz = h2f2(dsz[j]);
        float v = sz.x * dot32_q4(dq[j], hc) + sz.y * hsum;
        v = group_sum(v, SH::CH);
        if (cl == 0) yp[jj * NLX + k] = mi->wl[k] * v;
      }
      __syncthreads();
      // the next step's inputs (this XCD's step s + 8) arrive while y is summed
      fetch_rows(s_next);
      // y = sum over list positions of the weighted down rows and LoRA terms
      if (jo < SH::DR) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < SH::NEF; ++i) {
          const int k = part + 8 * i;
          if (k >= n_list) continue;
          acc += yp[jo * NLX + k];
          const float sc = mi->dsc[k];
          if (sc != 0.f) {
            float t = 0.f;
#pragma unroll
            for (int v = 0; v < BV; ++v) {
              const uint32_t wb[4] = {bd[i][v].x, bd[i][v].y, bd[i][v].z, bd[i][v].w};
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
    }
  }

  // ---- finish: the last workgroup moves the tag base past this launch --------
  __syncthreads();
  if (tid == 0) {
    const uint32_t old = atomicAdd(&a.ctl[1], 1u);
    if (old == NWG - 1) {
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
  a->xs_logr = (size_t)(E + 31) / 32 * 32;
  a->xo_logr = take(tok::NX * a->xs_logr);
  a->xo_loghm = take(tok::NX * a->xs_logr);
  a->xs_av = (size_t)n_list * 2 * rr;
  a->xo_av = take(tok::NX * a->xs_av);
  a->xs_hv = (size_t)n_list * I;
  a->xo_hv = take(tok::NX * a->xs_hv);
  a->xs_adp = (size_t)tok::NM * 2 * rr;
  a->xo_adp = take(tok::NX * a->xs_adp);
  return off;
}

hipError_t launch_engine_tokens(EngineArgs& a, int d, int I, int r, hipStream_t st) {
  if (d == 2048 && I == 512 && r == 16) return tok::launch<tok::TShapeMoe35b>(a, st);
  if (d == 512 && I == 256 && r == 8) return tok::launch<tok::TShapeTiny>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace moe
