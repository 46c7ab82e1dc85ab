// Two-half pipelined decode chain for gfx950 (Sec. 3.2, Prediction-as-routing).
//
// One cooperative launch of 256 workgroups (one per CU, 32 per XCD) runs a
// whole decode chain. The chip is split into two halves of four XCDs (even
// and odd XCD ids), 128 workgroups each. Layer step s (token t, layer N) is
// computed by half s & 1, so consecutive layers alternate between the halves.
//
// While one half computes layer N, the other half loads the expert weights
// of its next step (layer N + 1) into registers and LDS. Those experts are
// known before layer N finishes: layer N + 1 at token t routes by the
// prediction that the head of layer N made at token t - 1. Weight streaming
// is therefore off the chain's critical path, and a half never streams while
// it waits on an exchange (polls on a CU whose load queue is full of weight
// copies take several times longer).
//
// Work split of one step on a half (4 XCDs x 32 workgroups):
//   The K routed + S shared experts' intermediate rows lie end to end
//   (n_list I rows); XCD xg of the half owns GX = n_list I / 4 of them (at
//   most NSEGX expert segments). Workgroup m of that XCD holds RM = GX / 32
//   gate/up row pairs in registers.
//   - LoRA-A rows of gate/up: spread over the XCD's workgroups, exchanged in
//     the XCD; then h = silu(g) u of the workgroup's rows, published to the
//     whole half rounded once to fp16 (the precision the down products take
//     it in), two rows per exchange word.
//   - Down: workgroup gw of the half owns the D/128 output rows
//     [gw D/128, (gw+1) D/128) over every expert's columns (codes in
//     registers), so no partial sums cross workgroups. The A_down h dots (one
//     rank row of one expert per wave) are exchanged across the half; each
//     workgroup adds B_down (A_down h) to its own rows and publishes its slice
//     of the residual, which the other half reads to start the next layer.
//
// Exchange words are {tag, 32-bit payload} written and polled with
// agent-scope relaxed atomics; the tag is the step index on a counter that
// persists across launches. Every wait is bounded; a timeout raises
// MOE_STATUS_ENGINE_ABORT and every workgroup leaves.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "moe_engine.h"
#include "moe_xchg.h"

namespace moe {
namespace pipe {

using eng::block_topk;
using eng::claim_place;
using eng::dma16;
using eng::dma4;
using eng::dma_wait;
using eng::f64_to_h;
using eng::kSpinMax;
using eng::ld_tag;
using eng::ld_u32;
using eng::pair_pos;
using eng::release_places;
using eng::rsqrt_f64;
using eng::silu;
using eng::wave_sum_f64;

constexpr int NX = 8, NXG = 4, NM = 32, NWGG = NXG * NM, NWG = NX * NM, NT = 512, NWV = NT / 64;
constexpr int NPT = 256;   // polling threads (waves 0-3)
constexpr int kAheadW = NWV - 1;  // the wave that routes the half's next step ahead

typedef _Float16 hv2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Weight loads through the global address space (addresses come from LDS
// tables, where the compiler cannot tell them from LDS pointers), streamed
// once: non-temporal.
__device__ __forceinline__ U4 ldw16(const void* p) {
  const u32x4 v = __builtin_nontemporal_load((const __attribute__((address_space(1))) u32x4*)(p));
  return U4{v.x, v.y, v.z, v.w};
}
__device__ __forceinline__ uint32_t ldw4(const void* p) {
  return __builtin_nontemporal_load((const __attribute__((address_space(1))) uint32_t*)(p));
}

__device__ __forceinline__ void st_word(uint64_t* p, uint32_t tag, uint32_t payload) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | payload, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct AllWanted {
  __device__ bool operator()(int) const { return true; }
};

// Poll `count` tagged words (addr(i), i < count and want(i)) until all carry
// `tag`, then store(i, payload) each. Polling threads (threadIdx.x < NPT)
// take items threadIdx.x + q NPT; every thread meets the two barriers.
// Returns false (after the barrier) if any thread timed out or saw the abort
// word.
template <int MAXI, typename AddrF, typename StoreF, typename WantF = AllWanted>
__device__ bool poll_all(int count, uint32_t tag, AddrF addr, StoreF store, uint32_t* ctl,
                         uint32_t* status, int* sh_abort, WantF want = WantF()) {
  uint32_t pending = 0;
  if ((int)threadIdx.x < NPT) {
#pragma unroll
    for (int q = 0; q < MAXI; ++q) {
      const int i = (int)threadIdx.x + q * NPT;
      if (i < count && want(i)) pending |= 1u << q;
    }
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
        store(threadIdx.x + q * NPT, (uint32_t)v[q]);
        pending &= ~(1u << q);
      }
    if (!pending) break;
    if (++spin > kSpinMax) {
      if (status) atomicOr(status, MOE_STATUS_ENGINE_ABORT);
      __hip_atomic_store(&ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *sh_abort = 1;
      break;
    }
    if ((spin & 63) == 0 && ld_u32(&ctl[2])) {
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

// D: hidden size, IE: expert intermediate size, R: LoRA rank, NLX: most
// experts per token (K + S), EX: most routed experts, NSEGX: most expert
// segments of one XCD's rows.
template <int D_, int IE_, int R_, int NLX_, int EX_, int NSEGX_>
struct PShape {
  static constexpr int D = D_, IE = IE_, R = R_, NLX = NLX_, EX = EX_, NSEGX = NSEGX_;
  static constexpr int GXX = NLX * IE / NXG;                 // most rows per XCD
  static constexpr int RMX = GXX / NM;                       // most row pairs per workgroup
  static constexpr int LPR = D / 32 < 64 ? D / 32 : 64;      // lanes per gate/up row
  static constexpr int RPI = 64 / LPR;                       // gate/up rows per wave instruction
  static constexpr int CPL = D / 32 / LPR;                   // 16-byte code chunks per lane and row
  static constexpr int NGW = (2 * RMX / RPI + NWV - 1) / NWV;  // gate/up instructions per wave
  static constexpr int GXG = NLX * IE;                       // most rows of a step (h entries)
  static constexpr int NAX = (NSEGX * 2 * R + NM - 1) / NM;  // LoRA-A (gate/up) rows per workgroup
  static constexpr int NAP = (NLX * R + NWGG - 1) / NWGG;    // A_down rank rows per workgroup
  static constexpr int HRX = (EX + NWGG - 1) / NWGG;         // router / head rows per workgroup
  static constexpr int RR = D / NWGG;                        // output rows per workgroup
  // down rows: an instruction covers RPD rows of one expert, CPE lanes (32 columns each) per row
  static constexpr int CPE = IE / 32;
  static constexpr int RPD = 64 / CPE < RR ? 64 / CPE : RR;
  static constexpr int NDW = (NLX * (RR / RPD) + NWV - 1) / NWV;  // down instructions per wave
  static constexpr int MDN = D / NT;                         // residual entries per thread
  static constexpr int MAXI_R = (D + NPT - 1) / NPT;
  static constexpr int MAXI_H = (GXG / 2 + NPT - 1) / NPT;
  static constexpr int MAXI_A = (NSEGX * 2 * R + NPT - 1) / NPT;
  static constexpr int MAXI_E = (EX + NPT - 1) / NPT;
  static constexpr int MAXI_D = (NLX * R + NPT - 1) / NPT;
  static constexpr int TPR = NT / RR < 64 ? NT / RR : 64;    // threads per output row (B_down term)
  static_assert(D % NT == 0 && D % NWGG == 0 && IE % 64 == 0 && IE <= 2048 && CPE <= 64, "shape");
  static_assert(RR % RPD == 0, "whole down instructions");
  static_assert(NAX <= NWV && HRX <= NWV && NAP <= NWV, "rows per wave");
  static_assert(RMX * 8 <= NT, "eight threads per gate/up row pair");
  static_assert(EX <= 256 && HRX <= 2 && NLX <= 10, "routing");
  static_assert(TPR >= 8 && (TPR & (TPR - 1)) == 0 && TPR <= 64, "threads per output row");
  static constexpr int kb(int b) { return (b + 1023) / 1024 * 1024; }
  // LDS layout (bytes); DMA regions padded to whole 1 KiB wave copies
  static constexpr int O_AR = 0;                               // [NAX][D] fp16 LoRA-A rows
  static constexpr int O_RT = O_AR + kb(NAX * D * 2);          // [HRX][D] router rows
  static constexpr int O_HD = O_RT + kb(HRX * D * 2);          // [HRX][D] head rows
  static constexpr int O_BGU = O_HD + kb(HRX * D * 2);         // [2 RMX][R] fp16 LoRA-B (gate, up)
  static constexpr int O_GS = O_BGU + kb(2 * RMX * R * 2);     // [2 RMX][D / 64] (scale, zero) of gate/up
  static constexpr int O_AD = O_GS + kb(2 * RMX * (D / 64) * 4);  // [NAP][IE] fp16 A_down rank rows
  static constexpr int O_BD = O_AD + kb(NAP * IE * 2);         // [RR][NLX][R] fp16 B_down rows
  static constexpr int O_XH = O_BD + kb(RR * NLX * R * 2);     // [D] fp16 x
  static constexpr int O_XQ = O_XH + D * 2;                    // [D] fp16 x, pair order
  static constexpr int O_R = O_XQ + D * 2;                     // [D] fp32 residual in
  static constexpr int O_R1 = O_R + D * 4;                     // [D] fp32 residual after mixing
  static constexpr int O_HX = O_R1 + D * 4;                    // [GXG] fp16 h of the step
  static constexpr int O_HQ = O_HX + GXG * 2;                  // [GXG] fp16 the same h, pair order
  static constexpr int O_HI = O_HQ + GXG * 2;                  // [RMX] int: segment and adapter flags of a row pair
  static constexpr int O_GXU = O_HI + RMX * 4;                 // [2 RMX] fp32 raw gate, up
  static constexpr int O_AV = O_GXU + 2 * RMX * 4;             // [NSEGX][2R] fp32 LoRA-A products
  static constexpr int O_DP = O_AV + NSEGX * 2 * R * 4;        // [NLX][RR] fp32 weighted down rows per expert
  static constexpr int O_YL = O_DP + NLX * RR * 4;             // [NLX][R] fp32 A_down h per expert
  static constexpr int O_LG = O_YL + NLX * R * 4;              // [256] fp32 logits
  static constexpr int O_TK = O_LG + 256 * 4;                  // top-k scratch
  static constexpr int TK_BYTES = 256 * 8 + 256 * 4 + 128 * 8 + 32 * 8;
  static constexpr int O_GR = O_TK + TK_BYTES;                 // [NWV][NGW][64] fp32 gate/up lane partials
  static constexpr int O_RED = O_GR + (LPR == 64 ? NWV * NGW * 64 * 4 : 0);  // [NWV] f64
  static constexpr int O_MISC = (O_RED + NWV * 8 + 1023) / 1024 * 1024;
  static constexpr int MISC_BYTES = 5 * 1024;
  static constexpr int O_SRC = O_MISC + MISC_BYTES;
};

struct Seg {
  int k;     // list position (k < K routed, else shared expert E + k - K)
  int i0;    // first expert row of the segment
  int len;   // rows
  int col0;  // first column of the segment among the XCD's rows
};

// A step's routing, resolved for every list position k (k < K routed, then
// the shared experts). bd is the target of one wave's bundle copies (six
// 16-byte pieces per bundle, 64 lanes): whole 1 KiB.
struct alignas(16) Route {
  char bd[1024];       // moe_bundle [NLX]
  int step;            // the step it belongs to, -1: none
  int idx[32];
  float w[32];
  int slot[16];
  int ok[16];          // resolved to a resident bundle
  float wl[16];        // combine weight (0 when not resolved)
  int lg[16], lu[16], ld[16];  // gate / up / down adapter applies
  float dsc[16];       // wl * lora_scale where the down adapter applies, else 0
  __device__ const moe_bundle& b(int k) const { return reinterpret_cast<const moe_bundle*>(bd)[k]; }
};

struct Misc {
  Route rt[2];       // by (step >> 1) & 1: the step being computed, the next one of the half
  int nseg, abort, px, pm;
  Seg seg[NXG][4];   // segments of the four XCDs of the half
  int nsegx[NXG];
  int pidx[32];
  float pw[32];
};

// Source addresses of one step's weights for this workgroup.
template <class SH>
struct Src {
  const uint8_t* gu[2 * SH::RMX];   // gate (pairs < RM) then up code rows
  const uint8_t* gus[2 * SH::RMX];  // their (scale, zero) rows
  const uint8_t* bgu[2 * SH::RMX];  // their LoRA-B rows
  const uint8_t* ar[SH::NAX];       // LoRA-A rows of gate / up
  const uint8_t* dq[SH::NLX];       // down codes of list position k at the workgroup's first output row
  const uint8_t* dz[SH::NLX];       // their (scale, zero)
  const uint8_t* bd[SH::NLX];       // B_down of list position k at the first output row
  const uint8_t* ad[SH::NAP];       // A_down rank rows of the workgroup's (expert, rank) pairs
};

// LDS offset of the sigmoid-group selection scratch: after the whole layout
// (16-byte aligned)
template <class SH>
__host__ __device__ constexpr int sig_scratch_off() {
  return (SH::O_SRC + (int)sizeof(Src<SH>) + 15) / 16 * 16;
}

// LDS of the full prerouter head (HM instantiations, after the whole layout):
// the workgroup's fc1 rows (x part) and fc2 rows, the step's hidden values,
// its linear-path logits and the layer's routing at the previous token
template <class SH>
struct HmLayout {
  static constexpr int HPWX = kHidMax / NWGG;                   // hidden rows per workgroup
  static constexpr int O_W1 = 0;                                // [HPWX][D] fp16
  static constexpr int O_W2 = O_W1 + HPWX * SH::D * 2;          // [HRX][kHidMax] fp16
  static constexpr int O_HID = O_W2 + SH::HRX * kHidMax * 2;    // [kHidMax] fp32
  static constexpr int O_HL = O_HID + kHidMax * 4;              // [HRX] fp32 (padded)
  static constexpr int O_TM1 = O_HL + 16;                       // [32] int
  static constexpr int BYTES = O_TM1 + 32 * 4;
  static_assert(kHidMax % NWGG == 0 && HPWX <= NWV && (HPWX * (SH::D / 8)) % 64 == 0, "head rows");
};

constexpr int kProfMarks = 24;

struct StepInfo {
  int t, N;
  bool own, head, ok;
};

// SIG: the layers route by sigmoid-group selection (App. A) instead of
// softmax-top-k; a separate instantiation so that the softmax path carries none
// of its code
// HM: the head of every layer is the full prerouter head (fc1 -> erf-GELU ->
// fc2 plus the linear path, Sec. 3.2 Head), its one-hot features the routing
// this layer used at this token and the last; a separate instantiation too
template <class SH, bool SIG, bool HM>
__global__ void __launch_bounds__(NT) pipe_kernel(EngineArgs) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  // The arguments are read through a pointer into the kernel-argument segment
  // that each step launders, so that the compiler reloads them (scalar loads)
  // instead of holding every field in registers across the step loop.
  typedef const __attribute__((address_space(4))) EngineArgs* ArgPtr;
  ArgPtr apx = (ArgPtr)__builtin_amdgcn_kernarg_segment_ptr();
  // the thread index, laundered at each step too (so that per-lane addresses
  // are recomputed in the step rather than kept live across the step loop)
  int tx = (int)threadIdx.x;
  auto sinfo = [&](int s) {
    StepInfo f;
    f.t = apx->first_token + s / apx->L;
    f.N = s % apx->L;
    f.own = f.t == 0 || f.N < apx->consumer_lo || f.N > apx->consumer_hi;
    f.ok = f.N < apx->n_table_layers;
    if constexpr (HM)  // the full head of the layer (its fc1 and fc2 given)
      f.head = f.ok && f.N + 1 < apx->L && apx->heads[f.N].w1_x != nullptr && apx->heads[f.N].w2 != nullptr;
    else
      f.head = f.ok && apx->layers[f.N].head != nullptr && f.N + 1 < apx->L;
    return f;
  };
  constexpr int D = SH::D, IE = SH::IE, R = SH::R;
  __half* arow = reinterpret_cast<__half*>(smem + SH::O_AR);
  __half* rtrow = reinterpret_cast<__half*>(smem + SH::O_RT);
  __half* hdrow = reinterpret_cast<__half*>(smem + SH::O_HD);
  __half* bgu = reinterpret_cast<__half*>(smem + SH::O_BGU);
  const uint32_t* gsm = reinterpret_cast<const uint32_t*>(smem + SH::O_GS);
  __half* adm = reinterpret_cast<__half*>(smem + SH::O_AD);
  __half* bdm = reinterpret_cast<__half*>(smem + SH::O_BD);
  __half* xh = reinterpret_cast<__half*>(smem + SH::O_XH);
  __half* xq = reinterpret_cast<__half*>(smem + SH::O_XQ);
  float* rr0 = reinterpret_cast<float*>(smem + SH::O_R);
  float* rr1 = reinterpret_cast<float*>(smem + SH::O_R1);
  __half* hx = reinterpret_cast<__half*>(smem + SH::O_HX);
  __half* hq = reinterpret_cast<__half*>(smem + SH::O_HQ);
  int* hinfo = reinterpret_cast<int*>(smem + SH::O_HI);
  float* gxu = reinterpret_cast<float*>(smem + SH::O_GXU);
  float* av = reinterpret_cast<float*>(smem + SH::O_AV);
  float* dp = reinterpret_cast<float*>(smem + SH::O_DP);
  float* yl = reinterpret_cast<float*>(smem + SH::O_YL);
  float* lg = reinterpret_cast<float*>(smem + SH::O_LG);
  uint64_t* tk_keys = reinterpret_cast<uint64_t*>(smem + SH::O_TK);
  int* tk_part = reinterpret_cast<int*>(smem + SH::O_TK + 256 * 8);
  uint64_t* tk_cand = reinterpret_cast<uint64_t*>(smem + SH::O_TK + 256 * 12);
  uint64_t* tk_sorted = tk_cand + 128;
  // (sigmoid-group scratch past the end of the softmax layout, in the SIG
  // instantiation only)
  eng::SigmoidScratch& tk_sig = *reinterpret_cast<eng::SigmoidScratch*>(smem + sig_scratch_off<SH>());
  using HL = HmLayout<SH>;
  char* const hmb = smem + sig_scratch_off<SH>();  // (HM instantiations only; never with SIG)
  __half* const hw1 = reinterpret_cast<__half*>(hmb + HL::O_W1);
  __half* const hw2 = reinterpret_cast<__half*>(hmb + HL::O_W2);
  float* const hhid = reinterpret_cast<float*>(hmb + HL::O_HID);
  float* const hlin = reinterpret_cast<float*>(hmb + HL::O_HL);
  int* const htm1 = reinterpret_cast<int*>(hmb + HL::O_TM1);
  static_assert(!(HM && SIG), "the full head runs with softmax-top-k routing");
  double* red = reinterpret_cast<double*>(smem + SH::O_RED);
  float* grp_part = reinterpret_cast<float*>(smem + SH::O_GR);
  Misc* mi = reinterpret_cast<Misc*>(smem + SH::O_MISC);
  static_assert(sizeof(Misc) <= SH::MISC_BYTES, "misc block");
  Src<SH>* const S = reinterpret_cast<Src<SH>*>(smem + SH::O_SRC);

  // ---- place: XCD, half, member --------------------------------------------
  if (tx == 0) {
    mi->abort = 0;
    int px = 0, pm = 0;
    if (!claim_place(apx->ctl, NX, NM, &px, &pm)) {
      if (apx->status) atomicOr(apx->status, MOE_STATUS_ENGINE_ABORT);
      __hip_atomic_store(&apx->ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      mi->abort = 1;
    }
    mi->px = px;
    mi->pm = pm;
    mi->rt[0].step = mi->rt[1].step = -1;
    if (ld_u32(&apx->ctl[2])) mi->abort = 1;
  }
  __syncthreads();
  const int x = __builtin_amdgcn_readfirstlane(mi->abort ? 0 : mi->px);
  const int m = __builtin_amdgcn_readfirstlane(mi->abort ? 0 : mi->pm);
  const int grp = x & 1, xg = x >> 1;
  const int gw = xg + NXG * m;  // workgroup index in the half
  int wave = __builtin_amdgcn_readfirstlane(tx >> 6), lane = tx & 63;
  const int K = apx->K, E = apx->E;
  // the layer's selection on its logits (router or head): softmax-top-k, or
  // sigmoid-group selection where the spec asks for it
  auto select = [&](const float* l, int32_t* idx_out, float* w_out) {
    if constexpr (SIG)
      eng::block_topk_sigmoid_group(l, nullptr, E, K, apx->n_groups, apx->top_groups, apx->route_scale, idx_out, w_out,
                                    tk_sig, tk_keys, tk_part, tk_cand, tk_sorted);
    else
      block_topk(l, E, K, idx_out, w_out, tk_keys, tk_part, tk_cand, tk_sorted);
  };
  const int n_list = K + apx->S;
  const int GX = n_list * IE / NXG;
  const int RM = GX / NM;
  const int NGI = 2 * RM / SH::RPI;   // gate/up instructions of the workgroup
  const int NDI = n_list * (SH::RR / SH::RPD);  // down instructions of the workgroup
  const uint32_t base = ld_u32(&apx->ctl[0]);

  if (tx < NXG) {  // segments of XCD tx of the half
    const int xx = tx;
    int row = xx * GX, end = (xx + 1) * GX, n = 0, col = 0;
    while (row < end && n < SH::NSEGX) {
      const int k = row / IE, i0 = row % IE;
      const int len = min(IE - i0, end - row);
      mi->seg[xx][n] = Seg{k, i0, len, col};
      ++n;
      row += len;
      col += len;
    }
    mi->nsegx[xx] = n;
  }
  __syncthreads();
  const int nseg = __builtin_amdgcn_readfirstlane(mi->nsegx[xg]);
  const Seg* const sg = mi->seg[xg];
  auto row_seg = [&](int lr) {
    int q = 0;
    while (q + 1 < nseg && lr >= sg[q + 1].col0) ++q;
    return q;
  };
  auto mark = [&](int s, int k) {
    if (!apx->phase_ts || tx != 0) return;
    const int slot = gw == 0 ? 0 : (gw == 7 ? 1 : (gw == NWGG - 1 ? 2 : -1));
    if (slot >= 0) apx->phase_ts[((size_t)s * 3 + slot) * kProfMarks + k] = wall_clock64();
  };
  // Before a bulk poll: thread p < 128 spins on one word of producer p (the
  // last word it writes), so that the whole vector is read about once, after
  // every producer has stored. A timeout here falls through to the bulk poll,
  // which reports it.
  auto watch = [&](auto marker, uint32_t tg) {
    if ((int)tx < NWGG) {
      const uint64_t* p = marker((int)tx);
      long spin = 0;
      while ((uint32_t)(ld_tag(p) >> 32) != tg && ++spin < kSpinMax) {
        if ((spin & 63) == 0 && ld_u32(&apx->ctl[2])) break;
        __builtin_amdgcn_s_sleep(1);
      }
    }
    __syncthreads();
  };
  uint64_t* const X = apx->xw;
  auto pred_of = [&](int t, int N) { return X + apx->xo_pred + ((size_t)(t & 1) * apx->L + N) * apx->xs_pred; };
  auto logh_of = [&](int t, int N) {
    return X + apx->xo_logh + ((size_t)(t & 1) * apx->L + N) * apx->xs_logh_layer;
  };

  // ---- routing -> slots -> bundles (one wave; LDS results) -------------------
  // Lanes k < n_list look up their expert's slot (returned); the bundles go
  // to R.bd by direct copies (six 16-byte pieces each), in flight until the
  // wave's next dma_wait.
  auto route_issue = [&](Route& R, int lay) -> int {
    int slot = -1;
    if (lane < n_list) {
      const int k = lane;
      const int e = k < K ? R.idx[k] : E + (k - K);
      const bool bad = k < K && (e < 0 || e >= E);
      if (!bad) slot = apx->slot_of[(size_t)lay * apx->n_ids + e];
    }
    const int q = lane / 6, c = lane % 6;
    const int sq = __shfl(slot, q < n_list ? q : 0, 64);
    const char* src = reinterpret_cast<const char*>(apx->bundles);
    if (lane < 6 * n_list && sq >= 0)
      src = reinterpret_cast<const char*>(apx->bundles + (size_t)lay * apx->n_slots + sq) + 16 * c;
    dma16(src, R.bd);
    return slot;
  };
  // after the wave's dma_wait: flags of list position k = lane
  auto route_finish = [&](Route& R, int slot, int step) {
    if (lane < n_list) {
      const int k = lane;
      const int e = k < K ? R.idx[k] : E + (k - K);
      const bool bad = k < K && (e < 0 || e >= E);
      const bool ok = !bad && slot >= 0;
      const moe_bundle& b = R.b(k);
      R.slot[k] = slot;
      R.ok[k] = ok;
      R.wl[k] = ok ? (k < K ? R.w[k] : 1.f) : 0.f;
      const bool lora = ok && apx->r > 0;
      R.lg[k] = lora && b.gate.lora_a && b.gate.lora_b;
      R.lu[k] = lora && b.up.lora_a && b.up.lora_b;
      R.ld[k] = lora && b.down.lora_a && b.down.lora_b;
      R.dsc[k] = R.ld[k] ? R.wl[k] * apx->lora_scale : 0.f;
      if (gw == 0 && apx->status) {
        if (bad) atomicOr(apx->status, MOE_STATUS_BAD_INDEX);
        else if (slot < 0) atomicOr(apx->status, MOE_STATUS_SLOT_MISS);
      }
    }
    if (lane == 0) R.step = step;
  };
  // whole routing by wave 0 (R.idx / R.w set); one barrier
  auto resolve_route = [&](Route& R, int lay, int step) {
    if (wave == 0) {
      const int slot = route_issue(R, lay);
      dma_wait();
      route_finish(R, slot, step);
    }
    __syncthreads();
  };

  // Source table of routing Rt (every thread; LDS only); the caller's barrier follows.
  const uint8_t* const dummy = reinterpret_cast<const uint8_t*>(apx->xi);
  auto fill_src = [&](const Route& Rt) {
    if (tx < RM) {  // row pair tx: segment (bits 0-7), resolved (8), gate (9) and up (10) adapters
      const int q = row_seg(m * RM + tx), kl = sg[q].k;
      const int ok = Rt.ok[kl] ? 1 : 0;
      hinfo[tx] = q | (ok << 8) | ((ok && Rt.lg[kl]) << 9) | ((ok && Rt.lu[kl]) << 10);
    }
    const int nrow = 2 * RM;
    const int n_all = nrow + SH::NAX + SH::NLX + SH::NAP;
    for (int k = tx; k < n_all; k += NT) {
      if (k < nrow) {
        const int lr = m * RM + (k < RM ? k : k - RM);
        const int q = row_seg(lr), kl = sg[q].k;
        const uint8_t *cq = dummy, *cs = dummy, *cb = dummy;
        if (Rt.ok[kl]) {
          const moe_proj& pj = k < RM ? Rt.b(kl).gate : Rt.b(kl).up;
          const int er = sg[q].i0 + (lr - sg[q].col0);
          cq = reinterpret_cast<const uint8_t*>(pj.q) + (size_t)er * (D / 2);
          cs = reinterpret_cast<const uint8_t*>(pj.sz) + (size_t)er * (D / 16);
          if (pj.lora_b) cb = reinterpret_cast<const uint8_t*>(pj.lora_b) + (size_t)er * R * 2;
        }
        S->gu[k] = cq;
        S->gus[k] = cs;
        S->bgu[k] = cb;
        continue;
      }
      int kk = k - nrow;
      if (kk < SH::NAX) {  // LoRA-A row m + NM kk of the XCD's 2R rows per segment
        const int ar = m + NM * kk;
        const uint8_t* p = dummy;
        if (ar < nseg * 2 * R) {
          const int q = ar / (2 * R), rr = ar % (2 * R), kl = sg[q].k;
          if (Rt.ok[kl]) {
            const void* A = rr < R ? Rt.b(kl).gate.lora_a : Rt.b(kl).up.lora_a;
            if (A) p = reinterpret_cast<const uint8_t*>(A) + (size_t)(rr % R) * D * 2;
          }
        }
        S->ar[kk] = p;
        continue;
      }
      kk -= SH::NAX;
      if (kk < SH::NLX) {  // list position kk: down rows, their scales and B_down at the first output row
        const size_t j0 = (size_t)gw * SH::RR;
        const uint8_t *p = dummy, *pz = dummy, *pb = dummy;
        if (kk < n_list && Rt.ok[kk]) {
          const moe_proj& dn = Rt.b(kk).down;
          p = reinterpret_cast<const uint8_t*>(dn.q) + j0 * (IE / 2);
          pz = reinterpret_cast<const uint8_t*>(dn.sz) + j0 * (IE / 16);
          if (Rt.ld[kk]) pb = reinterpret_cast<const uint8_t*>(dn.lora_b) + j0 * R * 2;
        }
        S->dq[kk] = p;
        S->dz[kk] = pz;
        S->bd[kk] = pb;
        continue;
      }
      kk -= SH::NLX;
      {  // A_down rank row of pair gw + NWGG kk of the step's (expert, rank) pairs
        const int pr = gw + NWGG * kk;
        const uint8_t* p = dummy;
        if (pr < n_list * R) {
          const int k = pr / R, rr = pr % R;
          if (Rt.ok[k] && Rt.ld[k]) p = reinterpret_cast<const uint8_t*>(Rt.b(k).down.lora_a) + (size_t)rr * IE * 2;
        }
        S->ad[kk] = p;
      }
    }
  };

  // ---- weights held in registers between the staging and the step ----------
  U4 gq[SH::NGW][SH::CPL];
  U4 dq[SH::NDW];        // down codes: instruction j of this wave, this lane's row and chunk
  uint32_t dz[SH::NDW];  // their (scale, zero)
  __half mixd[SH::MDN];  // mixing scales
  int mixp[SH::MDN];     // mixing permutation
#pragma unroll
  for (int j = 0; j < SH::NGW; ++j)
#pragma unroll
    for (int cc = 0; cc < SH::CPL; ++cc) gq[j][cc] = U4{0, 0, 0, 0};
#pragma unroll
  for (int j = 0; j < SH::NDW; ++j) {
    dq[j] = U4{0, 0, 0, 0};
    dz[j] = 0;
  }
#pragma unroll
  for (int q = 0; q < SH::MDN; ++q) {
    mixd[q] = __ushort_as_half(0);
    mixp[q] = 0;
  }

  // Expert weights of the routing whose source table is filled: gate/up and
  // down codes into registers, the rest into LDS. Every wave issues its
  // loads; nothing waits here.
  auto stage_experts = [&]() {
#pragma unroll
    for (int j = 0; j < SH::NGW; ++j) {
      const int gi = j * NWV + wave;
      if (gi < NGI) {
        const int row = gi * SH::RPI + lane / SH::LPR;
#pragma unroll
        for (int cc = 0; cc < SH::CPL; ++cc) {
          const int ch = lane % SH::LPR + SH::LPR * cc;
          gq[j][cc] = ldw16(S->gu[row] + ch * 16);
        }
      }
    }
    // down rows: instruction di = j NWV + wave covers rows of expert di / (RR / RPD);
    // lane: row rg RPD + lane / CPE, 32-column chunk lane % CPE
#pragma unroll
    for (int j = 0; j < SH::NDW; ++j) {
      const int di = j * NWV + wave;
      if (di < NDI && lane < SH::RPD * SH::CPE) {
        const int k = di / (SH::RR / SH::RPD), rg = di % (SH::RR / SH::RPD);
        const int row = rg * SH::RPD + lane / SH::CPE, c = lane % SH::CPE;
        dq[j] = ldw16(S->dq[k] + (size_t)row * (IE / 2) + c * 16);
        dz[j] = ldw4(S->dz[k] + (size_t)row * (IE / 16) + (c >> 1) * 4);
      }
    }
    constexpr int GSP = D / 64 * 4 / 16;  // 16-byte pieces of a gate/up (scale, zero) row
    for (int b = wave; b * 64 < 2 * RM * GSP; b += NWV) {  // [2 RM][D / 64] gate/up scales
      const int i = b * 64 + lane, ii = i < 2 * RM * GSP ? i : 0;
      dma16(S->gus[ii / GSP] + (ii % GSP) * 16, const_cast<uint32_t*>(gsm) + b * 256);
    }
    constexpr int BCH = R * 2 / 16;  // 16-byte pieces of a LoRA-B row
    for (int b = wave; b * 64 < 2 * RM * BCH; b += NWV) {  // [2 RM][R] LoRA-B of gate / up
      const int i = b * 64 + lane, ii = i < 2 * RM * BCH ? i : 0;
      dma16(S->bgu[ii / BCH] + (ii % BCH) * 16, bgu + b * 512);
    }
    for (int b = wave; b * 64 < SH::NAX * (D / 8); b += NWV) {  // [NAX][D] LoRA-A rows
      const int i = b * 64 + lane, ii = i < SH::NAX * (D / 8) ? i : 0;
      dma16(S->ar[ii / (D / 8)] + (ii % (D / 8)) * 16, arow + b * 512);
    }
    for (int b = wave; b * 64 < SH::NAP * (IE / 8); b += NWV) {  // [NAP][IE] A_down rank rows
      const int i = b * 64 + lane, ii = i < SH::NAP * (IE / 8) ? i : 0;
      dma16(S->ad[ii / (IE / 8)] + (ii % (IE / 8)) * 16, adm + b * 512);
    }
    {  // [RR][NLX][R] B_down rows of the workgroup's output rows: piece i = (jr NLX + k) BCH + c
      constexpr int nbd = SH::RR * SH::NLX * BCH;
      for (int b = wave; b * 64 < nbd; b += NWV) {
        const int i = b * 64 + lane, ii = i < nbd ? i : 0;
        const int c = ii % BCH, jk = ii / BCH, k = jk % SH::NLX, jr = jk / SH::NLX;
        dma16(S->bd[k] + (size_t)jr * R * 2 + c * 16, bdm + b * 512);
      }
    }
  };
  auto stage_rows = [&](__half* dst, const void* W) {  // router or head rows of this workgroup
    const __half* Wh = reinterpret_cast<const __half*>(W);
    for (int b = wave; b * 64 < SH::HRX * (D / 8); b += NWV) {
      const int i = b * 64 + lane;
      const int ii = i < SH::HRX * (D / 8) ? i : 0;
      const int e = gw + NWGG * (ii / (D / 8));
      dma16(Wh + (size_t)(e < E ? e : 0) * D + (ii % (D / 8)) * 8, dst + b * 512);
    }
  };
  auto stage_layer = [&](int sn) {  // mixing data, router / head rows of step sn
    const StepInfo f = sinfo(sn);
    const __half* md = reinterpret_cast<const __half*>(apx->layers[f.N].mix_d);
    const int* mp = apx->layers[f.N].mix_perm;
#pragma unroll
    for (int q = 0; q < SH::MDN; ++q) {
      const int j = tx + q * NT;
      mixd[q] = md[j];
      mixp[q] = mp[j];
    }
    if (f.own) stage_rows(rtrow, apx->layers[f.N].router);
    if (f.head) {
      if constexpr (HM) {
        const moe_head_mlp* hm = apx->heads + f.N;
        const int H = apx->hidden;
        if (hm->w_l) stage_rows(hdrow, hm->w_l);  // the linear path, as head rows
        // fc1 rows h = gw + NWGG j (x part; row 0 stands in past H, never read)
        const __half* W1 = static_cast<const __half*>(hm->w1_x);
        for (int b = wave; b * 64 < HL::HPWX * (D / 8); b += NWV) {
          const int i = b * 64 + lane, j = i / (D / 8), h = gw + NWGG * j;
          dma16(W1 + (size_t)(h < H ? h : 0) * D + (i % (D / 8)) * 8, hw1 + b * 512);
        }
        // fc2 rows e = gw + NWGG q, padded to kHidMax (the pad is never read)
        const __half* W2 = static_cast<const __half*>(hm->w2);
        for (int b = wave; b * 64 < SH::HRX * (kHidMax / 8); b += NWV) {
          const int i = b * 64 + lane, q = i / (kHidMax / 8), c = i % (kHidMax / 8), e = gw + NWGG * q;
          dma16(W2 + (e < E && c < H / 8 ? (size_t)e * H + c * 8 : 0), hw2 + b * 512);
        }
      } else {
        stage_rows(hdrow, apx->layers[f.N].head);
      }
    }
  };

  // ---- the head's prediction of a step (one workgroup per step) -------------
  auto flush_pred = [&](int s) -> bool {
    const StepInfo f = sinfo(s);
    const uint64_t* lh = logh_of(f.t + 1, f.N + 1);
    const uint32_t htag = (uint32_t)f.t + 2u;
    if (!poll_all<SH::MAXI_E>(E, htag, [&](int i) { return lh + i; },
                              [&](int i, uint32_t v) { lg[i] = __uint_as_float(v); }, apx->ctl, apx->status,
                              &mi->abort))
      return false;
    select(lg, mi->pidx, mi->pw);
    if ((int)tx < K) {
      const int i = tx;
      uint64_t* pw = pred_of(f.t + 1, f.N + 1);
      st_word(pw + i, htag, (uint32_t)mi->pidx[i]);
      st_word(pw + K + i, htag, __float_as_uint(mi->pw[i]));
      if (apx->pidx_rec) apx->pidx_rec[(size_t)s * K + i] = mi->pidx[i];
      if (apx->pw_rec) apx->pw_rec[(size_t)s * K + i] = mi->pw[i];
    }
    __syncthreads();
    return true;
  };
  // Route step s from its published prediction (polled); false on abort.
  auto route_from_pred = [&](Route& Rt, int s) -> bool {
    const StepInfo f = sinfo(s);
    uint64_t* pw = pred_of(f.t, f.N);
    if (!poll_all<1>(2 * K, (uint32_t)f.t + 1u, [&](int i) { return pw + i; },
                     [&](int i, uint32_t v) {
                       if (i < K) Rt.idx[i] = (int)v;
                       else Rt.w[i - K] = __uint_as_float(v);
                     },
                     apx->ctl, apx->status, &mi->abort))
      return false;
    resolve_route(Rt, f.N, s);
    return true;
  };

  // ---- step loop of this half ------------------------------------------------
  bool staged = false;   // the experts of the current step are in registers / LDS
  bool lstaged = false;  // its layer data (mixing, draws, router / head rows)
  for (int s = grp; s < apx->n_steps && !mi->abort; s += 2) {
    asm volatile("" : "+s"(apx));
    asm volatile("" : "+v"(tx));
    wave = __builtin_amdgcn_readfirstlane(tx >> 6);
    lane = tx & 63;
    const uint32_t tag = base + (uint32_t)s + 1u;
    const StepInfo f = sinfo(s);
    if (!f.ok) {
      if (gw == 0 && tx == 0 && apx->status) atomicOr(apx->status, MOE_STATUS_BAD_INDEX);
      break;
    }
    const int t = f.t, N = f.N, lay = f.N;
    Route& Rt = mi->rt[(s >> 1) & 1];
    Route& Rn = mi->rt[((s >> 1) & 1) ^ 1];
    if (!lstaged) {
      stage_layer(s);
      dma_wait();
      __syncthreads();
    }
    mark(s, 0);
    // ---- S0: the residual of the previous step (the other half's output) ----
    if (s == 0) {
      for (int j = tx; j < D; j += NT) rr0[j] = apx->r_state[j];
      __syncthreads();
    } else {
      uint64_t* rv = X + apx->xo_rv + (size_t)((s - 1) & 1) * apx->xs_rv;
      // The half usually arrives here well before the other half's output:
      // it watches one word per producer until all have stored (so that 128
      // workgroups do not poll the whole vector in repeated rounds while the
      // other half is still at work), then polls every word.
      watch([&](int p) { return rv + p * SH::RR + SH::RR - 1; }, tag - 1u);
      if (!poll_all<SH::MAXI_R>(D, tag - 1u, [&](int i) { return rv + i; },
                                [&](int i, uint32_t v) { rr0[i] = __uint_as_float(v); }, apx->ctl, apx->status,
                                &mi->abort))
        break;
    }
    mark(s, 1);
    if (N == 0) {  // token start: r = xi + rmsnorm(r)
      float xin[SH::MDN];
#pragma unroll
      for (int q = 0; q < SH::MDN; ++q) xin[q] = apx->xi[(size_t)(s / apx->L) * D + tx + q * NT];
      double acc = 0.0;
#pragma unroll
      for (int q = 0; q < SH::MDN; ++q) {
        const double v = rr0[tx + q * NT];
        acc += v * v;
      }
      acc = wave_sum_f64(acc);
      if (lane == 0) red[wave] = acc;
      __syncthreads();
      double tot = 0.0;
#pragma unroll
      for (int w = 0; w < NWV; ++w) tot += red[w];
      const double inv = rsqrt_f64(tot / (double)D + 1e-6);
      __syncthreads();
#pragma unroll
      for (int q = 0; q < SH::MDN; ++q) {
        const int j = tx + q * NT;
        rr0[j] = (float)((double)xin[q] + (double)rr0[j] * inv);
      }
      __syncthreads();
    }
    {  // r1 = r + d * r[perm]; x = fp16(rmsnorm(r1))
      float vv[SH::MDN];
      double acc = 0.0;
#pragma unroll
      for (int q = 0; q < SH::MDN; ++q) {
        const int j = tx + q * NT;
        const int p = mixp[q];
        const float v = (p >= 0 && p < D) ? rr0[p] : 0.f;
        vv[q] = fmaf(__half2float(mixd[q]), v, rr0[j]);
        rr1[j] = vv[q];
        acc += (double)vv[q] * (double)vv[q];
      }
      acc = wave_sum_f64(acc);
      if (lane == 0) red[wave] = acc;
      __syncthreads();
      double tot = 0.0;
#pragma unroll
      for (int w = 0; w < NWV; ++w) tot += red[w];
      const double inv = rsqrt_f64(tot / (double)D + 1e-6);
#pragma unroll
      for (int q = 0; q < SH::MDN; ++q) {
        const int j = tx + q * NT;
        const __half h = f64_to_h((double)vv[q] * inv);
        xh[j] = h;
        xq[pair_pos(j)] = h;
      }
    }
    __syncthreads();
    mark(s, 2);
    if (gw == 0 && apx->x_rec)
      for (int j = tx; j < D; j += NT) apx->x_rec[(size_t)s * D + j] = xh[j];
    if (gw == 1 && apx->r_rec)
      for (int j = tx; j < D; j += NT) apx->r_rec[(size_t)s * D + j] = rr1[j];

    // ---- S1: routing (own router, or the prediction when not routed ahead) ----
    if (f.own) {
      uint64_t* lr = X + apx->xo_logr + (size_t)grp * apx->xs_logr;
      for (int q = wave; q < SH::HRX; q += NWV) {
        const int e = gw + NWGG * q;
        float acc = 0.f;
#pragma unroll
        for (int c = 0; c < D / 512; ++c) {
          const int ch = lane + 64 * c;
          acc = dot8_h(*reinterpret_cast<const U4*>(rtrow + (size_t)q * D + ch * 8),
                       *reinterpret_cast<const U4*>(xh + ch * 8), acc);
        }
        acc = wave_sum(acc);
        if (lane == 0 && e < E) st_word(lr + e, tag, __float_as_uint(acc));
      }
      if (!poll_all<SH::MAXI_E>(E, tag, [&](int i) { return lr + i; },
                                [&](int i, uint32_t v) { lg[i] = __uint_as_float(v); }, apx->ctl, apx->status,
                                &mi->abort))
        break;
      select(lg, Rt.idx, Rt.w);
      __syncthreads();
      resolve_route(Rt, lay, s);
      staged = false;
    } else if (!staged && Rt.step != s) {
      if (!route_from_pred(Rt, s)) break;
    }
    if (!staged) {  // experts of this step not loaded ahead: load them now
      fill_src(Rt);
      __syncthreads();
      stage_experts();
      dma_wait();
      __syncthreads();
    }
    if (gw == 0 && (int)tx < K) {
      if (apx->idx_rec) apx->idx_rec[(size_t)s * K + tx] = Rt.idx[tx];
      if (apx->w_rec) apx->w_rec[(size_t)s * K + tx] = Rt.w[tx];
      // the full head of this layer at the next token reads this routing
      if constexpr (HM)
        if (f.head)
          st_word(X + apx->xo_rtm1 + ((size_t)(t & 1) * apx->L + N) * 32 + tx, (uint32_t)t + 1u,
                  (uint32_t)Rt.idx[tx]);
    }
    mark(s, 3);

    // ---- S2: LoRA-A rows of gate/up (published first), head rows ---------------
    uint64_t* AV = X + apx->xo_av + ((size_t)grp * NXG + xg) * apx->xs_av;
    if (wave < SH::NAX) {
      const int ar = m + NM * wave;
      if (ar < nseg * 2 * R) {
        const int q = ar / (2 * R), rr = ar % (2 * R), kl = sg[q].k;
        const bool has = rr < R ? Rt.lg[kl] : Rt.lu[kl];
        float acc = 0.f;
        if (has) {
#pragma unroll
          for (int c = 0; c < D / 512; ++c) {
            const int ch = lane + 64 * c;
            acc = dot8_h(*reinterpret_cast<const U4*>(arow + (size_t)wave * D + ch * 8),
                         *reinterpret_cast<const U4*>(xh + ch * 8), acc);
          }
          acc = wave_sum(acc);
        }
        if (lane == 0) st_word(AV + q * 2 * R + rr, tag, __float_as_uint(acc));
      }
    }
    if (f.head && wave >= NWV - SH::HRX) {  // head rows on the last waves
      const int q = wave - (NWV - SH::HRX);
      const int e = gw + NWGG * q;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < D / 512; ++c) {
        const int ch = lane + 64 * c;
        acc = dot8_h(*reinterpret_cast<const U4*>(hdrow + (size_t)q * D + ch * 8),
                     *reinterpret_cast<const U4*>(xh + ch * 8), acc);
      }
      acc = wave_sum(acc);
      if constexpr (HM) {  // the linear path of the full head, completed after the step
        if (lane == 0) hlin[q] = apx->heads[N].w_l ? acc : 0.f;
      } else {
        if (lane == 0 && e < E) st_word(logh_of(t + 1, N + 1) + e, (uint32_t)t + 2u, __float_as_uint(acc));
      }
    }

    // ---- S3: gate/up rows from registers ---------------------------------------
    // Codes become fp16 pairs (q, q') * 2^-24 (exact subnormals) under one mask;
    // masks 0x000F000F and 0x00F000F0 of a code word and of the word shifted
    // right by 8 give the four pairs of its eight codes, the second and fourth
    // scaled by 16 (their sum is taken apart and scaled back). x is held in the
    // matching pair order.
    {
      const int c0 = lane % SH::LPR;
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
      // every instruction slot is computed (no branch, so that the rows interleave);
      // slots past the workgroup's rows are not written
      float part[SH::NGW];
#pragma unroll
      for (int j = 0; j < SH::NGW; ++j) {
        const int gi = j * NWV + wave;
        const int row = gi * SH::RPI + lane / SH::LPR;
        float acc = 0.f;
#pragma unroll
        for (int cc = 0; cc < SH::CPL; ++cc) {
          const uint32_t wd[4] = {gq[j][cc].x, gq[j][cc].y, gq[j][cc].z, gq[j][cc].w};
          float da = 0.f, db = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t w8 = wd[i] >> 8;
            da = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, wd[i] & 0x000F000Fu), xp[cc][4 * i + 0], da,
                                        false);
            db = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, wd[i] & 0x00F000F0u), xp[cc][4 * i + 1], db,
                                        false);
            da = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w8 & 0x000F000Fu), xp[cc][4 * i + 2], da,
                                        false);
            db = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w8 & 0x00F000F0u), xp[cc][4 * i + 3], db,
                                        false);
          }
          const float d = fmaf(db, 0.0625f, da);
          const float2 sz = h2f2(gsm[(size_t)(row < 2 * RM ? row : 0) * (D / 64) + ((c0 + SH::LPR * cc) >> 1)]);
          acc += (sz.x * 16777216.f) * d + sz.y * xs[cc];
        }
        part[j] = acc;
      }
      if (SH::LPR == 64) {
        // one row per instruction: the lane partials of the wave's rows go
        // through LDS; eight lanes then sum each row's 64 partials (eight
        // each, then three lane swaps)
        float* gp = grp_part + wave * SH::NGW * 64;
#pragma unroll
        for (int j = 0; j < SH::NGW; ++j) gp[j * 64 + lane] = part[j];
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the wave reads its own writes
#pragma unroll
        for (int j0 = 0; j0 < SH::NGW; j0 += 8) {
          const int j = j0 + (lane >> 3), sub = lane & 7;
          float v = 0.f;
          if (j < SH::NGW) {
            const float4* src = reinterpret_cast<const float4*>(gp + j * 64 + sub * 8);
            const float4 p0 = src[0], p1 = src[1];
            v = ((p0.x + p0.y) + (p0.z + p0.w)) + ((p1.x + p1.y) + (p1.z + p1.w));
          }
          v += dpp_f<0xB1>(0.f, v);
          v += dpp_f<0x4E>(0.f, v);
          v += dpp_f<0x141>(0.f, v);
          const int gi = j * NWV + wave;
          if (sub == 0 && j < SH::NGW && gi < NGI) gxu[gi] = v;
        }
      } else {
#pragma unroll
        for (int j = 0; j < SH::NGW; ++j) {
          const int gi = j * NWV + wave;
          const int row = gi * SH::RPI + lane / SH::LPR;
          const float v = group_sum(part[j], SH::LPR);
          if (lane % SH::LPR == 0 && gi < NGI && row < 2 * RM) gxu[row] = v;
        }
      }
    }
    __syncthreads();
    mark(s, 4);

    // Route the half's next step ahead (its prediction was published at least
    // a token ago): the ahead wave loads the prediction words now, the slots
    // after the LoRA-A exchange, the bundles after the h exchange, and resolves
    // the routing after the down rows.
    const int sn = s + 2;
    bool ahead = false;
    if (sn < apx->n_steps) {
      const StepInfo fn = sinfo(sn);
      ahead = fn.ok && !fn.own;
    }
    uint64_t pfw = 0;
    if (ahead && wave == kAheadW && lane < 2 * K) {
      const StepInfo fn = sinfo(sn);
      pfw = ld_tag(pred_of(fn.t, fn.N) + lane);
    }

    // ---- S4: LoRA-A products of the XCD -> h of this workgroup's rows --------
    if (!poll_all<SH::MAXI_A>(nseg * 2 * R, tag, [&](int i) { return AV + i; },
                              [&](int i, uint32_t v) { av[i] = __uint_as_float(v); }, apx->ctl, apx->status,
                              &mi->abort))
      break;
    mark(s, 5);
    uint64_t* HV = X + apx->xo_hv + (size_t)grp * apx->xs_hv;  // h of the step's rows, in pairs
    {
      const int i = tx >> 3, kl8 = tx & 7;
      float hv = 0.f;
      if (i < RM) {
        const int info = hinfo[i];
        const int q = info & 0xff;
        const bool ok = (info >> 8) & 1, lgg = (info >> 9) & 1, lgu = (info >> 10) & 1;
        float sgt = 0.f, sut = 0.f;
#pragma unroll
        for (int kk = kl8; kk < R; kk += 8) {
          sgt = fmaf(__half2float(bgu[(size_t)i * R + kk]), av[q * 2 * R + kk], sgt);
          sut = fmaf(__half2float(bgu[(size_t)(RM + i) * R + kk]), av[q * 2 * R + R + kk], sut);
        }
        sgt = group_sum(sgt, 8);
        sut = group_sum(sut, 8);
        if (ok) {
          const float gg = lgg ? fmaf(apx->lora_scale, sgt, gxu[i]) : gxu[i];
          const float uu = lgu ? fmaf(apx->lora_scale, sut, gxu[RM + i]) : gxu[RM + i];
          hv = silu(gg) * uu;
        }
      }
      // rows 2i' and 2i' + 1 share a word; the odd row's value is 8 lanes up (same 16-lane row)
      const float hn = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(hv), 0x108, 0xf, 0xf, true));
      if (i < RM && kl8 == 0 && (i & 1) == 0) {
        const uint32_t w = (uint32_t)__half_as_ushort(__float2half_rn(hv)) |
                           ((uint32_t)__half_as_ushort(__float2half_rn(hn)) << 16);
        st_word(HV + (xg * GX + m * RM + i) / 2, tag, w);
      }
    }
    mark(s, 13);
    // ahead wave: the next step's routing words and slots
    int pf_slot = -1;
    bool pf_ok = false;
    if (ahead && wave == kAheadW) {
      const StepInfo fn = sinfo(sn);
      pf_ok = __all(lane >= 2 * K || (uint32_t)(pfw >> 32) == (uint32_t)fn.t + 1u);
      if (pf_ok) {
        if (lane < K) Rn.idx[lane] = (int)(uint32_t)pfw;
        else if (lane < 2 * K) Rn.w[lane - K] = __uint_as_float((uint32_t)pfw);
        if (lane < n_list) {
          const int e = lane < K ? (int)(uint32_t)pfw : E + (lane - K);
          const bool bad = lane < K && (e < 0 || e >= E);
          if (!bad) pf_slot = apx->slot_of[(size_t)fn.N * apx->n_ids + e];
        }
      }
    }

    // ---- S5: h of the step (all experts) -> A_down h of this workgroup's pairs ---
    if (!poll_all<SH::MAXI_H>(n_list * IE / 2, tag, [&](int i) { return HV + i; },
                              [&](int i, uint32_t v) {
                                reinterpret_cast<uint32_t*>(hx)[i] = v;
                                reinterpret_cast<uint16_t*>(hq)[pair_pos(2 * i)] = (uint16_t)v;
                                reinterpret_cast<uint16_t*>(hq)[pair_pos(2 * i + 1)] = (uint16_t)(v >> 16);
                              },
                              apx->ctl, apx->status, &mi->abort))
      break;
    mark(s, 6);
    if (pf_ok) {  // ahead wave: the next step's bundles, in flight during the down rows
      const StepInfo fn = sinfo(sn);
      const int q = lane / 6, c = lane % 6;
      const int sq = __shfl(pf_slot, q < n_list ? q : 0, 64);
      const char* src = reinterpret_cast<const char*>(apx->bundles);
      if (lane < 6 * n_list && sq >= 0)
        src = reinterpret_cast<const char*>(apx->bundles + (size_t)fn.N * apx->n_slots + sq) + 16 * c;
      dma16(src, Rn.bd);
    }
    uint64_t* ADX = X + apx->xo_adp + (size_t)grp * apx->xs_adp;  // A_down h, [list position][rank]
    if (wave < SH::NAP) {  // pair gw + NWGG wave: rank row rr of expert k's A_down, dot its h
      const int pr = gw + NWGG * wave;
      if (pr < n_list * R) {
        const int k = pr / R;
        float acc = 0.f;
        if (Rt.ok[k] && Rt.ld[k]) {
          for (int c8 = lane; c8 * 8 < IE; c8 += 64) {
            const U4 a8 = *reinterpret_cast<const U4*>(adm + (size_t)wave * IE + c8 * 8);
            const U4 h8 = *reinterpret_cast<const U4*>(hx + (size_t)k * IE + c8 * 8);
            acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, a8.x), __builtin_bit_cast(hv2, h8.x), acc, false);
            acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, a8.y), __builtin_bit_cast(hv2, h8.y), acc, false);
            acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, a8.z), __builtin_bit_cast(hv2, h8.z), acc, false);
            acc = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, a8.w), __builtin_bit_cast(hv2, h8.w), acc, false);
          }
          acc = wave_sum(acc);
        }
        if (lane == 0) st_word(ADX + pr, tag, __float_as_uint(acc));
      }
    }
    mark(s, 12);

    // ---- S6: this workgroup's output rows over every expert's columns ---------------
    // (codes in registers; the lane's h chunk read in pair order; CPE lanes per row)
    {
      const hv2 one2 = {(_Float16)1.0f, (_Float16)1.0f};
      const int rsub = lane / SH::CPE, c = lane % SH::CPE;
#pragma unroll
      for (int j = 0; j < SH::NDW; ++j) {
        const int di = j * NWV + wave;
        if (di < NDI) {
          const int k = di / (SH::RR / SH::RPD), rg = di % (SH::RR / SH::RPD);
          const float wk = Rt.wl[k];  // uniform
          if (wk != 0.f) {
            const U4* hsrc = reinterpret_cast<const U4*>(hq + (size_t)k * IE + c * 32);
            const uint32_t wd[4] = {dq[j].x, dq[j].y, dq[j].z, dq[j].w};
            float da = 0.f, db = 0.f, hsum = 0.f;
#pragma unroll
            for (int g8 = 0; g8 < 4; ++g8) {
              const U4 hk = hsrc[g8];
              const uint32_t w8 = wd[g8] >> 8;
              da = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, wd[g8] & 0x000F000Fu), __builtin_bit_cast(hv2, hk.x),
                                          da, false);
              db = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, wd[g8] & 0x00F000F0u), __builtin_bit_cast(hv2, hk.y),
                                          db, false);
              da = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w8 & 0x000F000Fu), __builtin_bit_cast(hv2, hk.z), da,
                                          false);
              db = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, w8 & 0x00F000F0u), __builtin_bit_cast(hv2, hk.w), db,
                                          false);
              hsum = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, hk.x), one2, hsum, false);
              hsum = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, hk.y), one2, hsum, false);
              hsum = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, hk.z), one2, hsum, false);
              hsum = __builtin_amdgcn_fdot2(__builtin_bit_cast(hv2, hk.w), one2, hsum, false);
            }
            const float d = fmaf(db, 0.0625f, da);
            const float2 sz = h2f2(dz[j]);
            float v = (sz.x * 16777216.f) * d + sz.y * hsum;
            v = group_sum(v, SH::CPE);
            if (c == 0 && rsub < SH::RPD) dp[k * SH::RR + rg * SH::RPD + rsub] = wk * v;
          } else if (c == 0 && rsub < SH::RPD) {
            dp[k * SH::RR + rg * SH::RPD + rsub] = 0.f;
          }
        }
      }
    }
    mark(s, 7);
    if (pf_ok) {  // ahead wave: the next step's routing, resolved
      dma_wait();
      route_finish(Rn, pf_slot, sn);
    }
    mark(s, 8);

    // ---- S7: A_down h of every expert -> B_down term; rows -> residual ----------
    if (!poll_all<SH::MAXI_D>(n_list * R, tag, [&](int i) { return ADX + i; },
                              [&](int i, uint32_t v) { yl[i] = __uint_as_float(v); }, apx->ctl, apx->status,
                              &mi->abort))
      break;
    mark(s, 14);
    if ((int)tx < SH::RR * SH::TPR) {
      const int jr = tx / SH::TPR, sub = tx % SH::TPR;
      const int j = gw * SH::RR + jr;
      // B_down (A_down h) of every expert with a down adapter, and the experts' rows
      float acc = 0.f;
      for (int term = sub; term < n_list * R; term += SH::TPR) {
        const int k = term / R, rr = term % R;
        acc = fmaf(Rt.dsc[k] * __half2float(bdm[((size_t)jr * SH::NLX + k) * R + rr]), yl[term], acc);
      }
      for (int k = sub; k < n_list; k += SH::TPR) acc += dp[k * SH::RR + jr];
      acc = group_sum(acc, SH::TPR);
      if (sub == 0) {
        const float rn = rr1[j] + acc;
        st_word(X + apx->xo_rv + (size_t)(s & 1) * apx->xs_rv + j, tag, __float_as_uint(rn));
        if (apx->y) apx->y[(size_t)s * D + j] = acc;
        if (s + 1 == apx->n_steps) apx->r_state[j] = rn;
      }
    }
    mark(s, 9);

    // ---- S7b: the full head (HM), after the residual is out ----------------------
    // fc1 rows of this workgroup on x and the one-hot features (the routing of
    // this step and of this layer at the last token), erf-GELU, fp16, published;
    // then every hidden value of the step, fc2 rows plus the linear path and
    // fc2's bias -> the logits of the next layer's prediction.
    if constexpr (HM) {
      if (f.head) {
        const moe_head_mlp* hm = apx->heads + N;
        const int H = apx->hidden;
        if (wave == 0) {
          int e = -1;
          if (lane < K && t > 0) {
            const uint64_t* p = X + apx->xo_rtm1 + ((size_t)((t - 1) & 1) * apx->L + N) * 32 + lane;
            uint64_t v = ld_tag(p);
            long spin = 0;
            while ((uint32_t)(v >> 32) != (uint32_t)t && ++spin < kSpinMax) {
              if ((spin & 63) == 0 && ld_u32(&apx->ctl[2])) break;
              __builtin_amdgcn_s_sleep(1);
              v = ld_tag(p);
            }
            if ((uint32_t)(v >> 32) == (uint32_t)t) {
              e = (int)(uint32_t)v;
            } else {  // timed out or aborted: leave (reported like every wait)
              if (apx->status && spin >= kSpinMax) atomicOr(apx->status, MOE_STATUS_ENGINE_ABORT);
              __hip_atomic_store(&apx->ctl[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              mi->abort = 1;
            }
          }
          if (lane < 32) htm1[lane] = e;
        }
        __syncthreads();
        if (mi->abort) break;
        uint64_t* const HID = X + apx->xo_hid + ((size_t)(s & 1) * 4 + ((s >> 1) & 3)) * kHidMax;
        if (wave < HL::HPWX) {
          const int h = gw + NWGG * wave;
          if (h < H) {
            float acc = 0.f;
#pragma unroll
            for (int c = 0; c < D / 512; ++c) {
              const int ch = lane + 64 * c;
              acc = dot8_h(*reinterpret_cast<const U4*>(hw1 + (size_t)wave * D + ch * 8),
                           *reinterpret_cast<const U4*>(xh + ch * 8), acc);
            }
            if (lane < 2 * K) {  // one-hot features: columns d + e (this step) and d + E + e (last token)
              const int e = lane < K ? Rt.idx[lane] : htm1[lane - K];
              if (e >= 0 && e < E)
                acc += __half2float(static_cast<const __half*>(hm->w1_r)[(size_t)(lane < K ? e : E + e) * H + h]);
            }
            acc = wave_sum(acc);
            if (hm->b1) acc += __half2float(static_cast<const __half*>(hm->b1)[h]);
            const float g = 0.5f * acc * (1.f + erff(acc * 0.70710678118654752f));
            if (lane == 0) st_word(HID + h, tag, __float_as_uint(__half2float(__float2half(g))));
          }
        }
        if (!poll_all<kHidMax / NPT>(H, tag, [&](int i) { return HID + i; },
                                     [&](int i, uint32_t v) { hhid[i] = __uint_as_float(v); }, apx->ctl, apx->status,
                                     &mi->abort))
          break;
        if (wave < SH::HRX) {
          const int q = wave, e = gw + NWGG * q;
          if (e < E) {
            float acc = 0.f;
            for (int i = lane; i < H; i += 64) acc = fmaf(__half2float(hw2[q * kHidMax + i]), hhid[i], acc);
            acc = wave_sum(acc) + hlin[q];
            if (hm->b2) acc += __half2float(static_cast<const __half*>(hm->b2)[e]);
            if (lane == 0) st_word(logh_of(t + 1, N + 1) + e, (uint32_t)t + 2u, __float_as_uint(acc));
          }
        }
      }
    }

    // ---- S8: load the half's next step while the other half computes -----------
    staged = false;
    lstaged = false;
    if (sn < apx->n_steps) {
      __syncthreads();
      const bool go = ahead && Rn.step == sn;
      if (go) {
        fill_src(Rn);
        __syncthreads();
      }
      stage_layer(sn);
      lstaged = true;
      if (go) {
        stage_experts();
        staged = true;
      } else {
        // not loaded ahead: the registers are rewritten before their next use
        // (this tells the compiler the current step's codes are dead here)
#pragma unroll
        for (int j = 0; j < SH::NGW; ++j)
#pragma unroll
          for (int cc = 0; cc < SH::CPL; ++cc) gq[j][cc] = U4{0, 0, 0, 0};
      }
      dma_wait();
      __syncthreads();
    }
    mark(s, 10);
    // the prediction of this step's head, by one workgroup of the half per step
    if (f.head && gw == (s >> 1) % NWGG) {
      if (!flush_pred(s)) break;
    }
    mark(s, 11);
  }

  // ---- finish ------------------------------------------------------------------
  dma_wait();
  __syncthreads();
  if (tx == 0) {
    const uint32_t old = atomicAdd(&apx->ctl[1], 1u);
    if (old == NWG - 1) {
      release_places(apx->ctl, NX);
      __hip_atomic_store(&apx->ctl[1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&apx->ctl[0], base + (uint32_t)apx->n_steps, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

using PShapeMoe35b = PShape<2048, 512, 16, 9, 256, 3>;
using PShapeTiny = PShape<512, 256, 8, 2, 16, 2>;
// the 8B-tier layer: d 4096, 64 experts top-4, I 1024; each XCD of a half
// owns one whole expert
using PShape8b = PShape<4096, 1024, 16, 4, 64, 1>;

template <class SH, bool SIG, bool HM>
static int lds_bytes() {
  if (HM) return sig_scratch_off<SH>() + HmLayout<SH>::BYTES;
  return SIG ? sig_scratch_off<SH>() + (int)sizeof(eng::SigmoidScratch) : SH::O_SRC + (int)sizeof(Src<SH>);
}

template <class SH, bool SIG, bool HM>
static hipError_t launch_as(EngineArgs& a, hipStream_t st) {
  const int lds = lds_bytes<SH, SIG, HM>();
  if (lds > 160 * 1024) return hipErrorInvalidValue;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)pipe_kernel<SH, SIG, HM>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  void* args[] = {&a};
  return hipLaunchCooperativeKernel((const void*)pipe_kernel<SH, SIG, HM>, dim3(NWG), dim3(NT), args, (size_t)lds,
                                    st);
}

template <class SH>
static hipError_t launch(EngineArgs& a, hipStream_t st) {
  if (a.heads) {  // the full head: softmax-top-k routing, shapes whose LDS holds its rows
    if constexpr (SH::D <= 2048) {
      if (a.n_groups > 0 || a.hidden < 64 || a.hidden > kHidMax || a.hidden % 64) return hipErrorInvalidValue;
      return launch_as<SH, false, true>(a, st);
    } else {
      return hipErrorInvalidValue;
    }
  }
  return a.n_groups > 0 ? launch_as<SH, true, false>(a, st) : launch_as<SH, false, false>(a, st);
}

// most expert segments over the four XCDs of a half
static int max_segments(int n_list, int I) {
  const int GX = n_list * I / NXG;
  int most = 0;
  for (int x = 0; x < NXG; ++x) {
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
static bool fits(int n_list, int I, int E, int K) {
  if (n_list > SH::NLX || E > SH::EX || K > 32 || n_list < 1) return false;
  if ((n_list * I) % (NXG * 64) != 0) return false;
  const int GX = n_list * I / NXG;
  if (GX % (NM * 2) != 0 || (2 * (GX / NM)) % SH::RPI != 0) return false;
  if (max_segments(n_list, I) > SH::NSEGX) return false;
  return true;
}

}  // namespace pipe

bool engine_pipe_supported(int d, int I, int r, int K, int S, int E) {
  const int n = K + S;
  if (d == 2048 && I == 512 && r == 16) return pipe::fits<pipe::PShapeMoe35b>(n, I, E, K);
  if (d == 512 && I == 256 && r == 8) return pipe::fits<pipe::PShapeTiny>(n, I, E, K);
  if (d == 4096 && I == 1024 && r == 16) return pipe::fits<pipe::PShape8b>(n, I, E, K);
  return false;
}

size_t engine_pipe_workspace_words(int E, int d, int I, int r, int n_list, int L, EngineArgs* a) {
  size_t off = 0;
  auto take = [&](size_t n) {
    const size_t o = off;
    off += (n + 31) / 32 * 32;
    return o;
  };
  const int NSEGX = 4;
  a->xs_logr = (size_t)(E + 31) / 32 * 32;
  a->xo_logr = take(2 * a->xs_logr);  // by half
  a->xs_av = (size_t)NSEGX * 2 * r;
  a->xo_av = take(2 * pipe::NXG * a->xs_av);  // by half and XCD
  a->xs_hv = (size_t)(n_list * I / 2 + 31) / 32 * 32;  // h of a step, two per word
  a->xo_hv = take(2 * a->xs_hv);                       // by half
  a->xs_adp = (size_t)(n_list * r + 31) / 32 * 32;     // A_down h of every expert
  a->xo_adp = take(2 * a->xs_adp);
  a->xs_rv = (size_t)d;
  a->xo_rv = take(2 * a->xs_rv);  // by step parity
  a->xs_logh_layer = (size_t)(E + 31) / 32 * 32;
  a->xo_logh = take(2 * (size_t)(L > 0 ? L : 1) * a->xs_logh_layer);
  a->xs_pred = 64;
  a->xo_pred = take(2 * (size_t)(L > 0 ? L : 1) * a->xs_pred);
  a->xo_hid = take((size_t)2 * 4 * kHidMax);                  // full head: by half and step
  a->xo_rtm1 = take((size_t)2 * (L > 0 ? L : 1) * 32);          // by token parity and layer
  return off;
}

hipError_t launch_engine_pipe(EngineArgs& a, int d, int I, int r, hipStream_t st) {
  if (d == 2048 && I == 512 && r == 16) return pipe::launch<pipe::PShapeMoe35b>(a, st);
  if (d == 512 && I == 256 && r == 8) return pipe::launch<pipe::PShapeTiny>(a, st);
  if (d == 4096 && I == 1024 && r == 16) return pipe::launch<pipe::PShape8b>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace moe
