// Batched decode / prefill expert path for gfx950.
//
// The math is the one-token expert FFN (Sec. 3.1, Math contract; Sec. 3.3
// unmerged LoRA) applied to every (token, expert) pair of a batch; grouping by
// expert is what makes it a dense contraction (the whole-layer executor path
// of Sec. 3.1 loads every expert of a layer for a prefill chunk).
//
//   permute   one workgroup: per-expert counts, scans, 64-row tiles, and the
//             permuted list of y_experts rows (token t, list position k).
//   prep      x in pair order (below), and per tile A_g x and A_u x (the
//             LoRA-A products, once per tile instead of once per column slab).
//   gate/up   per tile x 64 columns: G = X W_g^T, U = X W_u^T over the tile's
//             rows with v_mfma_f32_16x16x32_f16 (four waves the gate rows,
//             four the up rows of the same columns); int4 codes and the
//             activation rows stream into LDS through global_load_lds in
//             128-k chunks of whole row segments (a ring of two to four
//             chunks, by the tile's row count), the (s, z) rows once per
//             tile; codes are dequantized to fp16 in registers (w = s q + z,
//             one rounding); the LoRA delta is one MFMA step with K = the
//             rank (B rows against lora_scale * A x); epilogue h = silu(g) u
//             stored fp16 in pair order, and the slab's partial A_d h.
//   down      per tile x 128 columns: Y = H W_d^T the same way, LoRA-B of down
//             against lora_scale * (the sum of the slab partials of A_d h);
//             fp32 rows go straight to y_experts.
//
// A GEMM workgroup uses under half of the CU's LDS, so two share a CU: the
// loads that start and end a tile of one overlap the streaming of the other.
// A workgroup's first copies depend only on its tile record (which carries the
// bundle's pointers) and on the tile's token list, both written by the
// permutation; the operands of the epilogue (LoRA rows, A x, the output rows)
// are requested before the copies and consumed after the k loop.
//
// Pair order: inside each 8-element piece the elements run [0,4,1,5,2,6,3,7],
// the order in which the packed nibbles of one code dword come out of a
// 0x000F000F mask at shifts 0, 4, 8, 12. Both MFMA operands use it, so the
// activations (x, h) are kept in pair order and the codes need no shuffle.
// Every output row depends only on its own input row, so the order of rows
// inside a group does not change any result bit.
#include "moe_grouped.h"

namespace moe {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2v __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kGK = 128;                        // k per staged chunk
constexpr int kGT = 512;                        // threads of a GEMM workgroup (8 waves)
constexpr int kGW = kGT / 64;
constexpr int kCodeRow = kGK / 2;               // code bytes of one weight row in a chunk
constexpr int kActRow = kGK * 2;                // activation bytes of one row in a chunk
constexpr int kGateCols = kGroupSlab;           // gate (and up) columns per gate/up workgroup
constexpr int kGateRows = 2 * kGateCols;        // its weight rows: one 16-row block per wave
constexpr int kDownCols = 128;                  // down columns per down workgroup: one block per wave
// Ring of chunk slots (the slot count follows the tile's row blocks). With the
// (s, z) rows and the static arrays a workgroup stays under half the LDS, so
// two workgroups share a CU and one's latencies hide behind the other's
// streaming.
constexpr int kRingBytes = 56 * 1024;
static_assert(kGateRows == 16 * kGW && kDownCols == 16 * kGW, "one row block per wave");
// (s, z) rows of the workgroup's weight rows, staged once per tile: Kdim / 16
// bytes per row
inline int gate_sz_bytes(int d) { return kGateRows * (d / 16); }
inline int down_sz_bytes(int I) { return kDownCols * (I / 16); }
constexpr int kGateStatic = 0;   // static LDS of the GEMM kernels (their epilogues reuse the ring)
constexpr int kDownStatic = 0;
constexpr int kLdsMax = 160 * 1024;             // LDS of a CU: the most one workgroup may take
// (a launch asks only for what its shape needs: up to 80 KB, two workgroups
// share a CU; the d 4096 gate/up rows need more, and run one per CU)

__device__ __forceinline__ h2v as_h2(uint32_t u) { return __builtin_bit_cast(h2v, u); }
__device__ __forceinline__ h8 as_h8(U4 u) { return __builtin_bit_cast(h8, u); }

// [v0..v7] -> [v0,v4,v1,v5,v2,v6,v3,v7] (fp16 elements of a 16-byte piece)
__device__ __forceinline__ U4 perm8(U4 w) {
  U4 o;
  o.x = (w.x & 0xffffu) | (w.z << 16);
  o.y = (w.x >> 16) | (w.z & 0xffff0000u);
  o.z = (w.y & 0xffffu) | (w.w << 16);
  o.w = (w.y >> 16) | (w.w & 0xffff0000u);
  return o;
}
// position of element e (of 8) in pair order
__device__ __forceinline__ int pair_slot(int e) { return e < 4 ? 2 * e : 2 * (e - 4) + 1; }

// Eight int4 codes of one dword (nibble m = input m) -> fp16 weights
// s q + z in pair order. A nibble masked into the mantissa of the fp16 1024
// (0x6400) gives 1024 + q from bits 0-3 and 1024 + 16 q from bits 4-7, so
// nibbles 0, 4 and 1, 5 of v and 2, 6 and 3, 7 of v >> 8 come out with one
// shift and four three-input bit operations ((x & mask) | 0x6400, truth table
// 0xEA); q = (1024 + q) - 1024 or (1024 + 16 q) / 16 - 64, both exact, then the
// fma rounds once.
__device__ __forceinline__ h8 dequant8(uint32_t v, h2v s, h2v z) {
  const uint32_t v8 = v >> 8;
  const h2v off = {(_Float16)1024.0f, (_Float16)1024.0f};
  const h2v sixteenth = {(_Float16)0.0625f, (_Float16)0.0625f}, m64 = {(_Float16)-64.0f, (_Float16)-64.0f};
  const h2v q0 = as_h2(__builtin_amdgcn_bitop3_b32(v, 0x000F000Fu, 0x64006400u, 0xEA)) - off;
  const h2v q1 = __builtin_elementwise_fma(as_h2(__builtin_amdgcn_bitop3_b32(v, 0x00F000F0u, 0x64006400u, 0xEA)),
                                           sixteenth, m64);
  const h2v q2 = as_h2(__builtin_amdgcn_bitop3_b32(v8, 0x000F000Fu, 0x64006400u, 0xEA)) - off;
  const h2v q3 = __builtin_elementwise_fma(as_h2(__builtin_amdgcn_bitop3_b32(v8, 0x00F000F0u, 0x64006400u, 0xEA)),
                                           sixteenth, m64);
  const h2v w0 = __builtin_elementwise_fma(q0, s, z);
  const h2v w1 = __builtin_elementwise_fma(q1, s, z);
  const h2v w2 = __builtin_elementwise_fma(q2, s, z);
  const h2v w3 = __builtin_elementwise_fma(q3, s, z);
  return h8{w0[0], w0[1], w1[0], w1[1], w2[0], w2[1], w3[0], w3[1]};
}

__device__ __forceinline__ f4 mfma(h8 a, h8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// LoRA-B operand of the rank step: row `row` of B [out][r], elements
// kq*8 .. kq*8+7 of the rank (zero past r and for kq >= 2).
__device__ __forceinline__ h8 lora_b_operand(const __half* b, int row, int r, int kq) {
  h8 v = {};
  if (kq < 2) {
    const _Float16* p = reinterpret_cast<const _Float16*>(b) + (size_t)row * r + kq * 8;
    if (r == 16 || (r == 8 && kq == 0)) {
      v = as_h8(ld16(p));
    } else if (r != 8) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (kq * 8 + e < r) v[e] = p[e];
    }
  }
  return v;
}

// ---- copies into LDS --------------------------------------------------------
// global_load_lds: each lane of the wave moves 16 (or 4) bytes from its own
// address to lds + 16 * lane (4 * lane). The compiler does not see these as
// memory instructions; vm_wait orders them.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}
__device__ __forceinline__ void dma16(const void* g, const void* lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_addr(lds)), "v"(g)
      : "memory");
}
__device__ __forceinline__ void dma4(const void* g, const void* lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %2, off nt\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_addr(lds)), "v"(g)
      : "memory");
}
// wait until at most N of this wave's copies are outstanding (N an immediate)
template <int N>
__device__ __forceinline__ void vm_wait_n() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// the same for N = A * (hi ? PH : PL) with A = ahead in [0, 6): a short chain of
// scalar compares on uniform values instead of one case per count
template <int PH, int PL, int A = 0>
__device__ __forceinline__ void vm_wait_ahead(int ahead, bool hi) {
  if constexpr (A < 6) {
    if (ahead == A) {
      if (hi)
        vm_wait_n<A * PH>();
      else
        vm_wait_n<A * PL>();
      return;
    }
    vm_wait_ahead<PH, PL, A + 1>(ahead, hi);
  } else {
    vm_wait_n<0>();
  }
}

// ---- one tile's k loop --------------------------------------------------------
// acc[0][m] += X[rows of block m] . W[16 rows of this wave's block]^T over
// Kdim for the MB 16-row blocks of the tile (MB a compile-time count) and
// NROWS = 128 weight rows (one block of 16 per wave). Chunk c (k in
// [c kGK, (c+1) kGK)) of every weight row and activation row is staged into a
// ring slot with global_load_lds, each instruction copying whole row segments
// (16 rows x 64 bytes of codes, 4 rows x 256 bytes of activations). In LDS
// the 16-byte pieces of a row are XOR-swizzled by the row, so that the 16
// rows an MFMA operand reads sit on different banks. MFMA instruction j of a
// chunk takes, in lane (col, kq), the k values kq 32 + 8 j .. + 7 (one dword
// of codes; the same k order in both operands, so any order is fine); a lane
// uses one (s, z) group per chunk. The (s, z) rows of the whole k range are
// staged before chunk 0.
// wrow(row) / srow(row): the global code and (s, z) row of weight row `row`;
// xsrc(row, k): global address of 8 activations (pair order) of activation
// row `row` at k.
template <int MB, int NROWS, typename WRow, typename SRow, typename XSrc>
__device__ __forceinline__ void tile_gemm_mb(char* ring, char* szl, int Kdim, WRow wrow, SRow srow,
                                             XSrc xsrc, f4 (*acc)[4]) {
  static_assert(NROWS == 16 * kGW, "one block per wave");
  constexpr int CODE_B = NROWS * kCodeRow;                     // codes of a slot
  constexpr int SLOT = CODE_B + MB * 16 * kActRow;
  constexpr int NBUF = kRingBytes / SLOT < 6 ? kRingBytes / SLOT : 6;
  static_assert(NBUF >= 2, "two slots at least");
  constexpr int CODE_I = CODE_B / 1024 / kGW;                  // code copies per wave per chunk
  constexpr int XI = MB * 16 * kActRow / 1024;                 // activation copies per chunk
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int col = lane & 15, kq = lane >> 4;
  // this wave's copies per chunk: CODE_I codes and XHI or XLO activation copies
  constexpr int XLO = XI / kGW, XHI = (XI + kGW - 1) / kGW;
  const bool xhi = wave < XI % kGW;
  const int nch = Kdim / kGK;
  const int szr = Kdim / 16;                                   // (s, z) bytes per row
  auto slot = [&](int c) { return ring + (c % NBUF) * SLOT; };
  auto issue = [&](int c) {
    char* sl = slot(c);
#pragma unroll
    for (int i = 0; i < CODE_I; ++i) {  // rows 16b .. 16b+15, 64 bytes each
      const int b = wave * CODE_I + i;
      const int row = 16 * b + (lane >> 2), phys = lane & 3;
      const int piece = phys ^ ((row >> 2) & 3);
      dma16(wrow(row) + c * kCodeRow + piece * 16, sl + b * 1024);
    }
#pragma unroll
    for (int j = 0; j < XHI; ++j) {  // activation rows 4b .. 4b+3, 256 bytes each
      const int b = wave + j * kGW;
      if (b < XI) {
        const int row = 4 * b + (lane >> 4), phys = lane & 15;
        const int piece = phys ^ (row & 15);
        dma16(xsrc(row, c * kGK + piece * 8), sl + CODE_B + b * 1024);
      }
    }
  };
  // (loads of the caller still outstanding here are older than every copy:
  // they complete before the chunks in whose wait they are counted)
  for (int b = wave; b * 1024 < NROWS * szr; b += kGW) {  // (s, z) rows, natural layout
    const int o = b * 1024 + lane * 16;
    dma16(srow(o / szr) + o % szr, szl + b * 1024);
  }
  const int pre = nch < NBUF ? nch : NBUF;
  for (int c = 0; c < pre; ++c) issue(c);
  const int row = wave * 16 + col;                             // this lane's weight row
  const int sw = (row >> 2) & 3;
  for (int c = 0; c < nch; ++c) {
    // chunks issued after chunk c: all of the first NBUF at c = 0, then one
    // per chunk (into the slot of chunk c - 1)
    const int ahead = c == 0 ? pre - 1 : min(nch - 1 - c, NBUF - 2);
    vm_wait_ahead<CODE_I + XHI, CODE_I + XLO>(ahead, xhi);
    __syncthreads();  // chunk c is in LDS for every wave; chunk c - 1 is consumed
    if (c > 0 && c + NBUF - 1 < nch) issue(c + NBUF - 1);
    const char* sl = slot(c);
    const U4 q = *reinterpret_cast<const U4*>(sl + row * kCodeRow + (kq ^ sw) * 16);
    const uint32_t szw = *reinterpret_cast<const uint32_t*>(szl + row * szr + (2 * c + (kq >> 1)) * 4);
    h8 af[4][MB];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int m = 0; m < MB; ++m)
        af[j][m] = *reinterpret_cast<const h8*>(sl + CODE_B + (16 * m + col) * kActRow + ((kq * 4 + j) ^ col) * 16);
    const h2v sz = as_h2(szw);
    const h2v s2 = h2v{sz[0], sz[0]}, z2 = h2v{sz[1], sz[1]};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t word = j == 0 ? q.x : j == 1 ? q.y : j == 2 ? q.z : q.w;
      const h8 w = dequant8(word, s2, z2);
#pragma unroll
      for (int m = 0; m < MB; ++m) acc[0][m] = mfma(af[j][m], w, acc[0][m]);
    }
  }
  __syncthreads();  // the ring is free again
}
// mb (1 .. 4) is the same for every thread of the workgroup
template <int NROWS, typename WRow, typename SRow, typename XSrc>
__device__ __forceinline__ void tile_gemm(char* ring, char* szl, int Kdim, int mb, WRow wrow, SRow srow,
                                          XSrc xsrc, f4 (*acc)[4]) {
  switch (mb) {
    case 1: tile_gemm_mb<1, NROWS>(ring, szl, Kdim, wrow, srow, xsrc, acc); break;
    case 2: tile_gemm_mb<2, NROWS>(ring, szl, Kdim, wrow, srow, xsrc, acc); break;
    case 3: tile_gemm_mb<3, NROWS>(ring, szl, Kdim, wrow, srow, xsrc, acc); break;
    default: tile_gemm_mb<4, NROWS>(ring, szl, Kdim, wrow, srow, xsrc, acc); break;
  }
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(1024) grouped_permute_kernel(GroupedArgs a) {
  __shared__ int cnt[kGroupMaxG];
  __shared__ int goff[kGroupMaxG];   // first permuted row and first tile of each group
  __shared__ int gtoff[kGroupMaxG];
  __shared__ int scr[2][1024];
  __shared__ int sct[2][1024];
  const int tid = threadIdx.x;
  const int G = a.E + a.S;
  for (int g = tid; g < G; g += 1024) cnt[g] = g >= a.E ? a.T : 0;
  __syncthreads();
  const int TK = a.T * a.K;
  // the thread's first kIdxReg routing ids are read once, into registers, for
  // both passes over them (each pass would otherwise wait on its loads in turn)
  constexpr int kIdxReg = 8;
  int ev[kIdxReg];
#pragma unroll
  for (int j = 0; j < kIdxReg; ++j) ev[j] = tid + 1024 * j < TK ? a.idx[tid + 1024 * j] : -1;
  auto id_at = [&](int j, int i) {  // routing id i = tid + 1024 j
    int e = -1;
#pragma unroll
    for (int q = 0; q < kIdxReg; ++q)
      if (j == q) e = ev[q];
    return j < kIdxReg ? e : a.idx[i];
  };
  for (int i = tid, j = 0; i < TK; i += 1024, ++j) {
    const int e = id_at(j, i);
    if (e >= 0 && e < a.E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  // thread t owns groups 2t and 2t+1; inclusive scan of rows and tiles
  const int g0 = 2 * tid, g1 = g0 + 1;
  const int c0 = g0 < G ? cnt[g0] : 0, c1 = g1 < G ? cnt[g1] : 0;
  const int t0 = (c0 + kGroupRows - 1) / kGroupRows, t1 = (c1 + kGroupRows - 1) / kGroupRows;
  const int vr = c0 + c1, vt = t0 + t1;
  int pb = 0;
  scr[0][tid] = vr;
  sct[0][tid] = vt;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    int r = scr[pb][tid], t = sct[pb][tid];
    if (tid >= o) {
      r += scr[pb][tid - o];
      t += sct[pb][tid - o];
    }
    scr[pb ^ 1][tid] = r;
    sct[pb ^ 1][tid] = t;
    pb ^= 1;
    __syncthreads();
  }
  const int off0 = scr[pb][tid] - vr, toff0 = sct[pb][tid] - vt;
  const int total_tiles = sct[pb][1023];
  // the slots and bundles of both groups requested together (one dependent
  // pair of loads for the thread); a group that is not resident copies slot 0's
  // bundle (a table has at least one slot), which no kernel reads. The bundle
  // moves as 12 pointer words (held in registers).
  constexpr int kBW = (int)(sizeof(moe_bundle) / 8);
  static_assert(sizeof(moe_bundle) == 8 * kBW && sizeof(GroupTile) == 16 + sizeof(moe_bundle), "record layout");
  const int s0 = g0 < G && c0 ? a.slot_of[g0] : -1, s1 = g1 < G && c1 ? a.slot_of[g1] : -1;
  uint64_t w0[kBW], w1[kBW];
  {
    const uint64_t* p0 = reinterpret_cast<const uint64_t*>(a.bundles + (s0 > 0 ? s0 : 0));
    const uint64_t* p1 = reinterpret_cast<const uint64_t*>(a.bundles + (s1 > 0 ? s1 : 0));
#pragma unroll
    for (int q = 0; q < kBW; ++q) {
      w0[q] = p0[q];
      w1[q] = p1[q];
    }
  }
  auto emit = [&](int g, int c, int off, int toff, int slot, const uint64_t (&w)[kBW]) {
    if (g >= G) return;
    goff[g] = off;
    gtoff[g] = toff;
    if (c == 0) return;
    if (slot < 0 && a.status) atomicOr(a.status, MOE_STATUS_SLOT_MISS);
    for (int j = 0; j * kGroupRows < c; ++j) {
      GroupTile* o = a.tiles + toff + j;
      o->g = g;
      o->row0 = off + kGroupRows * j;
      o->nrows = min(kGroupRows, c - kGroupRows * j);
      o->slot = slot;
      uint64_t* ob = reinterpret_cast<uint64_t*>(&o->b);
#pragma unroll
      for (int q = 0; q < kBW; ++q) ob[q] = w[q];
    }
  };
  emit(g0, c0, off0, toff0, s0, w0);
  emit(g1, c1, off0 + c0, toff0 + t0, s1, w1);
  __syncthreads();  // every count is read: the array becomes the insertion cursors
  if (g0 < G) cnt[g0] = off0;
  if (g1 < G) cnt[g1] = off0 + c0;
  if (tid == 0) *a.n_tiles = total_tiles;
  __syncthreads();
  for (int i = tid, j = 0; i < TK; i += 1024, ++j) {
    const int e = id_at(j, i);
    const int t = i / a.K, k = i - t * a.K;
    const int row = t * a.n_list + k;
    if (e >= 0 && e < a.E) {
      const int pos = atomicAdd(&cnt[e], 1), rel = pos - goff[e];
      a.perm[pos] = row;
      a.tile_tok[(size_t)(gtoff[e] + rel / kGroupRows) * kGroupRows + rel % kGroupRows] = t;
    } else {  // an id outside [0, E) contributes zeros and is reported
      if (a.status) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      float* y = a.y_experts + (size_t)row * a.d;
      for (int j = 0; j < a.d; ++j) y[j] = 0.f;
    }
  }
  for (int i = tid; i < a.T * a.S; i += 1024) {
    const int s = i / a.T, t = i - s * a.T, g = a.E + s;
    a.perm[cnt[g] + t] = t * a.n_list + a.K + s;
    a.tile_tok[(size_t)(gtoff[g] + t / kGroupRows) * kGroupRows + t % kGroupRows] = t;
  }
}

// ---------------------------------------------------------------------------
// prep: blocks [0, xb) write x in pair order; blocks [xb, xb + 4 max_tiles)
// form A_g x and A_u x of one tile over one quarter of d (four workgroups per
// tile): waves 4c .. 4c+3 take projection c, each over a sixteenth of d, with
// MFMA (ranks as the 16 columns); the waves' sums add up in the workgroup as
// (w0 + w1) + (w2 + w3), the quarters' in gate/up the same way.
__global__ void __launch_bounds__(kGT, 6) grouped_prep_kernel(GroupedArgs a, int xb) {
  __shared__ float part[2][4][kGroupRows][16];
  const int tid = threadIdx.x;
  if ((int)blockIdx.x < xb) {
    const size_t pieces = (size_t)a.T * a.d / 8;
    const size_t p = (size_t)blockIdx.x * kGT + tid;
    if (p < pieces) {
      const U4 v = ld16(reinterpret_cast<const char*>(a.x) + p * 16);
      *reinterpret_cast<U4*>(reinterpret_cast<char*>(a.xp) + p * 16) = perm8(v);
    }
    return;
  }
  const int ti = (blockIdx.x - xb) >> 2, Q = (blockIdx.x - xb) & 3;
  if (ti >= *a.n_tiles) return;
  const GroupTile tl = a.tiles[ti];
  const int wave = tid >> 6, lane = tid & 63, col = lane & 15, kq = lane >> 4;
  // the tokens of this lane's rows (the tile's token list, read beside the record)
  int tok[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) tok[m] = a.tile_tok[(size_t)ti * kGroupRows + 16 * m + col];
  if (tl.slot < 0 || a.r <= 0) return;
  const moe_bundle& bd = tl.b;
  const int c = wave >> 2, quarter = wave & 3;
  const int d = a.d, r = a.r;
  const int mb = (tl.nrows + 15) >> 4;
  const void* A = c == 0 ? bd.gate.lora_a : bd.up.lora_a;
  const void* Bm = c == 0 ? bd.gate.lora_b : bd.up.lora_b;
  const bool on = A && Bm;
  f4 acc[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) acc[m] = f4{0.f, 0.f, 0.f, 0.f};
  if (on) {
    const _Float16* arow = col < r ? static_cast<const _Float16*>(A) + (size_t)col * d : nullptr;
    const _Float16* xrow[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int row = 16 * m + col;
      xrow[m] = row < tl.nrows ? reinterpret_cast<const _Float16*>(a.x) + (size_t)tok[m] * d : nullptr;
    }
    const int kbeg = Q * (d / 4) + quarter * (d / 16), kend = kbeg + d / 16;
#pragma unroll 1
    for (int k0 = kbeg + kq * 8; k0 < kend; k0 += 64) {  // two k steps: all loads, then the MFMAs
      h8 b[2], av[2][4];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int k = k0 + 32 * u;
        const bool in = k < kend;
        b[u] = arow && in ? as_h8(ld16(arow + k)) : h8{};
#pragma unroll
        for (int m = 0; m < 4; ++m) av[u][m] = m < mb && xrow[m] && in ? as_h8(ld16(xrow[m] + k)) : h8{};
      }
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int m = 0; m < 4; ++m)
          if (m < mb) acc[m] = mfma(av[u][m], b[u], acc[m]);
    }
  }
  // C layout: lane (col, kq) holds rows 4 kq + e of block m, rank col
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int e = 0; e < 4; ++e) part[c][quarter][16 * m + 4 * kq + e][col] = acc[m][e];
  __syncthreads();
  for (int p = tid; p < 2 * tl.nrows * 16; p += kGT) {
    const int cc = p / (tl.nrows * 16), rem = p % (tl.nrows * 16), row = rem >> 4, k = rem & 15;
    const float v = (part[cc][0][row][k] + part[cc][1][row][k]) + (part[cc][2][row][k] + part[cc][3][row][k]);
    a.ax[(((size_t)(tl.row0 + row) * 4 + Q) * 2 + cc) * 16 + k] = v;
  }
}

// ---------------------------------------------------------------------------
// gate/up: workgroup (tile, y) takes the gate and up rows of columns
// [64 y, 64 y + 64): wave w < 4 the gate rows of columns 64 y + 16 w + col,
// wave w + 4 the up rows of the same columns.
// Block b of a GEMM grid -> (token tile, column tile). The dispatcher deals
// blocks to the 8 XCDs in turn, so blocks b and b + 8 share an XCD: every
// column tile of token tile x gets a block that is congruent to x mod 8, the
// ny of them 8 apart. The tile's activations (and its row list) then go
// through one XCD's L2, fetched once instead of once per column tile. The
// grid is the tile count rounded up to a multiple of 8, times ny.
__device__ __forceinline__ void tile_of_block(int b, int ny, int& x, int& y) {
  const int grp = b / (8 * ny), r = b - grp * 8 * ny;
  x = grp * 8 + (r & 7);
  y = r >> 3;
}

__global__ void __launch_bounds__(kGT, 4) grouped_gateup_kernel(GroupedArgs a) {
  extern __shared__ __attribute__((aligned(16))) char ring[];
  char* const szl = ring + kRingBytes;
  // after the k loop the ring holds the up accumulators, h of the tile, the
  // A_d rows and lora_scale * (A x) of the tile's rows
  float* const uacc = reinterpret_cast<float*>(ring);  // [4 waves][4 m][4 e][64 lanes]
  _Float16(*hs)[kGateCols] = reinterpret_cast<_Float16(*)[kGateCols]>(ring + 16384);
  _Float16(*ads)[kGateCols] = reinterpret_cast<_Float16(*)[kGateCols]>(ring + 16384 + kGroupRows * kGateCols * 2);
  constexpr int kLaOff = 16384 + (kGroupRows + 16) * kGateCols * 2;
  _Float16(*la)[kGroupRows][16] = reinterpret_cast<_Float16(*)[kGroupRows][16]>(ring + kLaOff);
  static_assert(kLaOff + 2 * kGroupRows * 16 * 2 <= kRingBytes, "epilogue fits in the ring");
  int bx, by;
  tile_of_block(blockIdx.x, a.I / kGateCols, bx, by);
  const int tix = bx < a.max_tiles ? bx : 0;
  // (the record and the token list are read beside the count; one past the
  // count is never used)
  const GroupTile tl = a.tiles[tix];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  // tokens of this wave's activation copies: rows 4 b .. 4 b + 3 for b = wave
  // and wave + 8 (uniform per wave)
  const int32_t* tt = a.tile_tok + (size_t)tix * kGroupRows;
  const int tr0 = tt[0];
  const int t0 = tt[4 * wave], t1 = tt[4 * wave + 1], t2 = tt[4 * wave + 2], t3 = tt[4 * wave + 3];
  const int t4 = tt[4 * (wave + kGW)], t5 = tt[4 * (wave + kGW) + 1], t6 = tt[4 * (wave + kGW) + 2],
            t7 = tt[4 * (wave + kGW) + 3];
  if (bx >= *a.n_tiles) return;
  if (tl.slot < 0) return;  // not resident: the down kernel writes zero rows
  const moe_bundle& bd = tl.b;
  const int col = lane & 15, kq = lane >> 4;
  const int d = a.d, I = a.I, r = a.r;
  const int mb = (tl.nrows + 15) >> 4;
  const int c0 = by * kGateCols;                // first column of this workgroup
  const int cc = wave >> 2, wb = wave & 3;      // projection (0 gate, 1 up), column block
  const int i = c0 + wb * 16 + col;             // this lane's gate/up column
  const bool lg = r > 0 && bd.gate.lora_a && bd.gate.lora_b;
  const bool lu = r > 0 && bd.up.lora_a && bd.up.lora_b;
  const bool ld = r > 0 && bd.down.lora_a && bd.down.lora_b;

  // The epilogue's operands, requested now and consumed after the k loop:
  // A x of the tile's rows (4 values per thread), the LoRA-B operand and the
  // A_d rows of this workgroup's columns.
  static_assert(2 * kGroupRows * 16 == 4 * kGT, "four A x values per thread");
  float axv[4][4];  // [value][quarter of d]
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int p = tid + q * kGT, pc = p / (kGroupRows * 16), row = (p >> 4) % kGroupRows, k = p & 15;
    const bool on = row < tl.nrows && k < r && (pc == 0 ? lg : lu);
    const float* src = a.ax + ((size_t)(tl.row0 + row) * 4 * 2 + pc) * 16 + k;
#pragma unroll
    for (int h = 0; h < 4; ++h) axv[q][h] = on ? src[h * 32] : 0.f;
  }
  const bool lw = cc == 0 ? lg : lu;
  const h8 bop = lw ? lora_b_operand(static_cast<const __half*>(cc == 0 ? bd.gate.lora_b : bd.up.lora_b), i,
                                     r, kq)
                    : h8{};
  static_assert(16 * kGateCols == 2 * kGT, "two A_d values per thread");
  _Float16 adv[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int p = tid + q * kGT, k = p / kGateCols, c = p % kGateCols;
    adv[q] = (ld && k < r) ? reinterpret_cast<const _Float16*>(bd.down.lora_a)[(size_t)k * I + c0 + c]
                           : (_Float16)0.f;
  }

  // weight row w_row (0 .. 127): projection w_row / 64, column c0 + w_row % 64
  // (the projection pointers are in registers: a pointer loaded inside the
  // copy loop would be a vector load behind the chunks in flight, and its wait
  // would drain them)
  const uint8_t* const gq = static_cast<const uint8_t*>(bd.gate.q);
  const uint8_t* const uq = static_cast<const uint8_t*>(bd.up.q);
  const uint8_t* const gs = static_cast<const uint8_t*>(bd.gate.sz);
  const uint8_t* const us = static_cast<const uint8_t*>(bd.up.sz);
  auto wrow = [&](int w_row) -> const uint8_t* {
    return (w_row < kGateCols ? gq : uq) + (size_t)(c0 + (w_row % kGateCols)) * (d / 2);
  };
  auto srow = [&](int w_row) -> const uint8_t* {
    return (w_row < kGateCols ? gs : us) + (size_t)(c0 + (w_row % kGateCols)) * (d / 16);
  };
  // The activation copies of this wave are b = wave and wave + 8, lane rows
  // 4 b + (lane >> 4): each lane's two source rows are fixed for the tile. They
  // are resolved here from plain values (a token array indexed inside the copy
  // loop would live in scratch memory, and each read's wait would drain the
  // copies in flight).
  static_assert(kActRow == 256, "four activation rows per copy");
  // (rows past nrows hold no token: they take row 0's, and are never stored)
  const int q4 = lane >> 4;
  const int tlo = 4 * wave + q4 >= tl.nrows ? tr0 : q4 == 0 ? t0 : q4 == 1 ? t1 : q4 == 2 ? t2 : t3;
  const int thi = 4 * (wave + kGW) + q4 >= tl.nrows ? tr0 : q4 == 0 ? t4 : q4 == 1 ? t5 : q4 == 2 ? t6 : t7;
  const char* const xlo = reinterpret_cast<const char*>(a.xp) + (size_t)tlo * d * 2;
  const long long xdelta = ((long long)thi - tlo) * d * 2;
  auto xsrc = [=](int row, int k) -> const void* {
    return xlo + ((row >> 2) >= kGW ? xdelta : 0LL) + (size_t)k * 2;
  };

  f4 acc[1][4];
#pragma unroll
  for (int m = 0; m < 4; ++m) acc[0][m] = f4{0.f, 0.f, 0.f, 0.f};
  tile_gemm<kGateRows>(ring, szl, d, mb, wrow, srow, xsrc, acc);

  // lora_scale * (A x) of the tile's rows, fp16 (rank past r: zero)
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int p = tid + q * kGT, pc = p / (kGroupRows * 16), row = (p >> 4) % kGroupRows, k = p & 15;
    la[pc][row][k] = (_Float16)(a.lora_scale * ((axv[q][0] + axv[q][1]) + (axv[q][2] + axv[q][3])));
  }
  __syncthreads();
  // LoRA delta of this wave's projection: one MFMA step of K = rank against
  // lora_scale * (A x)
  if (lw) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (m >= mb) continue;
      h8 aop = {};
      if (kq < 2) aop = *reinterpret_cast<const h8*>(&la[cc][16 * m + col][kq * 8]);
      acc[0][m] = mfma(aop, bop, acc[0][m]);
    }
  }
  // the up waves hand their sums to the gate waves of the same columns (same
  // lane); A_d rows restricted to this workgroup's columns
  if (cc == 1) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (m >= mb) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) uacc[((wb * 4 + m) * 4 + e) * 64 + lane] = acc[0][m][e];
    }
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int p = tid + q * kGT;
    ads[p / kGateCols][p % kGateCols] = adv[q];
  }
  __syncthreads();
  // h = silu(g) u, fp16: to HBM in pair order, and to LDS for A_d h
  if (cc == 0) {
    const int ip = (i & ~7) | pair_slot(i & 7);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (m >= mb) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = 16 * m + 4 * kq + e;
        const float g = acc[0][m][e], u = uacc[((wb * 4 + m) * 4 + e) * 64 + lane];
        const __half h = __float2half(g / (1.0f + expf(-g)) * u);
        if (row < tl.nrows) a.h[(size_t)(tl.row0 + row) * I + ip] = h;
        hs[row][wb * 16 + col] = h;
      }
    }
  }
  __syncthreads();
  // the slab's partial A_d h: row x rank over this workgroup's columns
  if (ld) {
    for (int p = tid; p < tl.nrows * 16; p += kGT) {
      const int row = p >> 4, k = p & 15;
      float s = 0.f;
      for (int c = 0; c < kGateCols; ++c) s = fmaf((float)ads[k][c], (float)hs[row][c], s);
      a.adp[((size_t)(tl.row0 + row) * (I / kGroupSlab) + by) * 16 + k] = s;
    }
  }
}

__global__ void __launch_bounds__(kGT, 4) grouped_down_kernel(GroupedArgs a) {
  extern __shared__ __attribute__((aligned(16))) char ring[];
  // after the k loop the ring holds lora_scale * (A_d h) of the tile's rows and
  // their y_experts rows
  _Float16(*la)[16] = reinterpret_cast<_Float16(*)[16]>(ring);
  int* ydst = reinterpret_cast<int*>(ring + kGroupRows * 16 * 2);
  int bx, by;
  tile_of_block(blockIdx.x, a.d / kDownCols, bx, by);
  const GroupTile tl = a.tiles[bx < a.max_tiles ? bx : 0];  // (read beside the count, as in gate/up)
  if (bx >= *a.n_tiles) return;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, kq = lane >> 4;
  const int d = a.d, I = a.I, r = a.r;
  const int mb = (tl.nrows + 15) >> 4;
  const int n0 = by * kDownCols + wave * 16 + col;  // this lane's output column
  if (tl.slot < 0) {  // not resident: the pair contributes zeros (the miss is reported)
    for (int p = tid; p < tl.nrows * kDownCols; p += kGT) {
      const int row = p / kDownCols, c = p % kDownCols;
      a.y_experts[(size_t)a.perm[tl.row0 + row] * d + by * kDownCols + c] = 0.f;
    }
    return;
  }
  const moe_bundle& bd = tl.b;
  const bool ld = r > 0 && bd.down.lora_a && bd.down.lora_b;
  // The epilogue's operands, requested now and consumed after the k loop: the
  // output rows, the LoRA-B operand, and the slab partials of A_d h (thread p
  // holds (row, rank) = (p / 16, p % 16) and (p + 512) / 16; the first 16 slabs
  // here, any further ones after the loop).
  const int nsl = I / kGroupSlab;
  constexpr int kPreSl = 16;
  const int ydv = tid < tl.nrows ? a.perm[tl.row0 + tid] : -1;
  const h8 bop = ld ? lora_b_operand(static_cast<const __half*>(bd.down.lora_b), n0, r, kq) : h8{};
  static_assert(kGroupRows * 16 == 2 * kGT, "two A_d h sums per thread");
  float adv[2][kPreSl];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int p = tid + q * kGT, row = p >> 4, k = p & 15;
    const bool on = ld && row < tl.nrows && k < r;
    const float* src = a.adp + (size_t)(tl.row0 + row) * nsl * 16 + k;
#pragma unroll
    for (int sl = 0; sl < kPreSl; ++sl) adv[q][sl] = on && sl < nsl ? src[sl * 16] : 0.f;
  }
  // weight row w_row (0 .. 127): output column by * 128 + w_row (the pointers
  // in registers, as in gate/up)
  const size_t nbase = (size_t)by * kDownCols;
  const uint8_t* const dq = static_cast<const uint8_t*>(bd.down.q);
  const uint8_t* const dsz = static_cast<const uint8_t*>(bd.down.sz);
  auto wrow = [&](int w_row) -> const uint8_t* { return dq + (nbase + w_row) * (I / 2); };
  auto srow = [&](int w_row) -> const uint8_t* { return dsz + (nbase + w_row) * (I / 16); };
  const char* hbase = reinterpret_cast<const char*>(a.h);
  auto xsrc = [&](int row, int k) -> const void* {
    return hbase + ((size_t)(tl.row0 + (row < tl.nrows ? row : 0)) * I + k) * 2;
  };

  f4 acc[1][4];
#pragma unroll
  for (int m = 0; m < 4; ++m) acc[0][m] = f4{0.f, 0.f, 0.f, 0.f};
  tile_gemm<kDownCols>(ring, ring + kRingBytes, I, mb, wrow, srow, xsrc, acc);

  // lora_scale * (A_d h): the slab partials summed in slab order
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int p = tid + q * kGT, row = p >> 4, k = p & 15;
    float v = 0.f;
#pragma unroll
    for (int sl = 0; sl < kPreSl; ++sl) v += adv[q][sl];
    if (ld && row < tl.nrows && k < r) {
      const float* src = a.adp + (size_t)(tl.row0 + row) * nsl * 16 + k;
      for (int sl = kPreSl; sl < nsl; ++sl) v += src[sl * 16];
    }
    la[row][k] = (_Float16)(v * a.lora_scale);
  }
  if (tid < kGroupRows) ydst[tid] = ydv;
  __syncthreads();
  if (ld) {
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (m >= mb) continue;
      h8 aop = {};
      if (kq < 2) aop = *reinterpret_cast<const h8*>(&la[16 * m + col][kq * 8]);
      acc[0][m] = mfma(aop, bop, acc[0][m]);
    }
  }
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    if (m >= mb) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 16 * m + 4 * kq + e;
      if (row < tl.nrows) {
        float* y = a.y_experts + (size_t)ydst[row] * d;
        y[n0] = acc[0][m][e];
      }
    }
  }
}

}  // namespace

bool grouped_shape_supported(int d, int I, int r, int groups) {
  return d % kDownCols == 0 && I % kGateCols == 0 && d % kGK == 0 && I % kGK == 0 && r >= 0 &&
         r <= kGroupMaxR && groups <= kGroupMaxG &&
         kRingBytes + gate_sz_bytes(d) + kGateStatic <= kLdsMax &&
         kRingBytes + down_sz_bytes(I) + kDownStatic <= kLdsMax;
}

hipError_t launch_grouped_ffn(const GroupedArgs& a, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)grouped_gateup_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsMax - kGateStatic);
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)grouped_down_kernel,
                              hipFuncAttributeMaxDynamicSharedMemorySize, kLdsMax - kDownStatic);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int lds_gu = kRingBytes + gate_sz_bytes(a.d), lds_dn = kRingBytes + down_sz_bytes(a.I);
  hipLaunchKernelGGL(grouped_permute_kernel, dim3(1), dim3(1024), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int xb = (int)(((size_t)a.T * a.d / 8 + kGT - 1) / kGT);
  hipLaunchKernelGGL(grouped_prep_kernel, dim3(xb + 4 * a.max_tiles), dim3(kGT), 0, st, a, xb);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles8 = (a.max_tiles + 7) / 8 * 8;
  hipLaunchKernelGGL(grouped_gateup_kernel, dim3(tiles8 * (a.I / kGateCols)), dim3(kGT), lds_gu, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(grouped_down_kernel, dim3(tiles8 * (a.d / kDownCols)), dim3(kGT), lds_dn, st, a);
  return hipGetLastError();
}

}  // namespace moe
