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
//   gate/up   per tile x 128 columns: G = X W_g^T, U = X W_u^T over the tile's
//             rows with v_mfma_f32_16x16x32_f16; int4 codes and the activation
//             rows stream into LDS through global_load_lds (four 128-k chunks
//             in flight), the codes are dequantized to fp16 in registers
//             (w = s q + z, one rounding); the LoRA delta is one MFMA step with
//             K = the rank (B rows against lora_scale * A x); epilogue
//             h = silu(g) u stored fp16 in pair order, and the slab's partial
//             A_d h.
//   down      per tile x 256 columns: Y = H W_d^T the same way, LoRA-B of down
//             against lora_scale * (the sum of the slab partials of A_d h);
//             fp32 rows go straight to y_experts.
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
constexpr int kNBuf = 4;                        // ring slots (chunks) per workgroup
constexpr int kGT = 512;                        // threads of a GEMM workgroup (8 waves)
constexpr int kGW = kGT / 64;
constexpr int kXSlot = kGroupRows * kGK * 2;    // one chunk of 64 activation rows (16 KB)
constexpr int kWBlk = 1024 + 256;               // one column block of one wave: codes + (s, z)
constexpr int kNBlk = 2;                        // column blocks of 16 per wave
constexpr int kWSlot = kGW * kNBlk * kWBlk;     // one chunk of all waves' weights
constexpr int kRingBytes = kNBuf * (kXSlot + kWSlot);
constexpr int kGateCols = kGW * 16;             // gate/up columns per workgroup (each of g, u)
constexpr int kDownCols = kGW * kNBlk * 16;     // down columns per workgroup
constexpr int kSlab = 128;                      // columns per A_d h partial (= kGateCols)
static_assert(kGateCols == kSlab, "one A_d h partial per gate/up workgroup");

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
// s q + z in pair order. 0x6400 | q is the fp16 value 1024 + q, so
// subtracting 1024 gives q exactly; the fma rounds once.
__device__ __forceinline__ h8 dequant8(uint32_t v, h2v s, h2v z) {
  const h2v off = {(_Float16)1024.0f, (_Float16)1024.0f};
  const h2v q0 = as_h2((v & 0x000F000Fu) | 0x64006400u) - off;
  const h2v q1 = as_h2(((v >> 4) & 0x000F000Fu) | 0x64006400u) - off;
  const h2v q2 = as_h2(((v >> 8) & 0x000F000Fu) | 0x64006400u) - off;
  const h2v q3 = as_h2(((v >> 12) & 0x000F000Fu) | 0x64006400u) - off;
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
    if (r == 16) {
      v = as_h8(ld16(p));
    } else {
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
// memory instructions; vm_wait / vm_drain order them.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
}
__device__ __forceinline__ void dma16(const void* g, const void* lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off nt\n\t"
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
// Nothing of the compiler's own outstanding (a wait it would place for one of
// its loads inside a copy loop would drain the copies too). simm16 0x0F70:
// vmcnt 0, expcnt and lgkmcnt unconstrained.
__device__ __forceinline__ void vm_drain() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);
}
// wait until at most n of this wave's copies are outstanding (n <= 27)
__device__ __forceinline__ void vm_wait(int n) {
  switch (n) {
#define MOE_VMW(N) \
  case N:          \
    asm volatile("s_waitcnt vmcnt(" #N ")" ::: "memory"); \
    break;
    MOE_VMW(0) MOE_VMW(1) MOE_VMW(2) MOE_VMW(3) MOE_VMW(4) MOE_VMW(5) MOE_VMW(6) MOE_VMW(7)
    MOE_VMW(8) MOE_VMW(9) MOE_VMW(10) MOE_VMW(11) MOE_VMW(12) MOE_VMW(13) MOE_VMW(14)
    MOE_VMW(15) MOE_VMW(16) MOE_VMW(17) MOE_VMW(18) MOE_VMW(19) MOE_VMW(20) MOE_VMW(21)
    MOE_VMW(22) MOE_VMW(23) MOE_VMW(24) MOE_VMW(25) MOE_VMW(26) MOE_VMW(27)
#undef MOE_VMW
    default:
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
}

// ---- one tile's k loop --------------------------------------------------------
// acc[blk][m] += X[rows of block m] . W[16 columns of block blk]^T over Kdim.
// Ring slot c % kNBuf holds chunk c: the tile's activation rows (srows of
// them, 16-byte pieces XOR-swizzled by row so that the 16 rows an MFMA
// operand reads sit on different banks) and every wave's codes and (s, z).
// xsrc(row, k): global address of 8 activations (pair order) of row `row` at
// k; qsrc(blk, k): this lane's 16 bytes of codes (32 inputs from k);
// ssrc(blk, k): its (s, z) word.
template <typename XSrc, typename QSrc, typename SSrc>
__device__ __forceinline__ void tile_gemm(char* ring, int Kdim, int mb, XSrc xsrc, QSrc qsrc,
                                          SSrc ssrc, f4 (*acc)[4]) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int col = lane & 15, kq = lane >> 4;
  const int nch = Kdim / kGK;
  const int nxi = 4 * mb;                                  // activation copies per chunk
  const int my_x = (nxi - wave + kGW - 1) / kGW;           // this wave's share of them
  const int per_chunk = my_x + 2 * kNBlk;                  // this wave's copies per chunk
  auto xslot = [&](int c) { return ring + (c % kNBuf) * kXSlot; };
  auto wslot = [&](int c) {
    return ring + kNBuf * kXSlot + ((c % kNBuf) * kGW + wave) * kNBlk * kWBlk;
  };
  auto issue = [&](int c) {
    const int k0 = c * kGK;
    char* xs = xslot(c);
    for (int b = wave; b < nxi; b += kGW) {  // 64 pieces: rows 4b .. 4b+3
      const int p = b * 64 + lane, row = p >> 4, phys = p & 15;
      dma16(xsrc(row, k0 + 8 * (phys ^ (row & 15))), xs + b * 1024);
    }
    char* ws = wslot(c);
#pragma unroll
    for (int blk = 0; blk < kNBlk; ++blk) {
      dma16(qsrc(blk, k0 + kq * 32), ws + blk * kWBlk);
      dma4(ssrc(blk, k0 + kq * 32), ws + blk * kWBlk + 1024);
    }
  };
  vm_drain();
  for (int c = 0; c < nch && c < kNBuf - 1; ++c) issue(c);
  for (int c = 0; c < nch; ++c) {
    const int ahead = min(nch - 1 - c, kNBuf - 2);  // chunks issued after c
    vm_wait(ahead * per_chunk);
    __syncthreads();  // chunk c is in LDS for every wave; chunk c - 1 is consumed
    if (c + kNBuf - 1 < nch) issue(c + kNBuf - 1);  // into the slot of chunk c - 1
    const char* xs = xslot(c);
    const char* ws = wslot(c);
    U4 q[kNBlk];
    h2v s2[kNBlk], z2[kNBlk];
#pragma unroll
    for (int blk = 0; blk < kNBlk; ++blk) {
      q[blk] = *reinterpret_cast<const U4*>(ws + blk * kWBlk + lane * 16);
      const h2v sz = as_h2(*reinterpret_cast<const uint32_t*>(ws + blk * kWBlk + 1024 + lane * 4));
      s2[blk] = h2v{sz[0], sz[0]};
      z2[blk] = h2v{sz[1], sz[1]};
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      h8 af[4];
#pragma unroll
      for (int m = 0; m < 4; ++m)
        if (m < mb) {
          const int row = 16 * m + col;
          af[m] = *reinterpret_cast<const h8*>(xs + row * 256 + (((kq * 4 + j) ^ col) * 16));
        }
#pragma unroll
      for (int blk = 0; blk < kNBlk; ++blk) {
        const uint32_t word = j == 0 ? q[blk].x : j == 1 ? q[blk].y : j == 2 ? q[blk].z : q[blk].w;
        const h8 w = dequant8(word, s2[blk], z2[blk]);
#pragma unroll
        for (int m = 0; m < 4; ++m)
          if (m < mb) acc[blk][m] = mfma(af[m], w, acc[blk][m]);
      }
    }
  }
  __syncthreads();  // the ring is free again
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(1024) grouped_permute_kernel(GroupedArgs a) {
  __shared__ int cnt[kGroupMaxG];
  __shared__ int scr[2][1024];
  __shared__ int sct[2][1024];
  const int tid = threadIdx.x;
  const int G = a.E + a.S;
  for (int g = tid; g < G; g += 1024) cnt[g] = g >= a.E ? a.T : 0;
  __syncthreads();
  const int TK = a.T * a.K;
  for (int i = tid; i < TK; i += 1024) {
    const int e = a.idx[i];
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
  auto emit = [&](int g, int c, int off, int toff) {
    if (g >= G || c == 0) return;
    const int slot = a.slot_of[g];
    if (slot < 0 && a.status) atomicOr(a.status, MOE_STATUS_SLOT_MISS);
    for (int j = 0; j * kGroupRows < c; ++j)
      a.tiles[toff + j] = GroupTile{g, off + kGroupRows * j, min(kGroupRows, c - kGroupRows * j), slot};
  };
  emit(g0, c0, off0, toff0);
  emit(g1, c1, off0 + c0, toff0 + t0);
  __syncthreads();  // every count is read: the array becomes the insertion cursors
  if (g0 < G) cnt[g0] = off0;
  if (g1 < G) cnt[g1] = off0 + c0;
  if (tid == 0) *a.n_tiles = total_tiles;
  __syncthreads();
  for (int i = tid; i < TK; i += 1024) {
    const int e = a.idx[i];
    const int t = i / a.K, k = i - t * a.K;
    const int row = t * a.n_list + k;
    if (e >= 0 && e < a.E) {
      a.perm[atomicAdd(&cnt[e], 1)] = row;
    } else {  // an id outside [0, E) contributes zeros and is reported
      if (a.status) atomicOr(a.status, MOE_STATUS_BAD_INDEX);
      float* y = a.y_experts + (size_t)row * a.d;
      for (int j = 0; j < a.d; ++j) y[j] = 0.f;
    }
  }
  for (int i = tid; i < a.T * a.S; i += 1024) {
    const int s = i / a.T, t = i - s * a.T;
    a.perm[cnt[a.E + s] + t] = t * a.n_list + a.K + s;
  }
}

// ---------------------------------------------------------------------------
// prep: blocks [0, xb) write x in pair order; blocks [xb, xb + max_tiles) form
// A_g x and A_u x of one tile: waves 4c .. 4c+3 take projection c, each over a
// quarter of d, with MFMA (ranks as the 16 columns), then the quarters add up.
__global__ void __launch_bounds__(kGT) grouped_prep_kernel(GroupedArgs a, int xb) {
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
  const int ti = blockIdx.x - xb;
  if (ti >= *a.n_tiles) return;
  const GroupTile tl = a.tiles[ti];
  if (tl.slot < 0 || a.r <= 0) return;
  const moe_bundle* bd = a.bundles + tl.slot;
  const int wave = tid >> 6, lane = tid & 63, col = lane & 15, kq = lane >> 4;
  const int c = wave >> 2, quarter = wave & 3;
  const int d = a.d, r = a.r;
  const int mb = (tl.nrows + 15) >> 4;
  const void* A = c == 0 ? bd->gate.lora_a : bd->up.lora_a;
  const void* Bm = c == 0 ? bd->gate.lora_b : bd->up.lora_b;
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
      const int t = row < tl.nrows ? a.perm[tl.row0 + row] / a.n_list : -1;
      xrow[m] = t >= 0 ? reinterpret_cast<const _Float16*>(a.x) + (size_t)t * d : nullptr;
    }
    const int kbeg = quarter * (d / 4), kend = kbeg + d / 4;
    for (int k = kbeg + kq * 8; k < kend; k += 32) {
      const h8 b = arow ? as_h8(ld16(arow + k)) : h8{};
#pragma unroll
      for (int m = 0; m < 4; ++m)
        if (m < mb) {
          const h8 av = xrow[m] ? as_h8(ld16(xrow[m] + k)) : h8{};
          acc[m] = mfma(av, b, acc[m]);
        }
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
    a.ax[((size_t)(tl.row0 + row) * 2 + cc) * 16 + k] = v;
  }
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kGT) grouped_gateup_kernel(GroupedArgs a) {
  extern __shared__ __attribute__((aligned(16))) char ring[];
  __shared__ __attribute__((aligned(16))) _Float16 la[2][kGroupRows][16];
  __shared__ int rsrc[kGroupRows];
  // after the k loop the ring holds h of the tile and the A_d rows
  _Float16(*hs)[kGateCols] = reinterpret_cast<_Float16(*)[kGateCols]>(ring);
  _Float16(*ads)[kGateCols] = reinterpret_cast<_Float16(*)[kGateCols]>(ring + kGroupRows * kGateCols * 2);
  static_assert((kGroupRows + 16) * kGateCols * 2 <= kRingBytes, "h and A_d rows fit in the ring");
  if ((int)blockIdx.x >= *a.n_tiles) return;
  const GroupTile tl = a.tiles[blockIdx.x];
  if (tl.slot < 0) return;  // not resident: the down kernel writes zero rows
  const moe_bundle* bd = a.bundles + tl.slot;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, kq = lane >> 4;
  const int d = a.d, I = a.I, r = a.r;
  const int mb = (tl.nrows + 15) >> 4;
  const int c0 = blockIdx.y * kGateCols;        // first column of this workgroup
  const int i = c0 + wave * 16 + col;           // this lane's gate/up column
  if (tid < kGroupRows) rsrc[tid] = tid < tl.nrows ? a.perm[tl.row0 + tid] / a.n_list : -1;
  const bool lg = r > 0 && bd->gate.lora_a && bd->gate.lora_b;
  const bool lu = r > 0 && bd->up.lora_a && bd->up.lora_b;
  const bool ld = r > 0 && bd->down.lora_a && bd->down.lora_b;
  // lora_scale * (A x) of the tile's rows, fp16 (rank past r: zero)
  for (int p = tid; p < 2 * kGroupRows * 16; p += kGT) {
    const int cc = p / (kGroupRows * 16), row = (p >> 4) % kGroupRows, k = p & 15;
    float v = 0.f;
    if (row < tl.nrows && k < r && (cc == 0 ? lg : lu))
      v = a.lora_scale * a.ax[((size_t)(tl.row0 + row) * 2 + cc) * 16 + k];
    la[cc][row][k] = (_Float16)v;
  }
  __syncthreads();

  const uint8_t* qb[2] = {static_cast<const uint8_t*>(bd->gate.q) + (size_t)i * (d / 2),
                          static_cast<const uint8_t*>(bd->up.q) + (size_t)i * (d / 2)};
  const uint8_t* sb[2] = {static_cast<const uint8_t*>(bd->gate.sz) + (size_t)i * (d / 16),
                          static_cast<const uint8_t*>(bd->up.sz) + (size_t)i * (d / 16)};
  const char* xbase = reinterpret_cast<const char*>(a.xp);
  auto xsrc = [&](int row, int k) -> const void* {
    const int t = rsrc[row < tl.nrows ? row : 0];
    return xbase + ((size_t)t * d + k) * 2;
  };
  auto qsrc = [&](int blk, int k) -> const void* { return qb[blk] + k / 2; };
  auto ssrc = [&](int blk, int k) -> const void* { return sb[blk] + (k / 64) * 4; };

  f4 acc[2][4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    acc[0][m] = f4{0.f, 0.f, 0.f, 0.f};
    acc[1][m] = acc[0][m];
  }
  tile_gemm(ring, d, mb, xsrc, qsrc, ssrc, acc);

  // LoRA delta: one MFMA step of K = rank against lora_scale * (A x)
#pragma unroll
  for (int cc = 0; cc < 2; ++cc) {
    if (!(cc == 0 ? lg : lu)) continue;
    const h8 bop = lora_b_operand(static_cast<const __half*>(cc == 0 ? bd->gate.lora_b : bd->up.lora_b),
                                  i, r, kq);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (m >= mb) continue;
      h8 aop = {};
      if (kq < 2) aop = *reinterpret_cast<const h8*>(&la[cc][16 * m + col][kq * 8]);
      acc[cc][m] = mfma(aop, bop, acc[cc][m]);
    }
  }
  // A_d rows restricted to this workgroup's columns (the ring is free now)
  for (int p = tid; p < 16 * kGateCols; p += kGT) {
    const int k = p / kGateCols, cc = p % kGateCols;
    ads[k][cc] = (ld && k < r) ? reinterpret_cast<const _Float16*>(bd->down.lora_a)[(size_t)k * I + c0 + cc]
                               : (_Float16)0.f;
  }
  // h = silu(g) u, fp16: to HBM in pair order, and to LDS for A_d h
  const int ip = (i & ~7) | pair_slot(i & 7);
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    if (m >= mb) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 16 * m + 4 * kq + e;
      const float g = acc[0][m][e], u = acc[1][m][e];
      const __half h = __float2half(g / (1.0f + expf(-g)) * u);
      if (row < tl.nrows) a.h[(size_t)(tl.row0 + row) * I + ip] = h;
      hs[row][wave * 16 + col] = h;
    }
  }
  __syncthreads();
  // the slab's partial A_d h: row x rank over this workgroup's columns
  if (ld) {
    for (int p = tid; p < tl.nrows * 16; p += kGT) {
      const int row = p >> 4, k = p & 15;
      float s = 0.f;
      for (int cc = 0; cc < kGateCols; ++cc) s = fmaf((float)ads[k][cc], (float)hs[row][cc], s);
      a.adp[((size_t)(tl.row0 + row) * (I / kSlab) + blockIdx.y) * 16 + k] = s;
    }
  }
}

__global__ void __launch_bounds__(kGT) grouped_down_kernel(GroupedArgs a) {
  extern __shared__ __attribute__((aligned(16))) char ring[];
  __shared__ __attribute__((aligned(16))) _Float16 la[kGroupRows][16];
  __shared__ int ydst[kGroupRows];
  if ((int)blockIdx.x >= *a.n_tiles) return;
  const GroupTile tl = a.tiles[blockIdx.x];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, kq = lane >> 4;
  const int d = a.d, I = a.I, r = a.r;
  const int mb = (tl.nrows + 15) >> 4;
  const int n0 = blockIdx.y * kDownCols + wave * 32 + col;  // columns n0 and n0 + 16 of this lane
  if (tid < kGroupRows) ydst[tid] = tid < tl.nrows ? a.perm[tl.row0 + tid] : -1;
  __syncthreads();
  if (tl.slot < 0) {  // not resident: the pair contributes zeros (the miss is reported)
    for (int p = tid; p < tl.nrows * kDownCols; p += kGT) {
      const int row = p / kDownCols, c = p % kDownCols;
      a.y_experts[(size_t)ydst[row] * d + blockIdx.y * kDownCols + c] = 0.f;
    }
    return;
  }
  const moe_bundle* bd = a.bundles + tl.slot;
  const bool ld = r > 0 && bd->down.lora_a && bd->down.lora_b;
  // lora_scale * (A_d h) of the tile's rows: the slab partials in slab order
  for (int p = tid; p < kGroupRows * 16; p += kGT) {
    const int row = p >> 4, k = p & 15;
    float v = 0.f;
    if (ld && row < tl.nrows && k < r) {
      const float* q = a.adp + (size_t)(tl.row0 + row) * (I / kSlab) * 16 + k;
      for (int sl = 0; sl < I / kSlab; ++sl) v += q[sl * 16];
      v *= a.lora_scale;
    }
    la[row][k] = (_Float16)v;
  }
  const uint8_t* qb[2] = {static_cast<const uint8_t*>(bd->down.q) + (size_t)n0 * (I / 2),
                          static_cast<const uint8_t*>(bd->down.q) + (size_t)(n0 + 16) * (I / 2)};
  const uint8_t* sb[2] = {static_cast<const uint8_t*>(bd->down.sz) + (size_t)n0 * (I / 16),
                          static_cast<const uint8_t*>(bd->down.sz) + (size_t)(n0 + 16) * (I / 16)};
  const char* hbase = reinterpret_cast<const char*>(a.h);
  auto xsrc = [&](int row, int k) -> const void* {
    return hbase + ((size_t)(tl.row0 + (row < tl.nrows ? row : 0)) * I + k) * 2;
  };
  auto qsrc = [&](int blk, int k) -> const void* { return qb[blk] + k / 2; };
  auto ssrc = [&](int blk, int k) -> const void* { return sb[blk] + (k / 64) * 4; };

  f4 acc[2][4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    acc[0][m] = f4{0.f, 0.f, 0.f, 0.f};
    acc[1][m] = acc[0][m];
  }
  tile_gemm(ring, I, mb, xsrc, qsrc, ssrc, acc);  // its barriers also publish la

  if (ld) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const h8 bop = lora_b_operand(static_cast<const __half*>(bd->down.lora_b), n0 + 16 * c, r, kq);
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        if (m >= mb) continue;
        h8 aop = {};
        if (kq < 2) aop = *reinterpret_cast<const h8*>(&la[16 * m + col][kq * 8]);
        acc[c][m] = mfma(aop, bop, acc[c][m]);
      }
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
        y[n0 + 16] = acc[1][m][e];
      }
    }
  }
}

}  // namespace

bool grouped_shape_supported(int d, int I, int r, int groups) {
  return d % kDownCols == 0 && I % kGateCols == 0 && d % kGK == 0 && I % kGK == 0 && r >= 0 &&
         r <= kGroupMaxR && groups <= kGroupMaxG;
}

hipError_t launch_grouped_ffn(const GroupedArgs& a, hipStream_t st) {
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)grouped_gateup_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kRingBytes);
    if (e == hipSuccess)
      e = hipFuncSetAttribute((const void*)grouped_down_kernel,
                              hipFuncAttributeMaxDynamicSharedMemorySize, kRingBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(grouped_permute_kernel, dim3(1), dim3(1024), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int xb = (int)(((size_t)a.T * a.d / 8 + kGT - 1) / kGT);
  hipLaunchKernelGGL(grouped_prep_kernel, dim3(xb + a.max_tiles), dim3(kGT), 0, st, a, xb);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(grouped_gateup_kernel, dim3(a.max_tiles, a.I / kGateCols), dim3(kGT), kRingBytes,
                     st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(grouped_down_kernel, dim3(a.max_tiles, a.d / kDownCols), dim3(kGT), kRingBytes,
                     st, a);
  return hipGetLastError();
}

}  // namespace moe
