// Batched decode / prefill expert path for gfx950.
//
// The math is the one-token expert FFN (Sec. 3.1, Math contract; Sec. 3.3
// unmerged LoRA) applied to every (token, expert) pair of a batch; grouping by
// expert is what makes it a dense contraction (the whole-layer executor path
// of Sec. 3.1 loads every expert of a layer for a prefill chunk).
//
//   permute   one workgroup: per-expert counts, scans, 64-row tiles, and the
//             permuted list of y_experts rows (token t, list position k).
//   gate/up   per tile x 64 columns: G = X W_g^T, U = X W_u^T over the tile's
//             rows with v_mfma_f32_16x16x32_f16; the int4 codes are dequantized
//             to fp16 in registers (w = s q + z, one rounding); A_g x and A_u x
//             ride along as one more 16-column block on waves 0 and 1; the LoRA
//             delta is one extra MFMA step with K = the rank (B rows against
//             lora_scale * A x); epilogue h = silu(g) u, stored fp16.
//   down      per tile x 128 columns: Y = H W_d^T the same way, with A_d h on
//             wave 0 and the B_d step; fp32 rows go straight to y_experts.
//
// The k order inside each 8-element MFMA operand is permuted to
// [0,4,1,5,2,6,3,7] on both operands: that is the order in which the packed
// nibbles of one dword come out of two mask/or operations per pair, so the
// activations are permuted once when they are staged in LDS.  Every output
// row depends only on its own input row, so the order of rows inside a group
// does not change any result bit.
#include "moe_grouped.h"

namespace moe {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2v __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kGK = 128;                 // k per staged chunk
constexpr int kGRowB = kGK * 2 + 16;     // LDS bytes per staged row (16 B pad: no bank conflicts)
constexpr int kGThreads = 256;

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

// Eight int4 codes of one dword (nibble m = input m) -> fp16 weights
// s q + z in the order [0,4,1,5,2,6,3,7].  0x6400 | q is the fp16 value
// 1024 + q, so subtracting 1024 gives q exactly; the fma rounds once.
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
// Staging of one k-chunk of the tile's input rows into LDS, permuted.  Thread
// `tid` moves pieces p = tid + 256 q (row p / 16, 16-byte piece p % 16).
struct Stager {
  U4 v[4];
  template <typename RowPtr>
  __device__ __forceinline__ void load(RowPtr row_ptr, int srows, int k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int p = threadIdx.x + kGThreads * q;
      const int row = p >> 4, c = p & 15;
      const _Float16* src = row < srows ? row_ptr(row) : nullptr;
      v[q] = src ? ld16(src + k0 + c * 8) : U4{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(char* buf, int srows) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int p = threadIdx.x + kGThreads * q;
      const int row = p >> 4, c = p & 15;
      if (row < srows) *reinterpret_cast<U4*>(buf + row * kGRowB + c * 16) = perm8(v[q]);
    }
  }
};

// Operands of NB int4 column blocks plus an optional raw fp16 LoRA-A block
// for one k-chunk of one lane: lane (col, kq) holds the 32 codes of inputs
// k0 + kq*32 .. +32 of its weight row, and the (scale, zero) of their group.
template <int NB>
struct ChunkB {
  U4 q[NB];
  uint32_t sz[NB];
  U4 l[4];
};

template <int NB>
__device__ __forceinline__ void load_chunk(ChunkB<NB>& b, const uint8_t* const* qrow,
                                           const uint32_t* const* szrow, const _Float16* lrow,
                                           int k0) {
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    b.q[c] = ld16(qrow[c] + k0 / 2);
    b.sz[c] = szrow[c][k0 / 64];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j)  // ranks past r stay exactly zero (0 * NaN garbage would not)
    b.l[j] = lrow ? ld16(lrow + k0 + 8 * j) : U4{0, 0, 0, 0};
}

// One staged chunk: 4 MFMA k-steps of 32 over mb row blocks.
template <int NB>
__device__ __forceinline__ void compute_chunk(const char* buf, const ChunkB<NB>& b, bool lora,
                                              int mb, int col, int kq, f4 (*acc)[4], f4* acl) {
  h2v s2[NB], z2[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    const h2v sz = as_h2(b.sz[c]);
    s2[c] = h2v{sz[0], sz[0]};
    z2[c] = h2v{sz[1], sz[1]};
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    h8 af[4];
#pragma unroll
    for (int m = 0; m < 4; ++m)
      if (m < mb)
        af[m] = *reinterpret_cast<const h8*>(buf + (16 * m + col) * kGRowB + (kq * 32 + j * 8) * 2);
#pragma unroll
    for (int c = 0; c < NB; ++c) {
      const uint32_t word = j == 0 ? b.q[c].x : j == 1 ? b.q[c].y : j == 2 ? b.q[c].z : b.q[c].w;
      const h8 w = dequant8(word, s2[c], z2[c]);
#pragma unroll
      for (int m = 0; m < 4; ++m)
        if (m < mb) acc[c][m] = mfma(af[m], w, acc[c][m]);
    }
    if (lora) {
      const h8 w = as_h8(perm8(b.l[j]));
#pragma unroll
      for (int m = 0; m < 4; ++m)
        if (m < mb) acl[m] = mfma(af[m], w, acl[m]);
    }
  }
}

// Runs the k loop of one tile: rows from row_ptr(row) (fp16, K elements),
// NB int4 column blocks, optional LoRA-A block lrow.  Double-buffered LDS
// staging of the rows; the next chunk's weights are loaded before this
// chunk is computed.
template <int NB, typename RowPtr>
__device__ __forceinline__ void tile_k_loop(char (*xs)[kGroupRows * kGRowB], RowPtr row_ptr,
                                            int srows, int Kdim, const uint8_t* const* qrow,
                                            const uint32_t* const* szrow, const _Float16* lrow,
                                            bool lora, int mb, int col, int kq, f4 (*acc)[4],
                                            f4* acl) {
  const int nch = Kdim / kGK;
  Stager st;
  ChunkB<NB> cur, nxt;
  st.load(row_ptr, srows, 0);
  load_chunk<NB>(cur, qrow, szrow, lrow, kq * 32);
  st.store(xs[0], srows);
  for (int c = 0; c < nch; ++c) {
    const bool more = c + 1 < nch;
    if (more) {
      st.load(row_ptr, srows, (c + 1) * kGK);
      load_chunk<NB>(nxt, qrow, szrow, lrow, (c + 1) * kGK + kq * 32);
    }
    __syncthreads();
    compute_chunk<NB>(xs[c & 1], cur, lora, mb, col, kq, acc, acl);
    if (more) {
      st.store(xs[(c + 1) & 1], srows);
      cur = nxt;
    }
  }
}

__global__ void __launch_bounds__(kGThreads) grouped_gateup_kernel(GroupedArgs a) {
  __shared__ __attribute__((aligned(16))) char xs[2][kGroupRows * kGRowB];
  __shared__ __attribute__((aligned(16))) _Float16 la[2][kGroupRows][16];
  __shared__ int rsrc[kGroupRows];
  if ((int)blockIdx.x >= *a.n_tiles) return;
  const GroupTile tl = a.tiles[blockIdx.x];
  if (tl.slot < 0) return;  // not resident: the down kernel writes zero rows
  const moe_bundle* bd = a.bundles + tl.slot;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, kq = lane >> 4;
  const int d = a.d, I = a.I, r = a.r;
  const int mb = (tl.nrows + 15) >> 4, srows = mb * 16;
  const int i = blockIdx.y * 64 + wave * 16 + col;  // this lane's gate/up column
  if (tid < kGroupRows) rsrc[tid] = tid < tl.nrows ? a.perm[tl.row0 + tid] / a.n_list : -1;

  const uint8_t* qrow[2] = {static_cast<const uint8_t*>(bd->gate.q) + (size_t)i * (d / 2),
                            static_cast<const uint8_t*>(bd->up.q) + (size_t)i * (d / 2)};
  const uint32_t* szrow[2] = {static_cast<const uint32_t*>(bd->gate.sz) + (size_t)i * (d / 64),
                              static_cast<const uint32_t*>(bd->up.sz) + (size_t)i * (d / 64)};
  const bool lg = r > 0 && bd->gate.lora_a && bd->gate.lora_b;
  const bool lu = r > 0 && bd->up.lora_a && bd->up.lora_b;
  const bool mine = (wave == 0 && lg) || (wave == 1 && lu);  // LoRA-A block of this wave
  const _Float16* lrow = nullptr;
  if (mine && col < r)
    lrow = static_cast<const _Float16*>(wave == 0 ? bd->gate.lora_a : bd->up.lora_a) + (size_t)col * d;

  f4 acc[2][4], acl[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    acc[0][m] = f4{0.f, 0.f, 0.f, 0.f};
    acc[1][m] = acc[0][m];
    acl[m] = acc[0][m];
  }
  __syncthreads();
  auto row_ptr = [&](int row) -> const _Float16* {
    const int t = rsrc[row];
    return t >= 0 ? reinterpret_cast<const _Float16*>(a.x) + (size_t)t * d : nullptr;
  };
  tile_k_loop<2>(xs, row_ptr, srows, d, qrow, szrow, lrow, mine, mb, col, kq, acc, acl);

  // LoRA delta: one MFMA step of K = rank against lora_scale * (A x)
  if (mine) {
#pragma unroll
    for (int m = 0; m < 4; ++m)
      if (m < mb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          la[wave][16 * m + 4 * kq + e][col] = (_Float16)(a.lora_scale * acl[m][e]);
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    if (!(c == 0 ? lg : lu)) continue;
    const h8 bop = lora_b_operand(static_cast<const __half*>(c == 0 ? bd->gate.lora_b : bd->up.lora_b),
                                  i, r, kq);
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (m >= mb) continue;
      h8 aop = {};
      if (kq < 2) aop = *reinterpret_cast<const h8*>(&la[c][16 * m + col][kq * 8]);
      acc[c][m] = mfma(aop, bop, acc[c][m]);
    }
  }
  // SwiGLU epilogue: h = silu(g) * u, fp16 by permuted row
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    if (m >= mb) continue;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 16 * m + 4 * kq + e;
      if (row < tl.nrows) {
        const float g = acc[0][m][e], u = acc[1][m][e];
        const float h = g / (1.0f + expf(-g)) * u;
        a.h[(size_t)(tl.row0 + row) * I + i] = __float2half(h);
      }
    }
  }
}

__global__ void __launch_bounds__(kGThreads) grouped_down_kernel(GroupedArgs a) {
  __shared__ __attribute__((aligned(16))) char xs[2][kGroupRows * kGRowB];
  __shared__ __attribute__((aligned(16))) _Float16 la[kGroupRows][16];
  __shared__ int ydst[kGroupRows];
  if ((int)blockIdx.x >= *a.n_tiles) return;
  const GroupTile tl = a.tiles[blockIdx.x];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, kq = lane >> 4;
  const int d = a.d, I = a.I, r = a.r;
  const int mb = (tl.nrows + 15) >> 4, srows = mb * 16;
  const int n0 = blockIdx.y * 128 + wave * 32 + col;  // columns n0 and n0 + 16 of this lane
  if (tid < kGroupRows) ydst[tid] = tid < tl.nrows ? a.perm[tl.row0 + tid] : -1;
  __syncthreads();
  if (tl.slot < 0) {  // not resident: the pair contributes zeros (the miss is reported)
    for (int p = tid; p < tl.nrows * 128; p += kGThreads) {
      const int row = p >> 7, c = p & 127;
      a.y_experts[(size_t)ydst[row] * d + blockIdx.y * 128 + c] = 0.f;
    }
    return;
  }
  const moe_bundle* bd = a.bundles + tl.slot;
  const uint8_t* qrow[2] = {static_cast<const uint8_t*>(bd->down.q) + (size_t)n0 * (I / 2),
                            static_cast<const uint8_t*>(bd->down.q) + (size_t)(n0 + 16) * (I / 2)};
  const uint32_t* szrow[2] = {static_cast<const uint32_t*>(bd->down.sz) + (size_t)n0 * (I / 64),
                              static_cast<const uint32_t*>(bd->down.sz) + (size_t)(n0 + 16) * (I / 64)};
  const bool ld = r > 0 && bd->down.lora_a && bd->down.lora_b;
  const bool mine = wave == 0 && ld;
  const _Float16* lrow = nullptr;
  if (mine && col < r) lrow = static_cast<const _Float16*>(bd->down.lora_a) + (size_t)col * I;

  f4 acc[2][4], acl[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    acc[0][m] = f4{0.f, 0.f, 0.f, 0.f};
    acc[1][m] = acc[0][m];
    acl[m] = acc[0][m];
  }
  auto row_ptr = [&](int row) -> const _Float16* {
    return row < tl.nrows ? reinterpret_cast<const _Float16*>(a.h) + (size_t)(tl.row0 + row) * I
                          : nullptr;
  };
  tile_k_loop<2>(xs, row_ptr, srows, I, qrow, szrow, lrow, mine, mb, col, kq, acc, acl);

  if (mine) {
#pragma unroll
    for (int m = 0; m < 4; ++m)
      if (m < mb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          la[16 * m + 4 * kq + e][col] = (_Float16)(a.lora_scale * acl[m][e]);
  }
  __syncthreads();
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
  return d % 128 == 0 && I % 128 == 0 && r >= 0 && r <= kGroupMaxR && groups <= kGroupMaxG;
}

hipError_t launch_grouped_ffn(const GroupedArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(grouped_permute_kernel, dim3(1), dim3(1024), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(grouped_gateup_kernel, dim3(a.max_tiles, a.I / 64), dim3(kGThreads), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(grouped_down_kernel, dim3(a.max_tiles, a.d / 128), dim3(kGThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace moe
