// prefill_common.h -- pieces shared by the chunked prefill kernels (gfx950):
// chunk numbering, tile shapes, the in-chunk token order of the contractions,
// the swizzled K/Q/V tile layout in LDS and the matrix-operand builders that
// read it.
#pragma once

#include "gdn_device.h"

namespace gdn {

// ============================================================ chunk numbering
// Chunks get global slots without a scan: sequence n owns the slots
// cu[n] / C + n + [0, ceil(len_n / C)). Consecutive ranges never overlap
// (cu[n+1] / C + n + 1 >= cu[n] / C + n + ceil(len_n / C)) and every slot is
// below ceil(T / C) + N, so per-chunk tables sized by that bound suffice.
__device__ __forceinline__ int64_t first_slot(const int32_t *cu, int n, int chunk) {
  return (int64_t)cu[n] / chunk + n;
}

template <int D, int C>
struct Cfg {
  static constexpr int NIB = C / 16;           // 16-token blocks per chunk
  static constexpr int KS = (C + 31) / 32;     // 32-token contraction steps
  static constexpr int CP = KS * 32;           // chunk padded to the step
  static constexpr int DS = D / 32;            // 32-wide steps over the head dim
  static constexpr int NKT = D / 16;           // 16-wide key tiles of the state
  static constexpr int KTW = (NKT + 3) / 4;    // key tiles per wavefront
  static constexpr int NVT = D / 16;           // 16-row value tiles per head
  static constexpr int LDK = D + 8;            // bf16 pitch, padded K/Q tiles
  static constexpr int LDA = C + 4;            // f32 pitch, C x C tiles
  static constexpr int LDV = CP + 8;           // bf16 pitch, [value][token] tiles
  static constexpr int FRAG = NIB * KS * 512;  // bf16 elements per C x C operand
  static constexpr int PIECES = (C / 4) * (D / 8);  // 4-row x 8-column K pieces
  static_assert(PIECES <= 256, "one K piece per thread");
  static_assert(C % 16 == 0 && C <= 64 && D % 32 == 0 && D <= 128, "shape");
};

// Every contraction over the tokens of a chunk (T Y, P U, K^T Uh) uses one
// order of the tokens inside each 32-token block: position p = 8 g + 4 h + e
// holds token j = 16 h + 4 g + e (g, e in [0, 4), h in {0, 1}). It is the
// order in which a 16x16 accumulator tile pair hands out its rows, so tiles
// produced by one product feed the next without a transpose.
__device__ __forceinline__ int tok_pos(int j) {
  const int r = j & 31;
  return (j & ~31) + 8 * ((r >> 2) & 3) + 4 * (r >> 4) + (r & 3);
}

// ============================================================ swizzled tiles
// Element index of (row, column) in a swizzled row-major [rows][D] bf16 tile:
// 16-byte chunks are XORed with a row function so that 16 consecutive rows
// at one column (matrix-operand reads) fall on distinct bank groups.
template <int D>
__device__ __forceinline__ int kn_swizzle(int row) {
  return ((row & 15) ^ ((row >> 4) & 3)) & (D / 8 - 1);
}
template <int D>
__device__ __forceinline__ int kn_index(int row, int col) {
  return row * D + 8 * ((col >> 3) ^ kn_swizzle<D>(row)) + (col & 7);
}

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ uint2 pack4_bf16(float a, float b, float c, float d) {
  return make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// K^T as the A operand of the state update for key tile t, token step s:
// lane (l16, g4) gets K[j][16 t + l16] for the 8 tokens at positions
// 32 s + 8 g4 + [0, 8). Each transpose load serves 4 tokens: lanes 4m..4m+3
// of a 16-lane group point at token j_m, key columns 16 t + 4 (l16 % 4) + [0,4).
template <int D>
__device__ __forceinline__ uint4 kt_operand(const uint16_t *Kn, int t, int s,
                                            int l16, int g4) {
  uint32_t w[4];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int j = 32 * s + 16 * hh + 4 * g4 + (l16 >> 2);
    const uint16_t *p = Kn + kn_index<D>(j, 16 * t + 4 * (l16 & 3));
    const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4i16 *)(const_cast<uint16_t *>(p)));
    w[2 * hh] = (uint32_t)(uint16_t)x[0] | ((uint32_t)(uint16_t)x[1] << 16);
    w[2 * hh + 1] = (uint32_t)(uint16_t)x[2] | ((uint32_t)(uint16_t)x[3] << 16);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

constexpr uint32_t kOutOfRange = 0x80000000u;  // beyond every resource: reads 0

// Waits until at most N of this wavefront's vector-memory operations are
// outstanding (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work-group barrier that lets the youngest N LDS operations of this
// wavefront stay in flight. LDS operations complete in issue order, so every
// LDS access issued before those N (a state write, say) is complete and
// visible to the other wavefronts after the barrier.
template <int N>
__device__ __forceinline__ void lds_barrier_keep() {
  static_assert(N >= 0 && N <= 15, "LDS counter range");
  asm volatile("s_waitcnt lgkmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// T' (and P) fragments of block row ib that are not all zero: steps s <= ib/2.
template <int C>
__device__ __forceinline__ constexpr int frag_steps(int ib) {
  return (ib / 2 + 1) < (C + 31) / 32 ? (ib / 2 + 1) : (C + 31) / 32;
}

// B operand of a contraction over the chunk's tokens, step st: blocks 2 st
// (slots 0-3) and 2 st + 1 (slots 4-7) of accumulator tiles X, each element
// times w[block][e] (or as is when w is null), rounded to bf16.
template <int NIB>
__device__ __forceinline__ uint4 u_operand(const f32x4 (&X)[NIB], int st, const f32x4 *w) {
  const int b0 = 2 * st, b1 = 2 * st + 1;
  f32x4 lo = X[b0 % NIB], hi = (b1 < NIB) ? X[b1 % NIB] : f32x4{0.f, 0.f, 0.f, 0.f};
  if (w != nullptr) {
    lo = lo * w[b0 % NIB];
    if (b1 < NIB) hi = hi * w[b1 % NIB];
  }
  return make_uint4(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]),
                    pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]));
}

// 16 x 32 A operand of a key contraction, rows from a row-major matrix:
// lane (l16, g4) gives row l16, keys 32 s + 4 g4 + [0, 4) and
// 32 s + 16 + 4 g4 + [0, 4).
__device__ __forceinline__ uint4 key_operand(uint2 lo, uint2 hi) {
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

// 16-byte piece m of a K (or Q, V) chunk copied into a swizzled LDS tile by
// buffer-to-LDS loads: lane i of copy m fills bytes [16 i, 16 i + 16) of the
// tile's 1 KB piece m, so its source offset picks the global 16-byte piece
// that belongs at that swizzled position. `stride` is the element distance
// between consecutive token rows in global memory.
template <int D>
__device__ __forceinline__ uint32_t tile_copy_offset(int m, int lane, int stride) {
  constexpr int KPR = D / 8;  // 16-byte pieces per row
  const int u = 64 * m + lane, row = u / KPR;
  const int jl = (u % KPR) ^ kn_swizzle<D>(row);
  return (uint32_t)((row * stride + 8 * jl) * 2);
}

}  // namespace gdn
