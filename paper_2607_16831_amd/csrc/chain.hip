// chain.hip -- the inter-chunk state carry of the chunked prefill, as
// whole-chain work-groups over segments of a sequence (gfx950, bf16 inputs).
//
// For one chunk of a (sequence, value head) chain with incoming state S
// (d_v x d_k), the chunk-local kernel has stored T' = (I + A)^-1 diag(beta),
// P = lower(E ⊙ Q K^T) and the decay factors exp(gamma), exp(gamma_last -
// gamma). The carry then computes, per chunk,
//
//   X  = K S^T,   U = T' (V - exp(gamma) X),   O = exp(gamma) (Q S^T) + P U,
//   S' = exp(gamma_last) S + (exp(gamma_last - gamma) U)^T K.
//
// Rows of S (value channels) evolve independently, and every row uses the
// same chunk operands (K, Q, T', P, decay). One work-group therefore carries
// ALL d_v rows of a chain: its compute wavefronts own 16 or 32 rows each and
// read the chunk operands from one LDS copy, which a loader wavefront streams
// in ahead of use. The chunk operands are read once per work-group instead of
// once per row tile.
//
// Segments. Whole-chain work-groups leave few work-groups when chains are few
// and long (one sequence of 4096 tokens and 32 value heads: 32 chains of 64
// chunks). The carry is affine in the incoming state: over a segment of
// chunks, S_out = S_in M + B, where M (d_k x d_k) is the product of the
// chunks' transition maps and B is the segment's result from a zero state.
// A sequence is cut into G segments of L chunks, and the work runs in three
// launches:
//   1. the maps of segments 0..G-2, all at once: the B rows of segment s run
//      from the true initial state (s = 0) or from zero, the M rows (s >= 1)
//      from the identity with no value input, so that they become the rows
//      of the product of the chunks' transition maps;
//   2. compose_kernel: S_in(s + 1) = S_in(s) M_s + B_s for s = 1..G-2, in
//      fp32 accumulation with hi/lo bf16 operand splits (S_in(1) = B_0);
//   3. every segment from its incoming state, with outputs.
// The sequential depth drops from the number of chunks to about 2L + G, at
// the price of the M rows and of a second pass over K, V and T'. When no
// sequence can exceed one segment, only launch 3 runs.
//
// Global reads go through buffer resources: rows past the end of a sequence
// read as zero (beta is zero there, so they add exact zeros), and output rows
// past the end are dropped by the resource extent.
#include "gdn_launch.h"
#include "prefill_common.h"

namespace gdn {

// MAPS = true: the first launch, which forms the maps of segments 0..G-2:
// one set of compute wavefronts carries the B rows (the segment from its
// incoming state, which is the true initial state for segment 0 and zero
// otherwise) and a second set the M rows (from the identity, no value
// input; idle for segment 0). MAPS = false: the output launch, one set of
// compute wavefronts carrying every segment from its composed incoming state
// with outputs.
template <int D, int C, bool MAPS>
struct ChainCfg {
  using F = Cfg<D, C>;
  // 16-row value tiles per compute wavefront. One in the output launch: its
  // eight compute wavefronts put two on each SIMD, which hides the latency
  // of the chunk step's dependent LDS reads and products better than four
  // wavefronts of two tiles each (measured on the 66K-token batch of 16
  // sequences: 1.20 -> 1.07 ms per call). Two in the map launch at d = 128,
  // which carries twice the rows and would exceed the work-group size.
  static constexpr int NJ = (D == 128 && MAPS) ? 2 : 1;
  static constexpr int NWR = D / (16 * NJ);     // compute wavefronts per set of D rows
  static constexpr int NCW = MAPS ? 2 * NWR : NWR;  // compute wavefronts
  static constexpr int NT = 64 * (NCW + 2);     // threads: compute, a loader and a prefetcher
  // K, Q and V tiles: rows of P = D + 8 bf16 (see chain_tile_copy_offset),
  // CP rows (those past C stay zero), and room for the last 1 KB copy.
  static constexpr int P = D + 8;               // row pitch, elements
  static constexpr int PPR = D / 8 + 1;         // 16-byte pieces per row, the last one padding
  static constexpr int NKI = (C * PPR + 63) / 64;  // 1 KB copies of a K / Q / V chunk
  static constexpr int TILE = NKI * 512 > F::CP * P ? NKI * 512 : F::CP * P;  // elements
  static constexpr int NB = 2;                  // LDS buffers (chunk i uses buffer i % 2)
  // L2 prefetch of the chunk PFD ahead of the one in use: one 128-byte line
  // per lane and load, over the K, Q and V rows and the T', P and decay
  // tables of that chunk.
  static constexpr int PFD = 2;
  static constexpr int LPR = (D * 2 + 127) / 128;          // lines per token row
  static constexpr int NPT = (C * LPR + 63) / 64;          // prefetch loads per tile
  static constexpr int NPF = 3 * NPT + 3;                  // per chunk
};

template <int D, int C, bool MAPS>
struct ChainLds;

// Output launch: every chunk operand.
template <int D, int C>
struct ChainLds<D, C, false> {
  using F = Cfg<D, C>;
  using H = ChainCfg<D, C, false>;
  uint16_t K[H::NB][H::TILE];  // rows at pitch P; rows C..CP-1 stay zero
  // 16 bytes between the K and Q tiles: at a distance of a multiple of 512
  // bytes the compiler pairs each K-row read with the Q-row read of the same
  // lane address into one two-address LDS read, whose results then need 64
  // register copies per chunk to form the A operands; apart, each read lands
  // in its operand's registers (66K-token batch: 1017 -> 974 us per call).
  uint16_t kq_gap[8];
  uint16_t Q[H::NB][H::TILE];
  uint16_t V[H::NB][H::TILE];
  uint16_t T[H::NB][F::FRAG];  // T' as A-operand fragments (only those on or below the diagonal)
  uint16_t P[H::NB][F::FRAG];  // P, same order
  float dec[H::NB][256];       // exp(gamma_i) [0, C), exp(gamma_last - gamma_i) [C, 2C)
  uint32_t sink[64];           // landing place of the L2 prefetch loads
};

// Map launch: no outputs, so no Q and no P.
template <int D, int C>
struct ChainLds<D, C, true> {
  using F = Cfg<D, C>;
  using H = ChainCfg<D, C, true>;
  uint16_t K[H::NB][H::TILE];
  uint16_t V[H::NB][H::TILE];
  uint16_t T[H::NB][F::FRAG];
  float dec[H::NB][256];
  uint32_t sink[64];
};

// Segment numbering, scan-free like the chunk slots: with span = C L tokens
// per segment, sequence n has G_n = max(1, ceil(len_n / span)) segments in
// slots cu[n] / span + n + [0, G_n) (disjoint; below T / span + N), and the
// maps of its segments 0..G_n-2 live in slots cu[n] / span + [0, G_n - 1)
// (disjoint; below T / span, since G_n - 1 <= floor(len_n / span)).
__device__ __forceinline__ int64_t seg_count(int64_t len, int64_t span) {
  return len <= span ? 1 : (len + span - 1) / span;
}

// ============================================================ chunk tiles
// The K, Q and V tiles of a chunk sit in LDS row by row at a pitch of D + 8
// bf16 (16 bytes of padding per row). The pitch in 16-byte units, D/8 + 1,
// is odd, so the 16 rows of a matrix-operand read (one 16-byte piece per
// row) fall on 16 distinct groups of four banks, as an XOR swizzle would
// arrange; unlike a swizzle, the address of every operand read of a chunk is
// one lane base plus a constant, which the compiler folds into the
// instruction's offset instead of forming an address per read.
//
// The tiles are filled by buffer-to-LDS copies, 16 bytes per lane, lane i of
// copy m landing at piece 64 m + i: the source offset of a piece is that of
// its row and column, and padding pieces (and pieces past the chunk's C
// rows) read out of range, as zeros.
template <int D, int C>
__device__ __forceinline__ uint32_t chain_tile_copy_offset(int m, int lane, int stride) {
  constexpr int PPR = D / 8 + 1;
  const int p = 64 * m + lane, row = p / PPR, pc = p - row * PPR;
  return (pc < D / 8 && row < C) ? (uint32_t)((row * stride + 8 * pc) * 2) : kOutOfRange;
}

// Element index of (row, column) in a tile.
template <int D>
__device__ __forceinline__ int ptile_index(int row, int col) {
  return row * (D + 8) + col;
}

// Rows of a tile as the transposed operand of a contraction over its rows
// (K^T for the state update, V for Y): lane (l16, g4) gets T[j][16 t + l16]
// for the 8 rows at positions 32 s + 8 g4 + [0, 8), in the token order of
// tok_pos. Each transpose load serves 4 rows: lanes 4m..4m+3 of a 16-lane
// group point at row j_m, columns 16 t + 4 (l16 % 4) + [0, 4).
template <int D>
__device__ __forceinline__ uint4 ptile_t_operand(const uint16_t *T, int t, int s, int l16, int g4) {
  uint32_t w[4];
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const int j = 32 * s + 16 * hh + 4 * g4 + (l16 >> 2);
    const uint16_t *p = T + ptile_index<D>(j, 16 * t + 4 * (l16 & 3));
    const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4i16 *)(const_cast<uint16_t *>(p)));
    w[2 * hh] = (uint32_t)(uint16_t)x[0] | ((uint32_t)(uint16_t)x[1] << 16);
    w[2 * hh + 1] = (uint32_t)(uint16_t)x[2] | ((uint32_t)(uint16_t)x[3] << 16);
  }
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// ============================================================ dispatch order
// The output launch runs one work-group per CU (its LDS), and work-groups
// start in block order as CUs free up. In block order (sequence order) a long
// sequence late in the batch starts late and finishes last: 16 sequences of
// U[64, 8192] tokens with 32 value heads give a 175-step span of chunk steps
// where the work is 122 steps per CU. Started longest first (list scheduling
// with the longest jobs first), the same batch spans 130 steps.
//
// chain_order_kernel lists the segment slots in decreasing order of their
// chunk count, for one work-group: a histogram over buckets of the count
// (exact below 960 chunks, then one bucket per power of two), a scan, and a
// scatter through per-bucket cursors (the order inside a bucket is whatever
// the atomics give). Slots that no sequence owns follow as -1. Each slot is
// still carried by exactly one set of work-groups, so the results do not
// depend on the order.
constexpr int kOrderThreads = 1024;
constexpr int kOrderBuckets = 1024;

// Bucket of a segment of `len` chunks, longest first.
__device__ __forceinline__ int order_rank_bucket(int64_t len) {
  const int b = len < 960 ? (int)len : 960 + (63 - __clzll((unsigned long long)len));
  return kOrderBuckets - 1 - b;
}

// Builds the list in one work-group of NTH threads. cursor (kOrderBuckets
// ints) and part (NTH ints) are LDS arrays of the caller.
template <int NTH>
__device__ void build_order(const int32_t *__restrict__ cu, int n_seqs, int chunk, int seg_chunks,
                            int64_t nseg, int32_t *__restrict__ order, int *cursor, int *part) {
  static_assert(kOrderBuckets % NTH == 0, "whole buckets per thread");
  constexpr int BPT = kOrderBuckets / NTH;  // consecutive buckets per thread in the scan
  const int tid = threadIdx.x;
  const int64_t span = (int64_t)chunk * seg_chunks;
  // Every segment s < G of sequence n: slot cu[n] / span + n + s, with
  // min(nch, (s + 1) L) - s L chunks (the slot numbering of chain_kernel).
  auto for_segments = [&](auto &&f) {
    for (int n = tid; n < n_seqs; n += NTH) {
      const int64_t a = cu[n], len = cu[n + 1] - a;
      const int64_t G = seg_count(len, span), nch = (len + chunk - 1) / chunk;
      const int64_t base = a / span + n;
      for (int64_t sg = 0; sg < G; ++sg) {
        const int64_t l = min(nch, (sg + 1) * seg_chunks) - sg * seg_chunks;
        f(base + sg, order_rank_bucket(max(l, (int64_t)0)));
      }
    }
  };
  for (int b = tid; b < kOrderBuckets; b += NTH) cursor[b] = 0;
  __syncthreads();
  for_segments([&](int64_t, int rb) { atomicAdd(&cursor[rb], 1); });
  __syncthreads();
  int loc[BPT], sum = 0;
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    loc[i] = cursor[BPT * tid + i];
    sum += loc[i];
  }
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < NTH; off <<= 1) {  // inclusive scan of the per-thread sums
    const int add = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += add;
    __syncthreads();
  }
  int run = part[tid] - sum;  // first rank of bucket BPT * tid
#pragma unroll
  for (int i = 0; i < BPT; ++i) {
    cursor[BPT * tid + i] = run;
    run += loc[i];
  }
  const int used = part[NTH - 1];
  __syncthreads();
  for_segments([&](int64_t slot, int rb) {
    const int r = atomicAdd(&cursor[rb], 1);
    if (r < nseg) order[r] = (int32_t)slot;  // (always, when cu[N] is the token count)
  });
  for (int64_t r = used + tid; r < nseg; r += NTH) order[r] = -1;
}

// The list on its own, when no composition launch runs to carry it.
__global__ __launch_bounds__(kOrderThreads) void chain_order_kernel(
    const int32_t *__restrict__ cu, int n_seqs, int chunk, int seg_chunks, int64_t nseg,
    int32_t *__restrict__ order) {
  __shared__ int cursor[kOrderBuckets];
  __shared__ int part[kOrderThreads];
  build_order<kOrderThreads>(cu, n_seqs, chunk, seg_chunks, nseg, order, cursor, part);
}

// Y operand of U = T' Y for token step st: Y = V - exp(gamma) X in the token
// order of tok_pos, from the bf16 V operand (transpose reads of the V tile)
// and the X accumulator tiles 2 st (slots 0-3) and 2 st + 1 (slots 4-7).
template <int NIB>
__device__ __forceinline__ uint4 y_operand(uint4 vb, const f32x4 (&X)[NIB], const f32x4 (&ga)[NIB],
                                           int st) {
  const int b0 = 2 * st, b1 = 2 * st + 1;
  const uint32_t w[4] = {vb.x, vb.y, vb.z, vb.w};
  float y[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const uint32_t bits = (e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16);
    y[e] = __uint_as_float(bits);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) y[e] -= ga[b0 % NIB][e] * X[b0 % NIB][e];
  if (b1 < NIB) {
#pragma unroll
    for (int e = 0; e < 4; ++e) y[4 + e] -= ga[b1 % NIB][e] * X[b1 % NIB][e];
  }
  return make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                    pack_bf16x2(y[6], y[7]));
}

// Scheduling: N pairs of (one LDS read, one matrix product) in a scheduling
// region, so that a wavefront issues its operand reads between its matrix
// products instead of stalling on a burst of reads before them.
#define GDN_INTERLEAVE_DS_MFMA(N)                            \
  _Pragma("unroll") for (int ilv_ = 0; ilv_ < (N); ++ilv_) { \
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);       \
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);       \
  }

// What one work-group's compute wavefronts do (uniform over it).
struct ChainTask {
  const float *src;    // incoming state [D][D] (null: zero, unless identity)
  bool identity;       // incoming "state" = I (the rows of a segment map)
  int nlc, lc0;        // chunks of the segment: lc0 .. lc0 + nlc - 1
  int64_t seq_t0, seq_t1;
  int h, hv;
  float *dst;          // outgoing state [D][D], or null
  uint16_t *dhi, *dlo; // outgoing map, transposed, bf16 hi / lo parts, or null
};

// Compute wavefront `wave` owns value rows v0 + 16 j + [0, 16), j < NJ. State
// tile t of row block j lives in the accumulator layout of the S^T update:
// lane (l16, g4) element e holds S[v0 + 16 j + l16][16 t + 4 g4 + e].
// OUT: outputs (Q S^T and P U, o stored); USE_V: V enters Y (false for the
// rows of a segment map, whose value input is zero).
template <int D, int C, int NJ, bool OUT, bool USE_V, typename Lds>
__device__ __forceinline__ void chain_compute(Lds &L, int wave, int lane, const ChainTask &tk,
                                              __bf16 *__restrict__ o) {
  using F = Cfg<D, C>;
  constexpr int NB = 2, NIB = F::NIB, KS = F::KS, DS = F::DS, NKT = F::NKT;
  const int l16 = lane & 15, g4 = lane >> 4;
  const int v0 = 16 * NJ * wave;
  f32x4 Sacc[NJ][NKT];
  if (tk.src != nullptr) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int t = 0; t < NKT; ++t) {
        const float4 x =
            *reinterpret_cast<const float4 *>(tk.src + (v0 + 16 * j + l16) * D + 16 * t + 4 * g4);
        Sacc[j][t] = f32x4{x.x, x.y, x.z, x.w};
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int t = 0; t < NKT; ++t) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          Sacc[j][t][e] = (tk.identity && v0 + 16 * j + l16 == 16 * t + 4 * g4 + e) ? 1.f : 0.f;
      }
    }
  }
  lds_barrier();

  // Every LDS read of a chunk is issued one step ahead of the matrix
  // products that use it (two steps in the state update, whose steps are
  // shorter), with scheduling barriers that keep the compiler from hoisting
  // them further (registers) or sinking the products above them (latency).
  for (int i = 0; i < tk.nlc; ++i) {
    const int bb = i % NB;
    // The lane id re-derived through an empty asm every chunk: otherwise the
    // compiler hoists every lane-dependent LDS address out of the loop and
    // keeps them all in registers.
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int l16 = ln & 15, g4 = ln >> 4;
    const uint16_t *Kt = L.K[bb], *Vt = L.V[bb];
    const float *dc = L.dec[bb];
    const int64_t t0 = tk.seq_t0 + (int64_t)(tk.lc0 + i) * C;
    const uint16_t *Qt = Kt;
    if constexpr (OUT) Qt = L.Q[bb];

    // rows of block ib of a row-major tile as A operands of a key contraction
    auto rows = [&](const uint16_t *Tl, int ib, uint4 (&a)[DS]) {
#pragma unroll
      for (int st = 0; st < DS; ++st) {
        const int row = 16 * ib + l16, col = 32 * st + 4 * g4;
        a[st] = key_operand(*reinterpret_cast<const uint2 *>(&Tl[ptile_index<D>(row, col)]),
                            *reinterpret_cast<const uint2 *>(&Tl[ptile_index<D>(row, col + 16)]));
      }
    };
    auto frag = [&](const uint16_t *Fl, int ib, int st) {
      return *reinterpret_cast<const uint4 *>(&Fl[((ib * KS + st) * 64 + ln) * 8]);
    };

    // The state enters both products as the bf16 B operand of S^T, its key
    // order that of tok_pos: slots 0-3 of step st are tile 2 st, slots 4-7
    // tile 2 st + 1.
    f32x4 X[NJ][NIB], O[NJ][NIB];
    uint4 vb[NJ][KS], ta[NIB][KS];
    auto read_v = [&]() {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int st = 0; st < KS; ++st)
          vb[j][st] = USE_V ? ptile_t_operand<D>(Vt, v0 / 16 + j, st, l16, g4) : make_uint4(0, 0, 0, 0);
      }
    };
    if constexpr (OUT) {
      // ---- X = K S^T and Q S^T, block by block, the next block's K and Q
      // rows read ahead; the last block's step reads the V operands instead
      uint4 SB[NJ][DS];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int st = 0; st < DS; ++st)
          SB[j][st] = make_uint4(pack_bf16x2(Sacc[j][2 * st][0], Sacc[j][2 * st][1]),
                                 pack_bf16x2(Sacc[j][2 * st][2], Sacc[j][2 * st][3]),
                                 pack_bf16x2(Sacc[j][2 * st + 1][0], Sacc[j][2 * st + 1][1]),
                                 pack_bf16x2(Sacc[j][2 * st + 1][2], Sacc[j][2 * st + 1][3]));
      }
      uint4 ka[DS], qa[DS];
      rows(Kt, 0, ka);
      rows(Qt, 0, qa);
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
        uint4 kn[DS], qn[DS];
        __builtin_amdgcn_sched_barrier(0);
        if (ib + 1 < NIB) {
          rows(Kt, ib + 1, kn);
          rows(Qt, ib + 1, qn);
        } else {
          read_v();
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          X[j][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
          O[j][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int st = 0; st < DS; ++st) {
#pragma unroll
          for (int j = 0; j < NJ; ++j) {
            X[j][ib] = mfma_16x16x32(ka[st], SB[j][st], X[j][ib]);
            O[j][ib] = mfma_16x16x32(qa[st], SB[j][st], O[j][ib]);
          }
        }
        GDN_INTERLEAVE_DS_MFMA(2 * DS * NJ)
        __builtin_amdgcn_sched_barrier(0);
        if (ib + 1 < NIB) {
#pragma unroll
          for (int st = 0; st < DS; ++st) {
            ka[st] = kn[st];
            qa[st] = qn[st];
          }
        }
      }
    } else {
      // ---- X = K S^T, key step by key step (the state's B operand packed
      // one step at a time), the K operands of the step R ahead read first;
      // fewer registers than the output launch's order, which the map
      // launch's wavefront count requires
      constexpr int NS = DS * NIB, R = 3;
      auto krd = [&](int n) {
        const int st = n / NIB, ib = n % NIB;
        const int row = 16 * ib + l16, col = 32 * st + 4 * g4;
        return key_operand(*reinterpret_cast<const uint2 *>(&Kt[ptile_index<D>(row, col)]),
                           *reinterpret_cast<const uint2 *>(&Kt[ptile_index<D>(row, col + 16)]));
      };
      uint4 kr[NS];
#pragma unroll
      for (int n = 0; n < R && n < NS; ++n) kr[n] = krd(n);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) X[j][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
      uint4 sb[NJ];
#pragma unroll
      for (int n = 0; n < NS; ++n) {
        const int st = n / NIB, ib = n % NIB;
        __builtin_amdgcn_sched_barrier(0);
        if (n + R < NS) kr[n + R] = krd(n + R);
        if (n + 1 == NS) read_v();
        if (ib == 0) {
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            sb[j] = make_uint4(pack_bf16x2(Sacc[j][2 * st][0], Sacc[j][2 * st][1]),
                               pack_bf16x2(Sacc[j][2 * st][2], Sacc[j][2 * st][3]),
                               pack_bf16x2(Sacc[j][2 * st + 1][0], Sacc[j][2 * st + 1][1]),
                               pack_bf16x2(Sacc[j][2 * st + 1][2], Sacc[j][2 * st + 1][3]));
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) X[j][ib] = mfma_16x16x32(kr[n], sb[j], X[j][ib]);
        GDN_INTERLEAVE_DS_MFMA(NJ)
        __builtin_amdgcn_sched_barrier(0);
      }
    }

    // ---- U = T' (V - exp(gamma) X)   (beta is folded into T')
#pragma unroll
    for (int jb = 0; jb < NIB; ++jb) {
#pragma unroll
      for (int st = 0; st < frag_steps<C>(jb); ++st) ta[jb][st] = frag(L.T[bb], jb, st);
    }
    f32x4 ga[NIB];
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      const float4 x = *reinterpret_cast<const float4 *>(&dc[16 * ib + 4 * g4]);
      ga[ib] = f32x4{x.x, x.y, x.z, x.w};
    }
    uint4 Yb[NJ][KS];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int st = 0; st < KS; ++st) Yb[j][st] = y_operand<NIB>(vb[j][st], X[j], ga, st);
    }
    // the P fragments and the first K^T operands of the update, read while
    // U is formed
    uint4 pa[NIB][KS], kt0[KS], kt1[KS];
    if constexpr (OUT) {
#pragma unroll
      for (int jb = 0; jb < NIB; ++jb) {
#pragma unroll
        for (int st = 0; st < frag_steps<C>(jb); ++st) pa[jb][st] = frag(L.P[bb], jb, st);
      }
    }
    auto read_kt01 = [&]() {
#pragma unroll
      for (int st = 0; st < KS; ++st) {
        kt0[st] = ptile_t_operand<D>(Kt, 0, st, l16, g4);
        kt1[st] = ptile_t_operand<D>(Kt, NKT > 1 ? 1 : 0, st, l16, g4);
      }
    };
    if constexpr (OUT) read_kt01();  // (the map launch reads them after U: registers)
    __builtin_amdgcn_sched_barrier(0);
    f32x4 U[NJ][NIB];
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) U[j][ib] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < frag_steps<C>(ib); ++st) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) U[j][ib] = mfma_16x16x32(ta[ib][st], Yb[j][st], U[j][ib]);
      }
    }
    if constexpr (!OUT) read_kt01();

    // ---- O = exp(gamma) Q S^T + P U, stored as bf16 (rows past the end of
    // the sequence dropped)
    if constexpr (OUT) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        uint4 Ub[KS];
#pragma unroll
        for (int st = 0; st < KS; ++st) Ub[st] = u_operand<NIB>(U[j], st, nullptr);
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) {
          O[j][ib] = O[j][ib] * ga[ib];
#pragma unroll
          for (int st = 0; st < frag_steps<C>(ib); ++st)
            O[j][ib] = mfma_16x16x32(pa[ib][st], Ub[st], O[j][ib]);
        }
      }
      const int nv = (int)min((int64_t)C, tk.seq_t1 - t0);
      const rsrc_t ro = make_rsrc(o + (t0 * tk.hv + tk.h) * D, (uint32_t)(nv * tk.hv * D * 2));
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            BufElem<__bf16>::store1_stream(
                ro, (uint32_t)((16 * ib + 4 * g4 + e) * tk.hv * D + v0 + 16 * j + l16), O[j][ib][e]);
        }
      }
    }

    // ---- S^T <- exp(gamma_last) S^T + K^T (exp(gamma_last - gamma) U),
    // key tile by key tile, the K^T operands two tiles ahead
    {
      f32x4 he[NIB];
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
        const float4 x = *reinterpret_cast<const float4 *>(&dc[C + 16 * ib + 4 * g4]);
        he[ib] = f32x4{x.x, x.y, x.z, x.w};
      }
      const float glast = dc[C - 1];
      uint4 Uh[NJ][KS];
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
#pragma unroll
        for (int st = 0; st < KS; ++st) Uh[j][st] = u_operand<NIB>(U[j], st, he);
      }
#pragma unroll
      for (int t = 0; t < NKT; ++t) {
        uint4 kn[KS];
        __builtin_amdgcn_sched_barrier(0);
        if (t + 2 < NKT) {
#pragma unroll
          for (int st = 0; st < KS; ++st) kn[st] = ptile_t_operand<D>(Kt, t + 2, st, l16, g4);
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          f32x4 acc = Sacc[j][t] * glast;
#pragma unroll
          for (int st = 0; st < KS; ++st) acc = mfma_16x16x32(kt0[st], Uh[j][st], acc);
          Sacc[j][t] = acc;
        }
        GDN_INTERLEAVE_DS_MFMA(NJ * KS)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int st = 0; st < KS; ++st) {
          kt0[st] = kt1[st];
          if (t + 2 < NKT) kt1[st] = kn[st];
        }
      }
    }
    lds_barrier();  // end of chunk i: buffer bb may be refilled
  }

  // ---- the state leaving the segment
  if (tk.dst != nullptr) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
#pragma unroll
      for (int t = 0; t < NKT; ++t)
        store_stream(tk.dst + (v0 + 16 * j + l16) * D + 16 * t + 4 * g4, Sacc[j][t]);
    }
  } else if (tk.dhi != nullptr) {
    // Rows i = v0 + 16 j + l16 of the segment's map M, stored transposed,
    // MT[key][pos(i)] = M[i][key], split into bf16 hi + lo (hi = M rounded,
    // lo = the rounding error rounded): the A operand of the composition. The
    // columns are in the order tok_pos gives the keys of a contraction step,
    // so that each lane's 8 contraction slots are 16 contiguous bytes there.
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int pos = tok_pos(v0 + 16 * j + l16);
#pragma unroll
      for (int t = 0; t < NKT; ++t) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = Sacc[j][t][e];
          const uint16_t hi = f32_to_bf16_bits(x);
          const uint16_t lo = f32_to_bf16_bits(x - bf16_bits_to_f32(hi));
          const int64_t idx = (int64_t)(16 * t + 4 * g4 + e) * D + pos;
          __builtin_nontemporal_store(hi, tk.dhi + idx);
          __builtin_nontemporal_store(lo, tk.dlo + idx);
        }
      }
    }
  }
}

template <int D, int C, bool MAPS>
__global__ __launch_bounds__((ChainCfg<D, C, MAPS>::NT)) void chain_kernel(
    const __bf16 *__restrict__ q, const __bf16 *__restrict__ k, const __bf16 *__restrict__ v,
    const int32_t *__restrict__ cu, const float *__restrict__ dec_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag, const float *s0,
    float *sT, __bf16 *__restrict__ o, float *__restrict__ bslot, uint16_t *__restrict__ mt_hi,
    uint16_t *__restrict__ mt_lo, const int32_t *__restrict__ order, int n_seqs, int hqk, int hv,
    int group, int n_units, int seg_chunks) {
  using F = Cfg<D, C>;
  using H = ChainCfg<D, C, MAPS>;
  constexpr int NIB = F::NIB, KS = F::KS;
  constexpr bool OUT = !MAPS;
  __shared__ __attribute__((aligned(16))) ChainLds<D, C, MAPS> L;

  // Block id -> (segment rank, key head) unit and head of the group. Work-
  // groups are dealt to the eight XCDs round robin, so ids b and b + 8 share
  // one: the value heads of a group (which share K and Q) take ids
  // 8 (group j + gi) + x. The segment of rank r is order[r] (longest
  // first; -1: no segment), or slot r when there is no order.
  const int bid = blockIdx.x;
  const int xg = bid & 7, jj = bid >> 3;
  const int gi = jj % group;
  const int unit = (jj / group) * 8 + xg;
  if (unit >= n_units) return;
  const int rank = unit / hqk, hk = unit - rank * hqk;
  const int slot = order != nullptr ? order[rank] : rank;
  if (slot < 0) return;
  const int h = hk * group + gi;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
  const int64_t span = (int64_t)C * seg_chunks;

  // ---- the sequence owning segment slot `slot`: each wavefront tests the
  // sequences 64 at a time and takes the (single) hit from a ballot.
  int n = -1, cu_a = 0, cu_b = 0;
  for (int m0 = 0; m0 < n_seqs; m0 += 64) {
    const int m = m0 + lane;
    int a = 0, b = 0;
    bool hit = false;
    if (m < n_seqs) {
      a = cu[m];
      b = cu[m + 1];
      const int64_t base = (int64_t)a / span + m;
      hit = slot >= base && slot < base + seg_count(b - a, span);
    }
    const uint64_t bal = __ballot(hit);
    if (bal != 0) {
      const int src = __ffsll((unsigned long long)bal) - 1;
      n = m0 + src;
      cu_a = __builtin_amdgcn_readlane(a, src);
      cu_b = __builtin_amdgcn_readlane(b, src);
      break;
    }
  }
  if (n < 0) return;  // an unused slot: the same for every wavefront
  const int64_t seq_t0 = cu_a, seq_t1 = cu_b;
  const int G = (int)seg_count(seq_t1 - seq_t0, span);
  const int s = (int)(slot - (seq_t0 / span + n));
  const int64_t mslot = seq_t0 / span + s;  // map slot of this segment (s <= G - 2)
  if (MAPS && s > G - 2) return;  // the last segment has no map
  const int nch = (int)((seq_t1 - seq_t0 + C - 1) / C);
  const int lc0 = s * seg_chunks;
  const int nlc = max(0, min(nch, lc0 + seg_chunks) - lc0);
  const int64_t c0 = seq_t0 / C + n;  // first chunk slot of the sequence (tables)
  const int64_t pair = (int64_t)n * hv + h;
  const int64_t hblk = (int64_t)hv * D * D;  // one map slot, all heads

  // token rows C..CP-1 of the K and V tiles stay zero (transpose reads cover CP rows)
  if (C < F::CP) {
    for (int idx = C * H::P + tid; idx < F::CP * H::P; idx += H::NT) {
#pragma unroll
      for (int bb = 0; bb < H::NB; ++bb) {
        L.K[bb][idx] = 0;
        L.V[bb][idx] = 0;
      }
    }
  }

  if (wave >= H::NCW) {
    // ================================================= loader wavefronts
    const int kstride = hqk * D, vstride = hv * D;
    auto issue = [&](int lc, int bb) {  // copies of chunk lc into buffer bb
      const int64_t t0 = seq_t0 + (int64_t)lc * C;
      const int nv = (int)min((int64_t)C, seq_t1 - t0);
      const rsrc_t rk = make_rsrc(k + (t0 * hqk + hk) * D, (uint32_t)(nv * kstride * 2));
      const rsrc_t rv = make_rsrc(v + (t0 * hv + h) * D, (uint32_t)(nv * vstride * 2));
#pragma unroll
      for (int m = 0; m < H::NKI; ++m) {
        const uint32_t off = chain_tile_copy_offset<D, C>(m, lane, kstride);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void *)&L.K[bb][512 * m], 16, off, 0, 0, 0);
      }
#pragma unroll
      for (int m = 0; m < H::NKI; ++m) {
        const uint32_t off = chain_tile_copy_offset<D, C>(m, lane, vstride);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void *)&L.V[bb][512 * m], 16, off, 0, 0, 0);
      }
      if constexpr (OUT) {
        const rsrc_t rq = make_rsrc(q + (t0 * hqk + hk) * D, (uint32_t)(nv * kstride * 2));
#pragma unroll
        for (int m = 0; m < H::NKI; ++m) {
          const uint32_t off = chain_tile_copy_offset<D, C>(m, lane, kstride);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rq, (lds_void *)&L.Q[bb][512 * m], 16, off, 0, 0, 0);
        }
      }
      const int64_t cs = (c0 + lc) * hv + h;
      const rsrc_t rt = make_rsrc(tfrag + cs * F::FRAG, F::FRAG * 2);
      const rsrc_t rp = make_rsrc(pfrag + cs * F::FRAG, F::FRAG * 2);
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
        for (int st = 0; st < frag_steps<C>(ib); ++st) {
          const int f = ib * KS + st;
          const uint32_t off = (uint32_t)((f * 64 + lane) * 16);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(rt, (lds_void *)&L.T[bb][512 * f], 16, off, 0, 0, 0);
          if constexpr (OUT)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (lds_void *)&L.P[bb][512 * f], 16, off, 0, 0, 0);
        }
      }
      const rsrc_t rd = make_rsrc(dec_ws + cs * 2 * C, 2 * C * 4);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (lds_void *)&L.dec[bb][0], 16,
                                               4 * lane < 2 * C ? (uint32_t)(16 * lane) : kOutOfRange,
                                               0, 0, 0);
    };
    // One 4-byte load per 128-byte line of chunk lc's K, Q and V rows (the
    // map launch repeats K for Q) and of its T', P and decay tables: brings
    // them into L2 before their copies are issued. Chunks past the sequence
    // read nothing.
    auto prefetch = [&](int lc) {
      const int64_t t0 = seq_t0 + (int64_t)lc * C;
      const int nv = (int)max((int64_t)0, min((int64_t)C, seq_t1 - t0));
      const rsrc_t rk = make_rsrc(k + (t0 * hqk + hk) * D, (uint32_t)(nv * kstride * 2));
      const rsrc_t rq = make_rsrc(q + (t0 * hqk + hk) * D, (uint32_t)(nv * kstride * 2));
      const rsrc_t rv = make_rsrc(v + (t0 * hv + h) * D, (uint32_t)(nv * vstride * 2));
#pragma unroll
      for (int p = 0; p < 3 * H::NPT; ++p) {
        const int tile = p / H::NPT, u = (p % H::NPT) * 64 + lane;
        const int row = u / H::LPR, part = u % H::LPR;
        const bool in = u < C * H::LPR;
        const bool isq = tile == 1 && OUT, isv = tile == 2;
        const int stride = isv ? vstride : kstride;
        const uint32_t off = in ? (uint32_t)(row * stride * 2 + part * 128) : kOutOfRange;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(isv ? rv : (isq ? rq : rk), (lds_void *)&L.sink[0], 4,
                                                 off, 0, 0, 0);
      }
      const int64_t cs = (c0 + lc) * hv + h;
      const uint32_t tb = nv > 0 ? (uint32_t)(F::FRAG * 2) : 0u;
      const rsrc_t rt = make_rsrc(tfrag + cs * F::FRAG, tb);
      const rsrc_t rp = make_rsrc(pfrag + cs * F::FRAG, OUT ? tb : 0u);
      const rsrc_t rd = make_rsrc(dec_ws + cs * 2 * C, nv > 0 ? 2 * C * 4 : 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rt, (lds_void *)&L.sink[0], 4, (uint32_t)(128 * lane), 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (lds_void *)&L.sink[0], 4, (uint32_t)(128 * lane), 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (lds_void *)&L.sink[0], 4, (uint32_t)(128 * lane), 0, 0, 0);
    };
    // The copies of chunk i + 1 go into the buffer chunk i - 1 used and must
    // land before chunk i ends.
    if (wave == H::NCW) {
      if (nlc > 0) {
        issue(lc0, 0);
        wait_vm<0>();
      }
      lds_barrier();
      for (int i = 0; i < nlc; ++i) {
        if (i + 1 < nlc) {
          issue(lc0 + i + 1, (i + 1) % H::NB);
          wait_vm<0>();
        }
        lds_barrier();  // end of chunk i
      }
    } else {
      // The prefetching wavefront: chunk lc0 + 1 at the start, chunk
      // lc0 + i + PFD while chunk i is in use (every work-group starting with
      // several chunks at once would flood memory just when the first copies
      // are needed). It never waits for its loads (a wavefront's loads
      // complete in order, so the loader's waits would otherwise include
      // them), except before it exits.
      if (nlc > 1) prefetch(lc0 + 1);
      lds_barrier();
      for (int i = 0; i < nlc; ++i) {
        if (i + H::PFD < nlc) prefetch(lc0 + i + H::PFD);
        lds_barrier();
      }
      wait_vm<0>();
    }
    return;
  }

  // ================================================= compute wavefronts
  const int set = wave / H::NWR, w = wave - set * H::NWR;  // row set, wavefront within it
  ChainTask t;
  t.nlc = nlc;
  t.lc0 = lc0;
  t.seq_t0 = seq_t0;
  t.seq_t1 = seq_t1;
  t.h = h;
  t.hv = hv;
  t.src = nullptr;
  t.identity = false;
  t.dst = nullptr;
  t.dhi = t.dlo = nullptr;
  if (MAPS && set == 1) {  // the rows of the map M of segment s >= 1
    if (s == 0) {  // segment 0 needs no map: stay in step with the barriers
      for (int i = 0; i <= nlc; ++i) lds_barrier();
      return;
    }
    t.identity = true;
    t.dhi = mt_hi + mslot * hblk + (int64_t)h * D * D;
    t.dlo = mt_lo + mslot * hblk + (int64_t)h * D * D;
    chain_compute<D, C, H::NJ, false, false>(L, w, lane, t, o);
    return;
  }
  // the state rows: from the initial state (segment 0) or, in the map launch,
  // from zero, or, in the output launch, from the composed incoming state
  if (s == 0)
    t.src = s0 == nullptr ? nullptr : s0 + pair * D * D;
  else if (OUT)
    t.src = bslot + (mslot - 1) * hblk + (int64_t)h * D * D;
  if (MAPS)
    t.dst = bslot + mslot * hblk + (int64_t)h * D * D;
  else if (s == G - 1)
    t.dst = sT + pair * D * D;
  chain_compute<D, C, H::NJ, OUT, true>(L, w, lane, t, o);
}

// ============================================================ composition
// One work-group per (sequence, value head, 16-row value tile): the incoming
// states of segments 2..G-1,
//   S_in(s + 1) = S_in(s) M_s + B_s,   s = 1..G-2,   S_in(1) = B_0,
// written over B_s in place. In the S^T orientation of the carry,
// S_in(s + 1)^T = M_s^T S_in(s)^T + B_s^T: the A operand is M_s^T (stored
// that way by the M work-groups), the B operand the previous result straight
// from the accumulators (key order of tok_pos). Both are split into bf16 hi +
// lo and multiplied as hi hi + hi lo + lo hi with fp32 accumulation, which
// keeps the composition at about fp32 accuracy. Each wavefront computes
// KTW 16-key tiles of the result; the tiles are exchanged through LDS before
// the next step.
template <int D>
struct ComposeCfg {
  static constexpr int NKT = D / 16;
  static constexpr int KTW = NKT >= 8 ? 2 : 1;  // key tiles per wavefront
  static constexpr int NW = NKT / KTW;          // wavefronts
  static constexpr int DS = D / 32;
};

template <int D>
__global__ __launch_bounds__(64 * ComposeCfg<D>::NW) void compose_kernel(
    const int32_t *__restrict__ cu, float *__restrict__ bslot, const uint16_t *__restrict__ mt_hi,
    const uint16_t *__restrict__ mt_lo, int hv, int64_t span, int n_seqs, int chunk,
    int seg_chunks, int64_t nseg, int32_t *__restrict__ order) {
  using CC = ComposeCfg<D>;
  constexpr int NKT = CC::NKT, KTW = CC::KTW, DS = CC::DS, NVT = D / 16;
  constexpr int NTH = 64 * CC::NW;
  __shared__ __attribute__((aligned(16))) union {
    float xch[NKT][64 * 4];
    struct {
      int cursor[kOrderBuckets];
      int part[NTH];
    } ord;
  } sh;
  auto &xch = sh.xch;

  const int bid = blockIdx.x;
  // With `order`, one work-group past the compositions builds the output
  // launch's longest-first list (a launch saved; nothing here reads it).
  if (order != nullptr && bid == (int)gridDim.x - 1) {
    build_order<NTH>(cu, n_seqs, chunk, seg_chunks, nseg, order, sh.ord.cursor, sh.ord.part);
    return;
  }
  const int vt = bid % NVT, ph = bid / NVT;
  const int h = ph % hv, n = ph / hv;
  const int64_t a0 = cu[n], a1 = cu[n + 1];
  const int G = (int)seg_count(a1 - a0, span);
  if (G < 3) return;  // uniform over the work-group
  const int lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int v0 = 16 * vt;
  const int64_t mb0 = a0 / span;
  const int64_t hstride = (int64_t)hv * D * D;
  auto tile_ptr = [&](int64_t mb, int t) {  // rows v0..v0+15, keys of tile t, this lane's piece
    return bslot + mb * hstride + (int64_t)h * D * D + (v0 + l16) * D + 16 * t + 4 * g4;
  };

  // Operands of one step, loaded two steps ahead of use: the B_s^T tiles of
  // this wavefront and the M_s^T A operands (hi and lo) of its key tiles.
  struct StepOps {
    float4 b[KTW];
    uint4 ah[KTW][DS], al[KTW][DS];
  };
  // (Steps past the last reload the last step's operands: no branch in the
  // loop, so that the compiler's wait counts stay exact across it.)
  auto load = [&](int s, StepOps &op) {
    const int64_t mb = mb0 + min(s, G - 2);
    const uint16_t *mh = mt_hi + mb * hstride + (int64_t)h * D * D;
    const uint16_t *ml = mt_lo + mb * hstride + (int64_t)h * D * D;
#pragma unroll
    for (int w = 0; w < KTW; ++w) {
      const int t = KTW * wave + w;
      op.b[w] = *reinterpret_cast<const float4 *>(tile_ptr(mb, t));
#pragma unroll
      for (int st = 0; st < DS; ++st) {
        // the map's columns are stored in tok_pos order: 16 contiguous bytes
        const int64_t r = (int64_t)(16 * t + l16) * D + 32 * st + 8 * g4;
        op.ah[w][st] = *reinterpret_cast<const uint4 *>(mh + r);
        op.al[w][st] = *reinterpret_cast<const uint4 *>(ml + r);
      }
    }
  };

  f32x4 S[NKT];  // S_in^T, every key tile (accumulator layout)
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    const float4 x = *reinterpret_cast<const float4 *>(tile_ptr(mb0, t));
    S[t] = f32x4{x.x, x.y, x.z, x.w};
  }
  auto step = [&](int s, const StepOps &op) {
    const int64_t mb = mb0 + s;
    uint4 bhi[DS], blo[DS];
#pragma unroll
    for (int st = 0; st < DS; ++st) {
      const float x[8] = {S[2 * st][0], S[2 * st][1], S[2 * st][2], S[2 * st][3],
                          S[2 * st + 1][0], S[2 * st + 1][1], S[2 * st + 1][2], S[2 * st + 1][3]};
      uint32_t hb[8], lb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hb[e] = f32_to_bf16_bits(x[e]);
        lb[e] = f32_to_bf16_bits(x[e] - bf16_bits_to_f32(hb[e]));
      }
      bhi[st] = make_uint4(hb[0] | hb[1] << 16, hb[2] | hb[3] << 16, hb[4] | hb[5] << 16,
                           hb[6] | hb[7] << 16);
      blo[st] = make_uint4(lb[0] | lb[1] << 16, lb[2] | lb[3] << 16, lb[4] | lb[5] << 16,
                           lb[6] | lb[7] << 16);
    }
#pragma unroll
    for (int w = 0; w < KTW; ++w) {
      const int t = KTW * wave + w;
      f32x4 acc = f32x4{op.b[w].x, op.b[w].y, op.b[w].z, op.b[w].w};
#pragma unroll
      for (int st = 0; st < DS; ++st) {
        acc = mfma_16x16x32(op.ah[w][st], bhi[st], acc);
        acc = mfma_16x16x32(op.ah[w][st], blo[st], acc);
        acc = mfma_16x16x32(op.al[w][st], bhi[st], acc);
      }
      store_stream(tile_ptr(mb, t), acc);
      *reinterpret_cast<float4 *>(&xch[t][4 * lane]) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
    lds_barrier();
#pragma unroll
    for (int t = 0; t < NKT; ++t) {
      const float4 x = *reinterpret_cast<const float4 *>(&xch[t][4 * lane]);
      S[t] = f32x4{x.x, x.y, x.z, x.w};
    }
    lds_barrier();
  };
  StepOps opa, opb;
  load(1, opa);
  load(2, opb);
  int s = 1;
  for (; s + 1 <= G - 2; s += 2) {
    step(s, opa);
    load(s + 2, opa);
    step(s + 1, opb);
    load(s + 3, opb);
  }
  if (s <= G - 2) step(s, opa);
}

// ============================================================ host side
template <int D, int C>
hipError_t launch_chain(const PrefillArgs &a, const PrefillWorkspace &ws) {
  char *base = static_cast<char *>(a.workspace);
  const float *dec = reinterpret_cast<const float *>(base + ws.decay);
  const uint16_t *tf = reinterpret_cast<const uint16_t *>(base + ws.tfrag);
  const uint16_t *pf = reinterpret_cast<const uint16_t *>(base + ws.pfrag);
  const bool segmented = ws.n_maps > 0;
  float *bs = segmented ? reinterpret_cast<float *>(base + ws.bslot) : nullptr;
  uint16_t *mh = segmented ? reinterpret_cast<uint16_t *>(base + ws.mthi) : nullptr;
  uint16_t *ml = segmented ? reinterpret_cast<uint16_t *>(base + ws.mtlo) : nullptr;
  const int group = a.hv / a.hqk;
  const int64_t span = (int64_t)C * a.seg_chunks;
  const int64_t nseg = a.n_tokens / span + a.n_seqs;  // segment slots
  const int64_t units = nseg * a.hqk;
  const unsigned bx = (unsigned)(((units + 7) / 8) * 8 * group);
  const __bf16 *q = (const __bf16 *)a.q, *k = (const __bf16 *)a.k, *v = (const __bf16 *)a.v;
  __bf16 *o = (__bf16 *)a.o;

  // Longest segments first in the output launch, when there is more than
  // one sequence (the segments of one sequence are equal but for the last):
  // built by an extra work-group of the composition launch when that runs,
  // else by a launch of its own.
  int32_t *order = a.n_seqs > 1 ? reinterpret_cast<int32_t *>(base + ws.order) : nullptr;
  const bool compose = segmented && ws.n_maps >= 2;  // some sequence may have 3+ segments
  if (order != nullptr && !compose) {
    hipLaunchKernelGGL(chain_order_kernel, dim3(1), dim3(kOrderThreads), 0, a.stream,
                       a.cu_seqlens, a.n_seqs, C, a.seg_chunks, nseg, order);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (segmented) {  // every map segment has L chunks: block order
    hipLaunchKernelGGL((chain_kernel<D, C, true>), dim3(bx), dim3(ChainCfg<D, C, true>::NT), 0,
                       a.stream, q, k, v, a.cu_seqlens, dec, tf, pf, a.initial_state,
                       a.final_state, o, bs, mh, ml, nullptr, a.n_seqs, a.hqk, a.hv, group,
                       (int)units, a.seg_chunks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (compose) {
      const int64_t cblocks = (int64_t)a.n_seqs * a.hv * (D / 16) + (order != nullptr ? 1 : 0);
      hipLaunchKernelGGL((compose_kernel<D>), dim3((unsigned)cblocks),
                         dim3(64 * ComposeCfg<D>::NW), 0, a.stream, a.cu_seqlens, bs, mh, ml,
                         a.hv, span, a.n_seqs, C, a.seg_chunks, nseg, order);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
  }
  hipLaunchKernelGGL((chain_kernel<D, C, false>), dim3(bx), dim3(ChainCfg<D, C, false>::NT), 0,
                     a.stream, q, k, v, a.cu_seqlens, dec, tf, pf, a.initial_state, a.final_state,
                     o, bs, mh, ml, order, a.n_seqs, a.hqk, a.hv, group, (int)units,
                     a.seg_chunks);
  return hipGetLastError();
}

hipError_t launch_chain_d(const PrefillArgs &a, const PrefillWorkspace &ws) {
  switch (a.d * 1000 + a.chunk) {
    case 32016: return launch_chain<32, 16>(a, ws);
    case 32032: return launch_chain<32, 32>(a, ws);
    case 32064: return launch_chain<32, 64>(a, ws);
    case 64016: return launch_chain<64, 16>(a, ws);
    case 64032: return launch_chain<64, 32>(a, ws);
    case 64064: return launch_chain<64, 64>(a, ws);
    case 128016: return launch_chain<128, 16>(a, ws);
    case 128032: return launch_chain<128, 32>(a, ws);
    case 128064: return launch_chain<128, 64>(a, ws);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gdn
