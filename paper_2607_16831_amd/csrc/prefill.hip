// prefill.hip -- chunked (WY / UT) prefill of the gated delta rule on gfx950.
//
// The paper reports that the winning prefill designs replace the token-serial
// recurrence by per-chunk summaries with matrix-shaped work (Sections 5.1, 5.2
// and 5.5). This file implements that reformulation. For one chunk of n <= C
// tokens of a (sequence, value head) chain, with incoming state S (d_v x d_k),
// in-chunk cumulative log-decay gamma_i = g_0 + ... + g_i and
// E_ij = exp(gamma_i - gamma_j) for j <= i:
//
//   A  = strict_lower( beta_i E_ij k_i.k_j )            (C x C)
//   T  = (I + A)^-1                                      unit lower triangular
//   P  = lower( E_ij q_i.k_j )                           diagonal included
//   U  = T ( beta (V - exp(gamma) (K S^T)) )             (C x d_v)
//   O  = exp(gamma) (Q S^T) + P U
//   S' = exp(gamma_last) S + (exp(gamma_last - gamma) U)^T K
//
// which reproduces the token-serial recurrence exactly up to rounding.
//
// Two kernels on one stream:
//   chunk_local_kernel    chunk-parallel: gamma, K K^T and Q K^T on bf16 MFMA,
//                         A, the triangular inverse in LDS (fp32), P; T and P
//                         are stored as bf16 in MFMA operand order.
//   chunk_carry_kernel    one work-group per (sequence, value head, 16-row
//                         value tile): walks the chunks of its sequence, keeps
//                         its fp32 state tile in MFMA accumulators and does
//                         every product on bf16 MFMA with fp32 accumulation;
//                         dedicated wavefronts stream the next chunks into LDS.
//
// Every exponent is a non-positive difference (for g <= 0), masked before
// exp, so strongly decaying inputs cannot overflow.
#include <algorithm>
#include <type_traits>

#include "gdn_launch.h"
#include "prefill_common.h"

namespace gdn {


// ============================================================ chunk-local
// One work-group per (chunk, value head): gamma, K K^T and K Q^T, then A, P
// and T = (I + A)^-1, written as bf16 A-operand fragments. The two Gram
// products depend only on the key head; the value heads of a GQA group each
// recompute them (a few dozen matrix instructions) rather than share a
// longer work-group, and the launch order puts the heads of one group on
// the same XCD so that the second reads K and Q from its L2.
//
// The 16x16 tiles of the two lower-triangular Gram products are dealt out
// evenly: wavefront w computes block row w of Q K^T (its Q rows are in its
// registers) and block row NIB - 1 - w of K K^T, NIB + 1 tiles each.
//
// T is built from its 16x16 blocks in fp32. Diagonal block b is inverted
// either by forward substitution on the vector ALU (one lane per column, all
// blocks at once in one wavefront) or, with NEUMANN, by the Neumann product
// on the matrix cores (one block per wavefront, see neumann_diag); wavefront
// b then forms its block row from
//   T[b][c] = -(sum_{m=c+1..b} T[b][m] A[m][c]) T[c][c]^-1    (c < b),
// carried in transposed form so that every intermediate stays in the
// accumulator layout of the fp32 16x16x4 matrix instruction.
// HPW value heads per work-group (1 or 2): each head has its own A blocks,
// inverses and gate copies; the K tile and the Gram products are shared.
template <int D, int C, int HPW>
struct LocalLds {
  static constexpr int NIB = C / 16;
  static constexpr int NBLK = NIB * (NIB + 1) / 2;  // lower blocks, diagonal included
  static constexpr int AP = 20;                     // f32 pitch of an A block row
  union {
    uint16_t kq[C * D];  // K tile, swizzled rows (kn_index)
    struct {
      float A[HPW][NBLK][16 * AP];    // block (m, c) at m (m + 1) / 2 + c, row-major
      float linv[HPW][NIB][16 * 17];  // transposed diagonal inverses
    } inv;
  } u;
  float gam[HPW][4][64];  // per-wavefront copies of gamma and beta
  float bet[HPW][4][64];
};

// Block row QB of Q K^T and block row KB of K K^T with their decay masks,
// for one wavefront: first Q K^T, masked with each head's gates and stored
// as P fragments to global memory, then K K^T, whose masked tiles become
// each head's A blocks of row KB once the K tile's space is free (after the
// first of the two barriers every wavefront passes). The products depend
// only on the key head, so the HPW heads of the work-group share them.
// Wavefront w takes QB = w (its Q registers) and KB = NIB - 1 - w, so that
// every wavefront forms NIB + 1 tiles. Lane (l16, g4) element e of a tile
// holds k_j . q_i (or k_j . k_i), j = 16 jb + 4 g4 + e, i = 16 (row) + l16.
// The rows are template parameters so that only the tiles on or below the
// diagonal exist, and each tile's K rows are read right before its
// products, which keeps a wavefront's registers within what its occupancy
// allows.
template <int D, int C, int HPW, int QB, int KB, typename LL>
__device__ __forceinline__ void gram_row_masks(LL &L, const uint16_t *Kt, const uint4 (&qv)[D / 32],
                                               int wave, uint16_t *const (&pf_base)[HPW],
                                               int lane) {
  using F = Cfg<D, C>;
  constexpr int KS = F::KS, DS = F::DS, AP = LL::AP;
  const int l16 = lane & 15, g4 = lane >> 4;
  auto masked = [&](int hh, int ib, int jb, const f32x4 &g, bool isp) {
    const float *gw = L.gam[hh][wave], *bw = L.bet[hh][wave];
    const int i = 16 * ib + l16;
    const float gami = gw[i], bi = bw[i];
    const float4 gj = *reinterpret_cast<const float4 *>(&gw[16 * jb + 4 * g4]);
    const float gjv[4] = {gj.x, gj.y, gj.z, gj.w};
    f32x4 m;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = 16 * jb + 4 * g4 + e;
      const float dec = (j <= i) ? __expf(gami - gjv[e]) : 0.f;
      m[e] = isp ? dec * g[e] : ((j < i) ? bi * dec * g[e] : 0.f);
    }
    return m;
  };
  // K rows of block jb, step s. The lane id passes through an empty asm at
  // every read: otherwise the compiler computes every (jb, s) address up
  // front and holds them all in registers.
  auto krow = [&](int jb, int s) {
    int ln = lane;
    asm volatile("" : "+v"(ln));
    return *reinterpret_cast<const uint4 *>(
        &Kt[kn_index<D>(16 * jb + (ln & 15), 32 * s + 8 * (ln >> 4))]);
  };
  if constexpr (QB < F::NIB) {
    // ---- Q K^T and P
    f32x4 Pt[QB + 1];
#pragma unroll
    for (int jb = 0; jb <= QB; ++jb) {
      __builtin_amdgcn_sched_barrier(0);
      Pt[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < DS; ++s) Pt[jb] = mfma_16x16x32(krow(jb, s), qv[s], Pt[jb]);
    }
    // P as A-operand fragments: step s takes tile 2s (elements 0-3) and tile
    // 2s+1 (elements 4-7), i.e. the token order of tok_pos(). Device-scope
    // stores, like every table the carry reads.
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      const rsrc_t rpf = make_rsrc(pf_base[hh], F::FRAG * 2);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (2 * s > QB) continue;  // above the diagonal: zero, never stored or read
        const f32x4 lo4 = masked(hh, QB, 2 * s, Pt[2 * s], true);
        const f32x4 hi4 = (2 * s + 1 <= QB)
                              ? masked(hh, QB, 2 * s + 1, Pt[(2 * s + 1) % (QB + 1)], true)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
        buf_store_b128<kCachePolicyDevice>(
            rpf, (uint32_t)((((QB * KS + s) * 64 + lane) * 8) * 2),
            make_uint4(pack_bf16x2(lo4[0], lo4[1]), pack_bf16x2(lo4[2], lo4[3]),
                       pack_bf16x2(hi4[0], hi4[1]), pack_bf16x2(hi4[2], hi4[3])));
      }
    }
    // ---- K K^T (the B operand, K rows of block KB, read once)
    __builtin_amdgcn_sched_barrier(0);
    uint4 kb[DS];
#pragma unroll
    for (int s = 0; s < DS; ++s) kb[s] = krow(KB, s);
    f32x4 G[KB + 1];
#pragma unroll
    for (int jb = 0; jb <= KB; ++jb) {
      __builtin_amdgcn_sched_barrier(0);
      G[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < DS; ++s) G[jb] = mfma_16x16x32(krow(jb, s), kb[s], G[jb]);
    }
    lds_barrier();  // the K tile is dead; the space is reused for A
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
#pragma unroll
      for (int jb = 0; jb <= KB; ++jb) {
        const f32x4 m = masked(hh, KB, jb, G[jb], false);
        *reinterpret_cast<float4 *>(&L.u.inv.A[hh][KB * (KB + 1) / 2 + jb][l16 * AP + 4 * g4]) =
            make_float4(m[0], m[1], m[2], m[3]);
      }
    }
    lds_barrier();
  } else {
    lds_barrier();
    lds_barrier();
  }
}

// Inverse of one unit lower-triangular 16 x 16 block I + N by the Neumann
// series, exact because N is strictly lower and so N^16 = 0, in its product
// form (the chunk-solve variant the paper's Section 5.1 names):
//   (I + N)^-1 = (I - N)(I + N^2)(I + N^4)(I + N^8).
// One wavefront, fp32 16x16x4 matrix instructions. Matrices are held in the
// accumulator layout (lane (g, n) holds rows 4g..4g+3 of column n); a
// product X Y takes Y in that layout as its B operand and X^T in that layout
// as its A operand, so each power is carried with its transpose and no data
// moves between products: P^2 = mul(P^T, P) and (P^2)^T = mul(P, P^T). The
// factors commute, so each is applied from the left. Ab: the block in LDS,
// row-major with pitch AP; the inverse is returned in the accumulator layout.
template <int AP>
__device__ __forceinline__ f32x4 neumann_diag(const float *Ab, int g4, int l16) {
  auto mul = [](f32x4 at, f32x4 b) {  // (matrix of at)^T times (matrix of b)
    f32x4 r = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) r = mfma_16x16x4_f32(at[kk], b[kk], r);
    return r;
  };
  f32x4 eye, P, Pt;  // P = (-N)^(2^k) and its transpose
  const float4 nt = *reinterpret_cast<const float4 *>(&Ab[l16 * AP + 4 * g4]);
  Pt = f32x4{-nt.x, -nt.y, -nt.z, -nt.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    eye[e] = (4 * g4 + e == l16) ? 1.f : 0.f;
    P[e] = -Ab[(4 * g4 + e) * AP + l16];
  }
  f32x4 inv = eye + P;  // I - N
#pragma unroll
  for (int k = 1; k < 4; ++k) {
    const f32x4 P2 = mul(Pt, P), P2t = mul(P, Pt);
    P = P2;
    Pt = P2t;
    inv = mul(eye + Pt, inv);  // (I + N^(2^k)) times the product so far
  }
  return inv;
}

template <int D, int C, typename TIn, bool NEUMANN, int HPW>
__global__ __launch_bounds__(256, HPW == 1 ? 8 : 4) void chunk_local_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const float *__restrict__ g, const float *__restrict__ beta, GateArgs gate,
    const int32_t *__restrict__ cu, int n_seqs, int hqk, int hv, int group,
    int n_pairs, float *__restrict__ dec_ws, uint16_t *__restrict__ tfrag,
    uint16_t *__restrict__ pfrag, uint16_t *__restrict__ qfrag) {
  static_assert(sizeof(TIn) == 2, "bf16 inputs (float32 inputs take prefill_f32.hip)");
  static_assert(HPW == 1 || HPW == 2, "heads per work-group");
  using F = Cfg<D, C>;
  using LL = LocalLds<D, C, HPW>;
  constexpr int NIB = F::NIB, KS = F::KS, AP = LL::AP;
  constexpr int NKI = C * D / 512;  // 1 KB pieces of the K (or Q) tile
  constexpr int KPR = D / 8;        // 16-byte pieces per row
  static_assert(NIB == 1 || NIB == 2 || NIB == 4, "16-token blocks per chunk");
  __shared__ __attribute__((aligned(16))) LL L;
  uint16_t *Kt = L.u.kq;

  // Block id -> (chunk, key head) pair and set of HPW heads of the group.
  // Work-groups are dealt to the eight XCDs round robin, so ids b and b + 8
  // share one: the head sets of a group for one pair take ids
  // 8 (nsets j + gi) + x.
  const int nsets = group / HPW;
  const int bid = blockIdx.x;
  const int xg = bid & 7, jj = bid >> 3;
  const int gi = jj % nsets;
  const int pair = (jj / nsets) * 8 + xg;
  if (pair >= n_pairs) return;
  const int cidx = pair / hqk, hk = pair - cidx * hqk;
  const int h0 = hk * group + gi * HPW;  // heads h0 .. h0 + HPW - 1
  const int64_t slot0 = (int64_t)cidx * hv + h0;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
  const int l16 = lane & 15, g4 = lane >> 4;

  // ---- the sequence owning slot cidx, if any: each wavefront tests the
  // sequences 64 at a time and takes the (single) hit from a ballot.
  int n = -1, cu_n = 0, cu_n1 = 0;
  for (int m0 = 0; m0 < n_seqs; m0 += 64) {
    const int m = m0 + lane;
    int a = 0, b = 0;
    bool hit = false;
    if (m < n_seqs) {
      a = cu[m];
      b = cu[m + 1];
      const int64_t base = (int64_t)a / C + m;  // first_slot(cu, m, C)
      hit = cidx >= base && cidx < base + (b - a + C - 1) / C;
    }
    const uint64_t bal = __ballot(hit);
    if (bal != 0) {
      const int src = __ffsll((unsigned long long)bal) - 1;
      n = m0 + src;
      cu_n = __builtin_amdgcn_readlane(a, src);
      cu_n1 = __builtin_amdgcn_readlane(b, src);
      break;
    }
  }
  if (n < 0) return;  // an unused slot: the same for every wavefront
  const int64_t t0 = cu_n + (cidx - ((int64_t)cu_n / C + n)) * C;
  const int nvalid = (int)min((int64_t)C, (int64_t)cu_n1 - t0);

  // ---- loads: rows past the end of the sequence read as zero
  const uint32_t rowb = (uint32_t)(nvalid * hqk * D * sizeof(TIn));
  const rsrc_t rk = make_rsrc(k + (t0 * hqk + hk) * D, rowb);
  const rsrc_t rq = make_rsrc(q + (t0 * hqk + hk) * D, rowb);
  // g and beta of token `lane` (0 past the end) for each head, read or
  // formed from the raw gate inputs
  float gl[HPW], bta[HPW];
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
    const int h = h0 + hh;
    if (gate.a_log != nullptr) {  // uniform over the launch
      const rsrc_t ra = make_rsrc(gate.a + t0 * hv, (uint32_t)(nvalid * hv * 4));
      const rsrc_t rb = make_rsrc(gate.b + t0 * hv, (uint32_t)(nvalid * hv * 4));
      const float ga = buf_load_f32(ra, (uint32_t)(lane * hv + h) * 4u);
      const float gb = buf_load_f32(rb, (uint32_t)(lane * hv + h) * 4u);
      const bool in = lane < nvalid;
      gl[hh] = in ? gate_log_decay(ga, gate.a_log[h], gate.dt_bias[h]) : 0.f;
      bta[hh] = in ? gate_beta(gb) : 0.f;
    } else {
      const rsrc_t rg = make_rsrc(g + t0 * hv, (uint32_t)(nvalid * hv * 4));
      const rsrc_t rb = make_rsrc(beta + t0 * hv, (uint32_t)(nvalid * hv * 4));
      gl[hh] = buf_load_f32(rg, (uint32_t)(lane * hv + h) * 4u);
      bta[hh] = buf_load_f32(rb, (uint32_t)(lane * hv + h) * 4u);
    }
  }
  // K: buffer-to-LDS copies (lane i of a copy fills bytes [16 i, 16 i + 16)
  // of its 1 KB piece, so the source offset picks the global 16-byte piece
  // that belongs at that swizzled position).
#pragma unroll
  for (int it = 0; it < (NKI + 3) / 4; ++it) {
    const int m = wave + 4 * it;
    if (m >= NKI) break;
    const int u = 64 * m + lane, row = u / KPR;
    const int gp = (u % KPR) ^ kn_swizzle<D>(row);
    const uint32_t off = (uint32_t)((row * hqk * D + 8 * gp) * 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void *)(Kt + 512 * m), 16, off, 0, 0, 0);
  }
  // Q: only the B operand of Q K^T (and the Q fragments of the per-tile
  // carry), so it goes straight into registers: wavefront w holds block row
  // w (when the chunk has one), in that operand's order: lane (l16, g4) of
  // step s holds Q[16 w + l16][32 s + 8 g4 + (0..7)]. Keeping it out of LDS
  // halves the kernel's LDS, so more work-groups fit per CU.
  const bool qrow = wave < NIB;
  uint4 qv[F::DS];
#pragma unroll
  for (int s = 0; s < F::DS; ++s)
    qv[s] = qrow ? buf_load_b128(rq, (uint32_t)(((16 * wave + l16) * hqk * D + 32 * s + 8 * g4) * 2))
                 : make_uint4(0, 0, 0, 0);
  // gamma: inclusive prefix sum of g over the chunk, lane t holding token t
  // (lanes past the end and past C hold g = 0: they repeat the last value).
  // Decay factors for the carry, exp(gamma_i) and exp(gamma_last - gamma_i),
  // of head `wave`: stored after the barrier below, whose wait for the K and
  // Q loads would otherwise also wait for these stores to complete.
  float dec_a = 0.f, dec_b = 0.f;
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
    const float gam = wave_prefix_sum(gl[hh]);
    if (wave == hh) {
      const float glast = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gam), C - 1));
      dec_a = __expf(gam);
      dec_b = __expf(glast - gam);
    }
    // per-wavefront copies of gamma and beta for the decay masks (outside
    // the K tile's space: Q K^T is masked before the tile is released)
    L.gam[hh][wave][lane] = gam;
    L.bet[hh][wave][lane] = bta[hh];
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (wave < HPW && lane < C) {
    const int64_t slot = slot0 + wave;
    dec_ws[slot * 2 * C + lane] = dec_a;
    dec_ws[slot * 2 * C + C + lane] = dec_b;
  }

  // ---- for the per-tile carry (qfrag not null): Q of this chunk in the
  // A-operand order of Q S^T, block ib, step s, lane (l16, g4) holding
  // Q[16 ib + l16][32 s + 8 g4 + (0..7)]: the registers of wavefront ib. One
  // value head of the group writes them.
  if (gi == 0 && qrow && qfrag != nullptr) {  // one head set of the group
    const int64_t base = ((int64_t)cidx * hqk + hk) * (C * D);
    const rsrc_t rqf = make_rsrc(qfrag + base, C * D * 2);
#pragma unroll
    for (int s = 0; s < F::DS; ++s)
      buf_store_b128<kCachePolicyDevice>(rqf, (uint32_t)((((wave * F::DS + s) * 64 + lane) * 8) * 2),
                                         qv[s]);
  }

  // ---- Gram tiles and decay masks: row `wave` of Q K^T, row NIB-1-wave of K K^T
  {
    uint16_t *pfb[HPW];
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) pfb[hh] = pfrag + (slot0 + hh) * F::FRAG;
    constexpr int M = NIB - 1;  // K K^T row of wavefront w: M - w
    if (wave == 0)
      gram_row_masks<D, C, HPW, 0, M>(L, Kt, qv, wave, pfb, lane);
    else if (wave == 1)
      gram_row_masks<D, C, HPW, 1, (M >= 1 ? M - 1 : 0)>(L, Kt, qv, wave, pfb, lane);
    else if (wave == 2)
      gram_row_masks<D, C, HPW, 2, (M >= 2 ? M - 2 : 0)>(L, Kt, qv, wave, pfb, lane);
    else
      gram_row_masks<D, C, HPW, 3, (M >= 3 ? M - 3 : 0)>(L, Kt, qv, wave, pfb, lane);
  }

  // ---- diagonal blocks. Neumann product: wavefront b inverts block b and
  // stores it transposed (linv[b] row c = column c of the inverse).
  if (NEUMANN && wave < NIB) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      const f32x4 tb = neumann_diag<AP>(L.u.inv.A[hh][wave * (wave + 1) / 2 + wave], g4, l16);
#pragma unroll
      for (int e = 0; e < 4; ++e) L.u.inv.linv[hh][wave][l16 * 17 + 4 * g4 + e] = tb[e];
    }
  }
  // Forward substitution, wavefront hh for head hh: lane (b, c) = (g4, l16)
  // solves (I + A[b][b]) x = e_c, i.e. column c of T[b][b], and stores it as
  // row c of the transposed inverse.
  if (!NEUMANN && wave < HPW) {
    const int hh = wave;
    const int b = min(g4, NIB - 1);  // lanes past the last block repeat it
    const float *Ab = L.u.inv.A[hh][b * (b + 1) / 2 + b];
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float s0 = (i == l16) ? 1.f : 0.f, s1 = 0.f;
#pragma unroll
      for (int j = 0; j + 1 < i; j += 2) {
        s0 -= Ab[i * AP + j] * x[j];
        s1 -= Ab[i * AP + j + 1] * x[j + 1];
      }
      if (i & 1) s0 -= Ab[i * AP + i - 1] * x[i - 1];
      x[i] = s0 + s1;
    }
    if (g4 < NIB) {
#pragma unroll
      for (int i = 0; i < 16; ++i) L.u.inv.linv[hh][b][l16 * 17 + i] = x[i];
    }
  }
  lds_barrier();

  // ---- block row ib = wave of each head, right to left: Z[c] = (T[ib][c])^T.
#pragma unroll
  for (int hh = 0; hh < HPW; ++hh) {
    if (wave >= NIB) break;
    const int ib = wave;
    const int64_t slot = slot0 + hh;
    const float *bw = L.bet[hh][wave];
    f32x4 Z[NIB];
#pragma unroll
    for (int c = 0; c < NIB; ++c) {
      Z[c] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (c == ib) {
#pragma unroll
        for (int e = 0; e < 4; ++e) Z[c][e] = L.u.inv.linv[hh][ib][(4 * g4 + e) * 17 + l16];
      }
    }
#pragma unroll
    for (int c = NIB - 2; c >= 0; --c) {
      if (c >= ib) continue;
      f32x4 R = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 1; m < NIB; ++m) {
        if (m <= c || m > ib) continue;
        const float *Amc = L.u.inv.A[hh][m * (m + 1) / 2 + c];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          R = mfma_16x16x4_f32(Amc[(4 * g4 + kk) * AP + l16], Z[m][kk], R);
      }
      f32x4 Zc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        Zc = mfma_16x16x4_f32(L.u.inv.linv[hh][c][l16 * 17 + 4 * g4 + kk], R[kk], Zc);
      Z[c] = -Zc;
    }
    // Fold beta into the factor: the carry uses T' = T diag(beta), so that
    // U = T' (V - exp(gamma) X) needs no beta of its own.
#pragma unroll
    for (int c = 0; c < NIB; ++c) {
      if (c > ib) continue;
      const float4 bc = *reinterpret_cast<const float4 *>(&bw[16 * c + 4 * g4]);
      Z[c][0] *= bc.x;
      Z[c][1] *= bc.y;
      Z[c][2] *= bc.z;
      Z[c][3] *= bc.w;
    }
    // T' as A-operand fragments, same token order as P.
    const rsrc_t rtf = make_rsrc(tfrag + slot * F::FRAG, F::FRAG * 2);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (2 * s > ib) continue;  // above the diagonal: zero, never stored or read
      const f32x4 lo4 = Z[2 * s];
      const f32x4 hi4 = (2 * s + 1 < NIB) ? Z[(2 * s + 1) % NIB] : f32x4{0.f, 0.f, 0.f, 0.f};
      buf_store_b128<kCachePolicyDevice>(
          rtf, (uint32_t)((((ib * KS + s) * 64 + lane) * 8) * 2),
          make_uint4(pack_bf16x2(lo4[0], lo4[1]), pack_bf16x2(lo4[2], lo4[3]),
                     pack_bf16x2(hi4[0], hi4[1]), pack_bf16x2(hi4[2], hi4[3])));
    }
  }
}

// ============================================================ single-wave carry
// The carry for batches of short sequences: one wavefront per (sequence,
// value head, 16-row value tile), 4 independent wavefronts per work-group,
// no barrier and no exchange between wavefronts. It walks the chunks of its
// sequence like the work-group carry; it is chosen when the average
// sequence fits in one chunk, where the work-group carry's fixed cost per
// work-group (ten wavefronts, the LDS of four chunk buffers) dominates.
//
// The state tile lives in the wavefront's accumulators for all key tiles:
// lane (l16, g4) element e of tile t is S[v0 + l16][16 t + 4 g4 + e]. Every
// contraction over the keys names its slots so that step s, slot
// 8 g + 4 hh + e stands for key 32 s + 16 hh + 4 g + e (the order of tok_pos
// over the keys): the bf16 B operand of S^T is then packed straight from
// tiles 2 s and 2 s + 1, and the A operands (K rows from LDS, Q rows from
// global memory) supply their keys in the same order. Y and U come out of
// their products in the accumulator layout, which in the token order of
// tok_pos is already the B operand of T' Y, P U and K^T (e U). Only K goes
// through LDS, for the K^T operands of the state update (transpose reads).
template <int D, int C>
struct WaveCfg {
  using F = Cfg<D, C>;
  static constexpr int WAVES = 4;
  static constexpr int NKI = C * D / 512;  // 1 KB copies per K chunk
};

template <int D, int C, typename TIn>
__global__ __launch_bounds__(256) void chunk_wave_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k, const TIn *__restrict__ v,
    const int32_t *__restrict__ cu, const float *__restrict__ dec_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag,
    const float *s0, float *sT, TIn *__restrict__ o, int n_units, int hqk, int hv, int group) {
  static_assert(sizeof(TIn) == 2, "bf16 inputs (float32 inputs take prefill_f32.hip)");
  using F = Cfg<D, C>;
  using WC = WaveCfg<D, C>;
  constexpr int NIB = F::NIB, KS = F::KS, DS = F::DS, NKT = F::NKT, NVT = F::NVT;
  __shared__ __attribute__((aligned(16))) uint16_t Kw[WC::WAVES][F::CP * D];

  // Work-group id -> (sequence, key head) unit and its tiles: every unit's
  // work-groups go to one XCD (ids b, b + 8, ...), so the value heads and
  // tiles that share K, Q, T' and P share an L2.
  const int tiles = group * NVT;                     // tiles per unit
  const int wpu = (tiles + WC::WAVES - 1) / WC::WAVES;  // work-groups per unit
  const int id = blockIdx.x;
  const int xg = id & 7, jj = id >> 3;
  const int unit = (jj / wpu) * 8 + xg;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tix = (jj % wpu) * WC::WAVES + wave;
  const int lane = threadIdx.x & 63, l16 = lane & 15, g4 = lane >> 4;
  uint16_t *K = Kw[wave];
  if (C < F::CP) {  // token rows past the chunk stay zero (K^T reads cover CP rows)
    for (int idx = C * D + lane; idx < F::CP * D; idx += 64) K[idx] = 0;
  }
  if (unit >= n_units || tix >= tiles) return;  // whole wavefront
  const int n = unit / hqk, hk = unit % hqk;
  const int gi = tix / NVT, vt = tix % NVT;
  const int h = hk * group + gi, v0 = 16 * vt;
  const int64_t pair = (int64_t)n * hv + h;
  const int64_t seq_t0 = cu[n], seq_t1 = cu[n + 1];
  const int nch = (int)((seq_t1 - seq_t0 + C - 1) / C);
  const int64_t c0 = first_slot(cu, n, C);

  f32x4 Sacc[NKT];
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
    Sacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (s0 != nullptr) {
      const float4 x = *reinterpret_cast<const float4 *>(s0 + (pair * D + v0 + l16) * D + 16 * t + 4 * g4);
      Sacc[t] = f32x4{x.x, x.y, x.z, x.w};
    }
  }

  const uint16_t *ksrc = reinterpret_cast<const uint16_t *>(k);
  const int kstride = hqk * D;

  for (int lc = 0; lc < nch; ++lc) {
    const int64_t t0 = seq_t0 + (int64_t)lc * C;
    const int nv = (int)min((int64_t)C, seq_t1 - t0);
    const int64_t slot = (c0 + lc) * hv + h;
    // ---- loads: K chunk into LDS (rows past nv read as zero), the tables
    const rsrc_t rk = make_rsrc(ksrc + (t0 * hqk + hk) * D, (uint32_t)(nv * hqk * D * 2));
#pragma unroll
    for (int m = 0; m < WC::NKI; ++m) {
      // (the offset goes in as a plain scalar: with an array element as the
      // builtin's argument the host pass emitted no launch stub)
      const uint32_t off = tile_copy_offset<D>(m, lane, kstride);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void *)(K + 512 * m), 16, off, 0, 0, 0);
    }
    const rsrc_t rt = make_rsrc(tfrag + slot * F::FRAG, F::FRAG * 2);
    const rsrc_t rp = make_rsrc(pfrag + slot * F::FRAG, F::FRAG * 2);
    const rsrc_t rv = make_rsrc(v + (t0 * hv + h) * D + v0, (uint32_t)(nv * hv * D * sizeof(TIn)));
    const float *dec = dec_ws + slot * 2 * C;
    f32x4 ga[NIB], he[NIB], Y[NIB];
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      const float4 x = *reinterpret_cast<const float4 *>(dec + 16 * ib + 4 * g4);
      const float4 y = *reinterpret_cast<const float4 *>(dec + C + 16 * ib + 4 * g4);
      ga[ib] = f32x4{x.x, x.y, x.z, x.w};
      he[ib] = f32x4{y.x, y.y, y.z, y.w};
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Y[ib][e] = BufElem<TIn>::load1(rv, (uint32_t)((16 * ib + 4 * g4 + e) * hv * D + l16));
    }
    const float glast = dec[C - 1];
    // At C = 32 the T', P and Q operands of the whole chunk are loaded here
    // too, so that the chunk waits for memory once (64 x 32 tokens: 74.8 ->
    // 69.3 us). At C = 16 the extra registers cost more occupancy than the
    // wait (512 x 12 tokens: 314.8 -> 371.6 us), and at C = 64 they would not
    // fit; there the operands are loaded where they are used.
    constexpr bool PRELOAD = C == 32;
    const rsrc_t rq = make_rsrc(q + (t0 * hqk + hk) * D, (uint32_t)(nv * hqk * D * sizeof(TIn)));
    uint4 ta[PRELOAD ? NIB * KS : 1], pa[PRELOAD ? NIB * KS : 1];
    uint2 qa[PRELOAD ? NIB * DS * 2 : 1];
    if constexpr (PRELOAD) {
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
        for (int st = 0; st < frag_steps<C>(ib); ++st) {
          const uint32_t off = (uint32_t)(((ib * KS + st) * 64 + lane) * 16);
          ta[ib * KS + st] = buf_load_b128(rt, off);
          pa[ib * KS + st] = buf_load_b128(rp, off);
        }
#pragma unroll
        for (int st = 0; st < DS; ++st) {
          const uint32_t e0 = (uint32_t)((16 * ib + l16) * hqk * D + 32 * st + 4 * g4);
          qa[(ib * DS + st) * 2] = BufElem<TIn>::load4_bf16(rq, e0);
          qa[(ib * DS + st) * 2 + 1] = BufElem<TIn>::load4_bf16(rq, e0 + 16);
        }
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // K has landed in LDS

    // ---- the state as the bf16 B operand of S^T, key order as above
    uint4 SB[DS];
#pragma unroll
    for (int st = 0; st < DS; ++st)
      SB[st] = make_uint4(pack_bf16x2(Sacc[2 * st][0], Sacc[2 * st][1]),
                          pack_bf16x2(Sacc[2 * st][2], Sacc[2 * st][3]),
                          pack_bf16x2(Sacc[2 * st + 1][0], Sacc[2 * st + 1][1]),
                          pack_bf16x2(Sacc[2 * st + 1][2], Sacc[2 * st + 1][3]));

    // ---- Y = V - exp(gamma) (K S^T), block by block
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      if (!PRELOAD) asm volatile("" ::: "memory");  // operands read per block
      f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < DS; ++st) {
        const int row = 16 * ib + l16, col = 32 * st + 4 * g4;
        const uint2 lo = *reinterpret_cast<const uint2 *>(&K[kn_index<D>(row, col)]);
        const uint2 hi = *reinterpret_cast<const uint2 *>(&K[kn_index<D>(row, col + 16)]);
        x = mfma_16x16x32(key_operand(lo, hi), SB[st], x);
      }
      Y[ib] = Y[ib] - ga[ib] * x;
    }

    // ---- U = T' Y (beta is folded into T')
    f32x4 U[NIB];
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      U[ib] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < frag_steps<C>(ib); ++st) {
        const uint4 a = PRELOAD ? ta[(ib * KS + st) % (PRELOAD ? NIB * KS : 1)]
                                : buf_load_b128(rt, (uint32_t)(((ib * KS + st) * 64 + lane) * 16));
        U[ib] = mfma_16x16x32(a, u_operand<NIB>(Y, st, nullptr), U[ib]);
      }
    }

    // ---- O = exp(gamma) (Q S^T) + P U, stored by block
    const rsrc_t ro = make_rsrc(o + (t0 * hv + h) * D + v0, (uint32_t)(nv * hv * D * sizeof(TIn)));
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      // without preloading, keep each block's loads in its own iteration
      // (hoisted, the loads of all blocks held twice the registers)
      if (!PRELOAD) asm volatile("" ::: "memory");
      f32x4 qs = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < DS; ++st) {
        uint2 lo, hi;
        if constexpr (PRELOAD) {
          lo = qa[((ib * DS + st) * 2) % (PRELOAD ? NIB * DS * 2 : 1)];
          hi = qa[((ib * DS + st) * 2 + 1) % (PRELOAD ? NIB * DS * 2 : 1)];
        } else {
          const uint32_t e0 = (uint32_t)((16 * ib + l16) * hqk * D + 32 * st + 4 * g4);
          lo = BufElem<TIn>::load4_bf16(rq, e0);
          hi = BufElem<TIn>::load4_bf16(rq, e0 + 16);
        }
        qs = mfma_16x16x32(key_operand(lo, hi), SB[st], qs);
      }
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < frag_steps<C>(ib); ++st) {
        const uint4 a = PRELOAD ? pa[(ib * KS + st) % (PRELOAD ? NIB * KS : 1)]
                                : buf_load_b128(rp, (uint32_t)(((ib * KS + st) * 64 + lane) * 16));
        acc = mfma_16x16x32(a, u_operand<NIB>(U, st, nullptr), acc);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e)
        BufElem<TIn>::store1_stream(ro, (uint32_t)((16 * ib + 4 * g4 + e) * hv * D + l16),
                                    ga[ib][e] * qs[e] + acc[e]);
    }

    // ---- S^T <- exp(gamma_last) S^T + K^T (exp(gamma_last - gamma) U)
    uint4 bu[KS];
#pragma unroll
    for (int st = 0; st < KS; ++st) bu[st] = u_operand<NIB>(U, st, he);
#pragma unroll
    for (int t = 0; t < NKT; ++t) {
      if (!PRELOAD) asm volatile("" ::: "memory");  // K^T operands read per tile
      f32x4 acc = Sacc[t] * glast;
#pragma unroll
      for (int st = 0; st < KS; ++st) acc = mfma_16x16x32(kt_operand<D>(K, t, st, l16, g4), bu[st], acc);
      Sacc[t] = acc;
    }
    // every read of this chunk's K is done before the next chunk's copy
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
#pragma unroll
  for (int t = 0; t < NKT; ++t)
    store_stream(sT + (pair * D + v0 + l16) * D + 16 * t + 4 * g4, Sacc[t]);
}

// ============================================================ host side
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int chain_segment_chunks(int n_seqs, int64_t n_tokens, int hv, int chunk, int requested) {
  if (requested > 0) return requested;
  const int64_t nck = (n_tokens + chunk - 1) / chunk;  // chunks of the longest possible chain
  const int64_t chains = (int64_t)std::max(n_seqs, 1) * hv;
  int64_t l;
  if (chains >= kChainUnits) {
    // The chains fill the chip: only a chain far longer than the average is
    // cut, into segments of the length at which the whole batch as one chain
    // would give kChainUnits work-groups.
    l = (nck * hv + kChainUnits - 1) / kChainUnits;
  } else {
    // Sequences of the average length are cut into as many segments as keep
    // every (segment, value head) in one round of kChainUnits work-groups,
    // and not at all when two would not fit: 6 x 4096 tokens (192 chains) at
    // C = 32 ran 473 us in two segments per sequence, 360 us in one.
    const int64_t avg = (nck + std::max(n_seqs, 1) - 1) / std::max(n_seqs, 1);
    const int64_t g = kChainUnits / chains;
    l = (avg + g - 1) / g;
  }
  return (int)std::min<int64_t>(std::max<int64_t>(l, kMinSegmentChunks), 1 << 20);
}

bool uses_tile_carry(int n_seqs, int64_t n_tokens, int hv, int d, int chunk) {
  const int64_t chains = (int64_t)n_seqs * hv;
  if (chains >= kChainCarryMinChains ||
      chain_segment_chunks(n_seqs, n_tokens, hv, chunk, 0) >= kChainMinSegment)
    return false;
  if (d < 128 || n_seqs <= 0) return true;
  // d = 128: eight 16-row tiles per chain make the per-tile carry's
  // work-groups many once chains reach the low hundreds. Measured (16/32
  // heads, N equal sequences of L tokens, each carry with its best chunk):
  // 7 x 1024 tokens whole-chain 97 against 140 us, 6 x 512 57 against 74,
  // 5 x 256 37 against 45, 4 x 512 53 against 54; the per-tile carry stays
  // ahead at 4 x 256 (36 against 40 us) and 5 x 128 (31 against 32).
  const int64_t avg = (n_tokens + n_seqs - 1) / n_seqs;
  return !(chains >= 192 || (chains >= 160 && avg >= 256) || (chains >= 128 && avg >= 512));
}

PrefillWorkspace prefill_workspace_layout(int n_seqs, int64_t n_tokens, int hqk,
                                          int hv, int d, int chunk, int seg_chunks, bool tile) {
  PrefillWorkspace w;
  const int64_t nc = chunk_bound(n_seqs, n_tokens, chunk);
  size_t p = 0;
  w.decay = p;
  p = align256(p + sizeof(float) * (size_t)nc * hv * 2 * chunk);
  w.tfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hv * frag_elems(chunk));
  w.pfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hv * frag_elems(chunk));
  const bool wave = uses_wave_carry(n_seqs, n_tokens, chunk);
  w.qfrag = p;
  if (tile && !wave) p = align256(p + sizeof(uint16_t) * (size_t)nc * hqk * chunk * d);
  // Maps of every segment but the last of each sequence (whole-chain carry):
  // at most T / span slots, and none when every sequence fits in one segment.
  const int64_t span = (int64_t)chunk * seg_chunks;
  w.n_maps = (!wave && !tile && span < n_tokens) ? n_tokens / span : 0;
  const size_t mbytes = (size_t)w.n_maps * hv * d * d;
  w.bslot = p;
  p = align256(p + sizeof(float) * mbytes);
  w.mthi = p;
  p = align256(p + sizeof(uint16_t) * mbytes);
  w.mtlo = p;
  p = align256(p + sizeof(uint16_t) * mbytes);
  w.order = p;
  if (!wave && !tile && span > 0 && n_seqs > 1)  // (one sequence: block order)
    p = align256(p + sizeof(int32_t) * (size_t)(n_tokens / span + n_seqs));
  w.total = p;
  return w;
}

template <int D, int C, typename TIn>
static hipError_t launch_prefill_t(const PrefillArgs &a, const PrefillWorkspace &ws) {
  using F = Cfg<D, C>;
  char *base = static_cast<char *>(a.workspace);
  float *dec = reinterpret_cast<float *>(base + ws.decay);
  uint16_t *tf = reinterpret_cast<uint16_t *>(base + ws.tfrag);
  uint16_t *pf = reinterpret_cast<uint16_t *>(base + ws.pfrag);
  uint16_t *qf =
      (a.tile_carry && !a.wave_carry) ? reinterpret_cast<uint16_t *>(base + ws.qfrag) : nullptr;
  const int group = a.hv / a.hqk;

  const int64_t nc = chunk_bound(a.n_seqs, a.n_tokens, C);
  if (a.n_tokens > 0) {
    // (chunk, key head) pairs in groups of eight, times the heads of a group.
    const int64_t pairs = nc * a.hqk;
    // Two value heads per work-group when the group has an even size: they
    // share the K tile and the Gram products.
    const int hpw = (group % 2 == 0) ? 2 : 1;
    const int64_t lblocks = ((pairs + 7) / 8) * 8 * (group / hpw);
    auto local = hpw == 2 ? (a.neumann ? chunk_local_kernel<D, C, TIn, true, 2>
                                       : chunk_local_kernel<D, C, TIn, false, 2>)
                          : (a.neumann ? chunk_local_kernel<D, C, TIn, true, 1>
                                       : chunk_local_kernel<D, C, TIn, false, 1>);
    hipLaunchKernelGGL(local, dim3((unsigned)lblocks), dim3(256), 0, a.stream, (const TIn *)a.q,
                       (const TIn *)a.k, a.g, a.beta, a.gate, a.cu_seqlens, a.n_seqs, a.hqk, a.hv,
                       group, (int)pairs, dec, tf, pf, qf);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  // The per-tile carry for few chains, else the whole-chain carry, unless
  // the average sequence fits in one chunk: then the single-wave carry, which
  // walks sequences of any length.
  if (!a.wave_carry)
    return a.tile_carry ? launch_tile_carry(a, ws) : launch_chain_d(a, ws);
  const int n_groups = a.n_seqs * a.hqk;
  const int wpu = (group * F::NVT + WaveCfg<D, C>::WAVES - 1) / WaveCfg<D, C>::WAVES;
  const int64_t wblocks = (int64_t)8 * ((n_groups + 7) / 8) * wpu;
  hipLaunchKernelGGL((chunk_wave_kernel<D, C, TIn>), dim3((unsigned)wblocks), dim3(256), 0,
                     a.stream, (const TIn *)a.q, (const TIn *)a.k, (const TIn *)a.v,
                     a.cu_seqlens, dec, tf, pf, a.initial_state, a.final_state, (TIn *)a.o,
                     n_groups, a.hqk, a.hv, group);
  return hipGetLastError();
}

template <int D, typename TIn>
static hipError_t launch_prefill_d(const PrefillArgs &a, const PrefillWorkspace &ws) {
  switch (a.chunk) {
    case 16: return launch_prefill_t<D, 16, TIn>(a, ws);
    case 32: return launch_prefill_t<D, 32, TIn>(a, ws);
    case 64: return launch_prefill_t<D, 64, TIn>(a, ws);
    default: return hipErrorInvalidValue;
  }
}

template <typename TIn>
static hipError_t launch_prefill_e(const PrefillArgs &a, const PrefillWorkspace &ws) {
  switch (a.d) {
    case 32: return launch_prefill_d<32, TIn>(a, ws);
    case 64: return launch_prefill_d<64, TIn>(a, ws);
    case 128: return launch_prefill_d<128, TIn>(a, ws);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_prefill(const PrefillArgs &a, const PrefillWorkspace &ws) {
  // float32 inputs: the float32-throughout form (prefill_f32.hip), no workspace
  return a.dtype == GDN_BF16 ? launch_prefill_e<__bf16>(a, ws) : launch_prefill_f32(a);
}

}  // namespace gdn
