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
#include "gdn_device.h"
#include "gdn_launch.h"

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

// ============================================================ chunk-local
// One work-group per (chunk, value head): gamma, K K^T and K Q^T, then A, P
// and T = (I + A)^-1, written as bf16 A-operand fragments. The two Gram
// products depend only on the key head; the value heads of a GQA group each
// recompute them (a few dozen matrix instructions) rather than share a
// longer work-group, and the launch order puts the heads of one group on
// the same XCD so that the second reads K and Q from its L2.
//
// The 16x16 tiles of the two lower-triangular Gram products are dealt out
// evenly: wavefront w computes product (w & 1) (0: K K^T for A, 1: K Q^T
// for P) for the block rows of row set (w >> 1).
//
// T is built from its 16x16 blocks in fp32. Diagonal block b is inverted
// either by forward substitution on the vector ALU (one lane per column, all
// blocks at once in one wavefront) or, with NEUMANN, by the Neumann product
// on the matrix cores (one block per wavefront, see neumann_diag); wavefront
// b then forms its block row from
//   T[b][c] = -(sum_{m=c+1..b} T[b][m] A[m][c]) T[c][c]^-1    (c < b),
// carried in transposed form so that every intermediate stays in the
// accumulator layout of the fp32 16x16x4 matrix instruction.
template <int D, int C>
struct LocalLds {
  static constexpr int NIB = C / 16;
  static constexpr int NBLK = NIB * (NIB + 1) / 2;  // lower blocks, diagonal included
  static constexpr int AP = 20;                     // f32 pitch of an A block row
  union {
    uint16_t kq[2 * C * D];  // K tile, then Q tile; swizzled rows (kn_index)
    struct {
      float A[NBLK][16 * AP];     // block (m, c) at m (m + 1) / 2 + c, row-major
      float linv[NIB][16 * 17];   // transposed diagonal inverses
      float gam[4][64];           // per-wavefront copies of gamma and beta
      float bet[4][64];
    } inv;
  } u;
};

// Block rows of row set p (one row set per pair of wavefronts): the longest
// row with the shortest, so that every set holds the same number of tiles.
template <int NIB>
__device__ __forceinline__ int gram_row(int p, int r) {
  if (r == 0) return NIB - 1 - p;
  return NIB == 4 ? p : -1;
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

template <int D, int C, typename TIn, bool NEUMANN>
__global__ __launch_bounds__(256) void chunk_local_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const float *__restrict__ g, const float *__restrict__ beta, GateArgs gate,
    const int32_t *__restrict__ cu, int n_seqs, int hqk, int hv, int group,
    int n_pairs, float *__restrict__ dec_ws, uint16_t *__restrict__ tfrag,
    uint16_t *__restrict__ pfrag, uint16_t *__restrict__ qfrag,
    uint16_t *__restrict__ kcopy) {
  using F = Cfg<D, C>;
  using LL = LocalLds<D, C>;
  constexpr int NIB = F::NIB, KS = F::KS, AP = LL::AP;
  constexpr int NKI = C * D / 512;  // 1 KB pieces of the K (or Q) tile
  constexpr int KPR = D / 8;        // 16-byte pieces per row
  static_assert(NIB == 1 || NIB == 2 || NIB == 4, "row sets");
  __shared__ __attribute__((aligned(16))) LL L;
  uint16_t *Kt = L.u.kq, *Qt = L.u.kq + C * D;

  // Block id -> (chunk, key head) pair and head of the group. Work-groups are
  // dealt to the eight XCDs round robin, so ids b and b + 8 share one: the
  // heads of a group for one pair take ids 8 (group j + gi) + x.
  const int bid = blockIdx.x;
  const int xg = bid & 7, jj = bid >> 3;
  const int gi = jj % group;
  const int pair = (jj / group) * 8 + xg;
  if (pair >= n_pairs) return;
  const int cidx = pair / hqk, hk = pair - cidx * hqk;
  const int h = hk * group + gi;
  const int64_t slot = (int64_t)cidx * hv + h;

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
  // g and beta of token `lane` (0 past the end), read or formed from the raw
  // gate inputs
  float gl, bta;
  if (gate.a_log != nullptr) {  // uniform over the launch
    const rsrc_t ra = make_rsrc(gate.a + t0 * hv, (uint32_t)(nvalid * hv * 4));
    const rsrc_t rb = make_rsrc(gate.b + t0 * hv, (uint32_t)(nvalid * hv * 4));
    const float ga = buf_load_f32(ra, (uint32_t)(lane * hv + h) * 4u);
    const float gb = buf_load_f32(rb, (uint32_t)(lane * hv + h) * 4u);
    const bool in = lane < nvalid;
    gl = in ? gate_log_decay(ga, gate.a_log[h], gate.dt_bias[h]) : 0.f;
    bta = in ? gate_beta(gb) : 0.f;
  } else {
    const rsrc_t rg = make_rsrc(g + t0 * hv, (uint32_t)(nvalid * hv * 4));
    const rsrc_t rb = make_rsrc(beta + t0 * hv, (uint32_t)(nvalid * hv * 4));
    gl = buf_load_f32(rg, (uint32_t)(lane * hv + h) * 4u);
    bta = buf_load_f32(rb, (uint32_t)(lane * hv + h) * 4u);
  }
  if constexpr (sizeof(TIn) == 2) {
    // Buffer-to-LDS copies: lane i of a copy fills bytes [16 i, 16 i + 16) of
    // its 1 KB piece, so the source offset picks the global 16-byte piece that
    // belongs at that swizzled position.
#pragma unroll
    for (int it = 0; it < (2 * NKI + 3) / 4; ++it) {
      const int m = wave + 4 * it;
      if (m >= 2 * NKI) break;
      const bool isq = m >= NKI;
      const int mm = isq ? m - NKI : m;
      const int u = 64 * mm + lane, row = u / KPR;
      const int gp = (u % KPR) ^ kn_swizzle<D>(row);
      const uint32_t off = (uint32_t)((row * hqk * D + 8 * gp) * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isq ? rq : rk, (lds_void *)((isq ? Qt : Kt) + 512 * mm),
                                               16, off, 0, 0, 0);
    }
  } else {
    constexpr int NP = C * KPR;
    constexpr int NL = (NP + 255) / 256;
    uint4 kv[NL], qv[NL];
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const int idx = min(tid + 256 * u, NP - 1);
      const uint32_t e = (uint32_t)((idx / KPR) * hqk * D + (idx % KPR) * 8);
      kv[u] = BufElem<TIn>::load8(rk, e);
      qv[u] = BufElem<TIn>::load8(rq, e);
    }
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const int idx = tid + 256 * u;
      if (idx < NP) {
        const int x = kn_index<D>(idx / KPR, 8 * (idx % KPR));
        *reinterpret_cast<uint4 *>(&Kt[x]) = kv[u];
        *reinterpret_cast<uint4 *>(&Qt[x]) = qv[u];
      }
    }
  }
  // gamma: inclusive prefix sum of g over the chunk, lane t holding token t
  // (lanes past the end and past C hold g = 0: they repeat the last value).
  const float gam = wave_prefix_sum(gl);
  if (wave == 0 && lane < C) {
    // decay factors for the carry: exp(gamma_i) and exp(gamma_last - gamma_i)
    const float glast = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gam), C - 1));
    dec_ws[slot * 2 * C + lane] = __expf(gam);
    dec_ws[slot * 2 * C + C + lane] = __expf(glast - gam);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // ---- Q of this chunk for the carry, in the A-operand order of Q S^T:
  // block ib, step s, lane (l16, g4) holds Q[16 ib + l16][32 s + 8 g4 + (0..7)].
  // For f32 inputs also a bf16 copy of K, row-major [C][D], for the carry.
  // One value head of the group writes them.
  if (gi == 0 && wave < NIB) {
    const int64_t base = ((int64_t)cidx * hqk + hk) * (C * D);
    uint16_t *qf = qfrag + base + ((int64_t)wave * F::DS * 64 + lane) * 8;
#pragma unroll
    for (int s = 0; s < F::DS; ++s)
      *reinterpret_cast<uint4 *>(qf + s * 512) =
          *reinterpret_cast<const uint4 *>(&Qt[kn_index<D>(16 * wave + l16, 32 * s + 8 * g4)]);
    if (sizeof(TIn) == 4) {
      uint16_t *kc = kcopy + base + (int64_t)(16 * wave + l16) * D;
#pragma unroll
      for (int s = 0; s < F::DS; ++s)
        *reinterpret_cast<uint4 *>(kc + 32 * s + 8 * g4) =
            *reinterpret_cast<const uint4 *>(&Kt[kn_index<D>(16 * wave + l16, 32 * s + 8 * g4)]);
    }
  }

  // ---- Gram tiles (ib, jb), jb <= ib, of this wavefront's product. Lane
  // (l16, g4) element e holds  k_j . k_i  (or  k_j . q_i),  j = 16 jb + 4 g4 + e,
  // i = 16 ib + l16.
  const int prod = wave & 1;
  const int rset = wave >> 1;
  const uint16_t *Bt = prod ? Qt : Kt;
  int rows[2];
  f32x4 G[2][NIB];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    rows[r] = gram_row<NIB>(rset, r);
    const int ib = rows[r];
#pragma unroll
    for (int jb = 0; jb < NIB; ++jb) {
      G[r][jb] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (jb > ib) continue;
#pragma unroll
      for (int s = 0; s < F::DS; ++s) {
        const int col = 32 * s + 8 * g4;
        const uint4 a = *reinterpret_cast<const uint4 *>(&Kt[kn_index<D>(16 * jb + l16, col)]);
        const uint4 bb = *reinterpret_cast<const uint4 *>(&Bt[kn_index<D>(16 * ib + l16, col)]);
        G[r][jb] = mfma_16x16x32(a, bb, G[r][jb]);
      }
    }
  }
  lds_barrier();  // the K and Q tiles are dead; the space is reused below

  // ---- decay masks: A (product 0) to LDS, P (product 1) to global.
  float *gw = L.u.inv.gam[wave], *bw = L.u.inv.bet[wave];
  gw[lane] = gam;
  bw[lane] = bta;
  wave_lds_fence();
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int ib = rows[r];
    if (ib < 0) continue;
    const int i = 16 * ib + l16;
    const float gami = gw[i], bi = bw[i];
    f32x4 Pt[NIB];
#pragma unroll
    for (int jb = 0; jb < NIB; ++jb) {
      Pt[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (jb > ib) continue;
      const float4 gj = *reinterpret_cast<const float4 *>(&gw[16 * jb + 4 * g4]);
      const float gjv[4] = {gj.x, gj.y, gj.z, gj.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = 16 * jb + 4 * g4 + e;
        const float dec = (j <= i) ? __expf(gami - gjv[e]) : 0.f;
        Pt[jb][e] = prod ? dec * G[r][jb][e] : ((j < i) ? bi * dec * G[r][jb][e] : 0.f);
      }
      if (!prod)
        *reinterpret_cast<float4 *>(&L.u.inv.A[ib * (ib + 1) / 2 + jb][l16 * AP + 4 * g4]) =
            make_float4(Pt[jb][0], Pt[jb][1], Pt[jb][2], Pt[jb][3]);
    }
    if (prod) {
      // P as A-operand fragments: step s takes tile 2s (elements 0-3) and
      // tile 2s+1 (elements 4-7), i.e. the token order of tok_pos().
      uint16_t *pf = pfrag + slot * F::FRAG + ((int64_t)ib * KS * 64 + lane) * 8;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (2 * s > ib) continue;  // above the diagonal: zero, never stored or read
        const f32x4 lo4 = Pt[2 * s];
        const f32x4 hi4 = (2 * s + 1 < NIB) ? Pt[(2 * s + 1) % NIB] : f32x4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<uint4 *>(pf + s * 512) =
            make_uint4(pack_bf16x2(lo4[0], lo4[1]), pack_bf16x2(lo4[2], lo4[3]),
                       pack_bf16x2(hi4[0], hi4[1]), pack_bf16x2(hi4[2], hi4[3]));
      }
    }
  }
  lds_barrier();

  // ---- diagonal blocks. Neumann product: wavefront b inverts block b and
  // stores it transposed (linv[b] row c = column c of the inverse).
  if (NEUMANN && wave < NIB) {
    const f32x4 tb = neumann_diag<AP>(L.u.inv.A[wave * (wave + 1) / 2 + wave], g4, l16);
#pragma unroll
    for (int e = 0; e < 4; ++e) L.u.inv.linv[wave][l16 * 17 + 4 * g4 + e] = tb[e];
  }
  // Forward substitution: lane (b, c) = (g4, l16) solves (I + A[b][b]) x =
  // e_c, i.e. column c of T[b][b], and stores it as row c of the transposed
  // inverse.
  if (!NEUMANN && wave == 0) {
    const int b = min(g4, NIB - 1);  // lanes past the last block repeat it
    const float *Ab = L.u.inv.A[b * (b + 1) / 2 + b];
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
      for (int i = 0; i < 16; ++i) L.u.inv.linv[b][l16 * 17 + i] = x[i];
    }
  }
  lds_barrier();

  // ---- block row ib = wave, right to left: Z[c] = (T[ib][c])^T.
  if (wave < NIB) {
    const int ib = wave;
    f32x4 Z[NIB];
#pragma unroll
    for (int c = 0; c < NIB; ++c) {
      Z[c] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (c == ib) {
#pragma unroll
        for (int e = 0; e < 4; ++e) Z[c][e] = L.u.inv.linv[ib][(4 * g4 + e) * 17 + l16];
      }
    }
#pragma unroll
    for (int c = NIB - 2; c >= 0; --c) {
      if (c >= ib) continue;
      f32x4 R = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int m = 1; m < NIB; ++m) {
        if (m <= c || m > ib) continue;
        const float *Amc = L.u.inv.A[m * (m + 1) / 2 + c];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          R = mfma_16x16x4_f32(Amc[(4 * g4 + kk) * AP + l16], Z[m][kk], R);
      }
      f32x4 Zc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        Zc = mfma_16x16x4_f32(L.u.inv.linv[c][l16 * 17 + 4 * g4 + kk], R[kk], Zc);
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
    uint16_t *tf = tfrag + slot * F::FRAG + ((int64_t)ib * KS * 64 + lane) * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (2 * s > ib) continue;  // above the diagonal: zero, never stored or read
      const f32x4 lo4 = Z[2 * s];
      const f32x4 hi4 = (2 * s + 1 < NIB) ? Z[(2 * s + 1) % NIB] : f32x4{0.f, 0.f, 0.f, 0.f};
      *reinterpret_cast<uint4 *>(tf + s * 512) =
          make_uint4(pack_bf16x2(lo4[0], lo4[1]), pack_bf16x2(lo4[2], lo4[3]),
                     pack_bf16x2(hi4[0], hi4[1]), pack_bf16x2(hi4[2], hi4[3]));
    }
  }
}

// ============================================================ chunk carry
// One work-group per (sequence, value head, 16-row value tile): ten
// wavefronts, eight that compute and two that only move data.
//
// Compute wavefronts 0-3 own token block w of the chunk for X = K S^T, Y and
// U = T' Y; wavefronts 4-7 own token block w - 4 for Q S^T and O; all eight
// update one 16-key tile of the state each. The operands only one wavefront
// needs (its rows of T', P and Q, stored by the chunk-local kernel in operand
// order) are loaded straight into its registers one chunk ahead, 1 KB per
// contiguous load. What several wavefronts share goes through LDS: K (rows
// for X, columns for the state update), the V tile and the decay factors,
// copied by the two loader wavefronts with buffer-to-LDS loads into a buffer
// the compute wavefronts are not reading.
//
// Per chunk, three phases separated by work-group barriers carry the chain
// X -> Y -> U -> state; each phase reads from LDS only what the phase before
// produced (S^T, Y, U). Everything else a phase needs -- K rows and K^T
// operands, V and the decay factors -- is read into registers a phase or
// more ahead: waves 0-3 read those of chunk c + 1 right after the state
// update of chunk c (the reads stay in flight across the barrier), waves
// 4-7 their K^T operands in phase 1. Outputs go from registers straight to
// global memory.
//
// Global reads go through buffer resources: rows past the end of the
// sequence read as zero (beta is zero there, so they add exact zeros) and
// stores past the end are dropped by the resource extent.
template <int D, int C, typename TIn>
struct CarryCfg {
  using F = Cfg<D, C>;
  static constexpr int NCW = 8;                  // compute wavefronts
  static constexpr int NLW = 2;                  // loader wavefronts
  static constexpr int NT = 64 * (NCW + NLW);    // threads
  static constexpr int ESZ = (int)sizeof(TIn);
  static constexpr int KPR = D / 8;              // 16-byte units per bf16 K row
  static constexpr int NKI = C * D / 512;        // 1 KB copies per K chunk
  static constexpr int VPR = ESZ;                // 16-byte units per token of a V tile row
  static constexpr int VU = C * VPR;             // 16-byte units of the V tile
  static constexpr int NVI = (VU + 63) / 64;     // 1 KB copies per V tile
  static constexpr int NDI = (2 * C + 255) / 256;  // 1 KB copies of the 2C decay factors
  static constexpr int M = NKI + NVI + NDI;      // copies per chunk
  static constexpr int SLOTS = (M + NLW - 1) / NLW;
  static constexpr int NB = 4;                   // LDS buffers of the copied inputs
  static constexpr int NA = NB - 1;              // chunks issued ahead of the one in use
  static_assert(NT == 640, "launch bounds of the carry kernel");
};

constexpr int kCarryThreads = 640;

template <int D, int C, typename TIn>
struct CarryLds {
  using F = Cfg<D, C>;
  using CC = CarryCfg<D, C, TIn>;
  // The copied inputs of chunk lc live in buffer lc % NB.
  uint16_t Kn[CC::NB][F::CP * D];  // K chunk, row-major, swizzled; rows C..CP-1 stay zero
  uint4 Vl[CC::NB][CC::NVI * 64];  // V tile, [token][16 values], input element type
  float Dl[CC::NB][CC::NDI * 256];  // exp(gamma_i), then exp(gamma_last - gamma_i)
  uint16_t Sl[16 * F::LDK];     // bf16 copy of the state tile, [value][key]
  uint16_t Yl[16 * F::LDV];     // Y,  [value][token position]
  uint16_t Ul[16 * F::LDV];     // U,  [value][token position]
  uint16_t Uh[16 * F::LDV];     // exp(gamma_last - gamma) U, same layout
};

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

// ---------------------------------------------------------------- loaders
// Copy m of a chunk, in order: K, V tile, decay factors, each 16 bytes per
// lane (1 KB per copy). A buffer-to-LDS load writes lane i's bytes at
// LDS base + i * size, so the per-lane source offset chooses what lands
// where: for K it undoes the row swizzle. The offsets do not change from
// chunk to chunk.
template <int D, int C, typename TIn>
__device__ __forceinline__ uint32_t copy_offset(int m, int lane, int kstride, int hv) {
  using CC = CarryCfg<D, C, TIn>;
  if (m < CC::NKI) {
    const int u = 64 * m + lane, row = u / CC::KPR;
    const int jl = (u % CC::KPR) ^ kn_swizzle<D>(row);
    return (uint32_t)((row * kstride + 8 * jl) * 2);
  } else if (m < CC::NKI + CC::NVI) {
    const int u = 64 * (m - CC::NKI) + lane;
    if (u >= CC::VU) return kOutOfRange;
    return (uint32_t)(((u / CC::VPR) * hv * D + (u % CC::VPR) * (16 / CC::ESZ)) * CC::ESZ);
  } else if (m < CC::M) {
    const int u = 64 * (m - CC::NKI - CC::NVI) + lane;  // 4 factors per lane
    return 4 * u < 2 * C ? (uint32_t)(16 * u) : kOutOfRange;
  }
  return kOutOfRange;
}

struct CopyRes {
  rsrc_t k, v, d;
};

template <int D, int C, typename TIn>
__device__ __forceinline__ void issue_copy(CarryLds<D, C, TIn> &L, int bb, const CopyRes &R,
                                           int m, uint32_t off) {
  using CC = CarryCfg<D, C, TIn>;
  if (m < CC::NKI) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(R.k, (lds_void *)&L.Kn[bb][512 * m], 16, off, 0, 0, 0);
  } else if (m < CC::NKI + CC::NVI) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(R.v, (lds_void *)&L.Vl[bb][64 * (m - CC::NKI)], 16, off, 0, 0, 0);
  } else if (m < CC::M) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(R.d, (lds_void *)&L.Dl[bb][256 * (m - CC::NKI - CC::NVI)], 16, off, 0, 0, 0);
  }
}

// Copies loader LW issues per chunk.
template <int D, int C, typename TIn, int LW>
constexpr int loader_copies() {
  using CC = CarryCfg<D, C, TIn>;
  int n = 0;
  for (int i = 0; i < CC::SLOTS; ++i) n += (CC::NLW * i + LW < CC::M) ? 1 : 0;
  return n;
}

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

// Loader wavefront LW (a template parameter, so that the kind of each of its
// copies is known when compiling). The copies of chunk lc + NA are issued at
// the start of chunk lc into the buffer chunk lc - 1 used, and chunk lc + 1
// must have landed before the second barrier of chunk lc: waves 0-3 read it
// in phase 3.
template <int D, int C, typename TIn, int LW>
__device__ __forceinline__ void carry_loader(
    CarryLds<D, C, TIn> &L, int lane, const uint16_t *__restrict__ ksrc, int kstride,
    bool kcopied, const TIn *__restrict__ v, const float *__restrict__ dec_ws, int nch,
    int64_t seq_t0, int64_t seq_t1, int64_t c0, int h, int hk, int hqk, int hv, int v0) {
  using CC = CarryCfg<D, C, TIn>;
  constexpr int NS = CC::SLOTS;
  uint32_t off[NS];
#pragma unroll
  for (int i = 0; i < NS; ++i) off[i] = copy_offset<D, C, TIn>(CC::NLW * i + LW, lane, kstride, hv);

  auto res = [&](int lc) {
    const int64_t t0 = seq_t0 + (int64_t)lc * C;
    const int nv = (int)min((int64_t)C, seq_t1 - t0);
    CopyRes r;
    if (kcopied)  // bf16 copy in the workspace, [chunk slot][key head][C][D]
      r.k = make_rsrc(ksrc + ((c0 + lc) * hqk + hk) * (C * D), C * D * 2);
    else
      r.k = make_rsrc(ksrc + (t0 * hqk + hk) * D, (uint32_t)(nv * hqk * D * 2));
    r.v = make_rsrc(v + (t0 * hv + h) * D + v0, (uint32_t)(nv * hv * D * CC::ESZ));
    r.d = make_rsrc(dec_ws + ((c0 + lc) * hv + h) * 2 * C, 2 * C * 4);
    return r;
  };

  constexpr int NCP = loader_copies<D, C, TIn, LW>();
  constexpr int NA = CC::NA;
  auto issue = [&](int lc) {  // chunk lc into buffer lc % NB
    const CopyRes R = res(lc);
#pragma unroll
    for (int i = 0; i < NS; ++i) issue_copy<D, C, TIn>(L, lc % CC::NB, R, CC::NLW * i + LW, off[i]);
  };
#pragma unroll
  for (int j = 0; j < NA; ++j)
    if (j < nch) issue(j);
  if (nch >= NA)
    wait_vm<(NA - 1) * NCP>();  // chunk 0 has landed
  else
    wait_vm<0>();
  lds_barrier();

  for (int lc = 0; lc < nch; ++lc) {
    if (lc + NA < nch) issue(lc + NA);
    lds_barrier();
    // Chunk lc + 1 must have landed. While copies are still issued every
    // chunk, those of the NA - 1 later chunks may stay in flight; near the
    // end everything is waited for.
    if (lc + NA < nch)
      wait_vm<(NA - 1) * NCP>();
    else
      wait_vm<0>();
    lds_barrier();
    lds_barrier();
  }
}

// ---------------------------------------------------------------- compute
// Per chunk c, three phases separated by work-group barriers:
//   1. waves 0-3: X = K S^T for their token block, Y = V - exp(gamma) X.
//      waves 4-7: O of chunk c-1 = exp(gamma) Q S^T + P U (their operands
//      were kept from chunk c-1; U of chunk c-1 is still in LDS), stored to
//      global memory; the K^T operands of chunk c.
//   2. waves 0-3: U = T' Y and exp(gamma_last - gamma) U.
//      waves 4-7: Q S^T (S is still the state entering chunk c).
//   3. all eight: S^T <- exp(gamma_last) S^T + K^T (exp(gamma_last - gamma) U)
//      for their key tile; waves 0-3 then read chunk c + 1's operands.
// The chain from one state to the next runs through phases 1-3 on waves 0-3
// and the update; the output work fills the phases where it would idle.
template <int D, int C, typename TIn>
__device__ __forceinline__ void state_update(CarryLds<D, C, TIn> &L, f32x4 &S, const uint4 *kt,
                                             float glast, int wave, int l16, int g4) {
  using F = Cfg<D, C>;
  uint4 bu[F::KS];
#pragma unroll
  for (int s = 0; s < F::KS; ++s)
    bu[s] = *reinterpret_cast<const uint4 *>(&L.Uh[l16 * F::LDV + 32 * s + 8 * g4]);
  f32x4 acc = S * glast;
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int s = 0; s < F::KS; ++s) acc = mfma_16x16x32(kt[s], bu[s], acc);
  S = acc;
  *reinterpret_cast<uint2 *>(&L.Sl[l16 * F::LDK + 16 * wave + 4 * g4]) =
      pack4_bf16(acc[0], acc[1], acc[2], acc[3]);
}

// Wavefronts 0-3: X, Y and U for token block ib. Each role runs its own loop
// (with the same barriers) so that every register prefetched for the next
// chunk is consumed and then reloaded in place.
template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_compute_xu(
    CarryLds<D, C, TIn> &L, f32x4 &S, int wave, int lane, int nch, int64_t c0,
    const uint16_t *__restrict__ tfrag, int h, int hv) {
  using F = Cfg<D, C>;
  using CC = CarryCfg<D, C, TIn>;
  const int l16 = lane & 15, g4 = lane >> 4;
  const int ib = wave;
  const bool blk = (F::NIB == 4) || (ib < F::NIB);
  const bool own = (F::NKT == 8) || (wave < F::NKT);
  const int ibc = min(ib, F::NIB - 1);
  // T' fragments of block ibc on or below the diagonal; the others are zero,
  // never stored, and read through an offset past the resource (zeros).
  const int nks = min(ibc / 2 + 1, F::KS);
  const int tb = 16 * ibc + 4 * g4;                     // this lane's first token
  const int ypos = 32 * (ib >> 1) + 8 * g4 + 4 * (ib & 1);  // tok_pos(16 ib + 4 g4)
  const uint32_t foff = (uint32_t)(((ibc * F::KS) * 64 + lane) * 16);
  auto frag_res = [&](int lc) {
    return make_rsrc(tfrag + ((c0 + lc) * hv + h) * F::FRAG, F::FRAG * 2);
  };
  // operands of the chunk in use, read ahead
  uint4 fa[F::KS];   // T' rows of block ib (global)
  uint4 ka[F::DS];   // K rows of block ib (LDS)
  uint4 kt[F::KS];   // K^T operands of key tile `wave` (LDS)
  float vv[4], ge[4], he[4], glast = 0.f;
  auto fetch_lds = [&](int b) {  // V, decay factors, then K^T and K rows of buffer b
    if (blk) {
      const TIn *vt = reinterpret_cast<const TIn *>(L.Vl[b]);
#pragma unroll
      for (int e = 0; e < 4; ++e) vv[e] = Elem<TIn>::load1(&vt[(tb + e) * 16 + l16]);
      const float4 ge4 = *reinterpret_cast<const float4 *>(&L.Dl[b][tb]);
      const float4 he4 = *reinterpret_cast<const float4 *>(&L.Dl[b][C + tb]);
      ge[0] = ge4.x; ge[1] = ge4.y; ge[2] = ge4.z; ge[3] = ge4.w;
      he[0] = he4.x; he[1] = he4.y; he[2] = he4.z; he[3] = he4.w;
    }
    glast = L.Dl[b][C - 1];
    if (own) {
#pragma unroll
      for (int s = 0; s < F::KS; ++s) kt[s] = kt_operand<D>(L.Kn[b], wave, s, l16, g4);
    }
    if (blk) {
#pragma unroll
      for (int s = 0; s < F::DS; ++s)
        ka[s] = *reinterpret_cast<const uint4 *>(&L.Kn[b][kn_index<D>(16 * ib + l16, 32 * s + 8 * g4)]);
    }
  };
  {
    const rsrc_t rt = frag_res(0);
#pragma unroll
    for (int s = 0; s < F::KS; ++s) fa[s] = buf_load_b128(rt, s < nks ? foff + 1024u * s : kOutOfRange);
  }
  fetch_lds(0);
  for (int lc = 0; lc < nch; ++lc) {
    // ---- phase 1: X = K S^T, Y = V - exp(gamma) X (beta is folded into T')
    if (blk) {
      uint4 bs[F::DS];
#pragma unroll
      for (int s = 0; s < F::DS; ++s)
        bs[s] = *reinterpret_cast<const uint4 *>(&L.Sl[l16 * F::LDK + 32 * s + 8 * g4]);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 xs = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < F::DS; ++s) xs = mfma_16x16x32(ka[s], bs[s], xs);
      *reinterpret_cast<uint2 *>(&L.Yl[l16 * F::LDV + ypos]) =
          pack4_bf16(vv[0] - ge[0] * xs[0], vv[1] - ge[1] * xs[1], vv[2] - ge[2] * xs[2],
                     vv[3] - ge[3] * xs[3]);
    }
    lds_barrier();
    // ---- phase 2: U = T' Y and exp(gamma_last - gamma) U
    if (blk) {
      uint4 by[F::KS];
#pragma unroll
      for (int s = 0; s < F::KS; ++s)
        by[s] = *reinterpret_cast<const uint4 *>(&L.Yl[l16 * F::LDV + 32 * s + 8 * g4]);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 u = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < F::KS; ++s) u = mfma_16x16x32(fa[s], by[s], u);
      *reinterpret_cast<uint2 *>(&L.Ul[l16 * F::LDV + ypos]) = pack4_bf16(u[0], u[1], u[2], u[3]);
      *reinterpret_cast<uint2 *>(&L.Uh[l16 * F::LDV + ypos]) =
          pack4_bf16(he[0] * u[0], he[1] * u[1], he[2] * u[2], he[3] * u[3]);
      // reload after the last reader (the last chunk re-reads itself)
      __builtin_amdgcn_sched_barrier(0);
      const rsrc_t rt = frag_res(min(lc + 1, nch - 1));
#pragma unroll
      for (int s = 0; s < F::KS; ++s) fa[s] = buf_load_b128(rt, s < nks ? foff + 1024u * s : kOutOfRange);
    }
    lds_barrier();
    // ---- phase 3: state update, then chunk lc + 1's LDS operands, whose
    // K^T and K reads may stay in flight across the barrier
    if (own) {
      state_update<D, C, TIn>(L, S, kt, glast, wave, l16, g4);
      asm volatile("" ::"v"(S) : "memory");
    }
    if (lc + 1 < nch) {
      fetch_lds((lc + 1) % CC::NB);
      lds_barrier_keep<((F::NKT == 8) ? 2 * F::KS : 0) + ((F::NIB == 4) ? F::DS : 0)>();
    } else {
      lds_barrier();
    }
  }
}

// Wavefronts 4-7: the K^T operands of the chunk and the output of the
// previous one in phase 1, Q S^T in phase 2, O = exp(gamma) Q S^T + P U
// for token block ib (U of that chunk is still in LDS in the next phase 1).
template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_compute_o(
    CarryLds<D, C, TIn> &L, f32x4 &S, int wave, int lane, int nch, int64_t c0,
    const uint16_t *__restrict__ pfrag, const uint16_t *__restrict__ qfrag,
    TIn *__restrict__ o, int64_t seq_t0, int64_t seq_t1, int h, int hk, int hqk, int hv,
    int v0) {
  using F = Cfg<D, C>;
  using CC = CarryCfg<D, C, TIn>;
  const int l16 = lane & 15, g4 = lane >> 4;
  const int ib = wave - 4;
  const bool blk = (F::NIB == 4) || (ib < F::NIB);
  const bool own = (F::NKT == 8) || (wave < F::NKT);
  const int ibc = min(ib, F::NIB - 1);
  const int nks = min(ibc / 2 + 1, F::KS);  // P fragments on or below the diagonal, as T'
  const int tb = 16 * ibc + 4 * g4;
  const uint32_t foff = (uint32_t)(((ibc * F::KS) * 64 + lane) * 16);
  const uint32_t qoff = (uint32_t)(((ibc * F::DS) * 64 + lane) * 16);
  auto p_res = [&](int lc) {
    return make_rsrc(pfrag + ((c0 + lc) * hv + h) * F::FRAG, F::FRAG * 2);
  };
  auto q_res = [&](int lc) {
    return make_rsrc(qfrag + ((c0 + lc) * hqk + hk) * (C * D), C * D * 2);
  };
  // O of chunk lc from the kept Q S^T, P and the U of that chunk in LDS,
  // straight to global memory: lane (l16, g4) element e is row tb + e,
  // column v0 + l16.
  auto out = [&](const uint4 *pa, const f32x4 &qs, const float *gq, int lc) {
    uint4 bu[F::KS];
#pragma unroll
    for (int s = 0; s < F::KS; ++s)
      bu[s] = *reinterpret_cast<const uint4 *>(&L.Ul[l16 * F::LDV + 32 * s + 8 * g4]);
    __builtin_amdgcn_sched_barrier(0);
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < F::KS; ++s) acc = mfma_16x16x32(pa[s], bu[s], acc);
    const int64_t t0 = seq_t0 + (int64_t)lc * C;
    const int nv = (int)min((int64_t)C, seq_t1 - t0);
    const rsrc_t ro = make_rsrc(o + (t0 * hv + h) * D + v0, (uint32_t)(nv * hv * D * CC::ESZ));
#pragma unroll
    for (int e = 0; e < 4; ++e)
      BufElem<TIn>::store1_stream(ro, (uint32_t)((tb + e) * hv * D + l16), gq[e] * qs[e] + acc[e]);
  };
  uint4 qf[F::DS];   // Q rows of block ib, one chunk ahead
  uint4 pa[F::KS];   // P rows of block ib of the previous chunk
  uint4 kt[F::KS];   // K^T operands of key tile `wave`
  f32x4 qs = f32x4{0.f, 0.f, 0.f, 0.f};
  float gq[4] = {0.f, 0.f, 0.f, 0.f};
  {
    const rsrc_t rq = q_res(0);
#pragma unroll
    for (int s = 0; s < F::DS; ++s) qf[s] = buf_load_b128(rq, qoff + 1024u * s);
#pragma unroll
    for (int s = 0; s < F::KS; ++s) pa[s] = make_uint4(0, 0, 0, 0);
  }
  for (int lc = 0; lc < nch; ++lc) {
    const int b = lc % CC::NB;  // input buffer of chunk lc
    // ---- phase 1: output of chunk lc - 1, then P of this chunk and the K^T
    // operands of the state update
    if (blk) {
      if (lc > 0) out(pa, qs, gq, lc - 1);
      __builtin_amdgcn_sched_barrier(0);
      const rsrc_t rp = p_res(lc);
#pragma unroll
      for (int s = 0; s < F::KS; ++s) pa[s] = buf_load_b128(rp, s < nks ? foff + 1024u * s : kOutOfRange);
    }
    if (own) {
#pragma unroll
      for (int s = 0; s < F::KS; ++s) kt[s] = kt_operand<D>(L.Kn[b], wave, s, l16, g4);
      // these waves write nothing to LDS in phase 1: the K^T reads may stay
      // in flight across the barrier
      lds_barrier_keep<((F::NKT == 8) ? 2 * F::KS : 0)>();
    } else {
      lds_barrier();
    }
    // ---- phase 2: Q S^T (S is still the state entering chunk lc)
    if (blk) {
      uint4 bs[F::DS];
#pragma unroll
      for (int s = 0; s < F::DS; ++s)
        bs[s] = *reinterpret_cast<const uint4 *>(&L.Sl[l16 * F::LDK + 32 * s + 8 * g4]);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 x = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < F::DS; ++s) x = mfma_16x16x32(qf[s], bs[s], x);
      qs = x;
      const float4 g4v = *reinterpret_cast<const float4 *>(&L.Dl[b][tb]);
      gq[0] = g4v.x; gq[1] = g4v.y; gq[2] = g4v.z; gq[3] = g4v.w;
      // the product must be complete before the registers of Q are reloaded
      asm volatile("" ::"v"(x) : "memory");
      const rsrc_t rq = q_res(min(lc + 1, nch - 1));
#pragma unroll
      for (int s = 0; s < F::DS; ++s) qf[s] = buf_load_b128(rq, qoff + 1024u * s);
    }
    lds_barrier();
    // ---- phase 3
    if (own) state_update<D, C, TIn>(L, S, kt, L.Dl[b][C - 1], wave, l16, g4);
    lds_barrier();
  }
  if (blk) out(pa, qs, gq, nch - 1);  // output of the last chunk
}

template <int D, int C, typename TIn>
__global__ __launch_bounds__(kCarryThreads) void chunk_carry_kernel(
    const TIn *__restrict__ k, const TIn *__restrict__ v,
    const int32_t *__restrict__ cu, const float *__restrict__ dec_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag,
    const uint16_t *__restrict__ qfrag, const uint16_t *__restrict__ kcopy,
    const float *s0, float *sT, TIn *__restrict__ o, int hqk, int hv, int group,
    int n_groups) {
  using F = Cfg<D, C>;
  using CC = CarryCfg<D, C, TIn>;
  __shared__ __attribute__((aligned(16))) CarryLds<D, C, TIn> L;

  // Work-groups are dealt to the 8 XCDs round-robin by id. Give each XCD
  // whole (sequence, key head) groups, every value head of the group with
  // all its value tiles, so the tiles that share K and Q (the group) and T'
  // and P (one head) share one L2.
  const int Lb = blockIdx.x;
  const int jx = Lb >> 3;  // index among the work-groups of XCD Lb % 8
  const int gq = (jx / (group * F::NVT)) * 8 + (Lb & 7);  // sequence * hqk + key head
  const int gi = (jx / F::NVT) % group, vt = jx % F::NVT;
  if (gq >= n_groups) return;
  const int n = gq / hqk, hk = gq % hqk, h = hk * group + gi;
  const int pair = n * hv + h;
  const int v0 = 16 * vt;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g4 = lane >> 4;
  const int64_t seq_t0 = cu[n], seq_t1 = cu[n + 1];
  const int nch = (int)((seq_t1 - seq_t0 + C - 1) / C);
  const int64_t c0 = first_slot(cu, n, C);
  const bool compute = wave < CC::NCW;
  const bool own = compute && ((F::NKT == 8) || (wave < F::NKT));

  // State rows v0..v0+15, key tile `wave`: lane l holds
  // S[v0 + l%16][16 wave + 4 (l/16) + e] (the accumulator layout of the
  // S^T update).
  f32x4 S = f32x4{0.f, 0.f, 0.f, 0.f};
  if (own && s0 != nullptr) {
    const float4 x = *reinterpret_cast<const float4 *>(
        s0 + ((int64_t)pair * D + v0 + l16) * D + 16 * wave + 4 * g4);
    S = f32x4{x.x, x.y, x.z, x.w};
  }
  if (nch > 0) {  // uniform over the work-group
    if (compute) {
      if (C < F::CP) {  // zero the token positions past the chunk, once
        for (int idx = tid; idx < 16 * F::LDV; idx += 64 * CC::NCW) {
          L.Yl[idx] = 0;
          L.Ul[idx] = 0;
          L.Uh[idx] = 0;
        }
        for (int idx = C * D + tid; idx < F::CP * D; idx += 64 * CC::NCW) {
#pragma unroll
          for (int bb = 0; bb < CC::NB; ++bb) L.Kn[bb][idx] = 0;
        }
      }
      if (own)
        *reinterpret_cast<uint2 *>(&L.Sl[l16 * F::LDK + 16 * wave + 4 * g4]) =
            pack4_bf16(S[0], S[1], S[2], S[3]);
      lds_barrier();
      if (wave < 4)
        carry_compute_xu<D, C, TIn>(L, S, wave, lane, nch, c0, tfrag, h, hv);
      else
        carry_compute_o<D, C, TIn>(L, S, wave, lane, nch, c0, pfrag, qfrag, o, seq_t0, seq_t1,
                                   h, hk, hqk, hv, v0);
    } else {
      // bf16 K is copied straight from the input; f32 K from its bf16 copy.
      const bool kcopied = sizeof(TIn) != 2;
      const uint16_t *ksrc = kcopied ? kcopy : reinterpret_cast<const uint16_t *>(k);
      const int kstride = kcopied ? D : hqk * D;
      static_assert(CC::NLW == 2, "loader dispatch below");
      if (wave == CC::NCW)
        carry_loader<D, C, TIn, 0>(L, lane, ksrc, kstride, kcopied, v, dec_ws, nch, seq_t0,
                                   seq_t1, c0, h, hk, hqk, hv, v0);
      else
        carry_loader<D, C, TIn, 1>(L, lane, ksrc, kstride, kcopied, v, dec_ws, nch, seq_t0,
                                   seq_t1, c0, h, hk, hqk, hv, v0);
    }
  }

  if (own)
    store_stream(sT + ((int64_t)pair * D + v0 + l16) * D + 16 * wave + 4 * g4, S);
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

template <int D, int C, typename TIn>
__global__ __launch_bounds__(256) void chunk_wave_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k, const TIn *__restrict__ v,
    const int32_t *__restrict__ cu, const float *__restrict__ dec_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag,
    const uint16_t *__restrict__ kcopy, const float *s0, float *sT, TIn *__restrict__ o,
    int n_units, int hqk, int hv, int group) {
  using F = Cfg<D, C>;
  using WC = WaveCfg<D, C>;
  using CC = CarryCfg<D, C, TIn>;
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

  // bf16 K comes straight from the input, f32 K from its bf16 copy
  const bool kcopied = sizeof(TIn) != 2;
  const uint16_t *ksrc = kcopied ? kcopy : reinterpret_cast<const uint16_t *>(k);
  const int kstride = kcopied ? D : hqk * D;

  for (int lc = 0; lc < nch; ++lc) {
    const int64_t t0 = seq_t0 + (int64_t)lc * C;
    const int nv = (int)min((int64_t)C, seq_t1 - t0);
    const int64_t slot = (c0 + lc) * hv + h;
    // ---- loads: K chunk into LDS (rows past nv read as zero), the tables
    const rsrc_t rk = kcopied ? make_rsrc(ksrc + ((c0 + lc) * hqk + hk) * (C * D), C * D * 2)
                              : make_rsrc(ksrc + (t0 * hqk + hk) * D, (uint32_t)(nv * hqk * D * 2));
#pragma unroll
    for (int m = 0; m < WC::NKI; ++m) {
      // (the offset goes in as a plain scalar: with an array element as the
      // builtin's argument the host pass emitted no launch stub)
      const uint32_t off = copy_offset<D, C, TIn>(m, lane, kstride, hv);
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

PrefillWorkspace prefill_workspace_layout(int n_seqs, int64_t n_tokens, int hqk,
                                          int hv, int d, int chunk) {
  PrefillWorkspace w;
  const int64_t nc = chunk_bound(n_seqs, n_tokens, chunk);
  size_t p = 0;
  w.decay = p;
  p = align256(p + sizeof(float) * (size_t)nc * hv * 2 * chunk);
  w.tfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hv * frag_elems(chunk));
  w.pfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hv * frag_elems(chunk));
  w.qfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hqk * chunk * d);
  w.kcopy = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hqk * chunk * d);
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
  uint16_t *qf = reinterpret_cast<uint16_t *>(base + ws.qfrag);
  uint16_t *kc = reinterpret_cast<uint16_t *>(base + ws.kcopy);
  const int group = a.hv / a.hqk;

  const int64_t nc = chunk_bound(a.n_seqs, a.n_tokens, C);
  if (a.n_tokens > 0) {
    // (chunk, key head) pairs in groups of eight, times the heads of a group.
    const int64_t pairs = nc * a.hqk;
    const int64_t lblocks = ((pairs + 7) / 8) * 8 * group;
    auto local = a.neumann ? chunk_local_kernel<D, C, TIn, true>
                           : chunk_local_kernel<D, C, TIn, false>;
    hipLaunchKernelGGL(local, dim3((unsigned)lblocks), dim3(256), 0, a.stream, (const TIn *)a.q, (const TIn *)a.k, a.g, a.beta, a.gate,
                       a.cu_seqlens, a.n_seqs, a.hqk, a.hv, group, (int)pairs, dec, tf, pf,
                       qf, kc);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  const int n_groups = a.n_seqs * a.hqk;
  if (a.wave_carry) {
    const int wpu = (group * F::NVT + WaveCfg<D, C>::WAVES - 1) / WaveCfg<D, C>::WAVES;
    const int64_t wblocks = (int64_t)8 * ((n_groups + 7) / 8) * wpu;
    hipLaunchKernelGGL((chunk_wave_kernel<D, C, TIn>), dim3((unsigned)wblocks), dim3(256), 0,
                       a.stream, (const TIn *)a.q, (const TIn *)a.k, (const TIn *)a.v,
                       a.cu_seqlens, dec, tf, pf, kc, a.initial_state, a.final_state, (TIn *)a.o,
                       n_groups, a.hqk, a.hv, group);
    return hipGetLastError();
  }
  const int64_t blocks = (int64_t)8 * ((n_groups + 7) / 8) * group * F::NVT;
  hipLaunchKernelGGL((chunk_carry_kernel<D, C, TIn>), dim3((unsigned)blocks),
                     dim3(kCarryThreads), 0, a.stream, (const TIn *)a.k, (const TIn *)a.v,
                     a.cu_seqlens, dec, tf, pf, qf, kc, a.initial_state, a.final_state,
                     (TIn *)a.o, a.hqk, a.hv, group, n_groups);
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
  return a.dtype == GDN_BF16 ? launch_prefill_e<__bf16>(a, ws)
                             : launch_prefill_e<float>(a, ws);
}

}  // namespace gdn
