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
// Three kernels on one stream:
//   chunk_offsets_kernel  first global chunk index of every sequence (a scan
//                         of ceil(len/C) on the device; no host read).
//   chunk_local_kernel    chunk-parallel: gamma, K K^T and Q K^T on bf16 MFMA,
//                         A, the triangular inverse in LDS (fp32), P; T and P
//                         are stored as bf16 in MFMA operand order.
//   chunk_carry_kernel    one work-group per (sequence, value head, 16-row
//                         value tile): walks the chunks of its sequence, keeps
//                         its fp32 state tile in MFMA accumulators and does
//                         every product on bf16 MFMA with fp32 accumulation.
//
// Every exponent is a non-positive difference (for g <= 0), masked before
// exp, so strongly decaying inputs cannot overflow.
#include "gdn_device.h"
#include "gdn_launch.h"

namespace gdn {

// ============================================================ chunk offsets
__global__ __launch_bounds__(256) void chunk_offsets_kernel(
    const int32_t *__restrict__ cu, int32_t *__restrict__ off, int n_seqs,
    int chunk) {
  __shared__ int32_t wave_sum[4];
  __shared__ int32_t carry;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    off[0] = 0;
    carry = 0;
  }
  __syncthreads();
  for (int base = 0; base < n_seqs; base += 256) {
    const int n = base + tid;
    int x = 0;
    if (n < n_seqs) x = (cu[n + 1] - cu[n] + chunk - 1) / chunk;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (lane == 63) wave_sum[wave] = x;
    __syncthreads();
    int prefix = carry;
    for (int w = 0; w < wave; ++w) prefix += wave_sum[w];
    if (n < n_seqs) off[n + 1] = prefix + x;
    __syncthreads();
    if (tid == 255) carry = prefix + x;
    __syncthreads();
  }
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

// ============================================================ chunk-local
// One work-group per (chunk, key head): gamma, K K^T and K Q^T once, then for
// every value head of the group A, P and T = (I + A)^-1, written as bf16
// A-operand fragments. T is built from its 16x16 blocks in fp32: wavefront b
// inverts diagonal block b as (I - M)(I + M^2)(I + M^4)(I + M^8) (M strictly
// triangular, so the product is exact), then forms its block row from
//   T[b][c] = -(sum_{m=c+1..b} T[b][m] A[m][c]) T[c][c]^-1    (c < b),
// carried in transposed form so that every intermediate stays in the
// accumulator layout of the fp32 16x16x4 matrix instruction.
template <int D, int C>
struct LocalLds {
  union {
    struct {
      uint16_t K[C * Cfg<D, C>::LDK];
      uint16_t Q[C * Cfg<D, C>::LDK];
    } kq;
    struct {
      float A[C * Cfg<D, C>::LDA];
      float linv[C / 16][16 * 17];   // transposed diagonal inverses
      float sa[4][16 * 17], sb[4][16 * 17];
    } inv;
  } u;
};

template <int D, int C, typename TIn>
__global__ __launch_bounds__(256) void chunk_local_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const float *__restrict__ g, const float *__restrict__ beta,
    const int32_t *__restrict__ cu, const int32_t *__restrict__ off,
    int n_seqs, int hqk, int hv, int group, float *__restrict__ gam_ws,
    uint16_t *__restrict__ tfrag, uint16_t *__restrict__ pfrag) {
  using F = Cfg<D, C>;
  constexpr int NIB = F::NIB, KS = F::KS;
  constexpr int NP = C * (D / 8);  // 16-byte row pieces of K (and of Q)
  constexpr int NL = (NP + 255) / 256;
  __shared__ __attribute__((aligned(16))) LocalLds<D, C> L;

  const int cidx = blockIdx.x;
  const int hk = blockIdx.y;
  if (cidx >= off[n_seqs]) return;
  int lo = 0, hi = n_seqs;  // off[lo] <= cidx < off[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (off[mid] <= cidx) lo = mid; else hi = mid;
  }
  const int n = lo;
  const int64_t t0 = cu[n] + (int64_t)(cidx - off[n]) * C;
  const int nvalid = (int)min((int64_t)C, (int64_t)cu[n + 1] - t0);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g4 = lane >> 4;
  const int ib = wave;

  // ---- loads: rows past the end of the sequence read as zero
  const uint32_t rowb = (uint32_t)(nvalid * hqk * D * sizeof(TIn));
  const rsrc_t rk = make_rsrc(k + (t0 * hqk + hk) * D, rowb);
  const rsrc_t rq = make_rsrc(q + (t0 * hqk + hk) * D, rowb);
  const rsrc_t rg = make_rsrc(g + t0 * hv, (uint32_t)(nvalid * hv * 4));
  const rsrc_t rb = make_rsrc(beta + t0 * hv, (uint32_t)(nvalid * hv * 4));
  uint4 kv[NL], qv[NL];
#pragma unroll
  for (int u = 0; u < NL; ++u) {
    const int idx = min(tid + 256 * u, NP - 1);
    const uint32_t e = (uint32_t)((idx / (D / 8)) * hqk * D + (idx % (D / 8)) * 8);
    kv[u] = BufElem<TIn>::load8(rk, e);
    qv[u] = BufElem<TIn>::load8(rq, e);
  }
  const uint32_t grow = (uint32_t)(lane * hv + hk * group);
  float gnext = buf_load_f32(rg, grow * 4u);
  float bnext = buf_load_f32(rb, grow * 4u);
#pragma unroll
  for (int u = 0; u < NL; ++u) {
    const int idx = tid + 256 * u;
    if (idx < NP) {
      const int r = idx / (D / 8), seg = idx % (D / 8);
      *reinterpret_cast<uint4 *>(&L.u.kq.K[r * F::LDK + seg * 8]) = kv[u];
      *reinterpret_cast<uint4 *>(&L.u.kq.Q[r * F::LDK + seg * 8]) = qv[u];
    }
  }
  lds_barrier();

  // ---- Gram tiles for column block ib, row blocks jb <= ib. Lane (l16, g4)
  // element e holds  k_j . k_i  and  k_j . q_i,  j = 16 jb + 4 g4 + e,
  // i = 16 ib + l16.
  f32x4 Gk[NIB], Gq[NIB];
#pragma unroll
  for (int jb = 0; jb < NIB; ++jb) {
    Gk[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
    Gq[jb] = Gk[jb];
    if (ib < NIB && jb <= ib) {
#pragma unroll
      for (int s = 0; s < F::DS; ++s) {
        const int col = 32 * s + 8 * g4;
        const uint4 a = *reinterpret_cast<const uint4 *>(&L.u.kq.K[(16 * jb + l16) * F::LDK + col]);
        const uint4 bk = *reinterpret_cast<const uint4 *>(&L.u.kq.K[(16 * ib + l16) * F::LDK + col]);
        const uint4 bq = *reinterpret_cast<const uint4 *>(&L.u.kq.Q[(16 * ib + l16) * F::LDK + col]);
        Gk[jb] = mfma_16x16x32(a, bk, Gk[jb]);
        Gq[jb] = mfma_16x16x32(a, bq, Gq[jb]);
      }
    }
  }
  lds_barrier();  // the K and Q tiles are dead; the space is reused below

  for (int gi = 0; gi < group; ++gi) {
    const int h = hk * group + gi;
    const int64_t slot = (int64_t)cidx * hv + h;
    float gam = gnext;  // this lane's row: g (zero past the sequence end)
    const float bta = bnext;
    if (gi + 1 < group) {
      gnext = buf_load_f32(rg, (grow + gi + 1) * 4u);
      bnext = buf_load_f32(rb, (grow + gi + 1) * 4u);
    }
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {  // inclusive prefix sum: gamma
      const float y = __shfl_up(gam, d, 64);
      if (lane >= d) gam += y;
    }
    if (wave == 0 && lane < C) gam_ws[slot * C + lane] = gam;

    f32x4 At[NIB], Z[NIB];
#pragma unroll
    for (int jb = 0; jb < NIB; ++jb) {
      At[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
      Z[jb] = At[jb];
    }
    if (ib < NIB) {
      const int i = 16 * ib + l16;
      const float gami = __shfl(gam, i, 64), bi = __shfl(bta, i, 64);
      f32x4 Pt[NIB];
#pragma unroll
      for (int jb = 0; jb < NIB; ++jb) {
        Pt[jb] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (jb > ib) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = 16 * jb + 4 * g4 + e;
          const float gamj = __shfl(gam, j, 64);
          const float dec = (j <= i) ? __expf(gami - gamj) : 0.f;
          Pt[jb][e] = dec * Gq[jb][e];
          At[jb][e] = (j < i) ? bi * dec * Gk[jb][e] : 0.f;
        }
        *reinterpret_cast<float4 *>(&L.u.inv.A[i * F::LDA + 16 * jb + 4 * g4]) =
            make_float4(At[jb][0], At[jb][1], At[jb][2], At[jb][3]);
      }
      // P as A-operand fragments: step s takes tile 2s (elements 0-3) and
      // tile 2s+1 (elements 4-7), i.e. the token order of tok_pos().
      uint16_t *pf = pfrag + slot * F::FRAG + ((int64_t)ib * KS * 64 + lane) * 8;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f32x4 lo4 = Pt[2 * s];
        const f32x4 hi4 = (2 * s + 1 < NIB) ? Pt[(2 * s + 1) % NIB] : f32x4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<uint4 *>(pf + s * 512) =
            make_uint4(pack_bf16x2(lo4[0], lo4[1]), pack_bf16x2(lo4[2], lo4[3]),
                       pack_bf16x2(hi4[0], hi4[1]), pack_bf16x2(hi4[2], hi4[3]));
      }
    }
    lds_barrier();

    // ---- diagonal block: M = A[b][b]^T (lane element e: M[4 g4 + e][l16]).
    if (ib < NIB) {
      const float *Ab = &L.u.inv.A[(16 * ib) * F::LDA + 16 * ib];
      float *sa = L.u.inv.sa[wave], *sb = L.u.inv.sb[wave];
      const f32x4 M = At[ib];
      f32x4 X = f32x4{0.f, 0.f, 0.f, 0.f}, M2 = X;
#pragma unroll
      for (int e = 0; e < 4; ++e) X[e] = ((4 * g4 + e) == l16 ? 1.f : 0.f) - M[e];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        M2 = mfma_16x16x4_f32(Ab[(4 * g4 + kk) * F::LDA + l16], M[kk], M2);
      // X <- X (I + M^2); then with M^4 and M^8. The A operand of X (I - M)
      // comes straight from the A tile.
#pragma unroll
      for (int e = 0; e < 4; ++e) sa[(4 * g4 + e) * 17 + l16] = M2[e];
      wave_lds_fence();
      f32x4 M4 = f32x4{0.f, 0.f, 0.f, 0.f};
      f32x4 X1 = X;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        M4 = mfma_16x16x4_f32(sa[l16 * 17 + 4 * g4 + kk], M2[kk], M4);
        const float x0 = ((4 * g4 + kk) == l16 ? 1.f : 0.f) - Ab[(4 * g4 + kk) * F::LDA + l16];
        X1 = mfma_16x16x4_f32(x0, M2[kk], X1);
      }
      wave_lds_fence();
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sa[(4 * g4 + e) * 17 + l16] = M4[e];
        sb[(4 * g4 + e) * 17 + l16] = X1[e];
      }
      wave_lds_fence();
      f32x4 M8 = f32x4{0.f, 0.f, 0.f, 0.f};
      f32x4 X2 = X1;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        M8 = mfma_16x16x4_f32(sa[l16 * 17 + 4 * g4 + kk], M4[kk], M8);
        X2 = mfma_16x16x4_f32(sb[l16 * 17 + 4 * g4 + kk], M4[kk], X2);
      }
      wave_lds_fence();
#pragma unroll
      for (int e = 0; e < 4; ++e) sb[(4 * g4 + e) * 17 + l16] = X2[e];
      wave_lds_fence();
      f32x4 X3 = X2;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        X3 = mfma_16x16x4_f32(sb[l16 * 17 + 4 * g4 + kk], M8[kk], X3);
      // X3 = (T[b][b])^T; publish it for the other block rows.
#pragma unroll
      for (int e = 0; e < 4; ++e) L.u.inv.linv[ib][(4 * g4 + e) * 17 + l16] = X3[e];
#pragma unroll
      for (int jb = 0; jb < NIB; ++jb)
        if (jb == ib) Z[jb] = X3;
    }
    lds_barrier();

    // ---- block row ib, right to left: Z[c] = (T[ib][c])^T.
    if (ib < NIB) {
#pragma unroll
      for (int c = NIB - 2; c >= 0; --c) {
        if (c >= ib) continue;
        f32x4 R = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 1; m < NIB; ++m) {
          if (m <= c || m > ib) continue;
          const float *Amc = &L.u.inv.A[(16 * m) * F::LDA + 16 * c];
#pragma unroll
          for (int kk = 0; kk < 4; ++kk)
            R = mfma_16x16x4_f32(Amc[(4 * g4 + kk) * F::LDA + l16], Z[m][kk], R);
        }
        f32x4 Zc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          Zc = mfma_16x16x4_f32(L.u.inv.linv[c][l16 * 17 + 4 * g4 + kk], R[kk], Zc);
        Z[c] = -Zc;
      }
      // T as A-operand fragments, same token order as P.
      uint16_t *tf = tfrag + slot * F::FRAG + ((int64_t)ib * KS * 64 + lane) * 8;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f32x4 lo4 = Z[2 * s];
        const f32x4 hi4 = (2 * s + 1 < NIB) ? Z[(2 * s + 1) % NIB] : f32x4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<uint4 *>(tf + s * 512) =
            make_uint4(pack_bf16x2(lo4[0], lo4[1]), pack_bf16x2(lo4[2], lo4[3]),
                       pack_bf16x2(hi4[0], hi4[1]), pack_bf16x2(hi4[2], hi4[3]));
      }
    }
    lds_barrier();  // A and the inverses are rewritten for the next head
  }
}

// ============================================================ chunk carry
// One work-group per (sequence, value head, 16-row value tile); wavefront w
// owns token block w of the chunk and key tiles w, w + 4 of the state. All
// global reads go through buffer resources rebuilt per chunk from scalars, so
// the per-lane offsets are loop invariant and rows past the end of the
// sequence read as zero (they then contribute exact zeros: beta = 0 there).
template <int D, int C>
struct ChunkRegs {
  using F = Cfg<D, C>;
  uint4 kr[4];       // K piece: rows 4 rg + [0, 4), columns 8 cg + [0, 8)
  uint4 qa[F::DS];   // Q rows as the A operand of Q S^T
  uint4 ta[F::KS];   // T fragments of this wave's token block
  uint4 pa[F::KS];   // P fragments of this wave's token block
  float vv[4], bb[4];
  float4 gg;
  float glast;
};

// Per-lane element offsets, fixed for the whole sequence.
struct CarryLane {
  uint32_t k, q, v, b, frag, gam;
};

template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_fetch(
    ChunkRegs<D, C> &r, const CarryLane &ln, const TIn *__restrict__ q,
    const TIn *__restrict__ k, const TIn *__restrict__ v,
    const float *__restrict__ beta, const float *__restrict__ gam_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag,
    int64_t t0, int nvalid, int64_t slot, int h, int hk, int hqk, int hv, int v0) {
  using F = Cfg<D, C>;
  const uint32_t kb = (uint32_t)(nvalid * hqk * D * sizeof(TIn));
  const rsrc_t rk = make_rsrc(k + (t0 * hqk + hk) * D, kb);
  const rsrc_t rq = make_rsrc(q + (t0 * hqk + hk) * D, kb);
  const rsrc_t rv = make_rsrc(v + (t0 * hv + h) * D + v0, (uint32_t)(nvalid * hv * D * sizeof(TIn)));
  const rsrc_t rb = make_rsrc(beta + t0 * hv + h, (uint32_t)(nvalid * hv * 4));
  const rsrc_t rt = make_rsrc(tfrag + slot * F::FRAG, F::FRAG * 2);
  const rsrc_t rp = make_rsrc(pfrag + slot * F::FRAG, F::FRAG * 2);
  const rsrc_t rg = make_rsrc(gam_ws + slot * C, C * 4);
#pragma unroll
  for (int rr = 0; rr < 4; ++rr)
    r.kr[rr] = BufElem<TIn>::load8(rk, ln.k + (uint32_t)(rr * hqk * D));
#pragma unroll
  for (int s = 0; s < F::DS; ++s) r.qa[s] = BufElem<TIn>::load8(rq, ln.q + 32 * s);
#pragma unroll
  for (int s = 0; s < F::KS; ++s) {
    r.ta[s] = buf_load_b128(rt, (ln.frag + s * 512) * 2);
    r.pa[s] = buf_load_b128(rp, (ln.frag + s * 512) * 2);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    r.vv[e] = BufElem<TIn>::load1(rv, ln.v + (uint32_t)(e * hv * D));
    r.bb[e] = buf_load_f32(rb, (ln.b + (uint32_t)(e * hv)) * 4);
  }
  r.gg = buf_load_f32x4(rg, ln.gam * 4);
  r.glast = buf_load_f32(rg, (C - 1) * 4);
}

template <int D, int C>
struct CarryLds {
  using F = Cfg<D, C>;
  uint16_t Kn[2][C * D];        // K chunk, row-major, 16-byte chunks swizzled
  uint16_t Kt[2][D * F::CP];    // K chunk transposed, tokens in tok_pos order
  uint16_t Sl[16 * F::LDK];     // bf16 copy of the state tile, [value][key]
  uint16_t Yl[16 * F::LDV];     // Y,  [value][token position]
  uint16_t Ul[16 * F::LDV];     // U,  [value][token position]
  uint16_t Uh[16 * F::LDV];     // exp(gamma_last - gamma) U, same layout
};

// 16-byte chunk swizzles (XOR with a row function), chosen so that both the
// 16-lane write pattern of the K commit and the 16-lane read pattern of the
// matrix operands touch 16 distinct bank groups.
template <int D>
__device__ __forceinline__ int kn_index(int row, int chunk) {
  const int sw = ((row & 15) ^ ((row >> 4) & 3)) & (D / 8 - 1);
  return row * D + 8 * (chunk ^ sw);
}
template <int CP>
__device__ __forceinline__ int kt_index(int row, int chunk) {
  const int sw = (row >> 1) & (CP / 8 - 1);
  return row * CP + 8 * (chunk ^ sw);
}

// Write a K piece into the row-major tile and the transposed tile.
template <int D, int C>
__device__ __forceinline__ void carry_commit_k(const ChunkRegs<D, C> &r,
                                               uint16_t *Kn, uint16_t *Kt,
                                               int tid) {
  using F = Cfg<D, C>;
  if (tid >= F::PIECES) return;
  const int rg = tid % (C / 4), cg = tid / (C / 4);
#pragma unroll
  for (int rr = 0; rr < 4; ++rr)
    *reinterpret_cast<uint4 *>(&Kn[kn_index<D>(4 * rg + rr, cg)]) = r.kr[rr];
  const int p = tok_pos(4 * rg);
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    const uint32_t w0 = r.kr[0][d], w1 = r.kr[1][d], w2 = r.kr[2][d], w3 = r.kr[3][d];
    const uint2 ev = make_uint2((w0 & 0xffffu) | (w1 << 16), (w2 & 0xffffu) | (w3 << 16));
    const uint2 od = make_uint2((w0 >> 16) | (w1 & 0xffff0000u), (w2 >> 16) | (w3 & 0xffff0000u));
    const int c0 = 8 * cg + 2 * d;
    *reinterpret_cast<uint2 *>(&Kt[kt_index<F::CP>(c0, p >> 3) + (p & 7)]) = ev;
    *reinterpret_cast<uint2 *>(&Kt[kt_index<F::CP>(c0 + 1, p >> 3) + (p & 7)]) = od;
  }
}

__device__ __forceinline__ uint2 pack4_bf16(float a, float b, float c, float d) {
  return make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
}

// One chunk of the carry for work-group (pair, value tile): consumes `cur`
// (fetched one chunk earlier) and prefetches the next chunk into `nxt`.
template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_step(
    CarryLds<D, C> &L, f32x4 (&S)[Cfg<D, C>::KTW], ChunkRegs<D, C> &cur,
    ChunkRegs<D, C> &nxt, const CarryLane &ln, int lc, int nch, int64_t seq_t0,
    int64_t seq_t1, int64_t c0, const TIn *__restrict__ q,
    const TIn *__restrict__ k, const TIn *__restrict__ v,
    const float *__restrict__ beta, const float *__restrict__ gam_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag,
    TIn *__restrict__ o, int h, int hk, int hqk, int hv, int v0, int tid) {
  using F = Cfg<D, C>;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const int ib = wave;
  const int b = lc & 1;
  const int64_t t0 = seq_t0 + (int64_t)lc * C;
  const int nvalid = (int)min((int64_t)C, seq_t1 - t0);
  {
    // Prefetch the next chunk (the last chunk re-reads itself, so every
    // iteration issues the same loads).
    const int lnx = min(lc + 1, nch - 1);
    const int64_t t1 = seq_t0 + (int64_t)lnx * C;
    carry_fetch<D, C, TIn>(nxt, ln, q, k, v, beta, gam_ws, tfrag, pfrag, t1,
                           (int)min((int64_t)C, seq_t1 - t1), (c0 + lnx) * hv + h,
                           h, hk, hqk, hv, v0);
  }
  const float gcur[4] = {cur.gg.x, cur.gg.y, cur.gg.z, cur.gg.w};
  const int ypos = 32 * (ib >> 1) + 8 * g4 + 4 * (ib & 1);  // tok_pos(16 ib + 4 g4)

  // X = K S^T and Q S^T for token block ib; Y = beta (V - exp(gamma) X).
  f32x4 qs = f32x4{0.f, 0.f, 0.f, 0.f};
  if (ib < F::NIB) {
    f32x4 x = qs;
#pragma unroll
    for (int s = 0; s < F::DS; ++s) {
      const uint4 bs = *reinterpret_cast<const uint4 *>(&L.Sl[l16 * F::LDK + 32 * s + 8 * g4]);
      const uint4 ak = *reinterpret_cast<const uint4 *>(&L.Kn[b][kn_index<D>(16 * ib + l16, 4 * s + g4)]);
      x = mfma_16x16x32(ak, bs, x);
      qs = mfma_16x16x32(cur.qa[s], bs, qs);
    }
    float y[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) y[e] = cur.bb[e] * (cur.vv[e] - __expf(gcur[e]) * x[e]);
    *reinterpret_cast<uint2 *>(&L.Yl[l16 * F::LDV + ypos]) = pack4_bf16(y[0], y[1], y[2], y[3]);
  }
  lds_barrier();

  // U = T Y; also the decay-to-chunk-end scaled copy used by the update.
  if (ib < F::NIB) {
    f32x4 u = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < F::KS; ++s) {
      const uint4 by = *reinterpret_cast<const uint4 *>(&L.Yl[l16 * F::LDV + 32 * s + 8 * g4]);
      u = mfma_16x16x32(cur.ta[s], by, u);
    }
    float uh[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) uh[e] = __expf(cur.glast - gcur[e]) * u[e];
    *reinterpret_cast<uint2 *>(&L.Ul[l16 * F::LDV + ypos]) = pack4_bf16(u[0], u[1], u[2], u[3]);
    *reinterpret_cast<uint2 *>(&L.Uh[l16 * F::LDV + ypos]) = pack4_bf16(uh[0], uh[1], uh[2], uh[3]);
  }
  lds_barrier();

  // O = exp(gamma) Q S^T + P U; rows past the sequence end are dropped by
  // the buffer extent.
  if (ib < F::NIB) {
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < F::KS; ++s) {
      const uint4 bu = *reinterpret_cast<const uint4 *>(&L.Ul[l16 * F::LDV + 32 * s + 8 * g4]);
      acc = mfma_16x16x32(cur.pa[s], bu, acc);
    }
    const rsrc_t ro = make_rsrc(o + (t0 * hv + h) * D + v0, (uint32_t)(nvalid * hv * D * sizeof(TIn)));
#pragma unroll
    for (int e = 0; e < 4; ++e)
      BufElem<TIn>::store1(ro, (uint32_t)((16 * ib + 4 * g4 + e) * hv * D + l16),
                           __expf(gcur[e]) * qs[e] + acc[e]);
  }

  // S^T <- exp(gamma_last) S^T + K^T Uh, one 16-key tile at a time.
  const float dl = __expf(cur.glast);
#pragma unroll
  for (int m = 0; m < F::KTW; ++m) {
    const int t = wave + 4 * m;
    if (t >= F::NKT) continue;
    f32x4 acc = S[m] * dl;
#pragma unroll
    for (int s = 0; s < F::KS; ++s) {
      const uint4 ak = *reinterpret_cast<const uint4 *>(&L.Kt[b][kt_index<F::CP>(16 * t + l16, 4 * s + g4)]);
      const uint4 bu = *reinterpret_cast<const uint4 *>(&L.Uh[l16 * F::LDV + 32 * s + 8 * g4]);
      acc = mfma_16x16x32(ak, bu, acc);
    }
    S[m] = acc;
    *reinterpret_cast<uint2 *>(&L.Sl[l16 * F::LDK + 16 * t + 4 * g4]) =
        pack4_bf16(acc[0], acc[1], acc[2], acc[3]);
  }
  if (lc + 1 < nch) carry_commit_k<D, C>(nxt, L.Kn[b ^ 1], L.Kt[b ^ 1], tid);
  lds_barrier();
}

template <int D, int C, typename TIn>
__global__ __launch_bounds__(256) void chunk_carry_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const TIn *__restrict__ v, const float *__restrict__ beta,
    const int32_t *__restrict__ cu, const int32_t *__restrict__ off,
    const float *__restrict__ gam_ws, const uint16_t *__restrict__ tfrag,
    const uint16_t *__restrict__ pfrag, const float *s0, float *sT,
    TIn *__restrict__ o, int hqk, int hv, int group, int n_pairs) {
  using F = Cfg<D, C>;
  __shared__ __attribute__((aligned(16))) CarryLds<D, C> L;

  // Work-groups are dealt to the 8 XCDs round-robin by id. Give each XCD
  // whole (sequence, head) pairs with their value tiles adjacent, so the
  // tiles that share K, Q, T and P share one L2.
  const int Lb = blockIdx.x;
  const int jx = Lb >> 3;
  const int pair = (jx / F::NVT) * 8 + (Lb & 7);
  const int vt = jx % F::NVT;
  if (pair >= n_pairs) return;
  const int n = pair / hv, h = pair % hv, hk = h / group;
  const int v0 = 16 * vt;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g4 = lane >> 4;
  const int64_t seq_t0 = cu[n], seq_t1 = cu[n + 1];
  const int nch = off[n + 1] - off[n];
  const int64_t c0 = off[n];

  // Loop-invariant lane offsets (clamped so idle lanes issue valid loads).
  CarryLane ln;
  {
    const int ibc = min(wave, F::NIB - 1);
    const int piece = min(tid, F::PIECES - 1);
    const int rg = piece % (C / 4), cg = piece / (C / 4);
    ln.k = (uint32_t)(4 * rg * hqk * D + 8 * cg);
    ln.q = (uint32_t)((16 * ibc + l16) * hqk * D + 8 * g4);
    ln.v = (uint32_t)((16 * ibc + 4 * g4) * hv * D + l16);
    ln.b = (uint32_t)((16 * ibc + 4 * g4) * hv);
    ln.frag = (uint32_t)((ibc * F::KS * 64 + lane) * 8);
    ln.gam = (uint32_t)(16 * ibc + 4 * g4);
  }

  if (C < F::CP) {  // zero the token positions past the chunk, once
    for (int idx = tid; idx < 16 * F::LDV; idx += 256) {
      L.Yl[idx] = 0;
      L.Ul[idx] = 0;
      L.Uh[idx] = 0;
    }
    for (int idx = tid; idx < 2 * D * F::CP; idx += 256) (&L.Kt[0][0])[idx] = 0;
  }

  // State tile rows v0..v0+15; this wave owns key tiles wave + 4m. Lane l
  // holds S[v0 + l%16][16 t + 4 (l/16) + e] (the accumulator layout of the
  // S^T update).
  f32x4 S[F::KTW];
#pragma unroll
  for (int m = 0; m < F::KTW; ++m) {
    S[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int t = wave + 4 * m;
    if (t < F::NKT && s0 != nullptr) {
      const float4 x = *reinterpret_cast<const float4 *>(
          s0 + ((int64_t)pair * D + v0 + l16) * D + 16 * t + 4 * g4);
      S[m] = f32x4{x.x, x.y, x.z, x.w};
    }
  }
  if (nch > 0) {  // uniform over the work-group
    ChunkRegs<D, C> ra, rb;
    carry_fetch<D, C, TIn>(ra, ln, q, k, v, beta, gam_ws, tfrag, pfrag, seq_t0,
                           (int)min((int64_t)C, seq_t1 - seq_t0), c0 * hv + h, h,
                           hk, hqk, hv, v0);
    lds_barrier();  // zero fills done before the first K commit
#pragma unroll
    for (int m = 0; m < F::KTW; ++m) {
      const int t = wave + 4 * m;
      if (t < F::NKT)
        *reinterpret_cast<uint2 *>(&L.Sl[l16 * F::LDK + 16 * t + 4 * g4]) =
            pack4_bf16(S[m][0], S[m][1], S[m][2], S[m][3]);
    }
    carry_commit_k<D, C>(ra, L.Kn[0], L.Kt[0], tid);
    lds_barrier();

    for (int lc = 0; lc < nch; lc += 2) {
      carry_step<D, C, TIn>(L, S, ra, rb, ln, lc, nch, seq_t0, seq_t1, c0, q, k,
                            v, beta, gam_ws, tfrag, pfrag, o, h, hk, hqk, hv, v0,
                            tid);
      if (lc + 1 < nch)
        carry_step<D, C, TIn>(L, S, rb, ra, ln, lc + 1, nch, seq_t0, seq_t1, c0,
                              q, k, v, beta, gam_ws, tfrag, pfrag, o, h, hk, hqk,
                              hv, v0, tid);
    }
  }

#pragma unroll
  for (int m = 0; m < F::KTW; ++m) {
    const int t = wave + 4 * m;
    if (t < F::NKT)
      *reinterpret_cast<float4 *>(sT + ((int64_t)pair * D + v0 + l16) * D + 16 * t + 4 * g4) =
          make_float4(S[m][0], S[m][1], S[m][2], S[m][3]);
  }
}

// ============================================================ host side
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

PrefillWorkspace prefill_workspace_layout(int n_seqs, int64_t n_tokens, int hv,
                                          int chunk) {
  PrefillWorkspace w;
  const int64_t nc = chunk_bound(n_seqs, n_tokens, chunk);
  size_t p = 0;
  w.chunk_off = p;
  p = align256(p + sizeof(int32_t) * (size_t)(n_seqs + 1));
  w.gamma = p;
  p = align256(p + sizeof(float) * (size_t)nc * hv * chunk);
  w.tfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hv * frag_elems(chunk));
  w.pfrag = p;
  p = align256(p + sizeof(uint16_t) * (size_t)nc * hv * frag_elems(chunk));
  w.total = p;
  return w;
}

template <int D, int C, typename TIn>
static hipError_t launch_prefill_t(const PrefillArgs &a, const PrefillWorkspace &ws) {
  using F = Cfg<D, C>;
  char *base = static_cast<char *>(a.workspace);
  int32_t *off = reinterpret_cast<int32_t *>(base + ws.chunk_off);
  float *gam = reinterpret_cast<float *>(base + ws.gamma);
  uint16_t *tf = reinterpret_cast<uint16_t *>(base + ws.tfrag);
  uint16_t *pf = reinterpret_cast<uint16_t *>(base + ws.pfrag);
  const int group = a.hv / a.hqk;

  hipLaunchKernelGGL(chunk_offsets_kernel, dim3(1), dim3(256), 0, a.stream,
                     a.cu_seqlens, off, a.n_seqs, C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;

  const int64_t nc = chunk_bound(a.n_seqs, a.n_tokens, C);
  if (a.n_tokens > 0) {
    hipLaunchKernelGGL((chunk_local_kernel<D, C, TIn>), dim3((unsigned)nc, (unsigned)a.hqk),
                       dim3(256), 0, a.stream, (const TIn *)a.q, (const TIn *)a.k,
                       a.g, a.beta, a.cu_seqlens, off, a.n_seqs, a.hqk, a.hv,
                       group, gam, tf, pf);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  const int n_pairs = a.n_seqs * a.hv;
  const int64_t blocks = (int64_t)8 * ((n_pairs + 7) / 8) * F::NVT;
  hipLaunchKernelGGL((chunk_carry_kernel<D, C, TIn>), dim3((unsigned)blocks), dim3(256),
                     0, a.stream, (const TIn *)a.q, (const TIn *)a.k,
                     (const TIn *)a.v, a.beta, a.cu_seqlens, off, gam, tf, pf,
                     a.initial_state, a.final_state, (TIn *)a.o, a.hqk, a.hv,
                     group, n_pairs);
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
