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
    int n_seqs, int hqk, int hv, int group, float *__restrict__ dec_ws,
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
    const float glast = __shfl(gam, C - 1, 64);
    if (wave == 0 && lane < C) {
      // decay factors for the carry: exp(gamma_i) and exp(gamma_last - gamma_i)
      dec_ws[slot * 2 * C + lane] = __expf(gam);
      dec_ws[slot * 2 * C + C + lane] = __expf(glast - gam);
    }

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
      // Fold beta into the factor: the carry uses T' = T diag(beta), so that
      // U = T' (V - exp(gamma) X) needs no beta of its own.
#pragma unroll
      for (int c = 0; c < NIB; ++c) {
        if (c > ib) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) Z[c][e] *= __shfl(bta, 16 * c + 4 * g4 + e, 64);
      }
      // T' as A-operand fragments, same token order as P.
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
// One work-group of 8 wavefronts per (sequence, value head, 16-row value
// tile), two wavefronts per SIMD. Wavefronts 0-3 own token block w of the
// chunk for X = K S^T, Y and U = T Y; wavefronts 4-7 own token block w - 4 for
// Q S^T and O; all eight update one 16-key tile of the state each. The next
// chunk is prefetched into registers while the current one is computed; K and
// Q go through row-major LDS tiles (16-byte chunks XOR-swizzled by row) and
// K^T is read from the same tile with the LDS transpose load.
//
// All global reads go through buffer resources rebuilt per chunk from
// scalars, so per-lane offsets are loop invariant and rows past the end of
// the sequence read as zero (beta is zero there, so they contribute exact
// zeros); stores past the end are dropped by the resource extent.
template <int D, int C, typename TIn = __bf16>
struct CarryCfg {
  using F = Cfg<D, C>;
  static constexpr int NT = 512;                      // threads
  static constexpr int NP = C * (D / 8);              // 16-byte pieces of K (or Q)
  // Wavefronts 0-3 fetch K, wavefronts 4-7 fetch Q: KP pieces per thread.
  static constexpr int KP = (NP + NT / 2 - 1) / (NT / 2);
  // Per-chunk small data, fetched by the first threads: the 16-value V tile
  // of every token (VPR 16-byte pieces per token) and the 2C decay factors.
  static constexpr int VPR = (16 * (int)sizeof(TIn)) / 16;
  static constexpr int VP = C * VPR;
  static constexpr int SP = VP + (2 * C) / 4;
  static_assert(SP <= NT, "small data fits one piece per thread");
};

template <int D, int C>
struct ChunkRegs {
  using F = Cfg<D, C>;
  uint4 kq[CarryCfg<D, C>::KP];   // K pieces (waves 0-3) or Q pieces (4-7)
  uint4 fa[F::KS];   // T' fragments (waves 0-3) or P fragments (waves 4-7)
  uint4 sd;          // one piece of the V tile or of the decay factors
};

// Per-lane offsets, fixed for the whole sequence.
template <int KP>
struct CarryLane {
  uint32_t kq[KP];   // elements
  uint32_t frag;     // elements
  uint32_t sd;       // bytes, into V (sd_v) or the decay row
  bool sd_v, sd_any;
};

template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_fetch(
    ChunkRegs<D, C> &r, const CarryLane<CarryCfg<D, C>::KP> &ln, bool tgroup,
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const TIn *__restrict__ v, const float *__restrict__ dec_ws,
    const uint16_t *__restrict__ tfrag, const uint16_t *__restrict__ pfrag,
    int64_t t0, int nvalid, int64_t slot, int h, int hk, int hqk, int hv,
    int v0) {
  using F = Cfg<D, C>;
  const rsrc_t rkq = make_rsrc((tgroup ? k : q) + (t0 * hqk + hk) * D,
                               (uint32_t)(nvalid * hqk * D * sizeof(TIn)));
  const rsrc_t rf = make_rsrc((tgroup ? tfrag : pfrag) + slot * F::FRAG, F::FRAG * 2);
#pragma unroll
  for (int u = 0; u < CarryCfg<D, C>::KP; ++u) r.kq[u] = BufElem<TIn>::load8(rkq, ln.kq[u]);
#pragma unroll
  for (int s = 0; s < F::KS; ++s) r.fa[s] = buf_load_b128(rf, (ln.frag + s * 512) * 2);
  if (ln.sd_any) {
    const rsrc_t rs = ln.sd_v
        ? make_rsrc(v + (t0 * hv + h) * D + v0, (uint32_t)(nvalid * hv * D * sizeof(TIn)))
        : make_rsrc(dec_ws + slot * 2 * C, 2 * C * 4);
    r.sd = buf_load_b128(rs, ln.sd);
  }
}

template <int D, int C, typename TIn>
struct CarryLds {
  using F = Cfg<D, C>;
  uint16_t Kn[2][F::CP * D];    // K chunk, row-major, swizzled (double buffered);
                                // rows C..CP-1 stay zero for chunks below 32
  uint16_t Qn[C * D];           // Q chunk, same layout (read before the first
                                // barrier of a chunk, refilled after it)
  TIn Vl[2][16][C + 8];         // V tile, [value][token], input element type
  float Dl[2][2 * C];           // exp(gamma_i), then exp(gamma_last - gamma_i)
  uint16_t Sl[16 * F::LDK];     // bf16 copy of the state tile, [value][key]
  uint16_t Yl[16 * F::LDV];     // Y,  [value][token position]
  uint16_t Ul[16 * F::LDV];     // U,  [value][token position]
  uint16_t Uh[16 * F::LDV];     // exp(gamma_last - gamma) U, same layout
  uint32_t Ol[4][16 * 16 * 4 / 4];  // per-wavefront output staging (fp32 worst case)
};

// Element index of (row, column) in a swizzled row-major [C][D] tile: 16-byte
// chunks are XORed with a row function so that both 16 consecutive rows at
// one column (matrix-operand reads) and 16 chunks of one row (the commit)
// fall on distinct bank groups.
template <int D>
__device__ __forceinline__ int kn_index(int row, int col) {
  const int sw = ((row & 15) ^ ((row >> 4) & 3)) & (D / 8 - 1);
  return row * D + 8 * ((col >> 3) ^ sw) + (col & 7);
}

// Pieces p = tid4 + 256 u of K (waves 0-3) or Q (waves 4-7), tid4 = tid % 256.
template <int D, int C>
__device__ __forceinline__ void carry_commit(const ChunkRegs<D, C> &r,
                                             uint16_t *dst, int tid4) {
  using CC = CarryCfg<D, C>;
#pragma unroll
  for (int u = 0; u < CC::KP; ++u) {
    const int p = tid4 + (CC::NT / 2) * u;
    if (CC::NP % (CC::NT / 2) != 0 && p >= CC::NP) continue;
    *reinterpret_cast<uint4 *>(&dst[kn_index<D>(p / (D / 8), 8 * (p % (D / 8)))]) = r.kq[u];
  }
}

// Small-data piece p of the thread: V pieces go to the [value][token] tile,
// decay quads to their row.
template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_commit_small(const ChunkRegs<D, C> &r,
                                                   TIn (*Vl)[C + 8], float *Dl,
                                                   int p) {
  using CC = CarryCfg<D, C, TIn>;
  if (p < CC::VP) {
    const int tok = p / CC::VPR, part = p % CC::VPR;
    const uint32_t w[4] = {r.sd.x, r.sd.y, r.sd.z, r.sd.w};
    if (sizeof(TIn) == 2) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        reinterpret_cast<uint16_t *>(&Vl[8 * part + e][tok])[0] =
            (uint16_t)((w[e >> 1] >> (16 * (e & 1))) & 0xffffu);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) reinterpret_cast<uint32_t *>(&Vl[4 * part + e][tok])[0] = w[e];
    }
  } else if (p < CC::SP) {
    *reinterpret_cast<uint4 *>(&Dl[4 * (p - CC::VP)]) = r.sd;
  }
}

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

// One chunk of the carry: consumes `cur` (fetched one chunk earlier) and
// prefetches the next chunk into `nxt`.
template <int D, int C, typename TIn>
__device__ __forceinline__ void carry_step(
    CarryLds<D, C, TIn> &L, f32x4 &S, ChunkRegs<D, C> &cur, ChunkRegs<D, C> &nxt,
    const CarryLane<CarryCfg<D, C>::KP> &ln, int lc, int nch, int64_t seq_t0,
    int64_t seq_t1, int64_t c0, const TIn *__restrict__ q,
    const TIn *__restrict__ k, const TIn *__restrict__ v,
    const float *__restrict__ dec_ws, const uint16_t *__restrict__ tfrag,
    const uint16_t *__restrict__ pfrag, TIn *__restrict__ o, int h, int hk,
    int hqk, int hv, int v0, int tid) {
  using F = Cfg<D, C>;
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, g4 = lane >> 4;
  const bool tgroup = wave < 4;           // X / Y / U wavefronts
  const int ib = wave & 3;                // token block
  const bool blk = (F::NIB == 4) || (ib < F::NIB);
  const bool own = (F::NKT == 8) || (wave < F::NKT);   // owns key tile `wave`
  const int b = lc & 1;
  const int64_t t0 = seq_t0 + (int64_t)lc * C;
  const int nvalid = (int)min((int64_t)C, seq_t1 - t0);
  {
    // Prefetch the next chunk (the last chunk re-reads itself, so every
    // iteration issues the same loads).
    const int lnx = min(lc + 1, nch - 1);
    const int64_t t1 = seq_t0 + (int64_t)lnx * C;
    carry_fetch<D, C, TIn>(nxt, ln, tgroup, q, k, v, dec_ws, tfrag, pfrag, t1,
                           (int)min((int64_t)C, seq_t1 - t1), (c0 + lnx) * hv + h,
                           h, hk, hqk, hv, v0);
  }
  const int tb = 16 * min(ib, F::NIB - 1) + 4 * g4;  // this lane's first token
  const float4 ge4 = *reinterpret_cast<const float4 *>(&L.Dl[b][tb]);
  const float4 he4 = *reinterpret_cast<const float4 *>(&L.Dl[b][C + tb]);
  const float ge[4] = {ge4.x, ge4.y, ge4.z, ge4.w};
  const float he[4] = {he4.x, he4.y, he4.z, he4.w};
  const float dl = L.Dl[b][C - 1];
  const int ypos = 32 * (ib >> 1) + 8 * g4 + 4 * (ib & 1);  // tok_pos(16 ib + 4 g4)

  // X = K S^T (waves 0-3) or Q S^T (waves 4-7) for token block ib.
  f32x4 xs = f32x4{0.f, 0.f, 0.f, 0.f};
  if (blk) {
    const uint16_t *A = tgroup ? L.Kn[b] : L.Qn;
#pragma unroll
    for (int s = 0; s < F::DS; ++s) {
      const uint4 bs = *reinterpret_cast<const uint4 *>(&L.Sl[l16 * F::LDK + 32 * s + 8 * g4]);
      const uint4 a = *reinterpret_cast<const uint4 *>(&A[kn_index<D>(16 * ib + l16, 32 * s + 8 * g4)]);
      xs = mfma_16x16x32(a, bs, xs);
    }
    if (tgroup) {  // Y = V - exp(gamma) X  (beta is folded into T')
      float vv[4];
      Elem<TIn>::load4(&L.Vl[b][l16][tb], vv);
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = vv[e] - ge[e] * xs[e];
      *reinterpret_cast<uint2 *>(&L.Yl[l16 * F::LDV + ypos]) = pack4_bf16(y[0], y[1], y[2], y[3]);
    }
  }
  lds_barrier();

  if (tgroup) {
    // U = T Y, and the decay-to-chunk-end scaled copy used by the update.
    if (blk) {
      f32x4 u = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < F::KS; ++s) {
        const uint4 by = *reinterpret_cast<const uint4 *>(&L.Yl[l16 * F::LDV + 32 * s + 8 * g4]);
        u = mfma_16x16x32(cur.fa[s], by, u);
      }
      float uh[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) uh[e] = he[e] * u[e];
      *reinterpret_cast<uint2 *>(&L.Ul[l16 * F::LDV + ypos]) = pack4_bf16(u[0], u[1], u[2], u[3]);
      *reinterpret_cast<uint2 *>(&L.Uh[l16 * F::LDV + ypos]) = pack4_bf16(uh[0], uh[1], uh[2], uh[3]);
    }
  } else if (lc + 1 < nch) {
    carry_commit<D, C>(nxt, L.Qn, tid - 256);   // every Q read of this chunk is done
  }
  if (lc + 1 < nch) carry_commit_small<D, C, TIn>(nxt, L.Vl[b ^ 1], L.Dl[b ^ 1], tid);
  lds_barrier();

  // O = exp(gamma) Q S^T + P U (waves 4-7); rows past the sequence end are
  // dropped by the buffer extent.
  if (!tgroup && blk) {
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < F::KS; ++s) {
      const uint4 bu = *reinterpret_cast<const uint4 *>(&L.Ul[l16 * F::LDV + 32 * s + 8 * g4]);
      acc = mfma_16x16x32(cur.fa[s], bu, acc);
    }
    // Stage the 16 x 16 output block in LDS ([token][value]) so that it
    // leaves as 16-byte stores; rows past the sequence end are dropped by the
    // buffer extent.
    TIn *ol = reinterpret_cast<TIn *>(L.Ol[ib]);
#pragma unroll
    for (int e = 0; e < 4; ++e) Elem<TIn>::store1(&ol[(4 * g4 + e) * 16 + l16], ge[e] * xs[e] + acc[e]);
    wave_lds_fence();
    constexpr int PPR = (int)sizeof(TIn);        // 16-byte pieces per token row
    constexpr int EPP = 16 / (int)sizeof(TIn);   // elements per piece
    if (lane < 16 * PPR) {
      const int row = lane / PPR, part = lane % PPR;
      const uint4 x = *reinterpret_cast<const uint4 *>(&ol[row * 16 + part * EPP]);
      const rsrc_t ro = make_rsrc(o + (t0 * hv + h) * D + v0, (uint32_t)(nvalid * hv * D * sizeof(TIn)));
      __builtin_amdgcn_raw_buffer_store_b128(
          (__attribute__((ext_vector_type(4))) unsigned int){x.x, x.y, x.z, x.w}, ro,
          (uint32_t)(((16 * ib + row) * hv * D + part * EPP) * sizeof(TIn)), 0, 0);
    }
  }

  // S^T <- exp(gamma_last) S^T + K^T Uh for key tile `wave`.
  if (own) {
    f32x4 acc = S * dl;
#pragma unroll
    for (int s = 0; s < F::KS; ++s) {
      const uint4 a = kt_operand<D>(L.Kn[b], wave, s, l16, g4);
      const uint4 bu = *reinterpret_cast<const uint4 *>(&L.Uh[l16 * F::LDV + 32 * s + 8 * g4]);
      acc = mfma_16x16x32(a, bu, acc);
    }
    S = acc;
    *reinterpret_cast<uint2 *>(&L.Sl[l16 * F::LDK + 16 * wave + 4 * g4]) =
        pack4_bf16(acc[0], acc[1], acc[2], acc[3]);
  }
  if (tgroup && lc + 1 < nch) carry_commit<D, C>(nxt, L.Kn[b ^ 1], tid);
  lds_barrier();
}

template <int D, int C, typename TIn>
__global__ __launch_bounds__(512) void chunk_carry_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const TIn *__restrict__ v, const float *__restrict__ beta,
    const int32_t *__restrict__ cu, const int32_t *__restrict__ off,
    const float *__restrict__ dec_ws, const uint16_t *__restrict__ tfrag,
    const uint16_t *__restrict__ pfrag, const float *s0, float *sT,
    TIn *__restrict__ o, int hqk, int hv, int group, int n_pairs) {
  using F = Cfg<D, C>;
  using CC = CarryCfg<D, C>;
  __shared__ __attribute__((aligned(16))) CarryLds<D, C, TIn> L;

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
  const bool own = (F::NKT == 8) || (wave < F::NKT);

  // Loop-invariant lane offsets (clamped so idle lanes issue valid loads).
  // Thread tid fetches pieces p = tid % 256 + 256 u of K (waves 0-3) or of Q
  // (waves 4-7), the numbering carry_commit uses.
  CarryLane<CC::KP> ln;
  {
    using CS = CarryCfg<D, C, TIn>;
    const int ibc = min(wave & 3, F::NIB - 1);
#pragma unroll
    for (int u = 0; u < CC::KP; ++u) {
      const int p = min((tid & 255) + (CC::NT / 2) * u, CC::NP - 1);
      ln.kq[u] = (uint32_t)((p / (D / 8)) * hqk * D + 8 * (p % (D / 8)));
    }
    ln.frag = (uint32_t)((ibc * F::KS * 64 + lane) * 8);
    ln.sd_any = tid < CS::SP;
    ln.sd_v = tid < CS::VP;
    ln.sd = ln.sd_v ? (uint32_t)(((tid / CS::VPR) * hv * D + (tid % CS::VPR) * (16 / (int)sizeof(TIn))) * sizeof(TIn))
                    : (uint32_t)(16 * (tid - CS::VP));
  }

  if (C < F::CP) {  // zero the token positions past the chunk, once
    for (int idx = tid; idx < 16 * F::LDV; idx += CC::NT) {
      L.Yl[idx] = 0;
      L.Ul[idx] = 0;
      L.Uh[idx] = 0;
    }
    for (int idx = C * D + tid; idx < F::CP * D; idx += CC::NT) {
      L.Kn[0][idx] = 0;
      L.Kn[1][idx] = 0;
    }
    lds_barrier();
  }

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
    ChunkRegs<D, C> ra, rb;
    carry_fetch<D, C, TIn>(ra, ln, wave < 4, q, k, v, dec_ws, tfrag, pfrag,
                           seq_t0, (int)min((int64_t)C, seq_t1 - seq_t0),
                           c0 * hv + h, h, hk, hqk, hv, v0);
    if (own)
      *reinterpret_cast<uint2 *>(&L.Sl[l16 * F::LDK + 16 * wave + 4 * g4]) =
          pack4_bf16(S[0], S[1], S[2], S[3]);
    carry_commit<D, C>(ra, wave < 4 ? L.Kn[0] : L.Qn, tid & 255);
    carry_commit_small<D, C, TIn>(ra, L.Vl[0], L.Dl[0], tid);
    lds_barrier();

    for (int lc = 0; lc < nch; lc += 2) {
      carry_step<D, C, TIn>(L, S, ra, rb, ln, lc, nch, seq_t0, seq_t1, c0, q, k,
                            v, dec_ws, tfrag, pfrag, o, h, hk, hqk, hv, v0, tid);
      if (lc + 1 < nch)
        carry_step<D, C, TIn>(L, S, rb, ra, ln, lc + 1, nch, seq_t0, seq_t1, c0,
                              q, k, v, dec_ws, tfrag, pfrag, o, h, hk, hqk, hv,
                              v0, tid);
    }
  }

  if (own)
    *reinterpret_cast<float4 *>(sT + ((int64_t)pair * D + v0 + l16) * D + 16 * wave + 4 * g4) =
        make_float4(S[0], S[1], S[2], S[3]);
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
  w.decay = p;
  p = align256(p + sizeof(float) * (size_t)nc * hv * 2 * chunk);
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
  float *dec = reinterpret_cast<float *>(base + ws.decay);
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
                       group, dec, tf, pf);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }

  const int n_pairs = a.n_seqs * a.hv;
  const int64_t blocks = (int64_t)8 * ((n_pairs + 7) / 8) * F::NVT;
  hipLaunchKernelGGL((chunk_carry_kernel<D, C, TIn>), dim3((unsigned)blocks), dim3(512),
                     0, a.stream, (const TIn *)a.q, (const TIn *)a.k,
                     (const TIn *)a.v, a.beta, a.cu_seqlens, off, dec, tf, pf,
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
