// prefill_f32.hip -- the chunked prefill for float32 inputs, in float32
// throughout (gfx950).
//
// The same chunked (WY) form as the bf16 path, with every product on the
// float32 matrix instruction v_mfma_f32_16x16x4_f32 and every table in
// float32. For a chunk of n <= C tokens with incoming state S (d_v x d_k),
// gamma the in-chunk prefix sum of g, Gamma = exp(gamma),
// E_ij = exp(gamma_i - gamma_j) (j <= i) and ehat = exp(gamma_last - gamma):
//
//   A  = strict_lower(diag(beta) E ⊙ K K^T),  T = (I + A)^-1,
//   X  = K S^T,  U = T diag(beta) (V - Gamma ⊙ X),
//   O  = Gamma ⊙ (Q S^T) + (E ⊙ Q K^T) U,
//   S' = exp(gamma_last) S + (ehat ⊙ U)^T K.
//
// One work-group per (sequence, value head) walks the chunks of its
// sequence. It has one wavefront per 16-row value tile; each holds its rows
// of the state, transposed, in the accumulator layout of the matrix
// instruction for the whole sequence. The chunk's K, Q, A, T and P live in
// LDS, shared by the wavefronts: the Gram tiles are dealt over them, and
// wavefront 0 solves for T by forward substitution. With D/16 wavefronts
// and no workspace, it is meant for
// correctness at float32 precision (the "fp32 throughout" case), not speed.
//
// Operand layouts (v_mfma_f32_16x16x4_f32, see gdn_device.h): in step kk of
// a 16-wide contraction, slot g of lane (l16, g) stands for index 4 g + kk,
// so a B operand is a lane's own accumulator element kk, and A operands are
// single LDS reads.
#include "gdn_launch.h"
#include "prefill_common.h"

namespace gdn {

template <int D, int C>
struct F32Cfg {
  static constexpr int NW = D / 16;      // wavefronts: one per 16-row value tile
  static constexpr int NT = 64 * NW;
  static constexpr int NIB = C / 16;     // 16-token blocks per chunk
  static constexpr int NKT = D / 16;     // 16-key tiles of the state
  static constexpr int PK = D + 1;       // odd pitches spread the column reads
  static constexpr int PC = C + 1;
};

template <int D, int C>
struct F32Lds {
  using FC = F32Cfg<D, C>;
  float K[C * FC::PK];   // K rows of the chunk (zero past the sequence)
  float Q[C * FC::PK];
  float A[C * FC::PC];   // strict_lower(diag(beta) E ⊙ K K^T)
  float T[C * FC::PC];   // (I + A)^-1 (unit lower; beta applied on use)
  float P[C * FC::PC];   // E ⊙ Q K^T, diagonal included
  float bet[C];          // beta (zero past the sequence)
  float lg[C];           // g, then gamma (in-chunk prefix sum)
  float ge[C];           // exp(gamma_i)
  float he[C];           // exp(gamma_last - gamma_i)
};

template <int D, int C>
__global__ __launch_bounds__((F32Cfg<D, C>::NT)) void prefill_f32_kernel(
    const float *__restrict__ q, const float *__restrict__ k, const float *__restrict__ v,
    const float *__restrict__ g, const float *__restrict__ beta, GateArgs gate,
    const int32_t *__restrict__ cu, const float *s0, float *sT, float *__restrict__ o, int hqk,
    int hv) {
  using FC = F32Cfg<D, C>;
  constexpr int PK = FC::PK, PC = FC::PC, NIB = FC::NIB, NKT = FC::NKT;
  __shared__ F32Lds<D, C> L;

  const int pair = blockIdx.x;  // sequence * hv + value head
  const int n = pair / hv, h = pair - n * hv;
  const int hk = h / (hv / hqk);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g4 = lane >> 4;
  const int v0 = 16 * wave;  // value rows of this wavefront
  const int64_t t_begin = cu[n], t_end = cu[n + 1];
  const int nch = (int)((t_end - t_begin + C - 1) / C);

  // State rows v0..v0+15, transposed: tile t holds S^T[16 t + 4 g4 + e][l16],
  // i.e. S[v0 + l16][16 t + 4 g4 + e].
  f32x4 St[NKT];
  const int64_t sbase = (int64_t)pair * D * D + (int64_t)(v0 + l16) * D;
#pragma unroll
  for (int t = 0; t < NKT; ++t) {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      St[t][e] = s0 != nullptr ? s0[sbase + 16 * t + 4 * g4 + e] : 0.f;
  }

  // The upper triangles of A, T and P are never written: zero them once.
  for (int i = tid; i < C * PC; i += FC::NT) {
    L.A[i] = 0.f;
    L.T[i] = 0.f;
    L.P[i] = 0.f;
  }

  for (int c = 0; c < nch; ++c) {
    const int64_t t0 = t_begin + (int64_t)c * C;
    const int nv = (int)min((int64_t)C, t_end - t0);
    __syncthreads();  // the previous chunk's LDS reads are done

    // ---- K and Q rows, g and beta (zero past the sequence: exact identity
    // steps, beta = 0 and k = 0)
    for (int i = tid; i < C * D; i += FC::NT) {
      const int r = i / D, col = i - r * D;
      const bool in = r < nv;
      const int64_t src = ((t0 + r) * hqk + hk) * D + col;
      L.K[r * PK + col] = in ? k[src] : 0.f;
      L.Q[r * PK + col] = in ? q[src] : 0.f;
    }
    if (tid < C) {
      float gv = 0.f, bv = 0.f;
      if (tid < nv) {
        const int64_t e = (t0 + tid) * hv + h;
        if (gate.a != nullptr) {
          gv = gate_log_decay(gate.a[e], gate.a_log[h], gate.dt_bias[h]);
          bv = gate_beta(gate.b[e]);
        } else {
          gv = g[e];
          bv = beta[e];
        }
      }
      L.lg[tid] = gv;
      L.bet[tid] = bv;
    }
    __syncthreads();
    if (tid < C) {  // gamma_i = sum_{m <= i} g_m, summed in token order
      float s = 0.f;
      for (int m = 0; m <= tid; ++m) s += L.lg[m];
      L.ge[tid] = s;  // gamma for now
    }
    __syncthreads();
    if (tid < C) {
      const float gl = L.ge[C - 1];  // padding adds g = 0: gamma of the last token
      const float gm = L.ge[tid];
      L.lg[tid] = gm;
      L.ge[tid] = expf(gm);
      L.he[tid] = expf(gl - gm);
    }
    __syncthreads();

    // ---- Gram tiles (i, j), j <= i, of K K^T and Q K^T, dealt over the
    // wavefronts; masked and decayed into A and P. Every exponent is a
    // non-positive difference gamma_r - gamma_c with c <= r.
    constexpr int NTILE = NIB * (NIB + 1) / 2;
    for (int job = wave; job < 2 * NTILE; job += FC::NW) {
      const bool isq = job >= NTILE;
      int tt = isq ? job - NTILE : job, ib = 0;
      while (tt > ib) {
        tt -= ib + 1;
        ++ib;
      }
      const int jb = tt;
      const float *X = isq ? L.Q : L.K;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
      for (int s = 0; s < D / 4; ++s) {
        // A = rows of X (block ib), B = K^T (block jb); index 4 g4 + (s % 4)
        // of key tile s / 4
        const int key = 16 * (s >> 2) + 4 * g4 + (s & 3);
        acc = mfma_16x16x4_f32(X[(16 * ib + l16) * PK + key], L.K[(16 * jb + l16) * PK + key],
                               acc);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * ib + 4 * g4 + e, cc = 16 * jb + l16;
        const float dec = cc <= r ? expf(L.lg[r] - L.lg[cc]) : 0.f;
        if (isq)
          L.P[r * PC + cc] = cc <= r ? dec * acc[e] : 0.f;
        else
          L.A[r * PC + cc] = cc < r ? L.bet[r] * dec * acc[e] : 0.f;
      }
    }
    __syncthreads();

    // ---- K S^T and Q S^T for this wavefront's rows; then T = (I + A)^-1 on
    // wavefront 0 (lane j: column j, row by row,
    // T[i][j] = -sum_{m=j..i-1} A[i][m] T[m][j] with T[j][j] = 1).
    f32x4 X[NIB], QS[NIB];
    auto state_products = [&]() {
#pragma unroll
      for (int ib = 0; ib < NIB; ++ib) {
        f32x4 xa = f32x4{0.f, 0.f, 0.f, 0.f}, qa = xa;
#pragma unroll
        for (int t = 0; t < NKT; ++t) {
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const int key = 16 * t + 4 * g4 + kk;
            xa = mfma_16x16x4_f32(L.K[(16 * ib + l16) * PK + key], St[t][kk], xa);
            qa = mfma_16x16x4_f32(L.Q[(16 * ib + l16) * PK + key], St[t][kk], qa);
          }
        }
        X[ib] = xa;
        QS[ib] = qa;
        // one 16-token block at a time: keeps the scheduler from hoisting
        // every block's LDS reads (register spills at d = 128, C = 64)
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    state_products();
    if (wave == 0) {
      if (lane < C) {
        const int j = lane;
        L.T[j * PC + j] = 1.f;
        for (int i = j + 1; i < C; ++i) {
          float s = 0.f;
          for (int m = j; m < i; ++m) s = fmaf(L.A[i * PC + m], L.T[m * PC + j], s);
          L.T[i * PC + j] = -s;
        }
      }
    }
    __syncthreads();

    // ---- Y = V - Gamma ⊙ X (tile rows 16 ib + 4 g4 + e, value v0 + l16);
    // U = T diag(beta) Y
    f32x4 Y[NIB], U[NIB];
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * ib + 4 * g4 + e;
        const float vv = r < nv ? v[((t0 + r) * hv + h) * D + v0 + l16] : 0.f;
        Y[ib][e] = vv - L.ge[r] * X[ib][e];
      }
    }
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jb = 0; jb <= ib; ++jb) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int j = 16 * jb + 4 * g4 + kk;
          acc = mfma_16x16x4_f32(L.T[(16 * ib + l16) * PC + j] * L.bet[j], Y[jb][kk], acc);
        }
      }
      U[ib] = acc;
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- O = Gamma ⊙ (Q S^T) + P U, rows past the sequence not stored
#pragma unroll
    for (int ib = 0; ib < NIB; ++ib) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jb = 0; jb <= ib; ++jb) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          acc = mfma_16x16x4_f32(L.P[(16 * ib + l16) * PC + 16 * jb + 4 * g4 + kk], U[jb][kk],
                                 acc);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 16 * ib + 4 * g4 + e;
        if (r < nv) o[((t0 + r) * hv + h) * D + v0 + l16] = L.ge[r] * QS[ib][e] + acc[e];
      }
      __builtin_amdgcn_sched_barrier(0);
    }

    // ---- S^T <- exp(gamma_last) S^T + K^T (ehat ⊙ U), key tile by key tile
    const float glast = L.ge[C - 1];
#pragma unroll
    for (int t = 0; t < NKT; ++t) {
      f32x4 acc = St[t] * glast;
#pragma unroll
      for (int jb = 0; jb < NIB; ++jb) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int j = 16 * jb + 4 * g4 + kk;
          acc = mfma_16x16x4_f32(L.K[j * PK + 16 * t + l16] * L.he[j], U[jb][kk], acc);
        }
      }
      St[t] = acc;
      __builtin_amdgcn_sched_barrier(0);
    }
  }

#pragma unroll
  for (int t = 0; t < NKT; ++t) {
#pragma unroll
    for (int e = 0; e < 4; ++e) sT[sbase + 16 * t + 4 * g4 + e] = St[t][e];
  }
}

template <int D, int C>
static hipError_t launch_f32_t(const PrefillArgs &a) {
  if (a.n_seqs <= 0) return hipSuccess;
  hipLaunchKernelGGL((prefill_f32_kernel<D, C>), dim3((unsigned)(a.n_seqs * a.hv)),
                     dim3(F32Cfg<D, C>::NT), 0, a.stream, (const float *)a.q,
                     (const float *)a.k, (const float *)a.v, a.g, a.beta, a.gate, a.cu_seqlens,
                     a.initial_state, a.final_state, (float *)a.o, a.hqk, a.hv);
  return hipGetLastError();
}

hipError_t launch_prefill_f32(const PrefillArgs &a) {
  switch (a.d * 1000 + a.chunk) {
    case 32016: return launch_f32_t<32, 16>(a);
    case 32032: return launch_f32_t<32, 32>(a);
    case 32064: return launch_f32_t<32, 64>(a);
    case 64016: return launch_f32_t<64, 16>(a);
    case 64032: return launch_f32_t<64, 32>(a);
    case 64064: return launch_f32_t<64, 64>(a);
    case 128016: return launch_f32_t<128, 16>(a);
    case 128032: return launch_f32_t<128, 32>(a);
    case 128064: return launch_f32_t<128, 64>(a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gdn
