// tile_carry.hip -- the inter-chunk carry of the chunked prefill with one
// work-group per (sequence, value head, 16-row value tile), for batches with
// few (sequence, value head) chains: it spreads every chain over eight
// work-groups without cutting it into segments, so the operands are read once
// from HBM (and eight times from L2). Batches with many chains take the
// whole-chain carry (chain.hip), which reads each chunk's operands once per
// chain.
//
// Per chunk, with the chunk-local tables T' = (I + A)^-1 diag(beta),
// P = lower(E ⊙ Q K^T), Q in operand order and the decay factors:
//   X = K S^T,  U = T' (V - exp(gamma) X),  O = exp(gamma) Q S^T + P U,
//   S <- exp(gamma_last) S + (exp(gamma_last - gamma) U)^T K.
#include "gdn_launch.h"
#include "prefill_common.h"

namespace gdn {

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
// more ahead: waves 0-3 read the K rows, V and exp(gamma) of chunk c + 1
// in phase 2 of chunk c (the K-row reads stay in flight across the barrier)
// and their K^T operands in phase 1, waves 4-7 their K^T operands in
// phase 1 too. Outputs go from registers straight to global
// memory.
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
  // The tiles exchanged between wavefronts, stored in the B-operand order of
  // the products that read them: contraction step s is 64 lanes x 16 bytes,
  // contiguous, so each operand read is one conflict-free 1 KB block
  // (row-major tiles with padded rows took two LDS passes per read).
  uint16_t Sl[F::DS * 512];     // bf16 copy of the state tile (key order)
  uint16_t Yl[F::KS * 512];     // Y (token order of tok_pos)
  uint16_t Ul[F::KS * 512];     // U
  uint16_t Uh[F::KS * 512];     // exp(gamma_last - gamma) U
};


// Element index, in a B-operand-ordered tile, of the 4 values a lane holds
// in accumulator layout:
//  - state tile `t` (keys 16 t + 4 g4 + [0, 4) of row l16): step t / 2,
//    operand lane 16 (2 (t % 2) + g4 / 2) + l16, half g4 % 2. The 64 lanes of
//    one key tile write 512 contiguous bytes (conflict-free 8-byte stores).
//  - token block `ib` (tokens 16 ib + 4 g4 + [0, 4), row l16): step ib / 2,
//    operand lane 16 g4 + l16, half ib % 2 (the token order of tok_pos).
__device__ __forceinline__ int s_slot(int t, int l16, int g4) {
  return ((t >> 1) * 64 + 16 * (2 * (t & 1) + (g4 >> 1)) + l16) * 8 + 4 * (g4 & 1);
}
__device__ __forceinline__ int y_slot(int ib, int l16, int g4) {
  return ((ib >> 1) * 64 + 16 * g4 + l16) * 8 + 4 * (ib & 1);
}
// Operand of step s for lane `lane`.
__device__ __forceinline__ uint4 op_read(const uint16_t *T, int s, int lane) {
  return *reinterpret_cast<const uint4 *>(&T[(s * 64 + lane) * 8]);
}

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
// A loader issues a chunk's copies in three parts, one per phase: slots
// [part_lo(p), part_lo(p + 1)) in part p.
template <int D, int C, typename TIn>
constexpr int part_lo(int p) { return (CarryCfg<D, C, TIn>::SLOTS * p) / 3; }
template <int D, int C, typename TIn, int LW>
constexpr int part_copies(int p) {
  using CC = CarryCfg<D, C, TIn>;
  int n = 0;
  for (int i = part_lo<D, C, TIn>(p); i < part_lo<D, C, TIn>(p + 1); ++i)
    n += (CC::NLW * i + LW < CC::M) ? 1 : 0;
  return n;
}

// Loader wavefront LW (a template parameter, so that the kind of each of its
// copies is known when compiling). The copies of chunk lc + NA go into the
// buffer chunk lc - 1 used, a third of them before each barrier of chunk lc,
// and chunk lc + 1 must have landed before the first barrier of chunk lc:
// waves 0-3 read it in phase 2. Issuing a buffer-to-LDS copy takes a
// wavefront tens of cycles while the compute wavefronts load and store too;
// issued all at the start of the chunk, the copies held the first barrier
// past the compute wavefronts' phase 1 (carry kernel at 4096 tokens 54.0 ->
// 52.5 us; two parts, before the second and third barriers: 53.5 us).
template <int D, int C, typename TIn, int LW>
__device__ __forceinline__ void carry_loader(
    CarryLds<D, C, TIn> &L, int lane, const uint16_t *__restrict__ ksrc, int kstride,
    const TIn *__restrict__ v, const float *__restrict__ dec_ws, int nch,
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

  auto issue_part = [&](int lc, auto part) {  // part p of chunk lc's copies
    constexpr int p = decltype(part)::value;
    const CopyRes R = res(lc);
#pragma unroll
    for (int i = part_lo<D, C, TIn>(p); i < part_lo<D, C, TIn>(p + 1); ++i)
      issue_copy<D, C, TIn>(L, lc % CC::NB, R, CC::NLW * i + LW, off[i]);
  };
  for (int lc = 0; lc < nch; ++lc) {
    const bool more = lc + NA < nch;
    if (more) issue_part(lc + NA, std::integral_constant<int, 0>{});
    // Chunk lc + 1 must have landed. While copies are still issued every
    // chunk, those of chunk lc + 2 and the part of chunk lc + NA just issued
    // may stay in flight; near the end everything is waited for.
    static_assert(NA == 3, "chunks in flight");
    if (more)
      wait_vm<NCP + part_copies<D, C, TIn, LW>(0)>();
    else
      wait_vm<0>();
    lds_barrier();
    if (more) issue_part(lc + NA, std::integral_constant<int, 1>{});
    lds_barrier();
    if (more) issue_part(lc + NA, std::integral_constant<int, 2>{});
    lds_barrier();
  }
}

// ---------------------------------------------------------------- compute
// Per chunk c, three phases separated by work-group barriers:
//   1. waves 0-3: X = K S^T for their token block, Y = V - exp(gamma) X;
//      then T' of chunk c + 1 and the K^T operands of chunk c.
//      waves 4-7: O of chunk c-1 = exp(gamma) Q S^T + P U (their operands
//      were kept from chunk c-1; U of chunk c-1 is still in LDS), stored to
//      global memory; the K^T operands of chunk c.
//   2. waves 0-3: U = T' Y and exp(gamma_last - gamma) U; then chunk
//      c + 1's K rows, V and exp(gamma).
//      waves 4-7: Q S^T (S is still the state entering chunk c).
//   3. all eight: S^T <- exp(gamma_last) S^T + K^T (exp(gamma_last - gamma) U)
//      for their key tile.
// The chain from one state to the next runs through phases 1-3 on waves 0-3
// and the update; the output work fills the phases where it would idle.
template <int D, int C, typename TIn>
__device__ __forceinline__ void state_update(CarryLds<D, C, TIn> &L, f32x4 &S, const uint4 *kt,
                                             float glast, int wave, int l16, int g4) {
  using F = Cfg<D, C>;
  uint4 bu[F::KS];
#pragma unroll
  for (int s = 0; s < F::KS; ++s)
    bu[s] = op_read(L.Uh, s, 16 * g4 + l16);
  f32x4 acc = S * glast;
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int s = 0; s < F::KS; ++s) acc = mfma_16x16x32(kt[s], bu[s], acc);
  S = acc;
  *reinterpret_cast<uint2 *>(&L.Sl[s_slot(wave, l16, g4)]) =
      pack4_bf16(acc[0], acc[1], acc[2], acc[3]);
}

// Wavefronts 0-3: X, Y and U for token block ib. Each role runs its own loop
// (with the same barriers) so that every register prefetched for the next
// chunk is consumed and then reloaded in place, but for T', which alternates
// between two register sets.
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
  const uint32_t foff = (uint32_t)(((ibc * F::KS) * 64 + lane) * 16);
  auto frag_res = [&](int lc) {
    return make_rsrc(tfrag + ((c0 + lc) * hv + h) * F::FRAG, F::FRAG * 2);
  };
  // operands of the chunk in use, read ahead
  uint4 fa[F::KS];   // T' rows of block ib (global), chunks of even index
  uint4 ka[F::DS];   // K rows of block ib (LDS)
  uint4 kt[F::KS];   // K^T operands of key tile `wave` (LDS)
  // V is kept as the input's bits until phase 1 uses it: converting it where
  // it is read (then phase 3 of the chunk before, now phase 2) made each
  // conversion wait for its LDS read there, on the chunk's critical path
  // (4096 tokens: 76.6 -> 75.5 us per call). Reading the output wavefronts'
  // decay factor a phase early instead was slower (77.4 us).
  uint32_t vb[4];
  float ge[4], he[4], glast = 0.f;
  auto fetch_lds = [&](int b) {  // V, exp(gamma), then K rows of buffer b
    if (blk) {
      const TIn *vt = reinterpret_cast<const TIn *>(L.Vl[b]);
#pragma unroll
      for (int e = 0; e < 4; ++e) vb[e] = RawElem<TIn>::load(&vt[(tb + e) * 16 + l16]);
      const float4 ge4 = *reinterpret_cast<const float4 *>(&L.Dl[b][tb]);
      ge[0] = ge4.x; ge[1] = ge4.y; ge[2] = ge4.z; ge[3] = ge4.w;
    }
    if (blk) {
#pragma unroll
      for (int s = 0; s < F::DS; ++s)
        ka[s] = *reinterpret_cast<const uint4 *>(&L.Kn[b][kn_index<D>(16 * ib + l16, 32 * s + 8 * g4)]);
    }
  };
  // T' of chunk lc + 1 is read in phase 1 of chunk lc, where these
  // wavefronts wait for the output ones, into the second of two register
  // sets (the chunk loop is unrolled by two to alternate them). Reading it
  // after phase 2's product instead, into the set just consumed, put the
  // read's issue on the chunk's critical path (4096 tokens: carry kernel
  // 53.8 -> 53.5 us).
  auto load_t = [&](uint4 (&f)[F::KS], int lc) {  // the last chunk re-reads itself
    const rsrc_t rt = frag_res(min(lc, nch - 1));
#pragma unroll
    for (int s = 0; s < F::KS; ++s) f[s] = buf_load_b128(rt, s < nks ? foff + 1024u * s : kOutOfRange);
  };
  uint4 fb[F::KS];
  load_t(fa, 0);
  fetch_lds(0);
  auto step = [&](int lc, uint4 (&fcur)[F::KS], uint4 (&fnext)[F::KS]) {
    // ---- phase 1: X = K S^T, Y = V - exp(gamma) X (beta is folded into T')
    if (blk) {
      uint4 bs[F::DS];
#pragma unroll
      for (int s = 0; s < F::DS; ++s)
        bs[s] = op_read(L.Sl, s, lane);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 xs = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < F::DS; ++s) xs = mfma_16x16x32(ka[s], bs[s], xs);
      *reinterpret_cast<uint2 *>(&L.Yl[y_slot(ib, l16, g4)]) =
          pack4_bf16(RawElem<TIn>::cvt(vb[0]) - ge[0] * xs[0], RawElem<TIn>::cvt(vb[1]) - ge[1] * xs[1],
                     RawElem<TIn>::cvt(vb[2]) - ge[2] * xs[2], RawElem<TIn>::cvt(vb[3]) - ge[3] * xs[3]);
      __builtin_amdgcn_sched_barrier(0);
      load_t(fnext, lc + 1);
    }
    // Operands used later in this chunk: exp(gamma_last - gamma) for phase 2,
    // gamma_last and the K^T operands for phase 3. Read here, in the wait for
    // the output wavefronts, rather than with the next chunk's operands at
    // the end of phase 3, whose barrier they delayed (carry kernel at 4096
    // tokens 55.2 -> 54.4 us; outputs bitwise unchanged). The next chunk's
    // operands themselves are read in phase 2 (52.1 -> 51.3 us once the
    // loaders issued their copies over the three phases).
    {
      const int b = lc % CC::NB;
      if (blk) {
        const float4 he4 = *reinterpret_cast<const float4 *>(&L.Dl[b][C + tb]);
        he[0] = he4.x; he[1] = he4.y; he[2] = he4.z; he[3] = he4.w;
      }
      glast = L.Dl[b][C - 1];
      if (own) {
#pragma unroll
        for (int s = 0; s < F::KS; ++s) kt[s] = kt_operand<D>(L.Kn[b], wave, s, l16, g4);
      }
    }
    // the Y stores are complete; the K^T reads may stay in flight
    lds_barrier_keep<((F::NKT == 8) ? 2 * F::KS : 0)>();
    // ---- phase 2: U = T' Y and exp(gamma_last - gamma) U
    if (blk) {
      uint4 by[F::KS];
#pragma unroll
      for (int s = 0; s < F::KS; ++s)
        by[s] = op_read(L.Yl, s, lane);
      __builtin_amdgcn_sched_barrier(0);
      f32x4 u = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < F::KS; ++s) u = mfma_16x16x32(fcur[s], by[s], u);
      *reinterpret_cast<uint2 *>(&L.Ul[y_slot(ib, l16, g4)]) = pack4_bf16(u[0], u[1], u[2], u[3]);
      *reinterpret_cast<uint2 *>(&L.Uh[y_slot(ib, l16, g4)]) =
          pack4_bf16(he[0] * u[0], he[1] * u[1], he[2] * u[2], he[3] * u[3]);
    }
    // chunk lc + 1's LDS operands, whose K-row reads may stay in flight
    // across the barrier; its copies landed before the first barrier
    if (lc + 1 < nch) {
      __builtin_amdgcn_sched_barrier(0);
      fetch_lds((lc + 1) % CC::NB);
      lds_barrier_keep<((F::NIB == 4) ? F::DS : 0)>();
    } else {
      lds_barrier();
    }
    // ---- phase 3: state update
    if (own) {
      state_update<D, C, TIn>(L, S, kt, glast, wave, l16, g4);
      asm volatile("" ::"v"(S) : "memory");
    }
    lds_barrier();
  };
  for (int lc = 0; lc < nch; lc += 2) {
    step(lc, fa, fb);
    if (lc + 1 < nch) step(lc + 1, fb, fa);
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
      bu[s] = op_read(L.Ul, s, 16 * g4 + l16);
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
        bs[s] = op_read(L.Sl, s, lane);
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
    const uint16_t *__restrict__ qfrag, const float *s0, float *sT, TIn *__restrict__ o, int hqk, int hv, int group,
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
        for (int idx = tid; idx < F::KS * 512; idx += 64 * CC::NCW) {
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
        *reinterpret_cast<uint2 *>(&L.Sl[s_slot(wave, l16, g4)]) =
            pack4_bf16(S[0], S[1], S[2], S[3]);
      lds_barrier();
      if (wave < 4) {
        // The X -> Y -> U chain is the critical path of every chunk: its
        // wavefronts issue first when they compete with the output ones on
        // a SIMD (4096 tokens: 77.6 -> 77.1 us per call, 16 calls each).
        // The output wavefronts in turn issue before the loaders (carry
        // kernel 51.5 -> 51.15 us; the two compute roles at one priority:
        // 51.7 us).
        __builtin_amdgcn_s_setprio(2);
        carry_compute_xu<D, C, TIn>(L, S, wave, lane, nch, c0, tfrag, h, hv);
      } else {
        __builtin_amdgcn_s_setprio(1);
        carry_compute_o<D, C, TIn>(L, S, wave, lane, nch, c0, pfrag, qfrag, o, seq_t0, seq_t1,
                                   h, hk, hqk, hv, v0);
      }
    } else {
      const uint16_t *ksrc = reinterpret_cast<const uint16_t *>(k);
      const int kstride = hqk * D;
      static_assert(CC::NLW == 2, "loader dispatch below");
      if (wave == CC::NCW)
        carry_loader<D, C, TIn, 0>(L, lane, ksrc, kstride, v, dec_ws, nch, seq_t0, seq_t1, c0,
                                   h, hk, hqk, hv, v0);
      else
        carry_loader<D, C, TIn, 1>(L, lane, ksrc, kstride, v, dec_ws, nch, seq_t0, seq_t1, c0,
                                   h, hk, hqk, hv, v0);
    }
  }

  if (own)
    store_stream(sT + ((int64_t)pair * D + v0 + l16) * D + 16 * wave + 4 * g4, S);
}

// ============================================================ host side
template <int D, int C, typename TIn>
static hipError_t launch_tile_carry_t(const PrefillArgs &a, const PrefillWorkspace &ws) {
  using F = Cfg<D, C>;
  char *base = static_cast<char *>(a.workspace);
  const float *dec = reinterpret_cast<const float *>(base + ws.decay);
  const uint16_t *tf = reinterpret_cast<const uint16_t *>(base + ws.tfrag);
  const uint16_t *pf = reinterpret_cast<const uint16_t *>(base + ws.pfrag);
  const uint16_t *qf = reinterpret_cast<const uint16_t *>(base + ws.qfrag);
  const int group = a.hv / a.hqk;
  const int n_groups = a.n_seqs * a.hqk;
  const int64_t blocks = (int64_t)8 * ((n_groups + 7) / 8) * group * F::NVT;
  hipLaunchKernelGGL((chunk_carry_kernel<D, C, TIn>), dim3((unsigned)blocks),
                     dim3(kCarryThreads), 0, a.stream, (const TIn *)a.k, (const TIn *)a.v,
                     a.cu_seqlens, dec, tf, pf, qf, a.initial_state, a.final_state,
                     (TIn *)a.o, a.hqk, a.hv, group, n_groups);
  return hipGetLastError();
}

hipError_t launch_tile_carry(const PrefillArgs &a, const PrefillWorkspace &ws) {
  switch (a.d * 1000 + a.chunk) {
    case 32016: return launch_tile_carry_t<32, 16, __bf16>(a, ws);
    case 32032: return launch_tile_carry_t<32, 32, __bf16>(a, ws);
    case 32064: return launch_tile_carry_t<32, 64, __bf16>(a, ws);
    case 64016: return launch_tile_carry_t<64, 16, __bf16>(a, ws);
    case 64032: return launch_tile_carry_t<64, 32, __bf16>(a, ws);
    case 64064: return launch_tile_carry_t<64, 64, __bf16>(a, ws);
    case 128016: return launch_tile_carry_t<128, 16, __bf16>(a, ws);
    case 128032: return launch_tile_carry_t<128, 32, __bf16>(a, ws);
    case 128064: return launch_tile_carry_t<128, 64, __bf16>(a, ws);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gdn
