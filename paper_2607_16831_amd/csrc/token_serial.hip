// token_serial.hip -- prefill of short sequences, one token at a time.
//
// The recurrence of the paper's Section 3.2 is applied token by token along
// each sequence. For every state row r (value channel) of a (sequence, value
// head) pair:
//     sk = S[r,:] . k_t,   sq = S[r,:] . q_t            (old state)
//     delta = beta_t (v_t[r] - alpha_t sk)
//     o_t[r] = alpha_t sq + delta (q_t . k_t)          (= S_t[r,:] . q_t)
//     S[r,:] = alpha_t S[r,:] + delta k_t
// The state rows stay in registers from a sequence's first token to its last,
// so every state element is read once and written once per call, whatever the
// length, and no workspace is touched. Each token costs 6 d^2 vector-ALU
// flops per head, against matrix-core work in the chunked form, so this path
// pays only for sequences of a few tokens: the narrow short-shape fallback of
// the paper's Sections 5.3 and 5.5, chosen by the measured dispatch in gdn_api.hip.
//
// Launch shape as in the decode kernel: a state row of D fp32 values is held
// by D/4 lanes, 16 bytes each; a wavefront holds PASSES such row groups of one
// (sequence, value head) pair. The per-token inputs (k, q, the wavefront's v
// entries) are fetched TB tokens ahead into registers (TB = 1 when sequences
// hold about one token), each slot refilled right after it is consumed, and
// the gates of the next block of TB tokens in one vector load; loads past the
// sequence end are clamped to its last token and never used. Whole blocks run
// in the loop, the remaining tokens after it.
#include "gdn_device.h"
#include "gdn_launch.h"

namespace gdn {

namespace {

// Four consecutive elements, kept in their storage type until used so that a
// prefetch is not waited for at the load.
template <typename T>
struct Raw4;
template <>
struct Raw4<__bf16> {
  using type = uint2;
  static __device__ __forceinline__ type load(const __bf16 *p) {
    return *reinterpret_cast<const uint2 *>(p);
  }
  static __device__ __forceinline__ void unpack(type r, float out[4]) {
    out[0] = bf16_bits_to_f32(r.x & 0xffffu);
    out[1] = bf16_bits_to_f32(r.x >> 16);
    out[2] = bf16_bits_to_f32(r.y & 0xffffu);
    out[3] = bf16_bits_to_f32(r.y >> 16);
  }
};
template <>
struct Raw4<float> {
  using type = float4;
  static __device__ __forceinline__ type load(const float *p) {
    return *reinterpret_cast<const float4 *>(p);
  }
  static __device__ __forceinline__ void unpack(type r, float out[4]) {
    out[0] = r.x;
    out[1] = r.y;
    out[2] = r.z;
    out[3] = r.w;
  }
};

template <typename T>
struct Raw1;
template <>
struct Raw1<__bf16> {
  using type = uint16_t;
  static __device__ __forceinline__ type load(const __bf16 *p) {
    return *reinterpret_cast<const uint16_t *>(p);
  }
  static __device__ __forceinline__ float unpack(type r) { return bf16_bits_to_f32(r); }
};
template <>
struct Raw1<float> {
  using type = float;
  static __device__ __forceinline__ type load(const float *p) { return *p; }
  static __device__ __forceinline__ float unpack(type r) { return r; }
};

// Compiler fence over the unpacked operands of one token: they are
// materialised before it, and no memory access moves across it.
template <int P>
__device__ __forceinline__ void slot_fence(float (&kk)[4], float (&qq)[4], float (&vv)[P]) {
  asm volatile("" : "+v"(kk[0]), "+v"(kk[1]), "+v"(kk[2]), "+v"(kk[3]), "+v"(qq[0]),
               "+v"(qq[1]), "+v"(qq[2]), "+v"(qq[3])::"memory");
#pragma unroll
  for (int p = 0; p < P; ++p) asm volatile("" : "+v"(vv[p])::"memory");
}

}  // namespace

template <int D, int PASSES, int TB, typename TIn, bool GATED>
__global__ __launch_bounds__(256) void token_serial_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k, const TIn *__restrict__ v,
    const float *__restrict__ g, const float *__restrict__ beta, GateArgs gate,
    const int32_t *__restrict__ cu_seqlens, const float *initial_state,
    TIn *__restrict__ o, float *final_state, int64_t total_rows, int hqk, int hv,
    int group) {
  constexpr int LPR = D / 4;        // lanes per state row
  constexpr int RPP = kWave / LPR;  // rows per pass
  constexpr int RPW = RPP * PASSES;
  static_assert(D % RPW == 0, "a wavefront must stay in one head");
  using R4 = Raw4<TIn>;
  using R1 = Raw1<TIn>;

  const int lane = threadIdx.x & (kWave - 1);
  // Wavefront-uniform values in scalar registers, so that the token loop's
  // control flow is scalar.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t row0 = ((int64_t)blockIdx.x * (blockDim.x / kWave) + wave) * RPW;
  if (row0 >= total_rows) return;  // whole wavefront out of range

  const int64_t pair = row0 / D;  // (n, h) flattened, sequence-major
  const int r0 = (int)(row0 % D);
  const int n = (int)(pair / hv);
  const int h = (int)(pair % hv);
  const int hk = h / group;
  const int col = (lane % LPR) * 4;
  const int sub = lane / LPR;
  const int t0 = cu_seqlens[n], t1 = cu_seqlens[n + 1];

  const int64_t soff = (pair * D + r0 + sub) * (int64_t)D + col;
  f32x4 s[PASSES];
#pragma unroll
  for (int p = 0; p < PASSES; ++p)
    s[p] = initial_state ? load_stream(initial_state + soff + (int64_t)p * RPP * D)
                         : f32x4{0.f, 0.f, 0.f, 0.f};

  const float a_log = GATED ? gate.a_log[h] : 0.f;
  const float dt_bias = GATED ? gate.dt_bias[h] : 0.f;
  const float *gsrc = GATED ? gate.a : g;
  const float *bsrc = GATED ? gate.b : beta;

  typename R4::type kr[TB], qr[TB];
  typename R1::type vr[TB][PASSES];
  // Fills slot j with k, q and v of token t (clamped to the sequence).
  auto fetch = [&](int j, int t) {
    const int64_t tl = min(t, t1 - 1);
    kr[j] = R4::load(k + (tl * hqk + hk) * D + col);
    qr[j] = R4::load(q + (tl * hqk + hk) * D + col);
#pragma unroll
    for (int p = 0; p < PASSES; ++p) vr[j][p] = R1::load(v + (tl * hv + h) * D + r0 + p * RPP + sub);
  };
  // The gates of a block of TB tokens in one vector load: lane l < TB holds
  // g (or a) of token tb + l, lane TB + l holds beta (or b). Read out per
  // token with readlane.
  const int glane = lane % (2 * TB);
  auto fetch_gates = [&](int tb) {
    const int64_t tl = min(tb + glane % TB, t1 - 1);
    return glane < TB ? gsrc[tl * hv + h] : bsrc[tl * hv + h];
  };
  float gcur = 0.f, gnext = 0.f;
  // Token t from slot j; refills the slot with token t + TB when asked.
  auto step = [&](int j, int t, bool refill) {
    float kk[4], qq[4], vv[PASSES];
    R4::unpack(kr[j], kk);
    R4::unpack(qr[j], qq);
#pragma unroll
    for (int p = 0; p < PASSES; ++p) vv[p] = R1::unpack(vr[j][p]);
    float gl = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gcur), j));
    float bt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gcur), TB + j));
    if (GATED) {
      gl = gate_log_decay(gl, a_log, dt_bias);
      bt = gate_beta(bt);
    }
    const float alpha = __expf(gl);
    // The slot's last use ends here: its refill below cannot be hoisted above
    // this point, so the new values may take the old values' registers (no
    // copy at the loop latch, which would wait for the refills).
    slot_fence(kk, qq, vv);
    if (refill) fetch(j, t + TB);

    float qk = qq[0] * kk[0] + qq[1] * kk[1] + qq[2] * kk[2] + qq[3] * kk[3];
    qk = group_sum<LPR>(qk);
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      float sk = s[p][0] * kk[0] + s[p][1] * kk[1] + s[p][2] * kk[2] + s[p][3] * kk[3];
      float sq = s[p][0] * qq[0] + s[p][1] * qq[1] + s[p][2] * qq[2] + s[p][3] * qq[3];
      sk = group_sum<LPR>(sk);
      sq = group_sum<LPR>(sq);
      const float delta = bt * (vv[p] - alpha * sk);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[p][e] = alpha * s[p][e] + delta * kk[e];
      if ((lane % LPR) == 0)
        Elem<TIn>::store1(o + ((int64_t)t * hv + h) * D + r0 + p * RPP + sub,
                          alpha * sq + delta * qk);
    }
  };

  if (t0 < t1) {
    gcur = fetch_gates(t0);
#pragma unroll
    for (int j = 0; j < TB; ++j) fetch(j, t0 + j);
  }
  int t = t0;
  for (; t + TB <= t1; t += TB) {  // whole blocks
    gnext = fetch_gates(t + TB);
#pragma unroll
    for (int j = 0; j < TB; ++j) step(j, t + j, true);
    gcur = gnext;
  }
  // Fewer than TB tokens remain; token t + j sits in slot j.
  const int rem = t1 - t;
#pragma unroll
  for (int j = 0; j < TB - 1; ++j)
    if (j < rem) step(j, t + j, false);

#pragma unroll
  for (int p = 0; p < PASSES; ++p) store_stream(final_state + soff + (int64_t)p * RPP * D, s[p]);
}

template <int D, int PASSES, int TB, typename TIn>
static hipError_t launch_serial_p(const PrefillArgs &a, int64_t total_rows) {
  constexpr int RPW = (kWave / (D / 4)) * PASSES;
  const int64_t rows_per_block = RPW * 4;
  const int64_t blocks = (total_rows + rows_per_block - 1) / rows_per_block;
  auto kern = a.gate.a_log != nullptr ? token_serial_kernel<D, PASSES, TB, TIn, true>
                                      : token_serial_kernel<D, PASSES, TB, TIn, false>;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, a.stream, (const TIn *)a.q,
                     (const TIn *)a.k, (const TIn *)a.v, a.g, a.beta, a.gate, a.cu_seqlens,
                     a.initial_state, (TIn *)a.o, a.final_state, total_rows, a.hqk, a.hv,
                     a.hv / a.hqk);
  return hipGetLastError();
}

template <int D, int PASSES, typename TIn>
static hipError_t launch_serial_pb(const PrefillArgs &a, int64_t total_rows) {
  // With at most one token per sequence on average, prefetching more tokens
  // only costs registers (the loads past a sequence's end are clamped).
  if (a.n_tokens <= a.n_seqs) return launch_serial_p<D, PASSES, 1, TIn>(a, total_rows);
  return launch_serial_p<D, PASSES, 4, TIn>(a, total_rows);
}

template <int D, typename TIn>
static hipError_t launch_serial_t(const PrefillArgs &a) {
  const int64_t total_rows = (int64_t)a.n_seqs * a.hv * D;
  if (total_rows == 0) return hipSuccess;
  // As for decode: four passes per wavefront when that still gives every
  // compute unit two work-groups, else two; eight (head sizes of 64 and up)
  // for the largest batches, where each wavefront's input loads are then
  // shared by more state rows.
  const int64_t blocks4 = (total_rows + (kWave / (D / 4)) * 16 - 1) / ((kWave / (D / 4)) * 16);
  const int64_t cus = device_compute_units();
  if constexpr (D >= 64) {
    if (blocks4 >= 1024 * cus) return launch_serial_pb<D, 8, TIn>(a, total_rows);
  }
  if (blocks4 < 2 * cus) return launch_serial_pb<D, 2, TIn>(a, total_rows);
  return launch_serial_pb<D, 4, TIn>(a, total_rows);
}

template <typename TIn>
static hipError_t launch_serial_e(const PrefillArgs &a) {
  switch (a.d) {
    case 32: return launch_serial_t<32, TIn>(a);
    case 64: return launch_serial_t<64, TIn>(a);
    case 128: return launch_serial_t<128, TIn>(a);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_prefill_serial(const PrefillArgs &a) {
  return a.dtype == GDN_BF16 ? launch_serial_e<__bf16>(a) : launch_serial_e<float>(a);
}

}  // namespace gdn
