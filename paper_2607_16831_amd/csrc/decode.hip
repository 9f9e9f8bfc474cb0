// decode.hip -- one decode step of the gated delta rule, state updated in place.
//
// Uses the paper's one-pass form with the gate-scaled state (Section 3.2): for
// every state row r (value channel) of a (sequence, value head) pair,
//     sk = S[r,:] . k,   sq = S[r,:] . q          (both on the OLD state)
//     delta = beta * (v[r] - alpha * sk)
//     o[r]  = alpha * sq + delta * (q . k)        (= S'[r,:] . q)
//     S'[r,:] = alpha * S[r,:] + delta * k
// so each state element is read once and written once. Rows are independent,
// which makes the flattened (pair, row) index the parallel axis (the V split
// of Section 3.2 taken to its limit).
//
// Launch shape: 256-thread work-groups of 4 wavefronts. A state row of D fp32
// values is covered by D/4 lanes with one 16-byte access each, so a wavefront
// touches 64*4/D rows per pass and makes PASSES passes; all PASSES loads are
// issued before any reduction so every lane keeps PASSES x 16 bytes in flight.
// PASSES is chosen per call (the paper's decode lesson, Section 5.4: decode is
// a launch-shape problem per batch regime): 4 when that grid still gives every
// CU two work-groups, else 2, which doubles the work-groups of a small batch
// (measured on MI355X, d = 128, 32 value heads: B = 1 takes 3.4 us with 2
// passes against 3.8 us with 4; from B = 8 on, 4 passes are as fast or faster).
// State traffic uses non-temporal loads and stores: each byte is touched once.
//
// With raw gate inputs (a_log != NULL) the gate and beta are formed here from
// a, b, A_log and dt_bias (Section 3.2) instead of being read.
#include "gdn_device.h"
#include "gdn_launch.h"

namespace gdn {

template <int D, int PASSES, typename TIn>
__global__ __launch_bounds__(256) void decode_kernel(
    const TIn *__restrict__ q, const TIn *__restrict__ k,
    const TIn *__restrict__ v, const float *__restrict__ g,
    const float *__restrict__ beta, const float *__restrict__ ga,
    const float *__restrict__ gb, const float *__restrict__ a_log,
    const float *__restrict__ dt_bias, float *__restrict__ state,
    TIn *__restrict__ o, int64_t total_rows, int hqk, int hv, int group) {
  constexpr int LPR = D / 4;            // lanes per state row
  constexpr int RPP = kWave / LPR;      // rows per pass
  constexpr int ROWS_PER_WAVE = RPP * PASSES;
  static_assert(D % ROWS_PER_WAVE == 0, "a wavefront must stay in one head");

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int64_t row0 =
      ((int64_t)blockIdx.x * (blockDim.x / kWave) + wave) * ROWS_PER_WAVE;
  if (row0 >= total_rows) return;  // whole wavefront out of range

  const int64_t pair = row0 / D;  // (b, h) flattened, b-major
  const int r0 = (int)(row0 % D);
  const int64_t b = pair / hv;
  const int h = (int)(pair % hv);
  const int hk = h / group;
  const int col = (lane % LPR) * 4;
  const int sub = lane / LPR;

  float kk[4], qq[4];
  Elem<TIn>::load4(k + (b * hqk + hk) * D + col, kk);
  Elem<TIn>::load4(q + (b * hqk + hk) * D + col, qq);
  f32x4 s[PASSES];
  float vv[PASSES];
  float *srow = state + (pair * D + r0 + sub) * (int64_t)D + col;
#pragma unroll
  for (int p = 0; p < PASSES; ++p) s[p] = load_stream(srow + (int64_t)p * RPP * D);
#pragma unroll
  for (int p = 0; p < PASSES; ++p)
    vv[p] = Elem<TIn>::load1(v + pair * D + r0 + p * RPP + sub);
  float alpha, bt;
  if (a_log != nullptr) {  // uniform over the launch
    alpha = __expf(gate_log_decay(ga[pair], a_log[h], dt_bias[h]));
    bt = gate_beta(gb[pair]);
  } else {
    alpha = __expf(g[pair]);
    bt = beta[pair];
  }

  float qk = qq[0] * kk[0] + qq[1] * kk[1] + qq[2] * kk[2] + qq[3] * kk[3];
  qk = group_sum<LPR>(qk);

#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    float sk = s[p][0] * kk[0] + s[p][1] * kk[1] + s[p][2] * kk[2] + s[p][3] * kk[3];
    float sq = s[p][0] * qq[0] + s[p][1] * qq[1] + s[p][2] * qq[2] + s[p][3] * qq[3];
    sk = group_sum<LPR>(sk);
    sq = group_sum<LPR>(sq);
    const float delta = bt * (vv[p] - alpha * sk);
    f32x4 ns;
#pragma unroll
    for (int e = 0; e < 4; ++e) ns[e] = alpha * s[p][e] + delta * kk[e];
    store_stream(srow + (int64_t)p * RPP * D, ns);
    if ((lane % LPR) == 0)
      Elem<TIn>::store1(o + pair * D + r0 + p * RPP + sub, alpha * sq + delta * qk);
  }
}

template <int D, int PASSES, typename TIn>
static hipError_t launch_decode_p(const DecodeArgs &a, int64_t total_rows) {
  constexpr int ROWS_PER_WAVE = (kWave / (D / 4)) * PASSES;
  const int64_t rows_per_block = ROWS_PER_WAVE * 4;
  const int64_t blocks = (total_rows + rows_per_block - 1) / rows_per_block;
  hipLaunchKernelGGL((decode_kernel<D, PASSES, TIn>), dim3((unsigned)blocks), dim3(256),
                     0, a.stream, (const TIn *)a.q, (const TIn *)a.k,
                     (const TIn *)a.v, a.g, a.beta, a.gate.a, a.gate.b, a.gate.a_log,
                     a.gate.dt_bias, a.state, (TIn *)a.o, total_rows, a.hqk, a.hv,
                     a.hv / a.hqk);
  return hipGetLastError();
}

template <int D, typename TIn>
static hipError_t launch_decode_t(const DecodeArgs &a) {
  const int64_t total_rows = (int64_t)a.batch * a.hv * D;
  if (total_rows == 0) return hipSuccess;
  const int64_t blocks4 = (total_rows + (kWave / (D / 4)) * 16 - 1) / ((kWave / (D / 4)) * 16);
  if (blocks4 < 2 * (int64_t)device_compute_units()) return launch_decode_p<D, 2, TIn>(a, total_rows);
  return launch_decode_p<D, 4, TIn>(a, total_rows);
}

hipError_t launch_decode(const DecodeArgs &a) {
  const bool bf = a.dtype == GDN_BF16;
  switch (a.d) {
    case 32: return bf ? launch_decode_t<32, __bf16>(a) : launch_decode_t<32, float>(a);
    case 64: return bf ? launch_decode_t<64, __bf16>(a) : launch_decode_t<64, float>(a);
    case 128: return bf ? launch_decode_t<128, __bf16>(a) : launch_decode_t<128, float>(a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace gdn
