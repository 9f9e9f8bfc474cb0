// gdn_api.hip -- the C ABI of libgdn: validation, workspace sizing, dispatch.
//
// Every check runs on the host before the first HIP call, so a rejected call
// enqueues nothing and the checks can be exercised without a GPU.
#include <hip/hip_runtime.h>

#include "../../include/gdn.h"
#include "gdn_launch.h"

namespace {

bool supported_head(int32_t dk, int32_t dv) {
  return dk == dv && (dk == 32 || dk == 64 || dk == 128);
}
bool supported_chunk(int32_t c) { return c == 16 || c == 32 || c == 64; }
bool supported_dtype(gdn_dtype t) { return t == GDN_BF16 || t == GDN_F32; }

gdn_status check_heads(int32_t hqk, int32_t hv) {
  if (hqk <= 0 || hv <= 0 || hv % hqk != 0) return GDN_ERR_INVALID_ARG;
  return GDN_OK;
}

// The gate inputs: either g and beta, or all four raw inputs of the gated
// entry points.
bool gate_present(const float *g, const float *beta, const gdn::GateArgs &gate) {
  if (gate.a_log != nullptr || gate.a != nullptr || gate.b != nullptr || gate.dt_bias != nullptr)
    return gate.a && gate.b && gate.a_log && gate.dt_bias;
  return g && beta;
}

gdn_status prefill_impl(const void *q, const void *k, const void *v, const float *g,
                        const float *beta, const gdn::GateArgs &gate,
                        const int32_t *cu_seqlens, const float *initial_state, void *o,
                        float *final_state, int32_t n_seqs, int64_t n_tokens, int32_t hqk,
                        int32_t hv, int32_t dk, int32_t dv, int32_t chunk, gdn_dtype dtype,
                        void *workspace, size_t workspace_bytes, hipStream_t stream) {
  if (n_seqs < 0 || n_tokens < 0 || n_tokens > INT32_MAX) return GDN_ERR_INVALID_ARG;
  if (check_heads(hqk, hv) != GDN_OK) return GDN_ERR_INVALID_ARG;
  if (dk <= 0 || dv <= 0) return GDN_ERR_INVALID_ARG;
  if (!supported_head(dk, dv) || !supported_chunk(chunk) || !supported_dtype(dtype))
    return GDN_ERR_UNSUPPORTED;
  if (n_seqs == 0) return n_tokens == 0 ? GDN_OK : GDN_ERR_INVALID_ARG;
  if (!cu_seqlens || !final_state) return GDN_ERR_INVALID_ARG;
  if (n_tokens > 0 && (!q || !k || !v || !o || !gate_present(g, beta, gate)))
    return GDN_ERR_INVALID_ARG;
  const gdn::PrefillWorkspace ws =
      gdn::prefill_workspace_layout(n_seqs, n_tokens, hqk, hv, dk, chunk);
  if (!workspace || workspace_bytes < ws.total ||
      (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
    return GDN_ERR_WORKSPACE;

  gdn::PrefillArgs a;
  a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta;
  a.gate = gate;
  a.cu_seqlens = cu_seqlens;
  a.initial_state = initial_state;
  a.o = o;
  a.final_state = final_state;
  a.n_seqs = n_seqs;
  a.n_tokens = n_tokens;
  a.hqk = hqk; a.hv = hv; a.d = dk; a.chunk = chunk;
  a.dtype = dtype;
  a.workspace = workspace;
  a.stream = stream;
  return gdn::launch_prefill(a, ws) == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status decode_impl(const void *q, const void *k, const void *v, const float *g,
                       const float *beta, const gdn::GateArgs &gate, float *state, void *o,
                       int32_t batch, int32_t hqk, int32_t hv, int32_t dk, int32_t dv,
                       gdn_dtype dtype, hipStream_t stream) {
  if (batch < 0) return GDN_ERR_INVALID_ARG;
  if (check_heads(hqk, hv) != GDN_OK) return GDN_ERR_INVALID_ARG;
  if (dk <= 0 || dv <= 0) return GDN_ERR_INVALID_ARG;
  if (!supported_head(dk, dv) || !supported_dtype(dtype)) return GDN_ERR_UNSUPPORTED;
  if (batch == 0) return GDN_OK;
  if (!q || !k || !v || !state || !o || !gate_present(g, beta, gate))
    return GDN_ERR_INVALID_ARG;

  gdn::DecodeArgs a;
  a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta;
  a.gate = gate;
  a.state = state;
  a.o = o;
  a.batch = batch;
  a.hqk = hqk; a.hv = hv; a.d = dk;
  a.dtype = dtype;
  a.stream = stream;
  return gdn::launch_decode(a) == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

}  // namespace

extern "C" {

const char *gdn_status_string(gdn_status status) {
  switch (status) {
    case GDN_OK: return "ok";
    case GDN_ERR_INVALID_ARG: return "invalid argument";
    case GDN_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case GDN_ERR_WORKSPACE: return "workspace missing or too small";
    case GDN_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

int gdn_version(void) { return 1 * 10000 + 1 * 100 + 0; }

size_t gdn_prefill_workspace_size(int32_t n_seqs, int64_t n_tokens,
                                  int32_t hqk, int32_t hv, int32_t dk,
                                  int32_t dv, int32_t chunk) {
  if (n_seqs < 0 || n_tokens < 0 || n_tokens > INT32_MAX) return 0;
  if (check_heads(hqk, hv) != GDN_OK) return 0;
  if (!supported_head(dk, dv) || !supported_chunk(chunk)) return 0;
  return gdn::prefill_workspace_layout(n_seqs, n_tokens, hqk, hv, dk, chunk).total;
}

gdn_status gdn_prefill(const void *q, const void *k, const void *v,
                       const float *g, const float *beta,
                       const int32_t *cu_seqlens, const float *initial_state,
                       void *o, float *final_state, int32_t n_seqs,
                       int64_t n_tokens, int32_t hqk, int32_t hv, int32_t dk,
                       int32_t dv, int32_t chunk, gdn_dtype dtype,
                       void *workspace, size_t workspace_bytes,
                       hipStream_t stream) {
  return prefill_impl(q, k, v, g, beta, gdn::GateArgs(), cu_seqlens, initial_state, o,
                      final_state, n_seqs, n_tokens, hqk, hv, dk, dv, chunk, dtype, workspace,
                      workspace_bytes, stream);
}

gdn_status gdn_prefill_gated(const void *q, const void *k, const void *v,
                             const float *a, const float *b,
                             const float *A_log, const float *dt_bias,
                             const int32_t *cu_seqlens,
                             const float *initial_state, void *o,
                             float *final_state, int32_t n_seqs,
                             int64_t n_tokens, int32_t hqk, int32_t hv,
                             int32_t dk, int32_t dv, int32_t chunk,
                             gdn_dtype dtype, void *workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  gdn::GateArgs gate;
  gate.a = a;
  gate.b = b;
  gate.a_log = A_log;
  gate.dt_bias = dt_bias;
  return prefill_impl(q, k, v, nullptr, nullptr, gate, cu_seqlens, initial_state, o,
                      final_state, n_seqs, n_tokens, hqk, hv, dk, dv, chunk, dtype, workspace,
                      workspace_bytes, stream);
}

gdn_status gdn_decode(const void *q, const void *k, const void *v,
                      const float *g, const float *beta, float *state,
                      void *o, int32_t batch, int32_t hqk, int32_t hv,
                      int32_t dk, int32_t dv, gdn_dtype dtype,
                      hipStream_t stream) {
  return decode_impl(q, k, v, g, beta, gdn::GateArgs(), state, o, batch, hqk, hv, dk, dv,
                     dtype, stream);
}

gdn_status gdn_decode_gated(const void *q, const void *k, const void *v,
                            const float *a, const float *b,
                            const float *A_log, const float *dt_bias,
                            float *state, void *o, int32_t batch, int32_t hqk,
                            int32_t hv, int32_t dk, int32_t dv,
                            gdn_dtype dtype, hipStream_t stream) {
  gdn::GateArgs gate;
  gate.a = a;
  gate.b = b;
  gate.a_log = A_log;
  gate.dt_bias = dt_bias;
  return decode_impl(q, k, v, nullptr, nullptr, gate, state, o, batch, hqk, hv, dk, dv,
                     dtype, stream);
}

}  // extern "C"
