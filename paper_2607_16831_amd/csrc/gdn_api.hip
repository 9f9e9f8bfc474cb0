// gdn_api.hip -- the C ABI of libgdn: validation, workspace sizing, dispatch.
//
// Every check runs on the host before the first HIP call, so a rejected call
// enqueues nothing and the checks can be exercised without a GPU.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/gdn.h"
#include "gdn_launch.h"

namespace gdn {

int device_compute_units() {
  static const int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    return n;
  }();
  return cus;
}

}  // namespace gdn

namespace {

bool supported_head(int32_t dk, int32_t dv) {
  return dk == dv && (dk == 32 || dk == 64 || dk == 128);
}
// 1: token-serial path; 16, 32, 64: chunked path. 0 (automatic) is resolved
// by auto_chunk() before this check.
bool supported_chunk(int32_t c) { return c == 1 || c == 16 || c == 32 || c == 64; }
bool supported_dtype(gdn_dtype t) { return t == GDN_BF16 || t == GDN_F32; }

gdn_status check_heads(int32_t hqk, int32_t hv) {
  if (hqk <= 0 || hv <= 0 || hv % hqk != 0) return GDN_ERR_INVALID_ARG;
  return GDN_OK;
}

// Shape dispatch of the prefill (the paper's Section 5.1: the chunk size is
// chosen from the number of sequences, the total tokens and the average
// sequence length; Sections 5.3 and 5.5: a narrow short-shape fallback).
// The rule is a table per head size on the average length T/N (rounded up)
// and the number of sequences N: the token-serial path up to `serial`
// tokens, or up to `serial_big` when N >= n_big; then chunks of 16, 32 and
// 64 up to the next bounds. Bounds measured on MI355X (16 q/k and 32 v
// heads, bf16, T = 1024 and 8192, lengths 1 to 8192, each chunked run with
// the carry the dispatch below pairs with it): at every measured shape the
// chosen path is within 15% of the fastest of the four.
struct ChunkRule {
  int d, serial, serial_big, n_big, c16, c32;
};
constexpr ChunkRule kChunkRules[] = {
    {32, 24, 24, 0, 24, 32},      // chunk 16 never wins at d = 32
    {64, 4, 4, 0, 16, 32},
    {128, 1, 4, 1536, 16, 320},
};

// Past those bounds, 64-token chunks unless 32 would take the whole-chain
// carry (many chains, or long ones) -- at d = 32 only if 64 would take it
// too. Measured (16/32 heads): where both take it, 32 is 6-20% faster at
// every d (16 x 4096 tokens at d = 128: 858 against 941 us; 2 x 32768: 1293
// against 1370 us); where 64 would take the per-tile carry instead, 32 is
// 7-41% faster at d = 64 and 128 (4 x 4096 tokens: 263 against 377 us;
// 1 x 16384 at d = 64: 148 against 251 us) but slower at d = 32 (4 x 4096:
// 127 against 95 us, two tiles per chain there). Where 32 takes the per-tile
// carry too (1 x 8192 tokens: 144 against 224 us; 3 x 4096: 252 against
// 322 us), 64 stays.
int32_t auto_chunk(int32_t n_seqs, int64_t n_tokens, int32_t hv, int32_t d) {
  if (n_seqs <= 0) return 64;
  ChunkRule r = kChunkRules[2];
  for (const ChunkRule &c : kChunkRules)
    if (c.d == d) r = c;
  const int64_t avg = (n_tokens + n_seqs - 1) / n_seqs;
  if (avg <= r.serial || (avg <= r.serial_big && n_seqs >= r.n_big)) return 1;
  if (avg <= r.c16) return 16;
  if (avg <= r.c32) return 32;
  auto whole_chain = [&](int c) {
    return !gdn::uses_wave_carry(n_seqs, n_tokens, c) &&
           !gdn::uses_tile_carry(n_seqs, n_tokens, hv, d, c);
  };
  return (whole_chain(32) && (d >= 64 || whole_chain(64))) ? 32 : 64;
}

// The `chunk` argument: a size (0, 1, 16, 32, 64), optionally OR-ed with
// GDN_CHUNK_NEUMANN and GDN_CHUNK_SEGMENT(L). `ok` is false when other bits
// are set.
struct ChunkArg {
  int32_t size;
  bool neumann;
  bool tiles;   // GDN_CHUNK_TILE_CARRY: the per-tile carry
  int32_t seg;  // requested chunks per segment (whole-chain carry), 0 = automatic
  bool ok;
};
ChunkArg parse_chunk(int32_t chunk) {
  ChunkArg c;
  const uint32_t u = (uint32_t)chunk;
  const uint32_t seg_mask = 0xfffu << GDN_CHUNK_SEGMENT_SHIFT;
  c.size = (int32_t)(u & 0xffu);
  c.neumann = (u & GDN_CHUNK_NEUMANN) != 0;
  c.tiles = (u & GDN_CHUNK_TILE_CARRY) != 0;
  c.seg = (int32_t)((u & seg_mask) >> GDN_CHUNK_SEGMENT_SHIFT);
  c.ok = (u & ~(0xffu | (uint32_t)GDN_CHUNK_NEUMANN | (uint32_t)GDN_CHUNK_TILE_CARRY | seg_mask)) == 0 &&
         !(c.tiles && c.seg > 0);
  return c;
}

// The carry of a chunked call (chunk resolved): the per-tile carry when
// forced, or when no segment length is forced and the whole-chain carry
// would not fill the chip.
bool tile_carry(const ChunkArg &c, int32_t n_seqs, int64_t n_tokens, int32_t hv, int32_t d,
                int32_t chunk) {
  return c.tiles || (c.seg == 0 && gdn::uses_tile_carry(n_seqs, n_tokens, hv, d, chunk));
}

// Workspace bytes for a resolved chunk size. The token-serial path uses none;
// it reports the 256-byte minimum so that 0 keeps meaning "invalid sizes".
size_t required_workspace(int32_t n_seqs, int64_t n_tokens, int32_t hqk, int32_t hv, int32_t d,
                          int32_t chunk, const ChunkArg &c) {
  if (chunk == 1) return 256;
  const int L = gdn::chain_segment_chunks(n_seqs, n_tokens, hv, chunk, c.seg);
  return gdn::prefill_workspace_layout(n_seqs, n_tokens, hqk, hv, d, chunk, L,
                                       tile_carry(c, n_seqs, n_tokens, hv, d, chunk))
      .total;
}

// Scratch of gdn_prefill_scratch: the prefill workspace of every call on a
// device, held by the code object for as long as the process runs. In host
// code `scratch` names a host-side stand-in, not device memory: every use
// goes through the device address hipGetSymbolAddress returns, fetched once
// per device with that device current.
static __device__ __align__(256) unsigned char scratch[GDN_PREFILL_SCRATCH_MAX_BYTES];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device (nullptr on failure).
void *scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return nullptr;
    addr[dev] = p;
  }
  return addr[dev];
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
                        void *workspace, size_t workspace_bytes, hipStream_t stream,
                        bool use_scratch = false) {
  if (n_seqs < 0 || n_tokens < 0 || n_tokens > INT32_MAX) return GDN_ERR_INVALID_ARG;
  if (check_heads(hqk, hv) != GDN_OK) return GDN_ERR_INVALID_ARG;
  if (dk <= 0 || dv <= 0) return GDN_ERR_INVALID_ARG;
  // GDN_CHUNK_NEUMANN selects the Neumann-product diagonal inverse of the
  // chunked path; it is meaningless for the token-serial path. A segment
  // length applies to the chunked path and is ignored when the automatic
  // choice is the token-serial path.
  const ChunkArg ca = parse_chunk(chunk);
  if (!ca.ok) return GDN_ERR_UNSUPPORTED;
  const bool neumann = ca.neumann;
  chunk = ca.size;
  if (chunk == 0 && !neumann) chunk = auto_chunk(n_seqs, n_tokens, hv, dk);
  if (!supported_head(dk, dv) || !supported_chunk(chunk) || !supported_dtype(dtype) ||
      (neumann && chunk < 16) || ((ca.seg > 0 || ca.tiles) && ca.size == 1))
    return GDN_ERR_UNSUPPORTED;
  if (n_seqs == 0) return n_tokens == 0 ? GDN_OK : GDN_ERR_INVALID_ARG;
  if (!cu_seqlens || !final_state) return GDN_ERR_INVALID_ARG;
  if (n_tokens > 0 && (!q || !k || !v || !o || !gate_present(g, beta, gate)))
    return GDN_ERR_INVALID_ARG;
  const int seg_chunks = chunk == 1 ? 0 : gdn::chain_segment_chunks(n_seqs, n_tokens, hv, chunk, ca.seg);
  if (use_scratch) {
    // Size first (no HIP call for a refused size), then the device's array.
    if (required_workspace(n_seqs, n_tokens, hqk, hv, dk, chunk, ca) >
        (size_t)GDN_PREFILL_SCRATCH_MAX_BYTES)
      return GDN_ERR_WORKSPACE;
    workspace = scratch_address();
    if (workspace == nullptr) return GDN_ERR_HIP;
    workspace_bytes = (size_t)GDN_PREFILL_SCRATCH_MAX_BYTES;
  }
  if (!workspace ||
      workspace_bytes < required_workspace(n_seqs, n_tokens, hqk, hv, dk, chunk, ca) ||
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
  a.neumann = neumann;
  // The single-wave carry when the average sequence fits in one chunk: a
  // work-group carry's fixed cost then outweighs its per-chunk speed.
  a.wave_carry = gdn::uses_wave_carry(n_seqs, n_tokens, chunk);
  a.seg_chunks = seg_chunks;
  a.tile_carry = tile_carry(ca, n_seqs, n_tokens, hv, dk, chunk);
  a.dtype = dtype;
  a.workspace = workspace;
  a.stream = stream;
  const hipError_t e =
      chunk == 1 ? gdn::launch_prefill_serial(a)
                 : gdn::launch_prefill(a, gdn::prefill_workspace_layout(n_seqs, n_tokens, hqk,
                                                                        hv, dk, chunk, seg_chunks,
                                                                        a.tile_carry));
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
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

int gdn_version(void) { return 1 * 10000 + 3 * 100 + 0; }

size_t gdn_prefill_workspace_size(int32_t n_seqs, int64_t n_tokens,
                                  int32_t hqk, int32_t hv, int32_t dk,
                                  int32_t dv, int32_t chunk) {
  if (n_seqs < 0 || n_tokens < 0 || n_tokens > INT32_MAX) return 0;
  if (check_heads(hqk, hv) != GDN_OK) return 0;
  if (!supported_head(dk, dv)) return 0;
  const ChunkArg ca = parse_chunk(chunk);
  if (!ca.ok || (ca.neumann && ca.size < 16) || ((ca.seg > 0 || ca.tiles) && ca.size == 1))
    return 0;
  if (ca.size == 0 && !ca.neumann) {  // enough for whichever size the dispatch picks
    size_t m = 0;
    for (int32_t c : {1, 16, 32, 64}) {
      const size_t b = required_workspace(n_seqs, n_tokens, hqk, hv, dk, c, ca);
      m = b > m ? b : m;
    }
    return m;
  }
  if (!supported_chunk(ca.size)) return 0;
  return required_workspace(n_seqs, n_tokens, hqk, hv, dk, ca.size, ca);
}

int32_t gdn_prefill_auto_chunk(int32_t n_seqs, int64_t n_tokens, int32_t hqk, int32_t hv,
                               int32_t dk, int32_t dv) {
  if (n_seqs < 0 || n_tokens < 0 || n_tokens > INT32_MAX) return 0;
  if (check_heads(hqk, hv) != GDN_OK || !supported_head(dk, dv)) return 0;
  return auto_chunk(n_seqs, n_tokens, hv, dk);
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

gdn_status gdn_prefill_scratch(const void *q, const void *k, const void *v,
                               const float *g, const float *beta,
                               const int32_t *cu_seqlens, const float *initial_state,
                               void *o, float *final_state, int32_t n_seqs,
                               int64_t n_tokens, int32_t hqk, int32_t hv, int32_t dk,
                               int32_t dv, int32_t chunk, gdn_dtype dtype,
                               hipStream_t stream) {
  return prefill_impl(q, k, v, g, beta, gdn::GateArgs(), cu_seqlens, initial_state, o,
                      final_state, n_seqs, n_tokens, hqk, hv, dk, dv, chunk, dtype, nullptr, 0,
                      stream, true);
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
