// gdn_launch.h -- internal interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/gdn.h"

namespace gdn {

// Raw gate inputs of the *_gated entry points; all NULL when g and beta are
// passed directly.
struct GateArgs {
  const float *a = nullptr, *b = nullptr, *a_log = nullptr, *dt_bias = nullptr;
};

struct DecodeArgs {
  const void *q, *k, *v;
  const float *g, *beta;
  GateArgs gate;
  float *state;
  void *o;
  int batch, hqk, hv, d;
  gdn_dtype dtype;
  hipStream_t stream;
};

struct PrefillArgs {
  const void *q, *k, *v;
  const float *g, *beta;
  GateArgs gate;
  const int32_t *cu_seqlens;
  const float *initial_state;
  void *o;
  float *final_state;
  int n_seqs;
  int64_t n_tokens;
  int hqk, hv, d, chunk;
  bool neumann;  // diagonal blocks of the WY factor by the Neumann product
  bool wave_carry;  // single-wave carry (batches of short sequences)
  int seg_chunks;   // chunks per segment of the whole-chain carry
  bool tile_carry;  // bf16: the per-tile carry instead of the whole-chain carry
  gdn_dtype dtype;
  void *workspace;
  hipStream_t stream;
};

// Device workspace carved out of the caller's buffer (all offsets 256-aligned).
struct PrefillWorkspace {
  size_t decay;       // f32  [chunks, HV, 2, C]: exp(gamma_i), exp(gamma_last - gamma_i)
  size_t tfrag;       // bf16 [chunks, HV, FRAG]: (I + A)^-1 in operand order
  size_t pfrag;       // bf16 [chunks, HV, FRAG]: decay-masked Q K^T, same order
  size_t qfrag;       // bf16 [chunks, HQK, C * D]: Q in operand order (per-tile carry)
  // Segment maps of the whole-chain carry (n_maps slots; none when no
  // sequence can span more than one segment):
  size_t bslot;       // f32  [n_maps, HV, D, D]: B of a segment, then the composed state
  size_t mthi, mtlo;  // bf16 [n_maps, HV, D, D]: M^T of a segment, hi and lo parts
  int64_t n_maps;
  // Whole-chain carry with more than one sequence: the segment slots, longest
  // first (T / span + N int32).
  size_t order;
  size_t total;
};

// Elements of one C x C matrix stored as 16x16x32 A-operand fragments.
inline int64_t frag_elems(int chunk) {
  const int nib = chunk / 16;
  const int ks = (chunk + 31) / 32;
  return (int64_t)nib * ks * 64 * 8;
}
inline int64_t chunk_bound(int n_seqs, int64_t n_tokens, int chunk) {
  return (n_tokens + chunk - 1) / chunk + n_seqs;
}
// Chunks per segment of the whole-chain carry: `requested` if positive, else
// for batches of fewer than kChainUnits chains as many segments per
// average-length sequence as keep all (segment, value head) work-groups in
// one round of kChainUnits, and for more chains the length at which the whole
// batch as one chain would give kChainUnits work-groups (so that only chains
// far longer than the average are cut).
constexpr int kChainUnits = 256;
// The whole-chain carry fills the chip when the batch has at least this many
// (sequence, value head) chains, one work-group each, or when its automatic
// segments are at least kChainMinSegment chunks long (long chains, cut into
// enough segments, whose map and composition launches are then amortised),
// and at d = 128 from 128 chains on with medium lengths (uses_tile_carry).
// Otherwise the per-tile carry spreads every chain over D/16 work-groups.
// Measured (d = 128, 16/32 heads, C = 64): 66K tokens in 16 sequences (512
// chains) whole-chain 1.07-1.10 ms, per-tile 1.43 ms; 2 x 32768 tokens (64
// chains, segments of 128 chunks) 1.39 against 1.47 ms, with 64-chunk
// segments 1.47 (even); 4096 tokens (32 chains, segments of 8 chunks) 139
// against 82 us.
constexpr int64_t kChainCarryMinChains = 256;
constexpr int kChainMinSegment = 64;
constexpr int kMinSegmentChunks = 4;
int chain_segment_chunks(int n_seqs, int64_t n_tokens, int hv, int chunk, int requested);
// The whole-chain carry runs unless the average sequence fits in one chunk
// (then the single-wave carry does).
inline bool uses_wave_carry(int n_seqs, int64_t n_tokens, int chunk) {
  return n_tokens <= (int64_t)n_seqs * chunk;
}
// The per-tile carry unless the whole-chain carry fills the chip (see
// kChainCarryMinChains): every chain is then spread over D/16 work-groups
// without segments.
bool uses_tile_carry(int n_seqs, int64_t n_tokens, int hv, int d, int chunk);
PrefillWorkspace prefill_workspace_layout(int n_seqs, int64_t n_tokens, int hqk,
                                          int hv, int d, int chunk, int seg_chunks, bool tile);

hipError_t launch_decode(const DecodeArgs &a);
// Chunked prefill (chunk 16, 32 or 64; bf16 inputs through the chunk-local
// kernel and a carry, float32 inputs through launch_prefill_f32) and the
// token-serial prefill (chunk 1, no workspace).
hipError_t launch_prefill(const PrefillArgs &a, const PrefillWorkspace &ws);
// The whole-chain carry and the per-tile carry (bf16 inputs), after the
// chunk-local kernel.
hipError_t launch_chain_d(const PrefillArgs &a, const PrefillWorkspace &ws);
hipError_t launch_tile_carry(const PrefillArgs &a, const PrefillWorkspace &ws);
hipError_t launch_prefill_serial(const PrefillArgs &a);
// float32 inputs, chunk 16, 32 or 64: float32 matrix products and tables
// throughout (no workspace).
hipError_t launch_prefill_f32(const PrefillArgs &a);

// Compute units of the current device, read once per process.
int device_compute_units();

}  // namespace gdn
