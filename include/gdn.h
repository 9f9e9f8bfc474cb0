/*
 * gdn.h -- C ABI of libgdn: the Gated DeltaNet gated delta-rule recurrence on
 * AMD MI355X (gfx950).
 *
 * The operation (paper, Section 3.2, display equations for old_v, delta, S';
 * Section 2.2 for the decode / prefill split). For one sequence and one value
 * head, with the recurrent state S stored as a d_v x d_k matrix:
 *
 *     S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t q_t                            (output from the updated state)
 *     alpha_t = exp(g_t)
 *
 * g is passed as the LOG of the paper's multiplicative gate (g <= 0 in every
 * intended use; positive g is accepted but can overflow inside the chunked
 * form). beta is passed already activated, in [0, 1]. There is no q scale:
 * callers fold 1/sqrt(d_k) into q.
 *
 * Grouped heads: HQK query/key heads and HV value heads with HV % HQK == 0;
 * value head h reads query/key head h / (HV / HQK).
 *
 * Memory layouts (row-major, densely packed, element type per `dtype` for
 * q/k/v/o, float32 for g, beta and states):
 *   q, k            [T_total, HQK, DK]
 *   v, o            [T_total, HV, DV]
 *   g, beta         [T_total, HV]
 *   cu_seqlens      [N + 1] int32: cu[0] = 0, non-decreasing, cu[N] = T_total
 *   states          [N, HV, DV, DK]   ("k-last": the d_k index is contiguous)
 *
 * Ownership and execution: every pointer is DEVICE memory owned by the caller.
 * The library never allocates, frees or retains memory; scratch space for
 * prefill comes from the caller through `workspace` (destination-passing
 * style, as in the paper's Sections 3.2 and 5.2). All work is enqueued on
 * `stream` and returns without synchronising; cu_seqlens is never read on the
 * host. The library holds no global state: calls are re-entrant, and calls on
 * different streams are independent as long as their buffers do not overlap.
 *
 * Errors: argument validation happens on the host before any HIP call, so an
 * invalid call enqueues nothing. Launch failures are reported as GDN_ERR_HIP.
 * Device-side contract violations (cu_seqlens not non-decreasing, cu[N] !=
 * T_total, overlapping in/out buffers other than the aliases allowed below)
 * are undefined behaviour. NaN and Inf propagate without checks.
 *
 * Supported shapes: DK == DV in {32, 64, 128}; chunk in {0 (automatic), 1
 * (token-serial), 16, 32, 64}.
 */
#ifndef GDN_H_
#define GDN_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gdn_status {
  GDN_OK = 0,
  GDN_ERR_INVALID_ARG = 1, /* null pointer, negative size, HV % HQK != 0 */
  GDN_ERR_UNSUPPORTED = 2, /* head size / chunk size / dtype not built   */
  GDN_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
  GDN_ERR_HIP = 4          /* a HIP launch failed                        */
} gdn_status;

typedef enum gdn_dtype {
  GDN_BF16 = 0, /* q, k, v, o are bfloat16; o is rounded to nearest even */
  GDN_F32 = 1   /* q, k, v, o are float32; computed in float32 throughout  */
} gdn_dtype;

/*
 * Flag OR-ed into the `chunk` argument of gdn_prefill, gdn_prefill_gated and
 * gdn_prefill_workspace_size together with a chunk size of 16, 32 or 64: the
 * 16 x 16 diagonal blocks of the WY factor (I + A)^-1 are formed by the
 * Neumann series in its product form, (I - N)(I + N^2)(I + N^4)(I + N^8) for
 * a strictly lower block N, on the matrix cores (the chunk-solve variant of
 * the paper's Section 5.1), instead of by forward substitution. Same result
 * up to rounding; the workspace is the same. Any other combination returns
 * GDN_ERR_UNSUPPORTED (0 from gdn_prefill_workspace_size).
 */
#define GDN_CHUNK_NEUMANN 0x100

/*
 * Segment length of the whole-chain carry, OR-ed into the `chunk` argument of
 * gdn_prefill, gdn_prefill_gated and gdn_prefill_workspace_size together with
 * a chunk size of 0, 16, 32 or 64: GDN_CHUNK_SEGMENT(L), 1 <= L <= 4095,
 * cuts every sequence into segments of L chunks whose carries run in
 * parallel and are joined through their affine state maps (see gdn_prefill).
 * Without it the library picks L from the sizes. L changes only rounding and
 * speed; the workspace size depends on it, so pass the same value to
 * gdn_prefill_workspace_size. With chunk = 1 it is GDN_ERR_UNSUPPORTED (0 from
 * gdn_prefill_workspace_size); with chunk = 0 it is ignored when the
 * automatic choice is the token-serial path.
 */
/*
 * The carry from chunk to chunk comes in two forms (see gdn_prefill). Without
 * a flag the library picks one from the sizes. GDN_CHUNK_TILE_CARRY, OR-ed
 * into `chunk` with a size of 0, 16, 32 or 64, forces the per-tile carry;
 * GDN_CHUNK_SEGMENT(L) forces the whole-chain carry (both together is
 * GDN_ERR_UNSUPPORTED). Same results up to rounding; the workspace size
 * depends on the choice, so pass the same `chunk` to
 * gdn_prefill_workspace_size.
 */
#define GDN_CHUNK_TILE_CARRY 0x200
#define GDN_CHUNK_SEGMENT_SHIFT 16
#define GDN_CHUNK_SEGMENT(L) ((int32_t)(L) << GDN_CHUNK_SEGMENT_SHIFT)

/* Human-readable name of a status code (static string, never NULL). */
const char *gdn_status_string(gdn_status status);

/* Library version as major * 10000 + minor * 100 + patch. */
int gdn_version(void);

/*
 * Bytes of device workspace gdn_prefill needs for these sizes (0 on invalid
 * sizes). The size grows with N and T_total, so a caller may size it once for
 * the largest batch it will submit. chunk = 1 needs no workspace and reports
 * the 256-byte minimum; chunk = 0 reports the largest size over every choice
 * the automatic dispatch can make, so it also covers every smaller batch.
 */
size_t gdn_prefill_workspace_size(int32_t n_seqs, int64_t n_tokens,
                                  int32_t hqk, int32_t hv, int32_t dk,
                                  int32_t dv, int32_t chunk);

/*
 * The chunk size gdn_prefill uses when called with chunk = 0 for these
 * sizes: 1 (token-serial), 16, 32 or 64; 0 on invalid sizes. Shape dispatch
 * after the paper's Section 5.1 (dispatch axes) and Sections 5.3 and 5.5 (a
 * narrow short-shape fallback): the choice depends on the head size,
 * the average sequence length T_total / N (rounded up) and N, with bounds
 * measured on MI355X. Very short sequences take the token-serial path, where
 * the chunked form's per-chunk work does not pay; longer ones take 16, 32 or
 * 64 as the average length grows, except that batches with many or long
 * chains, which take the whole-chain carry at 32 (at d = 32: at 32 and 64),
 * take 32.
 * Pure host function; no HIP call.
 */
int32_t gdn_prefill_auto_chunk(int32_t n_seqs, int64_t n_tokens, int32_t hqk,
                               int32_t hv, int32_t dk, int32_t dv);

/*
 * Chunked prefill over N packed variable-length sequences (paper, Sections
 * 5.1, 5.2 and 5.5: the chunk / WY reformulation of the recurrence above).
 *
 * Each sequence is cut into chunks of `chunk` tokens starting at cu[n] (the
 * last chunk of a sequence may be shorter). `chunk` changes only rounding,
 * not the result. Per chunk, the intra-chunk recurrence is summarised by a
 * unit lower-triangular WY factor; the state is carried chunk to chunk in
 * float32.
 *
 * The carry from chunk to chunk takes one of two forms, chosen from the
 * sizes unless GDN_CHUNK_TILE_CARRY or GDN_CHUNK_SEGMENT(L) forces one: with
 * fewer than 256 (sequence, value head) chains, the per-tile carry spreads
 * every chain over DV/16 work-groups of 16 value rows; with more, the
 * whole-chain carry gives each chain (or each segment of a long chain,
 * joined through the segments' affine state maps) one work-group. Batches
 * whose average sequence fits in one chunk use a third, single-wavefront
 * carry. All three give the same result up to rounding.
 *
 * Precision of the chunked path: bf16 inputs enter the matrix products as
 * bf16 operands with float32 accumulation, and the state is carried in
 * float32 (rel-L2 against an fp64 evaluation of the recurrence about 2e-3
 * to 4e-3 on o and the final state at the benchmark sizes). float32 inputs
 * are computed in float32 throughout, products and tables included (rel-L2
 * about 1e-7 to 1e-6); for them GDN_CHUNK_NEUMANN changes nothing, the
 * carry forms above do not apply, and the workspace goes unused.
 *
 * chunk = 1 runs the token-serial form instead: the recurrence token by
 * token in float32 on the vector ALU, the state held in registers for the
 * whole sequence (the narrow short-shape fallback, paper Sections 5.3 and 5.5). chunk = 0 picks
 * one of the sizes as gdn_prefill_auto_chunk() reports.
 *
 *   q, k, v, g, beta, cu_seqlens : inputs, layouts above.
 *   initial_state : [N, HV, DV, DK] float32, or NULL for zero states.
 *   o             : [T_total, HV, DV] output (dtype as q).
 *   final_state   : [N, HV, DV, DK] float32 output; may alias initial_state
 *                   exactly (same pointer), in which case it is updated in
 *                   place. A zero-length sequence yields its initial state.
 *   workspace     : device scratch of at least gdn_prefill_workspace_size()
 *                   bytes, 256-byte aligned; contents on entry are ignored.
 *   stream        : HIP stream the work is enqueued on (NULL = default).
 */
gdn_status gdn_prefill(const void *q, const void *k, const void *v,
                       const float *g, const float *beta,
                       const int32_t *cu_seqlens, const float *initial_state,
                       void *o, float *final_state, int32_t n_seqs,
                       int64_t n_tokens, int32_t hqk, int32_t hv, int32_t dk,
                       int32_t dv, int32_t chunk, gdn_dtype dtype,
                       void *workspace, size_t workspace_bytes,
                       hipStream_t stream);

/*
 * gdn_prefill for callers that cannot allocate device memory or pass a
 * workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the same operation, arguments and results as
 * gdn_prefill, with the workspace taken from a fixed array of
 * GDN_PREFILL_SCRATCH_MAX_BYTES bytes that the library's code object holds
 * on each device it runs on until the process ends. The call allocates
 * nothing. It uses the array of the current device (hipGetDevice), whose
 * address it looks up on its first call there.
 *
 * Sizes whose workspace (gdn_prefill_workspace_size with the same `chunk`)
 * exceeds GDN_PREFILL_SCRATCH_MAX_BYTES are refused with GDN_ERR_WORKSPACE
 * before any HIP call; the 128 MiB hold, for example, one sequence of up
 * to 10240 tokens with 16 query/key and 32 value heads of size 128 at
 * chunk 64 (4096 tokens: 50 MiB). Every call on one device shares that device's array: calls that
 * overlap in time on one device (different streams, or different host
 * threads without ordering) race and give undefined results; calls ordered
 * on one stream do not. GDN_ERR_HIP if the array's address cannot be
 * obtained.
 */
#define GDN_PREFILL_SCRATCH_MAX_BYTES (128u << 20)

gdn_status gdn_prefill_scratch(const void *q, const void *k, const void *v,
                               const float *g, const float *beta,
                               const int32_t *cu_seqlens, const float *initial_state,
                               void *o, float *final_state, int32_t n_seqs,
                               int64_t n_tokens, int32_t hqk, int32_t hv, int32_t dk,
                               int32_t dv, int32_t chunk, gdn_dtype dtype,
                               hipStream_t stream);

/*
 * One decode step for a batch of B sequences, one token each (paper, Section
 * 3.2: the one-pass form with the gate-scaled state; Section 5.4 for decode
 * as a bandwidth/launch-shape problem). The state is read once and written
 * once, in place.
 *
 *   q, k  : [B, HQK, DK]    v, o : [B, HV, DV]    g, beta : [B, HV]
 *   state : [B, HV, DV, DK] float32, advanced in place.
 */
gdn_status gdn_decode(const void *q, const void *k, const void *v,
                      const float *g, const float *beta, float *state,
                      void *o, int32_t batch, int32_t hqk, int32_t hv,
                      int32_t dk, int32_t dv, gdn_dtype dtype,
                      hipStream_t stream);

/*
 * Gate activation (paper, Section 3.2, the first two lines of the one-pass
 * form: the multiplicative gate exp(-exp(A_log) softplus(a + b_dt)) and
 * beta = sigmoid(b)). The *_gated entry points take the raw per-token inputs
 * instead of g and beta and form them inside the kernels, per token t and
 * value head h:
 *
 *     g[t, h]    = -exp(A_log[h]) * softplus(a[t, h] + dt_bias[h])
 *     beta[t, h] = 1 / (1 + exp(-b[t, h]))
 *
 * with softplus(x) = log(1 + exp(x)); g is the log of the paper's gate, as
 * everywhere in this header. Layouts (float32, row-major):
 *   a, b              [T_total, HV]   (decode: [B, HV])
 *   A_log, dt_bias    [HV]
 * Everything else -- the other arguments, ownership, execution, errors and
 * the workspace (gdn_prefill_workspace_size) -- is as for gdn_prefill and
 * gdn_decode. A NULL a, b, A_log or dt_bias is GDN_ERR_INVALID_ARG when there
 * is at least one token.
 */
gdn_status gdn_prefill_gated(const void *q, const void *k, const void *v,
                             const float *a, const float *b,
                             const float *A_log, const float *dt_bias,
                             const int32_t *cu_seqlens,
                             const float *initial_state, void *o,
                             float *final_state, int32_t n_seqs,
                             int64_t n_tokens, int32_t hqk, int32_t hv,
                             int32_t dk, int32_t dv, int32_t chunk,
                             gdn_dtype dtype, void *workspace,
                             size_t workspace_bytes, hipStream_t stream);

gdn_status gdn_decode_gated(const void *q, const void *k, const void *v,
                            const float *a, const float *b,
                            const float *A_log, const float *dt_bias,
                            float *state, void *o, int32_t batch, int32_t hqk,
                            int32_t hv, int32_t dk, int32_t dv,
                            gdn_dtype dtype, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* GDN_H_ */
