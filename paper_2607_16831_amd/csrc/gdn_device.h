// gdn_device.h -- device-side helpers shared by the libgdn kernels (gfx950).
//
// Element types, bf16 packing, the 16x16x32 bf16 matrix-core instruction and
// wave-level reductions. Nothing here depends on the recurrence itself.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

constexpr int kWave = 64;  // CDNA wavefront width

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- bf16 bits
__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  __bf16 b = (__bf16)x;  // v_cvt_pk_bf16_f32: round to nearest even
  return __builtin_bit_cast(uint16_t, b);
}
// Two floats rounded to nearest even into one packed bf16 pair (lo in the
// low half): a single v_cvt_pk_bf16_f32.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

// Eight consecutive elements of a row, returned as packed bf16 (16 bytes).
// bf16 input is copied bit-exactly; f32 input is rounded to nearest even.
template <typename T>
struct Elem;

template <>
struct Elem<__bf16> {
  static __device__ __forceinline__ uint4 load8(const __bf16 *p) {
    return *reinterpret_cast<const uint4 *>(p);
  }
  static __device__ __forceinline__ float load1(const __bf16 *p) {
    return bf16_bits_to_f32(*reinterpret_cast<const uint16_t *>(p));
  }
  static __device__ __forceinline__ void load4(const __bf16 *p, float out[4]) {
    uint2 r = *reinterpret_cast<const uint2 *>(p);
    out[0] = bf16_bits_to_f32(r.x & 0xffffu);
    out[1] = bf16_bits_to_f32(r.x >> 16);
    out[2] = bf16_bits_to_f32(r.y & 0xffffu);
    out[3] = bf16_bits_to_f32(r.y >> 16);
  }
  static __device__ __forceinline__ void store1(__bf16 *p, float x) {
    *reinterpret_cast<uint16_t *>(p) = f32_to_bf16_bits(x);
  }
};

// The bits of one input element, read ahead of its use and converted there.
template <typename T>
struct RawElem;
template <>
struct RawElem<__bf16> {
  static __device__ __forceinline__ uint32_t load(const __bf16 *p) {
    return *reinterpret_cast<const uint16_t *>(p);
  }
  static __device__ __forceinline__ float cvt(uint32_t b) { return bf16_bits_to_f32(b); }
};
template <>
struct RawElem<float> {
  static __device__ __forceinline__ uint32_t load(const float *p) {
    return *reinterpret_cast<const uint32_t *>(p);
  }
  static __device__ __forceinline__ float cvt(uint32_t b) { return __uint_as_float(b); }
};

template <>
struct Elem<float> {
  static __device__ __forceinline__ uint4 load8(const float *p) {
    float4 a = reinterpret_cast<const float4 *>(p)[0];
    float4 b = reinterpret_cast<const float4 *>(p)[1];
    return make_uint4(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w),
                      pack_bf16x2(b.x, b.y), pack_bf16x2(b.z, b.w));
  }
  static __device__ __forceinline__ float load1(const float *p) { return *p; }
  static __device__ __forceinline__ void load4(const float *p, float out[4]) {
    float4 r = *reinterpret_cast<const float4 *>(p);
    out[0] = r.x;
    out[1] = r.y;
    out[2] = r.z;
    out[3] = r.w;
  }
  static __device__ __forceinline__ void store1(float *p, float x) { *p = x; }
};

// ---------------------------------------------------------------- MFMA
// v_mfma_f32_16x16x32_bf16, one wavefront:
//   A (16 x 32): lane l supplies row (l % 16), contraction slots 8*(l/16)+[0,8)
//   B (32 x 16): lane l supplies column (l % 16), the same contraction slots
//   D (16 x 16): lane l receives column (l % 16), rows 4*(l/16)+[0,4)
// A and B name contraction slots identically, so any assignment of true
// contraction indices to slots is valid as long as both operands use it.
__device__ __forceinline__ f32x4 mfma_16x16x32(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(
      __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// v_mfma_f32_16x16x4_f32, one wavefront:
//   A (16 x 4): lane l supplies A[l % 16][l / 16]
//   B (4 x 16): lane l supplies B[l / 16][l % 16]
//   D: as above. Four of these cover a 16 x 16 x 16 product; in step kk,
//   contraction slot g stands for index 4 g + kk, so a B operand can be taken
//   straight from a lane's own accumulator element kk.
__device__ __forceinline__ f32x4 mfma_16x16x4_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------- buffers
// Raw buffer resources: a base address and byte extent held in scalar
// registers, addressed with a 32-bit per-lane byte offset. Reads past the
// extent return zero and writes past it are dropped by the hardware; partial
// chunks rely on this instead of branches.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer, gfx9 family

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0,
                                           (int)bytes, kRsrcWord3);
}
__device__ __forceinline__ uint4 buf_load_b128(rsrc_t r, uint32_t off) {
  const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(x[0], x[1], x[2], x[3]);
}
__device__ __forceinline__ float buf_load_f32(rsrc_t r, uint32_t off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ float4 buf_load_f32x4(rsrc_t r, uint32_t off) {
  const uint4 x = buf_load_b128(r, off);
  return make_float4(__uint_as_float(x.x), __uint_as_float(x.y),
                     __uint_as_float(x.z), __uint_as_float(x.w));
}

// Cache-policy operand of the buffer intrinsics: the non-temporal (streaming)
// bit of gfx940-family targets (the position of SLC on earlier gfx9).
constexpr int kCachePolicyNT = 2;
// SC1 set, SC0 clear: a device-scope store on gfx940-family targets, written
// through the XCD's L2 to the memory side that every XCD shares. For tables
// that the next kernel reads on other XCDs it saves the write-back of dirty
// L2 lines at the end of the kernel.
constexpr int kCachePolicyDevice = 16;

template <int POL>
__device__ __forceinline__ void buf_store_b128(rsrc_t r, uint32_t off, uint4 v) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 x = {v.x, v.y, v.z, v.w};
  __builtin_amdgcn_raw_buffer_store_b128(x, r, off, 0, POL);
}

// Element access through a buffer resource; offsets are in elements.
template <typename T>
struct BufElem;

template <>
struct BufElem<__bf16> {
  static __device__ __forceinline__ uint4 load8(rsrc_t r, uint32_t e) {
    return buf_load_b128(r, e * 2u);
  }
  static __device__ __forceinline__ float load1(rsrc_t r, uint32_t e) {
    return bf16_bits_to_f32(__builtin_amdgcn_raw_buffer_load_b16(r, e * 2u, 0, 0));
  }
  // Four consecutive elements as packed bf16.
  static __device__ __forceinline__ uint2 load4_bf16(rsrc_t r, uint32_t e) {
    const auto x = __builtin_amdgcn_raw_buffer_load_b64(r, e * 2u, 0, 0);
    return make_uint2(x[0], x[1]);
  }
  static __device__ __forceinline__ void store1(rsrc_t r, uint32_t e, float x) {
    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_bits(x), r, e * 2u, 0, 0);
  }
  // Streaming store (non-temporal): written out to memory as the kernel runs
  // instead of staying dirty in L2 until the kernel ends.
  static __device__ __forceinline__ void store1_stream(rsrc_t r, uint32_t e, float x) {
    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_bits(x), r, e * 2u, 0, kCachePolicyNT);
  }
};

template <>
struct BufElem<float> {
  static __device__ __forceinline__ uint4 load8(rsrc_t r, uint32_t e) {
    const float4 a = buf_load_f32x4(r, e * 4u), b = buf_load_f32x4(r, e * 4u + 16u);
    return make_uint4(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w),
                      pack_bf16x2(b.x, b.y), pack_bf16x2(b.z, b.w));
  }
  static __device__ __forceinline__ float load1(rsrc_t r, uint32_t e) {
    return buf_load_f32(r, e * 4u);
  }
  static __device__ __forceinline__ uint2 load4_bf16(rsrc_t r, uint32_t e) {
    const float4 a = buf_load_f32x4(r, e * 4u);
    return make_uint2(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w));
  }
  static __device__ __forceinline__ void store1(rsrc_t r, uint32_t e, float x) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, e * 4u, 0, 0);
  }
  static __device__ __forceinline__ void store1_stream(rsrc_t r, uint32_t e, float x) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, e * 4u, 0, kCachePolicyNT);
  }
};

// ---------------------------------------------------------------- gates
// Gate activation of the raw inputs (paper, Section 3.2): the log-decay
// g = -exp(A_log) softplus(a + dt_bias) and beta = sigmoid(b). softplus is
// evaluated as max(x, 0) + log(1 + exp(-|x|)), which cannot overflow.
__device__ __forceinline__ float softplus_f32(float x) {
  return fmaxf(x, 0.f) + log1pf(__expf(-fabsf(x)));
}
__device__ __forceinline__ float gate_log_decay(float a, float a_log, float dt_bias) {
  return -__expf(a_log) * softplus_f32(a + dt_bias);
}
__device__ __forceinline__ float gate_beta(float b) { return 1.f / (1.f + __expf(-b)); }

// ---------------------------------------------------------------- reductions
// Lane move of a DPP control within each 16-lane row (every lane has a source).
template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}

// Sum over aligned groups of `W` consecutive lanes (W a power of two <= 64);
// every lane of a group receives the same total. Inside a 16-lane row the
// partial sums move by DPP (quad swaps of 1 and 2 lanes, then the 8-lane and
// 16-lane mirrors, each pairing a lane with one from the other half of its
// group); across rows by the gfx950 row swaps, which exchange rows 0 <-> 1
// and 2 <-> 3 (16 lanes) or the two 32-lane halves. No LDS instruction is used.
template <int W>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(W >= 2 && W <= kWave && (W & (W - 1)) == 0, "group width");
  x += dpp_move<0xB1>(x);                      // quad_perm [1,0,3,2]
  if constexpr (W >= 4) x += dpp_move<0x4E>(x);   // quad_perm [2,3,0,1]
  if constexpr (W >= 8) x += dpp_move<0x141>(x);  // row_half_mirror
  if constexpr (W >= 16) x += dpp_move<0x140>(x); // row_mirror
  if constexpr (W >= 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  if constexpr (W >= 64) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return x;
}

// Lane move of a DPP control (row shift or row broadcast); lanes without a
// source, and rows outside ROW_MASK, receive 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_or_zero(float x) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROW_MASK, 0xf, false));
}

// Inclusive prefix sum over the 64 lanes of a wavefront: row shifts by 1, 2,
// 4 and 8 scan each 16-lane row, then row broadcasts of lanes 15 and 31 carry
// the running totals into the later rows.
__device__ __forceinline__ float wave_prefix_sum(float x) {
  x += dpp_or_zero<0x111, 0xf>(x);  // row_shr:1
  x += dpp_or_zero<0x112, 0xf>(x);  // row_shr:2
  x += dpp_or_zero<0x114, 0xf>(x);  // row_shr:4
  x += dpp_or_zero<0x118, 0xf>(x);  // row_shr:8
  x += dpp_or_zero<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x += dpp_or_zero<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}

// ---------------------------------------------------------------- barriers
// Work-group barrier that orders LDS traffic only. Unlike __syncthreads() it
// does not wait for outstanding global loads and stores, so prefetches stay
// in flight across it; the memory clobber keeps the compiler from moving
// memory accesses across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Orders LDS accesses of one wavefront for the compiler. The hardware already
// executes a wavefront's LDS instructions in issue order, so data written by
// one lane is visible to other lanes of the same wavefront afterwards.
__device__ __forceinline__ void wave_lds_fence() { asm volatile("" ::: "memory"); }

// ---------------------------------------------------------------- streaming
__device__ __forceinline__ f32x4 load_stream(const float *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
}
__device__ __forceinline__ void store_stream(float *p, f32x4 x) {
  __builtin_nontemporal_store(x, reinterpret_cast<f32x4 *>(p));
}

}  // namespace gdn
