// Device primitives shared by the TReVS kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace trevs {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Input element tags.  Every operand fragment a lane holds is 64 bytes: 32
// bf16 values or 16 fp32 values.
struct BF16 {
  static constexpr int kBytes = 2;
};
struct F32 {
  static constexpr int kBytes = 4;
};

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float load_scalar(const void* p, size_t i, BF16) {
  return __uint_as_float(uint32_t(reinterpret_cast<const uint16_t*>(p)[i]) << 16);
}
__device__ __forceinline__ float load_scalar(const void* p, size_t i, F32) {
  return reinterpret_cast<const float*>(p)[i];
}

// Sum of squares of the values packed in a 16-byte vector.
__device__ __forceinline__ float sumsq(u32x4 v, BF16) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float lo = bf16_lo(v[j]), hi = bf16_hi(v[j]);
    s = fmaf(lo, lo, s);
    s = fmaf(hi, hi, s);
  }
  return s;
}
__device__ __forceinline__ float sumsq(u32x4 v, F32) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float x = __uint_as_float(v[j]);
    s = fmaf(x, x, s);
  }
  return s;
}

// C[32x32] += A[32 x k] * B[k x 32] over one fragment of NQ 16-byte chunks
// per lane.  Lane l supplies row (l % 32) of A and column (l % 32) of B; its
// half (l / 32) selects which half of a row slab it carries.  A and B lanes
// carry the same k values element for element, so any assignment of k to
// (half, chunk, element) that both operands share contracts correctly.
// Output layout: lane l holds column (l % 32), register r holds row
// 8*(r/4) + 4*(l/32) + (r%4).
template <int NQ>
__device__ __forceinline__ f32x16 mfma_frag(const u32x4 (&a)[NQ], const u32x4 (&b)[NQ], f32x16 c,
                                            BF16) {
#pragma unroll
  for (int s = 0; s < NQ; ++s)
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[s]),
                                                __builtin_bit_cast(bf16x8, b[s]), c, 0, 0, 0);
  return c;
}
template <int NQ>
__device__ __forceinline__ f32x16 mfma_frag(const u32x4 (&a)[NQ], const u32x4 (&b)[NQ], f32x16 c,
                                            F32) {
#pragma unroll
  for (int s = 0; s < NQ; ++s)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[s][j]), __uint_as_float(b[s][j]),
                                               c, 0, 0, 0);
  return c;
}

// Row of the 32x32 output block held by register r of a lane in half `half`.
__device__ __forceinline__ int mfma_row(int r, int half) { return 8 * (r >> 2) + 4 * half + (r & 3); }

__device__ __forceinline__ u32x4 ldg16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ u32x4 ldg16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void stg16_stream(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

// Valid text rows of sample b: len[b] clamped into 1..rows (rows when len is
// null).  The lengths live in device memory and cannot be validated on the
// host; clamping keeps every access of a bad length inside the buffers.
__device__ __forceinline__ int text_rows(const int32_t* len, int b, int rows) {
  return len ? min(max(len[b], 1), rows) : rows;
}

// Word 3 of a raw (unstructured, stride 0) buffer resource on gfx9-family
// GPUs: 32-bit data format, bounds checked against num_records.
constexpr int kBufferRsrcWord3 = 0x00020000;
// Cache-policy operand of buffer/global memory builtins: nontemporal (data
// streamed once, not worth keeping in the caches).
constexpr int kCachePolicyStream = 2;

// Wait until at most n vector-memory operations of this wave are outstanding
// (s_waitcnt immediate with expcnt and lgkmcnt unconstrained).  Placed where
// every path reaches it, it also tells the compiler that older loads have
// landed, so loads issued under uniform branches are not waited for one by
// one afterwards.
template <int n>
__device__ __forceinline__ void wait_vmem() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
}

// ---------------------------------------------------------------- reductions
// Wave-wide reductions and scans on DPP lane moves (no LDS traffic): four
// row_shr steps combine the 16 lanes of a row, then row_bcast:15 and
// row_bcast:31 carry across rows; lane 63 ends with the full result.
namespace dpp {
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ int mov(int old, int v) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, ROW_MASK, 0xf, false);
}
constexpr int kShr1 = 0x111, kShr2 = 0x112, kShr4 = 0x114, kShr8 = 0x118;
constexpr int kBcast15 = 0x142, kBcast31 = 0x143;
}  // namespace dpp

template <class Op>
__device__ __forceinline__ int wave_reduce_bits(int v, int identity, Op op) {
  v = op(v, dpp::mov<dpp::kShr1>(identity, v));
  v = op(v, dpp::mov<dpp::kShr2>(identity, v));
  v = op(v, dpp::mov<dpp::kShr4>(identity, v));
  v = op(v, dpp::mov<dpp::kShr8>(identity, v));
  v = op(v, dpp::mov<dpp::kBcast15, 0xa>(identity, v));
  v = op(v, dpp::mov<dpp::kBcast31, 0xc>(identity, v));
  return __builtin_amdgcn_readlane(v, 63);
}
__device__ __forceinline__ float wave_sum(float v) {
  return __int_as_float(wave_reduce_bits(__float_as_int(v), 0, [](int a, int b) {
    return __float_as_int(__int_as_float(a) + __int_as_float(b));
  }));
}
__device__ __forceinline__ float wave_max(float v) {
  return __int_as_float(wave_reduce_bits(__float_as_int(v), __float_as_int(-INFINITY), [](int a, int b) {
    return __float_as_int(fmaxf(__int_as_float(a), __int_as_float(b)));
  }));
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  return (uint32_t)wave_reduce_bits((int)v, -1, [](int a, int b) { return (int)min((uint32_t)a, (uint32_t)b); });
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  return (uint32_t)wave_reduce_bits((int)v, 0, [](int a, int b) { return (int)max((uint32_t)a, (uint32_t)b); });
}
// Inclusive prefix sum across the wave (lane argument kept for call sites).
__device__ __forceinline__ int wave_incl_scan(int v, int /*lane*/) {
  v += dpp::mov<dpp::kShr1>(0, v);
  v += dpp::mov<dpp::kShr2>(0, v);
  v += dpp::mov<dpp::kShr4>(0, v);
  v += dpp::mov<dpp::kShr8>(0, v);
  v += dpp::mov<dpp::kBcast15, 0xa>(0, v);
  v += dpp::mov<dpp::kBcast31, 0xc>(0, v);
  return v;
}

// The same inclusive scan in unsigned (wrapping) arithmetic.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
  auto add = [](uint32_t a, int b) { return a + (uint32_t)b; };
  v = add(v, dpp::mov<dpp::kShr1>(0, (int)v));
  v = add(v, dpp::mov<dpp::kShr2>(0, (int)v));
  v = add(v, dpp::mov<dpp::kShr4>(0, (int)v));
  v = add(v, dpp::mov<dpp::kShr8>(0, (int)v));
  v = add(v, dpp::mov<dpp::kBcast15, 0xa>(0, (int)v));
  v = add(v, dpp::mov<dpp::kBcast31, 0xc>(0, (int)v));
  return v;
}

// Order-preserving map from fp32 to uint32 (-0 taken as +0).
__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t u = __float_as_uint(f + 0.0f);  // -0 + +0 is +0: both zeros share one key
  return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Workgroup-id remap so that consecutive logical tiles land on the same XCD:
// the hardware hands workgroup w to XCD (w % 8); XCD x gets the contiguous
// logical range starting at x*(W/8) + min(x, W%8).
__device__ __forceinline__ int xcd_remap(int w, int W) {
  const int per = W >> 3, rem = W & 7, x = w & 7, local = w >> 3;
  return x * per + min(x, rem) + local;
}

}  // namespace trevs
