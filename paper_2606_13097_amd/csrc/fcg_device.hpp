// Device helpers shared by the gfx950 kernels of libfcg: storage-dtype
// conversion, 16-byte vector access, rotary angles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fcg {

typedef uint16_t bf16_t;  // raw bfloat16 bits

// bf16 -> fp32 is exact: the bits are the high half of the binary32 pattern.
__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Two fp32 -> packed pair of bf16 (lo in bits 0..15).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Storage traits: a 16-byte vector holds VEC elements.
template <typename T> struct Store;
template <> struct Store<float> {
  static constexpr int VEC = 4;
  __device__ static inline void unpack(const uint4& w, float* x) {
    x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
    x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
  }
  __device__ static inline uint4 pack(const float* x) {
    return make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3]));
  }
  __device__ static inline float load1(const float* p) { return *p; }
  __device__ static inline float round(float x) { return x; }
  __device__ static inline void store1(float* p, float x) { *p = x; }
};
template <> struct Store<bf16_t> {
  static constexpr int VEC = 8;
  __device__ static inline void unpack(const uint4& w, float* x) {
    x[0] = lo_bf16(w.x); x[1] = hi_bf16(w.x); x[2] = lo_bf16(w.y); x[3] = hi_bf16(w.y);
    x[4] = lo_bf16(w.z); x[5] = hi_bf16(w.z); x[6] = lo_bf16(w.w); x[7] = hi_bf16(w.w);
  }
  __device__ static inline uint4 pack(const float* x) {
    return make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                      pack_bf16x2(x[6], x[7]));
  }
  __device__ static inline float load1(const bf16_t* p) { return bf16_to_f32(*p); }
  __device__ static inline float round(float x) { return bf16_to_f32(f32_to_bf16(x)); }
  __device__ static inline void store1(bf16_t* p, float x) { *p = f32_to_bf16(x); }
};

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// 16-byte load with the nontemporal hint (global_load ... nt): for data read
// once, which then does not displace reused lines from the caches
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// 8-byte store with the nontemporal hint: for results another kernel reads
// (from another XCD's L2, so keeping them in this one buys nothing)
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void st8_nt(void* p, uint32_t lo, uint32_t hi) {
  const u32x2_t v = {lo, hi};
  __builtin_nontemporal_store(v, reinterpret_cast<u32x2_t*>(p));
}
__device__ __forceinline__ void st16(void* p, const uint4& v) { *reinterpret_cast<uint4*>(p) = v; }

// Device-coherent accesses for data that one block writes and another block
// of the same launch reads (the XCDs' L2 caches are not coherent with each
// other): relaxed device-scope atomic stores, and buffer loads with the
// device-scope cache policy.  Buffer loads past num_records return zeros.
__device__ __forceinline__ void st_dev(float* p, float x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev_u32(uint32_t* p, uint32_t x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
constexpr int kBufWord3 = 0x00020000;  // raw 32-bit buffer (no format conversion)
constexpr int kPolicyDevice = 16;      // sc1: coherent at device scope
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, kBufWord3);
}
__device__ __forceinline__ u32x4_t ld16_dev(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kPolicyDevice);
}
__device__ __forceinline__ u32x2_t ld8_dev(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kPolicyDevice);
}
// s_waitcnt vmcnt(0): every vector memory access of this wave has completed
__device__ __forceinline__ void wait_vm0() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);
  asm volatile("" ::: "memory");
}

// Reductions over the four lanes l, l ^ 16, l ^ 32, l ^ 48 of a wave (one
// value per 16-lane row), with the gfx950 lane-swap instructions instead of
// LDS permutes (__shfl_xor goes through ds_bpermute, an LDS round trip each).
// Called with one register as both operands, v_permlane16_swap hands every
// lane its own value and that of lane l ^ 16 as its two results (in an order
// that depends on the row), and v_permlane32_swap the same for lane l ^ 32;
// the operations below are commutative, so the order does not matter and all
// four lanes end with the same bits.
__device__ __forceinline__ float max_rows4(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum_rows4(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float m = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Reductions over each 32-lane half of a wave, every lane ending with the
// half's result (the same bits in all of them: each step combines symmetric
// pairs of lanes).  Lanes l ^ 1 and l ^ 2 by DPP quad permutes, then the
// mirrored lane within 8 and within 16 (DPP row_half_mirror, row_mirror),
// then lane l ^ 16 by v_permlane16_swap; no LDS round trip.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141; // lane 7 - l within 8
constexpr int kDppMirror = 0x140;     // lane 15 - l within 16
__device__ __forceinline__ float max_lanes32(float v) {
  v = fmaxf(v, dpp_f32<kDppXor1>(v));
  v = fmaxf(v, dpp_f32<kDppXor2>(v));
  v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f32<kDppMirror>(v));
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
}
__device__ __forceinline__ float sum_lanes32(float v) {
  v += dpp_f32<kDppXor1>(v);
  v += dpp_f32<kDppXor2>(v);
  v += dpp_f32<kDppHalfMirror>(v);
  v += dpp_f32<kDppMirror>(v);
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(a[0]) + __uint_as_float(a[1]);
}

// cos and sin of pos * w for the rotary pair with float64 frequency w: the
// angle is the float64 product and the float64 cos/sin are rounded to fp32.
__device__ __forceinline__ void rope_cs(double pos, double w, float* c, float* s) {
  double sd, cd;
  sincos(pos * w, &sd, &cd);
  *c = (float)cd;
  *s = (float)sd;
}

}  // namespace fcg
