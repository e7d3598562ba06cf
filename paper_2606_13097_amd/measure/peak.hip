// Probes of this GPU's ceilings, for the bench's roofline context (not steps
// of the grafting path): the matrix-core issue rate, and the HBM stream rates
// of plain copy, read and write kernels.
//
// Matrix-core issue rate.  Every wave runs `iters` rounds of eight
// independent bf16 v_mfma_f32_16x16x32 chains on register operands: no memory
// traffic, no dependent stalls (eight chains cover the instruction's
// latency), so the rate is what the matrix cores sustain at the clock the
// chip holds under that load.  One float per lane is stored at the end so the
// work is kept.
//
// extern "C" int fcg_measure_mfma_rate(int blocks, int iters, float* out, void* stream, int shape)
//   blocks: workgroups of 256 lanes (4 waves); out: device array of
//   blocks * 256 floats; stream: HIP stream (null: the default stream);
//   shape 0: 16x16x32 instructions, 1: 32x32x16 (four chains).  Returns 0, or
//   the HIP error of the launch.  FLOPs = blocks * 4 * iters * 131072 either way.
#include <hip/hip_runtime.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) mfma_rate_kernel(int iters, float* __restrict__ out) {
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)(threadIdx.x & 63) + 0.125f * (float)i);
    b[i] = (__bf16)(1.0f - 0.0625f * (float)i);
  }
  // eight chains with distinct starting values: equal ones let the compiler
  // treat the chains as one value, and it then rotated them through shared
  // registers with copies every round
  floatx4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {1.f, 0.f, 0.f, 0.f}, c2 = {2.f, 0.f, 0.f, 0.f},
          c3 = {3.f, 0.f, 0.f, 0.f}, c4 = {4.f, 0.f, 0.f, 0.f}, c5 = {5.f, 0.f, 0.f, 0.f},
          c6 = {6.f, 0.f, 0.f, 0.f}, c7 = {7.f, 0.f, 0.f, 0.f};
  // Each instruction accumulates in place (inline assembly: through the
  // builtin the compiler still rotated the chains through shared registers
  // with copies every round).  A chain's next instruction comes eight
  // instructions later, past the dependency's latency.
#define FCG_MFMA16(c) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b))
  // wait states the compiler does not insert around inline assembly: after
  // the accumulators' initial writes, and before their final reads
  asm volatile("s_nop 7" ::: "memory");
  for (int it = 0; it < iters; ++it) {
    FCG_MFMA16(c0);
    FCG_MFMA16(c1);
    FCG_MFMA16(c2);
    FCG_MFMA16(c3);
    FCG_MFMA16(c4);
    FCG_MFMA16(c5);
    FCG_MFMA16(c6);
    FCG_MFMA16(c7);
  }
#undef FCG_MFMA16
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  const floatx4 t = c0 + c1 + c2 + c3 + c4 + c5 + c6 + c7;
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = t[0] + t[1] + t[2] + t[3];
}

typedef float floatx16 __attribute__((ext_vector_type(16)));

// the same with v_mfma_f32_32x32x16_bf16 (32,768 FLOP per instruction)
__global__ void __launch_bounds__(256) mfma32_rate_kernel(int iters, float* __restrict__ out) {
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)(threadIdx.x & 63) + 0.125f * (float)i);
    b[i] = (__bf16)(1.0f - 0.0625f * (float)i);
  }
  floatx16 c[4];  // distinct starting values, as above
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) c[j][e] = e == 0 ? (float)j : 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += c[j][e];
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

// shape 0: 16x16x32 (FLOPs = blocks * 4 * iters * 8 * 16384); shape 1: 32x32x16
// (FLOPs = blocks * 4 * iters * 4 * 32768, the same count)
extern "C" int fcg_measure_mfma_rate(int blocks, int iters, float* out, void* stream, int shape) {
  if (blocks < 1 || iters < 1 || !out || shape < 0 || shape > 1) return (int)hipErrorInvalidValue;
  if (shape == 0)
    hipLaunchKernelGGL(mfma_rate_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, out);
  else
    hipLaunchKernelGGL(mfma32_rate_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, iters, out);
  return (int)hipGetLastError();
}

// HBM stream rates.  Each block moves V16 x 256 16-byte vectors, issuing every
// load before any store; the grid covers the buffer once.  The variants are the
// fastest ones of a sweep over block sizes (4-64 KB) and cache hints on this GPU:
//   copy:  32 KB per block, nontemporal loads and stores;
//   read:  64 KB per block, nontemporal loads, folded into one value per lane
//          (stored only if it matches a pattern zeroed input never gives);
//   write: 16 KB per block, plain stores.
typedef unsigned int u32x4_m __attribute__((ext_vector_type(4)));

template <int V16>
__global__ void __launch_bounds__(256) stream_copy_kernel(const u32x4_m* __restrict__ src, u32x4_m* __restrict__ dst,
                                                          long long nvec) {
  const long long base = (long long)blockIdx.x * V16 * 256 + threadIdx.x;
  u32x4_m r[V16];
#pragma unroll
  for (int i = 0; i < V16; ++i) {
    const long long j = base + i * 256;
    r[i] = __builtin_nontemporal_load(src + (j < nvec ? j : nvec - 1));
  }
#pragma unroll
  for (int i = 0; i < V16; ++i) {
    const long long j = base + i * 256;
    if (j < nvec) __builtin_nontemporal_store(r[i], dst + j);
  }
}

template <int V16>
__global__ void __launch_bounds__(256) stream_read_kernel(const u32x4_m* __restrict__ src, u32x4_m* __restrict__ sink,
                                                          long long nvec) {
  const long long base = (long long)blockIdx.x * V16 * 256 + threadIdx.x;
  u32x4_m a = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < V16; ++i) {
    const long long j = base + i * 256;
    a ^= __builtin_nontemporal_load(src + (j < nvec ? j : nvec - 1));
  }
  if (a.x == 0x12345678u && a.y == 0x9abcdef0u) sink[threadIdx.x] = a;
}

template <int V16>
__global__ void __launch_bounds__(256) stream_write_kernel(u32x4_m* __restrict__ dst, long long nvec) {
  const long long base = (long long)blockIdx.x * V16 * 256 + threadIdx.x;
#pragma unroll
  for (int i = 0; i < V16; ++i) {
    const long long j = base + i * 256;
    if (j < nvec) dst[j] = u32x4_m{(unsigned)j, 1u, 2u, 3u};
  }
}

// extern "C" int fcg_measure_stream(int mode, const void* src, void* dst, long long bytes, void* stream)
//   mode 0: copy bytes from src to dst; 1: read bytes of src (zeroed input;
//   dst: a sink of at least 4 KB that stays untouched); 2: write bytes to dst
//   (src unused).  bytes: a positive multiple of 16.  Returns 0, or the HIP error.
extern "C" int fcg_measure_stream(int mode, const void* src, void* dst, long long bytes, void* stream) {
  if (mode < 0 || mode > 2 || bytes < 16 || bytes % 16 || !dst || (mode < 2 && !src)) return (int)hipErrorInvalidValue;
  const long long nvec = bytes / 16;
  hipStream_t s = (hipStream_t)stream;
  const u32x4_m* in = (const u32x4_m*)src;
  u32x4_m* out = (u32x4_m*)dst;
  if (mode == 0)
    hipLaunchKernelGGL(stream_copy_kernel<8>, dim3((unsigned)((nvec + 2047) / 2048)), dim3(256), 0, s, in, out, nvec);
  else if (mode == 1)
    hipLaunchKernelGGL(stream_read_kernel<16>, dim3((unsigned)((nvec + 4095) / 4096)), dim3(256), 0, s, in, out, nvec);
  else
    hipLaunchKernelGGL(stream_write_kernel<4>, dim3((unsigned)((nvec + 1023) / 1024)), dim3(256), 0, s, out, nvec);
  return (int)hipGetLastError();
}
