// Device twin of the seeded input generator (paper_2606_13097_amd/synth):
// fills a strided [layer][row][head][dim] region with the same bits as the
// host generator, so multi-gigabyte segment libraries can be built in place.
// It holds no arithmetic of the grafting method.
//
// Definition (identical to the host module): SplitMix64 outputs
// mix64(key + n * GAMMA), key = mix64(seed + GAMMA), for n = 4c + 1, 4c + 2,
// 4c + 3 of the element counter
// c = (((tag * 2^8 + layer) * 2^16 + item) * 2^20 + row) * 2^13 + col; the
// twelve 16-bit fields h_j give x = (sum h_j - 393210) / 65536 (exact in fp32),
// times a power-of-two scale, times 8 on outlier rotary pairs, rounded to
// bf16 with round-to-nearest-even or kept as fp32.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t counter(uint64_t tag, uint64_t layer, uint64_t item, uint64_t row, uint64_t col) {
  return ((((tag << 8 | layer) << 16 | item) << 20 | row) << 13) | col;
}

__device__ __forceinline__ float normal_f32(uint64_t key, uint64_t c) {
  uint64_t acc = 0;
#pragma unroll
  for (uint64_t j = 1; j <= 3; ++j) {
    const uint64_t h = mix64(key + (4 * c + j) * GAMMA);
    acc += (h & 0xFFFF) + ((h >> 16) & 0xFFFF) + ((h >> 32) & 0xFFFF) + (h >> 48);
  }
  return (float)((int64_t)acc - 393210) * (1.0f / 65536.0f);
}

__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ void fill_kernel(void* dst, int dtype, uint64_t key, int tag, int layer0, int item, int row0, int n_rows,
                            int n_heads, int head_dim, int64_t stride_layer, int64_t stride_head, int64_t stride_row,
                            float scale, uint64_t outlier_thresh) {
  const int64_t per_layer = (int64_t)n_rows * n_heads * head_dim;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per_layer) return;
  const int l = blockIdx.y;
  const int d = (int)(i % head_dim);
  const int64_t rh = i / head_dim;
  const int h = (int)(rh % n_heads);
  const int r = (int)(rh / n_heads);
  const int layer = layer0 + l;
  const uint64_t c = counter(tag, layer, item, row0 + r, (uint64_t)h * head_dim + d);
  float x = normal_f32(key, c) * scale;
  if (outlier_thresh) {
    const int pair = d % (head_dim / 2);
    const uint64_t co = counter(8, layer, 0, h, pair);
    if ((mix64(key + (co * 4) * GAMMA) >> 11) < outlier_thresh) x *= 8.0f;
  }
  const int64_t off = l * stride_layer + h * stride_head + r * stride_row + d;
  if (dtype == 0)
    reinterpret_cast<float*>(dst)[off] = x;
  else
    reinterpret_cast<uint16_t*>(dst)[off] = to_bf16(x);
}

uint64_t host_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace

extern "C" {

// Fill dst[l * stride_layer + h * stride_head + r * stride_row + d] (elements
// of dtype 0 = fp32 / 1 = bf16) for l < n_layers, r < n_rows, h < n_heads,
// d < head_dim with the value of counter (tag, layer0 + l, item, row0 + r,
// h * head_dim + d).  outlier_rate > 0 applies the outlier pairs (tags of K and
// V only).  Returns 0 or a hipError_t.
int fcg_synth_fill(void* dst, int dtype, uint64_t seed, int tag, int layer0, int n_layers, int item, int row0,
                   int n_rows, int n_heads, int head_dim, int64_t stride_layer, int64_t stride_head,
                   int64_t stride_row, float scale, double outlier_rate, void* stream) {
  if (n_layers <= 0 || n_rows <= 0) return 0;
  if (tag < 0 || tag > 15 || layer0 < 0 || layer0 + n_layers > 256 || item < 0 || item >= 65536 || row0 < 0 ||
      row0 + n_rows > (1 << 20) || (int64_t)n_heads * head_dim > 8192)
    return (int)hipErrorInvalidValue;
  const uint64_t key = host_mix64(seed + GAMMA);
  uint64_t thresh = 0;
  if (outlier_rate > 0.0) thresh = (uint64_t)__builtin_floor(outlier_rate * 9007199254740992.0);
  const int64_t per_layer = (int64_t)n_rows * n_heads * head_dim;
  dim3 grid((unsigned)((per_layer + 255) / 256), n_layers);
  hipLaunchKernelGGL(fill_kernel, grid, dim3(256), 0, (hipStream_t)stream, dst, dtype, key, tag, layer0, item, row0,
                     n_rows, n_heads, head_dim, stride_layer, stride_head, stride_row, scale, thresh);
  return (int)hipGetLastError();
}

}  // extern "C"
