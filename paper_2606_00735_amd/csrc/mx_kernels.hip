// MXFP8 quantisation (OCP MX block scaling, mx.hpp) of activations and
// expert weights for the FP8 expert FFN.
#include "common.hpp"
#include "launch.hpp"
#include "mx.hpp"

namespace moe {

// x [batch][rows][K] (bf16 or fp32) -> codes [batch][rows][K] E4M3 (rows ldc
// bytes apart, ldc >= K a multiple of 16) and scale dwords [batch][K/128][rows]. Each lane takes 8 consecutive elements, so the
// 4 lanes of a 32-element block (a lane group aligned to 4) find the block's
// largest magnitude with two shuffles; the first of them writes the scale
// code. K % 128 == 0 keeps every group inside one row, and the element count
// is a multiple of 32, so a group is either wholly in range or wholly out.
// row_count (device, optional, batch 1 only): only rows [0, min(rows,
// *row_count)) are quantised; the others are left as they are.
template <bool F32IN>
__global__ __launch_bounds__(256) void mx_quantize_kernel(const void* __restrict__ x, int batch, int rows, int K,
                                                          int ldc, const int32_t* __restrict__ row_count,
                                                          uint8_t* __restrict__ codes,
                                                          uint32_t* __restrict__ scales) {
  const int n8k = K / 8;
  const int live = row_count != nullptr ? min(max(*row_count, 0), rows) : rows;
  const size_t n8 = (size_t)batch * live * n8k;
  for (size_t t = (size_t)blockIdx.x * 256 + threadIdx.x; t < n8; t += (size_t)gridDim.x * 256) {
    float v[8];
    if (F32IN) {
      const float4* p = static_cast<const float4*>(x) + 2 * t;
      const float4 a = p[0], b = p[1];
      v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = b.x, v[5] = b.y, v[6] = b.z, v[7] = b.w;
    } else {
      const uint4 u = static_cast<const uint4*>(x)[t];
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[2 * q] = __uint_as_float(w[q] << 16);
        v[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
      }
    }
    float amax = 0.0f;
#pragma unroll
    for (int q = 0; q < 8; ++q) amax = fmaxf(amax, fabsf(v[q]));
    amax = fmaxf(amax, __shfl_xor(amax, 1, kWave));
    amax = fmaxf(amax, __shfl_xor(amax, 2, kWave));
    const uint32_t code = mx_scale_code(amax);
    const float inv = mx_inv_scale(code);
    uint2 out;
    out.x = e4m3x4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
    out.y = e4m3x4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv);
    const int k8 = (int)(t % n8k);
    const size_t row = t / n8k;  // batch * rows + r
    *reinterpret_cast<uint2*>(codes + row * ldc + (size_t)k8 * 8) = out;
    if ((k8 & 3) == 0) {
      const size_t b = row / rows, r = row % rows;
      const int kb = k8 / 4;  // 32-element block within the row
      reinterpret_cast<uint8_t*>(scales + (b * (K / kMxChunk) + kb / 4) * rows + r)[kb & 3] =
          static_cast<uint8_t>(code);
    }
  }
}

hipError_t launch_mx_quantize(const void* x, bool f32, int batch, int rows, int K, int ldc,
                              const int32_t* row_count, uint8_t* codes, uint32_t* scales, hipStream_t s) {
  const size_t n8 = (size_t)batch * rows * (K / 8);
  if (n8 == 0) return hipSuccess;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) cus = n;
  }
  size_t grid = (n8 + 255) / 256;
  if (grid > (size_t)cus * 16) grid = (size_t)cus * 16;
  if (f32)
    mx_quantize_kernel<true><<<(unsigned)grid, 256, 0, s>>>(x, batch, rows, K, ldc, row_count, codes, scales);
  else
    mx_quantize_kernel<false><<<(unsigned)grid, 256, 0, s>>>(x, batch, rows, K, ldc, row_count, codes, scales);
  return hipGetLastError();
}

}  // namespace moe
