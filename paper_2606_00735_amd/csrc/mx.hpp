// OCP Microscaling FP8 (MXFP8) on gfx950: FP8 E4M3 elements (the OCP
// encoding: bias 7, no infinities, largest finite 448) sharing one E8M0
// scale 2^(c - 127) per 32 consecutive elements along the reduction
// dimension. The paper serves its models in FP8 (Table 2a) without naming a
// scaling scheme; MX block scaling is the one gfx950's scaled MFMA consumes
// directly.
//
// Scale layout used by every MX operand here: the four codes of a row's
// 128-element K chunk form one dword (byte b covers elements
// [32 b, 32 b + 32) of the chunk), and dwords are stored chunk-major:
// scales[chunk][row], so one chunk of a tile's rows is contiguous.
#pragma once

#include "common.hpp"

namespace moe {

constexpr int kMxBlock = 32;   // elements per scale code
constexpr int kMxChunk = 128;  // elements per scale dword

typedef int int32x8_t __attribute__((ext_vector_type(8)));

// Scale code of a block whose largest magnitude is amax (finite, >= 0): the
// shared exponent floor(log2 amax) - 8, 8 being the exponent of E4M3's
// largest power of two (so the block's largest element lands in [256, 512)
// before the clamp to 448), biased by 127 and clamped below at code 0. An
// fp32 with biased exponent E has floor(log2) = E - 127, so the code is
// E - 8; zero, denormal and tiny blocks take code 0 (2^-127).
__device__ __forceinline__ uint32_t mx_scale_code(float amax) {
  const int be = static_cast<int>((__float_as_uint(amax) >> 23) & 0xFFu);
  return be > 8 ? static_cast<uint32_t>(be - 8) : 0u;
}

// 2^-(c - 127) for scale code c: an exact power of two, normal for every code
// a finite fp32 block produces (c <= 246).
__device__ __forceinline__ float mx_inv_scale(uint32_t c) { return __uint_as_float((254u - c) << 23); }

// Four values already divided by their block scale, as E4M3 codes packed
// little-endian (v0 in the low byte): clamped to +-448, then rounded to
// nearest even by v_cvt_pk_fp8_f32 (OCP E4M3 on gfx950; the sign of a value
// that rounds to zero is kept).
__device__ __forceinline__ uint32_t e4m3x4(float v0, float v1, float v2, float v3) {
  auto sat = [](float v) { return fminf(fmaxf(v, -448.0f), 448.0f); };
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(sat(v0), sat(v1), 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(sat(v2), sat(v3), w, true);
  return static_cast<uint32_t>(w);
}

}  // namespace moe
