// Gating, activation profile, dispatch permutation and combine kernels (gfx950).
//
// The routed MoE layer of ViBE's Section 2: tokens pick k experts each; this
// GPU counts the picks per expert (the activation profile, Section 4.2.2),
// gathers the rows routed to its local experts (its token load, Section 4.2.3)
// and, after the expert FFN, scatters the weighted results back.
#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace moe {

// ---------------------------------------------------------------------------
// Block-wide helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ int wave_inclusive_scan(int v, int lane) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int n = __shfl_up(v, off, kWave);
    if (lane >= off) v += n;
  }
  return v;
}

// Exclusive scan of one int per thread over a 256-thread block.
__device__ __forceinline__ int block_exclusive_scan_256(int v, int* s_wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = wave_inclusive_scan(v, lane);
  if (lane == 63) s_wave_tot[wave] = inc;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    int t = s_wave_tot[w];
    if (w < wave) base += t;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return base + inc - v;
}

// ---------------------------------------------------------------------------
// Top-k over one row held by a group of GROUP lanes, NV values per lane; the
// value in slot q of lane g is column q * GROUP + g. Selection order is
// (value descending, column ascending). Every lane of the group ends with the
// same selection.
// ---------------------------------------------------------------------------
// Best (value, column) of each group of GROUP = 32 or 64 consecutive lanes,
// returned in every lane of the group, by DPP (a few cycles a step, where a
// lane shuffle through LDS takes tens): a running best along each row of 16
// lanes (row_shr 1, 2, 4, 8; lanes shifted in from outside the row offer
// (-inf, INT_MAX), which never wins), leaving each row's best in its lane
// 15; row_bcast:15 then gives lanes 31 and 63 the best of rows 0-1 and 2-3,
// and row_bcast:31 lane 63 the best of all four. The order (value
// descending, column ascending) is strict, so the winner does not depend on
// the reduction's shape.
// One DPP step of group_best: (v, i) becomes the better of itself and the
// pair DPP control CTRL brings from another lane of rows ROW_MASK.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void best_dpp(float& v, int& i) {
  const float ov = __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(-__builtin_huge_valf()), __float_as_int(v), CTRL, ROW_MASK, 0xf, false));
  const int oi = __builtin_amdgcn_update_dpp(0x7fffffff, i, CTRL, ROW_MASK, 0xf, false);
  if (better(ov, oi, v, i)) {
    v = ov;
    i = oi;
  }
}

template <int GROUP>
__device__ __forceinline__ void group_best(float& v, int& i) {
  static_assert(GROUP == 32 || GROUP == 64, "group of 32 or 64 lanes");
  best_dpp<0x111, 0xf>(v, i);  // row_shr:1
  best_dpp<0x112, 0xf>(v, i);  // row_shr:2
  best_dpp<0x114, 0xf>(v, i);  // row_shr:4
  best_dpp<0x118, 0xf>(v, i);  // row_shr:8
  best_dpp<0x142, 0xa>(v, i);  // row_bcast:15 into rows 1, 3
  if (GROUP == 64) {
    best_dpp<0x143, 0xc>(v, i);  // row_bcast:31 into rows 2, 3
    v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
    i = __builtin_amdgcn_readlane(i, 63);
  } else {
    const float v0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 31));
    const float v1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
    const int i0 = __builtin_amdgcn_readlane(i, 31), i1 = __builtin_amdgcn_readlane(i, 63);
    const bool hi = (threadIdx.x & 32) != 0;
    v = hi ? v1 : v0;
    i = hi ? i1 : i0;
  }
}

template <int GROUP, int NV>
__device__ __forceinline__ void topk_group(const float (&val)[NV], int g, int E, int k,
                                           float (&sel_v)[kMaxTopk], int (&sel_i)[kMaxTopk]) {
  uint32_t taken = 0;
#pragma unroll
  for (int j = 0; j < kMaxTopk; ++j) {
    if (j < k) {
      float lv = -__builtin_huge_valf();
      int li = 0x7fffffff;
#pragma unroll
      for (int q = 0; q < NV; ++q) {
        const int col = q * GROUP + g;
        if (!((taken >> q) & 1u) && col < E && better(val[q], col, lv, li)) {
          lv = val[q];
          li = col;
        }
      }
      group_best<GROUP>(lv, li);
      sel_v[j] = lv;
      sel_i[j] = li;
      if ((li % GROUP) == g) taken |= 1u << (li / GROUP);
    }
  }
}

// Renormalised softmax over the k selected logits; lane g < k of the group
// writes slot g of the row.
__device__ __forceinline__ void write_topk(const float (&sel_v)[kMaxTopk], const int (&sel_i)[kMaxTopk],
                                           int g, int k, int row, int32_t* __restrict__ ids,
                                           float* __restrict__ wts) {
  float p[kMaxTopk];
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < kMaxTopk; ++j) {
    if (j < k) {
      p[j] = expf(sel_v[j] - sel_v[0]);
      s = s + p[j];
    }
  }
  if (g < k) {
    float pj = 0.0f;
    int ij = 0;
#pragma unroll
    for (int j = 0; j < kMaxTopk; ++j) {
      if (j == g) {
        pj = p[j];
        ij = sel_i[j];
      }
    }
    ids[(size_t)row * k + g] = ij;
    wts[(size_t)row * k + g] = pj / s;
  }
}

// ---------------------------------------------------------------------------
// Router, bf16: logits on MFMA (v_mfma_f32_32x32x16_bf16), top-k in registers.
//
// A block of 4 waves takes 128 tokens; each wave owns 32 tokens and all
// E_pad = 32 * NCB expert columns. Token rows and router weights are loaded
// straight into three swizzled LDS stages, one 64-wide K chunk at a time
// (see pipeline).
// ---------------------------------------------------------------------------
constexpr int kGateBK = 64;
constexpr int kSmallRouterT = 8192;  // largest batch for gate_topk_bf16_small_kernel

template <int NCB>
__global__ __launch_bounds__(256) void gate_topk_bf16_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, const float* __restrict__ bias,
    int T, int H, int E, int k, float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ wts) {
  constexpr int BROWS = NCB * 32;
  constexpr int STAGE = (128 + BROWS) * 64;
  __shared__ __align__(16) bf16_t smem[3 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 31, half = lane >> 5;
  const int row0 = blockIdx.x * 128 + wave * 32;
  const bf16_t* xa = x + (size_t)blockIdx.x * 128 * H;
  const int a_rows = T - blockIdx.x * 128;
  const int nK = H / kGateBK;

  f32x16_t acc[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) acc[c] = f32x16_t{};

  auto issue = [&](int kc, bool live, bf16_t* st) {
    dma_rows<128, 4, kGateBK>(xa, H, kc * kGateBK, a_rows, live, st, wave, lane);
    dma_rows<BROWS, 4, kGateBK>(wr, H, kc * kGateBK, E, live, st + 128 * 64, wave, lane);
  };
  auto compute = [&](const bf16_t* st) {
#pragma unroll
    for (int i = 0; i < kGateBK / 16; ++i) {
      const int chunk = 2 * i + half;
      const bf16x8_t a = lds_frag<kGateBK>(st, wave * 32 + r, chunk);
#pragma unroll
      for (int c = 0; c < NCB; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, lds_frag<kGateBK>(st + 128 * 64, c * 32 + r, chunk), acc[c], 0,
                                                         0, 0);
    }
  };
  pipeline<3, 4 + NCB>(nK, smem, STAGE, issue, compute);

  float bias_r[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) {
    const int col = c * 32 + r;
    bias_r[c] = (bias != nullptr && col < E) ? bias[col] : 0.0f;
  }

  // 32x32 accumulator layout: register v of lane (r, half) is row
  // 8 * (v / 4) + 4 * half + (v % 4), column r of the block.
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int row = row0 + 8 * (v >> 2) + 4 * half + (v & 3);
    float val[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c) {
      const int col = c * 32 + r;
      val[c] = (col < E) ? acc[c][v] + bias_r[c] : -__builtin_huge_valf();
    }
    if (logits != nullptr && row < T) {
#pragma unroll
      for (int c = 0; c < NCB; ++c) {
        const int col = c * 32 + r;
        if (col < E) logits[(size_t)row * E + col] = val[c];
      }
    }
    float sel_v[kMaxTopk];
    int sel_i[kMaxTopk];
    topk_group<32, NCB>(val, r, E, k, sel_v, sel_i);
    if (row < T) write_topk(sel_v, sel_i, r, k, row, ids, wts);
  }
}

// ---------------------------------------------------------------------------
// Router, bf16, for small batches of few experts (E <= 128): 32 tokens per
// block, so that a batch of a few thousand tokens still spreads over the
// CUs. The 4 waves split every 64-wide K chunk (wave w takes k-step w), then
// sum their partial logits in wave order through LDS. On inputs whose
// partial sums are exact in fp32 the split gives the same logits as any
// other order.
// ---------------------------------------------------------------------------
template <int NCB>
__global__ __launch_bounds__(256) void gate_topk_bf16_ksplit_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, const float* __restrict__ bias,
    int T, int H, int E, int k, float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ wts) {
  constexpr int BROWS = NCB * 32;
  constexpr int STAGE = (32 + BROWS) * 64;
  constexpr int FIT = (96 * 1024) / (STAGE * 2);  // stages in 96 KB: small blocks need depth
  constexpr int NS = FIT > 8 ? 8 : FIT;
  constexpr int RED = 4 * NCB * 16 * kWave;  // fp32 partials of all waves
  constexpr int SMEM_BYTES = (NS * STAGE * 2 > RED * 4) ? NS * STAGE * 2 : RED * 4;
  __shared__ __align__(16) unsigned char smem_raw[SMEM_BYTES];
  bf16_t* smem = reinterpret_cast<bf16_t*>(smem_raw);
  float* red = reinterpret_cast<float*>(smem_raw);

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 31, half = lane >> 5;
  const int row0 = blockIdx.x * 32;
  const bf16_t* xa = x + (size_t)row0 * H;
  const int a_rows = T - row0;
  const int nK = H / kGateBK;

  f32x16_t acc[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) acc[c] = f32x16_t{};

  auto issue = [&](int kc, bool live, bf16_t* st) {
    dma_rows<32, 4, kGateBK>(xa, H, kc * kGateBK, a_rows, live, st, wave, lane);
    dma_rows<BROWS, 4, kGateBK>(wr, H, kc * kGateBK, E, live, st + 32 * 64, wave, lane);
  };
  auto compute = [&](const bf16_t* st) {
    const int chunk = 2 * wave + half;
    const bf16x8_t a = lds_frag<kGateBK>(st, r, chunk);
#pragma unroll
    for (int c = 0; c < NCB; ++c)
      acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, lds_frag<kGateBK>(st + 32 * 64, c * 32 + r, chunk),
                                                       acc[c], 0, 0, 0);
  };
  pipeline<NS, 1 + NCB>(nK, smem, STAGE, issue, compute);

  // partial logits of wave w -> red[w][c][v][lane]
#pragma unroll
  for (int c = 0; c < NCB; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) red[((wave * NCB + c) * 16 + v) * kWave + lane] = acc[c][v];
  __syncthreads();

  float bias_r[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) {
    const int col = c * 32 + r;
    bias_r[c] = (bias != nullptr && col < E) ? bias[col] : 0.0f;
  }
  // wave w finishes accumulator registers v = 4w .. 4w+3 (8 of the 32 rows)
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int v = 4 * wave + q;
    const int row = row0 + 8 * (v >> 2) + 4 * half + (v & 3);
    float val[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c) {
      float z = 0.0f;
#pragma unroll
      for (int w = 0; w < 4; ++w) z += red[((w * NCB + c) * 16 + v) * kWave + lane];
      const int col = c * 32 + r;
      val[c] = (col < E) ? z + bias_r[c] : -__builtin_huge_valf();
    }
    if (logits != nullptr && row < T) {
#pragma unroll
      for (int c = 0; c < NCB; ++c) {
        const int col = c * 32 + r;
        if (col < E) logits[(size_t)row * E + col] = val[c];
      }
    }
    float sel_v[kMaxTopk];
    int sel_i[kMaxTopk];
    topk_group<32, NCB>(val, r, E, k, sel_v, sel_i);
    if (row < T) write_topk(sel_v, sel_i, r, k, row, ids, wts);
  }
}

// ---------------------------------------------------------------------------
// Router, bf16, for batches of a few hundred tokens (decode) and E <= 128:
// 32 tokens per block and NW waves, each taking an equal, contiguous share of
// the K range straight from global memory into registers (no LDS stages, so
// no barriers in the K loop: one block's K range is streamed by all its
// waves at once instead of chunk by chunk). A wave loads GK k-steps of
// operands per group, the next group while the MFMAs of the current one run;
// the four k-steps of a 64-wide chunk cover whole 128-byte lines of each row.
// Partial logits are summed through LDS in wave order; on inputs whose
// partial sums are exact in fp32 that equals any other order.
// ---------------------------------------------------------------------------
template <int NCB, int NW, int GK>
__global__ __launch_bounds__(NW * 64) void gate_topk_bf16_small_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, const float* __restrict__ bias,
    int T, int H, int E, int k, float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ wts, int S = 1, float* __restrict__ part = nullptr) {
  __shared__ float red[NW * NCB * 16 * kWave];  // partial logits of every wave
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 31, half = lane >> 5;
  const int row0 = blockIdx.x * 32;
  // lane (r, half) holds elements 16 s + 8 half .. + 8 of k-step s of token
  // row r (A operand) and of router row 32 c + r (B operand, block c);
  // rows past the batch or past E re-read the last one and are masked below
  const bf16x8_t* xp =
      reinterpret_cast<const bf16x8_t*>(x + (size_t)min(row0 + r, T - 1) * H) + half;
  const bf16x8_t* wp[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c)
    wp[c] = reinterpret_cast<const bf16x8_t*>(wr + (size_t)min(c * 32 + r, E - 1) * H) + half;
  // block (x, y) sums K range y of S (part != nullptr: fp32 partial logits
  // of its 32 tokens go to part[y][row][0, 32 NCB) for the top-k pass)
  const int nkb = H / 16 / S, per = nkb / NW;  // the launcher checks per % (2 GK) == 0
  const int s0 = (int)blockIdx.y * nkb + wave * per;

  f32x16_t acc[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) acc[c] = f32x16_t{};
  bf16x8_t a0[GK], b0[GK][NCB], a1[GK], b1[GK][NCB];
  auto load = [&](int s, bf16x8_t(&a)[GK], bf16x8_t(&b)[GK][NCB]) {
#pragma unroll
    for (int g = 0; g < GK; ++g) {
      a[g] = xp[2 * (s + g)];
#pragma unroll
      for (int c = 0; c < NCB; ++c) b[g][c] = wp[c][2 * (s + g)];
    }
  };
  auto mma = [&](const bf16x8_t(&a)[GK], const bf16x8_t(&b)[GK][NCB]) {
#pragma unroll
    for (int g = 0; g < GK; ++g)
#pragma unroll
      for (int c = 0; c < NCB; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[g], b[g][c], acc[c], 0, 0, 0);
  };
  load(s0, a0, b0);
  for (int s = s0; s < s0 + per; s += 2 * GK) {
    load(s + GK, a1, b1);
    mma(a0, b0);
    if (s + 2 * GK < s0 + per) load(s + 2 * GK, a0, b0);
    mma(a1, b1);
  }

#pragma unroll
  for (int c = 0; c < NCB; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) red[((wave * NCB + c) * 16 + v) * kWave + lane] = acc[c][v];
  __syncthreads();

  float bias_r[NCB];
#pragma unroll
  for (int c = 0; c < NCB; ++c) {
    const int col = c * 32 + r;
    bias_r[c] = (bias != nullptr && col < E) ? bias[col] : 0.0f;
  }
  // wave w finishes accumulator registers v = w, w + NW, ... (2 rows each)
  for (int v = wave; v < 16; v += NW) {
    const int row = row0 + 8 * (v >> 2) + 4 * half + (v & 3);
    float val[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c) {
      float z = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) z += red[((w * NCB + c) * 16 + v) * kWave + lane];
      const int col = c * 32 + r;
      val[c] = (col < E) ? z + bias_r[c] : -__builtin_huge_valf();
      if (part != nullptr && row < T) part[((size_t)blockIdx.y * T + row) * (32 * NCB) + col] = z;
    }
    if (part != nullptr) continue;  // wave-uniform
    if (logits != nullptr && row < T) {
#pragma unroll
      for (int c = 0; c < NCB; ++c) {
        const int col = c * 32 + r;
        if (col < E) logits[(size_t)row * E + col] = val[c];
      }
    }
    float sel_v[kMaxTopk];
    int sel_i[kMaxTopk];
    topk_group<32, NCB>(val, r, E, k, sel_v, sel_i);
    if (row < T) write_topk(sel_v, sel_i, r, k, row, ids, wts);
  }
}

// ---------------------------------------------------------------------------
// Router, bf16, for E > 32 when blocks of 128 tokens would leave CUs idle:
// 8 waves per block of BT = 64 tokens, the FFN GEMM's pipeline
// (pipeline_xk: operands read one k-step ahead across chunks, NS stages of x
// rows and router weights in swizzled LDS). Waves tile the BT x E_pad
// logits as (BT / 32) x (256 / BT) (32 tokens by a share of the experts
// each). The logits then go through LDS (fp32, BT x E_pad), and each wave
// selects the top k of BT / 8 tokens with all 64 lanes. Every block loads
// all E_pad router rows, and the load path, not the MFMAs, bounds both
// router kernels, so the launcher takes the block size for which one CU
// loads fewer rows: rounds of blocks x (E_pad + tokens per block).
// ---------------------------------------------------------------------------
template <int BT, int NCB>  // E_pad = 32 * NCB, NCB = 4 or 8
__global__ __launch_bounds__(512) void gate_topk_bf16_wide_kernel(
    const bf16_t* __restrict__ x, const bf16_t* __restrict__ wr, const float* __restrict__ bias,
    int T, int H, int E, int k, float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ wts) {
  static_assert(NCB == 4 || NCB == 8, "E_pad of 128 or 256");
  static_assert(BT == 64 || BT == 128, "tokens per block");
  constexpr int WAVES_M = BT / 32, WAVES_N = 8 / WAVES_M;
  constexpr int EP = NCB * 32, NI = NCB / WAVES_N;
  constexpr int ROWS = BT + EP;
  constexpr int STAGE = ROWS * kGateBK;                          // bf16 slots
  constexpr int NS = (144 * 1024) / (STAGE * 2) > 8 ? 8 : (144 * 1024) / (STAGE * 2);
  static_assert(NS >= 2, "stages");
  constexpr int LOADS = ROWS / 64;                               // 1 KB loads per wave per chunk
  constexpr int SMEM = (NS * STAGE * 2 > BT * EP * 4) ? NS * STAGE * 2 : BT * EP * 4;
  __shared__ __align__(16) unsigned char smem_raw[SMEM];
  bf16_t* smem = reinterpret_cast<bf16_t*>(smem_raw);
  float* tile = reinterpret_cast<float*>(smem_raw);

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int r = lane & 31, half = lane >> 5;
  const int row0 = blockIdx.x * BT;
  const bf16_t* xa = x + (size_t)row0 * H;
  const int a_rows = T - row0;
  const int nK = H / kGateBK;

  f32x16_t acc[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) acc[j] = f32x16_t{};

  auto issue = [&](int kc, bool live, bf16_t* st) {
    dma_rows<BT, 8, kGateBK>(xa, H, kc * kGateBK, a_rows, live, st, wave, lane);
    dma_rows<EP, 8, kGateBK>(wr, H, kc * kGateBK, E, live, st + BT * kGateBK, wave, lane);
  };
  bf16x8_t af[2], bfr[2][NI];
  auto read = [&](const bf16_t* st, int s, int buf) {
    const int chunk = 2 * s + half;
    af[buf] = lds_frag<kGateBK>(st, wm * 32 + r, chunk);
#pragma unroll
    for (int j = 0; j < NI; ++j) bfr[buf][j] = lds_frag<kGateBK>(st + BT * kGateBK, (wn * NI + j) * 32 + r, chunk);
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[buf], bfr[buf][j], acc[j], 0, 0, 0);
  };
  auto mix = [&]() {
#pragma unroll
    for (int q = 0; q < NI; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  };
  pipeline_xk<NS, LOADS, kGateBK / 16>(nK, smem, STAGE, issue, read, mma, mix);

  // logits + bias into the LDS tile (the stages are free): register v of lane
  // (r, half) holds token row 8 (v / 4) + 4 half + (v % 4), expert column r of
  // its 32-column block
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int col = (wn * NI + j) * 32 + r;
    const float b = (bias != nullptr && col < E) ? bias[col] : 0.0f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = wm * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
      tile[row * EP + col] = (col < E) ? acc[j][v] + b : -__builtin_huge_valf();
    }
  }
  __syncthreads();

  // wave w selects for tokens w BT / 8 .. (w + 1) BT / 8 - 1; lane g holds
  // columns q * 64 + g
  constexpr int NV = EP / 64;
  for (int t = 0; t < BT / 8; ++t) {
    const int lr = wave * (BT / 8) + t;
    const int row = row0 + lr;
    if (row >= T) break;  // wave-uniform
    float val[NV];
#pragma unroll
    for (int q = 0; q < NV; ++q) val[q] = tile[lr * EP + q * 64 + lane];
    if (logits != nullptr) {
#pragma unroll
      for (int q = 0; q < NV; ++q) {
        const int col = q * 64 + lane;
        if (col < E) logits[(size_t)row * E + col] = val[q];
      }
    }
    float sel_v[kMaxTopk];
    int sel_i[kMaxTopk];
    topk_group<64, NV>(val, lane, E, k, sel_v, sel_i);
    write_topk(sel_v, sel_i, lane, k, row, ids, wts);
  }
}

// ---------------------------------------------------------------------------
// Router, fp32: one wave per token, lanes over experts, VALU dot products in
// ascending h.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gate_topk_f32_kernel(
    const float* __restrict__ x, const float* __restrict__ wr, const float* __restrict__ bias,
    int T, int H, int E, int k, float* __restrict__ logits, int32_t* __restrict__ ids,
    float* __restrict__ wts) {
  constexpr int NV = kMaxExperts / kWave;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= T) return;
  const float* xr = x + (size_t)row * H;
  float val[NV];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    const int e = q * kWave + lane;
    float z = -__builtin_huge_valf();
    if (e < E) {
      const float* w = wr + (size_t)e * H;
      float s = 0.0f;
      for (int h = 0; h < H; ++h) s = __builtin_fmaf(xr[h], w[h], s);
      z = s + (bias != nullptr ? bias[e] : 0.0f);
      if (logits != nullptr) logits[(size_t)row * E + e] = z;
    }
    val[q] = z;
  }
  float sel_v[kMaxTopk];
  int sel_i[kMaxTopk];
  topk_group<kWave, NV>(val, lane, E, k, sel_v, sel_i);
  write_topk(sel_v, sel_i, lane, k, row, ids, wts);
}

// ---------------------------------------------------------------------------
// Activation profile: per-block expert counts (LDS atomics on integers, so
// the result does not depend on their order).
// ---------------------------------------------------------------------------
constexpr int kTokPerBlk = 256;  // tokens per block of the count table (T / 256 blocks)

__global__ __launch_bounds__(256) void hist_kernel(const int32_t* __restrict__ ids, int T, int k, int E,
                                                   int32_t* __restrict__ table) {
  __shared__ int cnt[kMaxExperts];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += 256) cnt[e] = 0;
  __syncthreads();
  const size_t first = (size_t)blockIdx.x * kTokPerBlk * k;
  const size_t last = min((size_t)T * k, first + (size_t)kTokPerBlk * k);
  for (size_t p = first + tid; p < last; p += 256) {
    const int e = ids[p];
    if ((unsigned)e < (unsigned)E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = tid; e < E; e += 256) table[(size_t)blockIdx.x * E + e] = cnt[e];
}

// Totals, local offsets (exclusive scan over slots) and per-block row bases.
__global__ __launch_bounds__(256) void scan_kernel(const int32_t* __restrict__ table, int n_blk,
                                                   SlotMap map, int32_t* __restrict__ counts,
                                                   int32_t* __restrict__ offsets,
                                                   int32_t* __restrict__ bases, int32_t* __restrict__ m_loc) {
  __shared__ int s_cnt[kMaxExperts];
  __shared__ int s_tot[4];
  const int tid = threadIdx.x;
  const int E = map.n_experts, L = map.n_local;
  for (int e = tid; e < E; e += 256) {
    int c = 0;
#pragma unroll 8
    for (int b = 0; b < n_blk; ++b) c += table[(size_t)b * E + e];
    counts[e] = c;
    s_cnt[e] = c;
  }
  __syncthreads();
  const int my_e = tid < L ? map.expert_of[tid] : 0;
  const int v = tid < L ? s_cnt[my_e] : 0;
  int total;
  const int excl = block_exclusive_scan_256(v, s_tot, &total);
  if (tid < L) {
    offsets[tid + 1] = excl + v;
    int run = excl;
#pragma unroll 8
    for (int b = 0; b < n_blk; ++b) {
      bases[(size_t)b * L + tid] = run;
      run += table[(size_t)b * E + my_e];
    }
  }
  if (tid == 0) {
    offsets[0] = 0;
    *m_loc = total;
  }
}

// scan_kernel for a count table of at most kScanLdsInts entries: the table
// is first copied into LDS with every thread's loads in flight together
// (16 a thread before the first wait), so the per-expert column sums and
// the row bases walk LDS instead of taking one dependent round trip to L2
// per 8 count blocks (Maverick-shaped T = 32768, 128 x 128 counts:
// 10.1 -> 8.5 us). Same integer results.
constexpr int kScanLdsInts = 16384;
__global__ __launch_bounds__(256) void scan_lds_kernel(const int32_t* __restrict__ table, int n_blk,
                                                       SlotMap map, int32_t* __restrict__ counts,
                                                       int32_t* __restrict__ offsets,
                                                       int32_t* __restrict__ bases, int32_t* __restrict__ m_loc) {
  __shared__ int s_tab[kScanLdsInts];
  __shared__ int s_cnt[kMaxExperts];
  __shared__ int s_tot[4];
  const int tid = threadIdx.x;
  const int E = map.n_experts, L = map.n_local;
  const int n = n_blk * E;
#pragma unroll 16
  for (int i = tid; i < n; i += 256) s_tab[i] = table[i];
  __syncthreads();
  for (int e = tid; e < E; e += 256) {
    int c = 0;
    for (int b = 0; b < n_blk; ++b) c += s_tab[b * E + e];
    counts[e] = c;
    s_cnt[e] = c;
  }
  __syncthreads();
  const int my_e = tid < L ? map.expert_of[tid] : 0;
  const int v = tid < L ? s_cnt[my_e] : 0;
  int total;
  const int excl = block_exclusive_scan_256(v, s_tot, &total);
  if (tid < L) {
    offsets[tid + 1] = excl + v;
    int run = excl;
    for (int b = 0; b < n_blk; ++b) {
      bases[(size_t)b * L + tid] = run;
      run += s_tab[b * E + my_e];
    }
  }
  if (tid == 0) {
    offsets[0] = 0;
    *m_loc = total;
  }
}

// One count block (T <= kTokPerBlk): the counts, the local offsets and the
// block's row bases in one launch (the count table is not needed).
__global__ __launch_bounds__(256) void hist_scan_one_block_kernel(const int32_t* __restrict__ ids, int T, int k,
                                                                  SlotMap map, int32_t* __restrict__ counts,
                                                                  int32_t* __restrict__ offsets,
                                                                  int32_t* __restrict__ bases,
                                                                  int32_t* __restrict__ m_loc) {
  __shared__ int cnt[kMaxExperts];
  __shared__ int s_tot[4];
  const int tid = threadIdx.x;
  const int E = map.n_experts, L = map.n_local;
  for (int e = tid; e < E; e += 256) cnt[e] = 0;
  __syncthreads();
  for (int p = tid; p < T * k; p += 256) {
    const int e = ids[p];
    if ((unsigned)e < (unsigned)E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = tid; e < E; e += 256) counts[e] = cnt[e];
  const int v = tid < L ? cnt[map.expert_of[tid]] : 0;
  int total;
  const int excl = block_exclusive_scan_256(v, s_tot, &total);
  if (tid < L) {
    offsets[tid + 1] = excl + v;
    bases[tid] = excl;
  }
  if (tid == 0) {
    offsets[0] = 0;
    *m_loc = total;
  }
}

// ---------------------------------------------------------------------------
// Dispatch permutation, step 1: positions. Block b re-reads the ids of its
// kTokPerBlk tokens in rounds of 256 (one token per thread). The rank of an
// assignment within its slot comes from 64-bit lane masks per (round, wave)
// -- lane order is token order -- never from atomic return order, so the
// permutation is the stable counting sort and is identical run to run.
// ---------------------------------------------------------------------------
constexpr int kRounds = kTokPerBlk / 256;

__global__ __launch_bounds__(256) void permute_index_kernel(const int32_t* __restrict__ ids, int T, int k,
                                                            SlotMap map, const int32_t* __restrict__ bases,
                                                            int M_cap, int32_t* __restrict__ perm_src,
                                                            int32_t* __restrict__ dest) {
  __shared__ unsigned long long s_mask[kRounds * 4][kMaxExperts];
  __shared__ int s_pre[kRounds * 4][kMaxExperts];
  __shared__ int16_t s_slot_of[kMaxExperts];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = map.n_experts, L = map.n_local;
  for (int i = tid; i < kRounds * 4 * kMaxExperts; i += 256) (&s_mask[0][0])[i] = 0ull;
  for (int e = tid; e < E; e += 256) s_slot_of[e] = map.slot_of[e];
  __syncthreads();

  auto slot_of = [&](int t, int j) {
    const int e = ids[(size_t)t * k + j];
    return ((unsigned)e < (unsigned)E) ? (int)s_slot_of[e] : -1;
  };
  for (int rd = 0; rd < kRounds; ++rd) {
    const int t = blockIdx.x * kTokPerBlk + rd * 256 + tid;
    if (t < T)
      for (int j = 0; j < k; ++j) {
        const int s = slot_of(t, j);
        if (s >= 0) atomicOr(&s_mask[rd * 4 + wave][s], 1ull << lane);
      }
  }
  __syncthreads();
  if (tid < L) {
    int run = 0;
    for (int q = 0; q < kRounds * 4; ++q) {
      s_pre[q][tid] = run;
      run += __popcll(s_mask[q][tid]);
    }
  }
  __syncthreads();
  const unsigned long long below = (1ull << lane) - 1ull;
  for (int rd = 0; rd < kRounds; ++rd) {
    const int t = blockIdx.x * kTokPerBlk + rd * 256 + tid;
    if (t >= T) break;
    const int q = rd * 4 + wave;
    for (int j = 0; j < k; ++j) {
      const int s = slot_of(t, j);
      int pos = -1;
      if (s >= 0) {
        pos = bases[(size_t)blockIdx.x * L + s] + s_pre[q][s] + __popcll(s_mask[q][s] & below);
        if (pos < 0 || pos >= M_cap) pos = -1;
      }
      dest[(size_t)t * k + j] = pos;
      if (pos >= 0) perm_src[pos] = t * k + j;
    }
  }
}

// Dispatch permutation, step 2: x_perm[pos] = x[perm_src[pos] / k] for
// pos < offsets[E_local]. One wave per row, 16-byte vectors, eight (then
// four) loads in flight per lane before the stores.
__global__ __launch_bounds__(256) void gather_rows_kernel(const uint4* __restrict__ x, int row_vecs, int T, int k,
                                                          const int32_t* __restrict__ perm_src,
                                                          const int32_t* __restrict__ m_loc, int M_cap,
                                                          uint4* __restrict__ x_perm) {
  constexpr int U = 8;
  const int lane = threadIdx.x & 63;
  const int m = min(max(*m_loc, 0), M_cap);
  const int waves = gridDim.x * 4;
  for (int pos = blockIdx.x * 4 + (threadIdx.x >> 6); pos < m; pos += waves) {
    const int tok = perm_src[pos] / k;
    if ((unsigned)tok >= (unsigned)T) continue;
    const uint4* src = x + (size_t)tok * row_vecs;
    uint4* dst = x_perm + (size_t)pos * row_vecs;
    int v0 = 0;
    for (; v0 + U * kWave <= row_vecs; v0 += U * kWave) {
      uint4 buf[U];
#pragma unroll
      for (int u = 0; u < U; ++u) buf[u] = src[v0 + u * kWave + lane];
#pragma unroll
      for (int u = 0; u < U; ++u) dst[v0 + u * kWave + lane] = buf[u];
    }
    if (v0 + (U / 2) * kWave <= row_vecs) {  // half a batch (rows of 2048 bf16, row tails)
      uint4 buf[U / 2];
#pragma unroll
      for (int u = 0; u < U / 2; ++u) buf[u] = src[v0 + u * kWave + lane];
#pragma unroll
      for (int u = 0; u < U / 2; ++u) dst[v0 + u * kWave + lane] = buf[u];
      v0 += (U / 2) * kWave;
    }
    for (int v = v0 + lane; v < row_vecs; v += kWave) dst[v] = src[v];
  }
}

// ---------------------------------------------------------------------------
// Combine: one wave per token, 16-byte vectors along H, fp32 accumulation in
// ascending slot order (no contraction, so each step rounds like the
// definition: a product, then a sum).
// ---------------------------------------------------------------------------
constexpr int kCombineVecs = 4;  // 16-byte row vectors per lane and slot in flight

__global__ __launch_bounds__(256) void combine_bf16_kernel(const uint4* __restrict__ y, const float* __restrict__ w,
                                                           const int32_t* __restrict__ dest, int T, int k,
                                                           int row_vecs, int M_cap, uint4* __restrict__ out) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int d[kMaxTopk];
  float wt[kMaxTopk];
#pragma unroll
  for (int j = 0; j < kMaxTopk; ++j) {
    d[j] = -1;
    wt[j] = 0.0f;
    if (j < k) {
      const int dj = dest[(size_t)t * k + j];
      d[j] = (dj >= 0 && dj < M_cap) ? dj : -1;
      wt[j] = w[(size_t)t * k + j];
    }
  }
  // each lane keeps kCombineVecs row vectors (kWave apart) of every slot in
  // flight; slots are still summed in ascending order per element
  for (int v0 = lane; v0 < row_vecs; v0 += kCombineVecs * kWave) {
    float acc[kCombineVecs][8];
#pragma unroll
    for (int u = 0; u < kCombineVecs; ++u)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[u][q] = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxTopk; ++j) {
      if (j < k && d[j] >= 0) {
        uint4 yv[kCombineVecs];
#pragma unroll
        for (int u = 0; u < kCombineVecs; ++u) {
          const int v = v0 + u * kWave;
          yv[u] = v < row_vecs ? y[(size_t)d[j] * row_vecs + v] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < kCombineVecs; ++u) {
          const uint32_t w4[4] = {yv[u].x, yv[u].y, yv[u].z, yv[u].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float lo = __uint_as_float(w4[q] << 16);
            const float hi = __uint_as_float(w4[q] & 0xffff0000u);
            const float plo = wt[j] * lo;
            const float phi = wt[j] * hi;
            acc[u][2 * q] = acc[u][2 * q] + plo;
            acc[u][2 * q + 1] = acc[u][2 * q + 1] + phi;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kCombineVecs; ++u) {
      const int v = v0 + u * kWave;
      if (v < row_vecs) {
        uint4 o;
        o.x = pack_bf16x2(acc[u][0], acc[u][1]);
        o.y = pack_bf16x2(acc[u][2], acc[u][3]);
        o.z = pack_bf16x2(acc[u][4], acc[u][5]);
        o.w = pack_bf16x2(acc[u][6], acc[u][7]);
        out[(size_t)t * row_vecs + v] = o;
      }
    }
  }
}

__global__ __launch_bounds__(256) void combine_f32_kernel(const float4* __restrict__ y, const float* __restrict__ w,
                                                          const int32_t* __restrict__ dest, int T, int k,
                                                          int row_vecs, int M_cap, float4* __restrict__ out) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  for (int v = lane; v < row_vecs; v += kWave) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < k; ++j) {
      const int dj = dest[(size_t)t * k + j];
      if (dj < 0 || dj >= M_cap) continue;
      const float wj = w[(size_t)t * k + j];
      const float4 yv = y[(size_t)dj * row_vecs + v];
      const float px = wj * yv.x, py = wj * yv.y, pz = wj * yv.z, pw = wj * yv.w;
      acc.x = acc.x + px;
      acc.y = acc.y + py;
      acc.z = acc.z + pz;
      acc.w = acc.w + pw;
    }
    out[(size_t)t * row_vecs + v] = acc;
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called from the C ABI after validation).
// ---------------------------------------------------------------------------
// ---------------------------------------------------------------------------
// Router top-k over K-split logits (router_logits_split_kernel): one wave per
// token; lane g sums its columns q * 64 + g over the S slices in split order,
// adds the bias and the wave selects as the other router kernels do. S is a
// template argument, so all NV x S loads of a wave are issued, unconditionally,
// before the first sum (same-process A/B, DSV3-shaped router at T = 16384:
// 141 -> 138 us, bitwise the same ids and weights).
// ---------------------------------------------------------------------------
constexpr int kMaxRouterSplit = 8;  // K ranges of the split routers, at most

// Partial rows are EP floats apart (E <= EP <= 64 NV); 1 <= S <= 8.
template <int NV, int S>
__global__ __launch_bounds__(256) void gate_topk_reduce_kernel(const float* __restrict__ part, int T, int E, int EP,
                                                               int k, const float* __restrict__ bias,
                                                               float* __restrict__ logits, int32_t* __restrict__ ids,
                                                               float* __restrict__ wts) {
  static_assert(S >= 1 && S <= kMaxRouterSplit, "slices");
  const int lane = threadIdx.x & 63;
  const int row = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (row >= T) return;  // wave-uniform
  // every slice's load in flight at once (columns past E read column E - 1),
  // then the sums in split order
  float p[NV][S];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    const int col = min(q * 64 + lane, E - 1);
#pragma unroll
    for (int sp = 0; sp < S; ++sp) p[q][sp] = part[((size_t)sp * T + row) * EP + col];
  }
  float val[NV];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    const int col = q * 64 + lane;
    float v = p[q][0];
#pragma unroll
    for (int sp = 1; sp < S; ++sp) v = v + p[q][sp];
    v = v + (bias != nullptr && col < E ? bias[col] : 0.0f);
    val[q] = col < E ? v : -__builtin_huge_valf();
  }
  if (logits != nullptr) {
#pragma unroll
    for (int q = 0; q < NV; ++q)
      if (q * 64 + lane < E) logits[(size_t)row * E + q * 64 + lane] = val[q];
  }
  float sel_v[kMaxTopk];
  int sel_i[kMaxTopk];
  topk_group<64, NV>(val, lane, E, k, sel_v, sel_i);
  write_topk(sel_v, sel_i, lane, k, row, ids, wts);
}

// The same pass for 256-column partial rows (E = 256): 16 lanes per token,
// four tokens per wave, lane g of a token holding columns [16 g, 16 g + 16)
// (four 16-byte loads per slice). A selection round then takes a 16-value
// scan in the lane and four DPP steps in its row instead of six steps over
// the whole wave for every token. Same sums in the same order, same
// selection order (value descending, then column ascending), same weights
// (same-process A/B, DSV3-shaped router at T = 16384: 138 -> 132 us).
template <int S>
__global__ __launch_bounds__(256) void gate_topk_reduce16_kernel(const float* __restrict__ part, int T, int E,
                                                                 int k, const float* __restrict__ bias,
                                                                 float* __restrict__ logits,
                                                                 int32_t* __restrict__ ids, float* __restrict__ wts) {
  static_assert(S >= 1 && S <= kMaxRouterSplit, "slices");
  constexpr int EP = 256;
  const int lane = threadIdx.x & 63, g = lane & 15;
  const int row = ((int)blockIdx.x * 4 + (int)(threadIdx.x >> 6)) * 4 + (lane >> 4);
  const bool live = row < T;
  const int rr = live ? row : T - 1;  // every lane takes part in the DPP steps
  float p[S][16];
#pragma unroll
  for (int sp = 0; sp < S; ++sp) {
    const float4* src = reinterpret_cast<const float4*>(part + ((size_t)sp * T + rr) * EP + 16 * g);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 f = src[q];
      p[sp][4 * q] = f.x;
      p[sp][4 * q + 1] = f.y;
      p[sp][4 * q + 2] = f.z;
      p[sp][4 * q + 3] = f.w;
    }
  }
  float v[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const int col = 16 * g + c;
    float x = p[0][c];
#pragma unroll
    for (int sp = 1; sp < S; ++sp) x = x + p[sp][c];
    x = x + (bias != nullptr && col < E ? bias[col] : 0.0f);
    v[c] = col < E ? x : -__builtin_huge_valf();
  }
  if (logits != nullptr && live) {
#pragma unroll
    for (int c = 0; c < 16; ++c)
      if (16 * g + c < E) logits[(size_t)row * E + 16 * g + c] = v[c];
  }
  float sel_v[kMaxTopk];
  int sel_i[kMaxTopk];
  uint32_t taken = 0;
#pragma unroll
  for (int j = 0; j < kMaxTopk; ++j) {
    if (j < k) {
      float lv = -__builtin_huge_valf();
      int li = 0x7fffffff;
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const int col = 16 * g + c;
        if (!((taken >> c) & 1u) && better(v[c], col, lv, li)) {
          lv = v[c];
          li = col;
        }
      }
      best_dpp<0x111, 0xf>(lv, li);  // row_shr:1
      best_dpp<0x112, 0xf>(lv, li);  // row_shr:2
      best_dpp<0x114, 0xf>(lv, li);  // row_shr:4
      best_dpp<0x118, 0xf>(lv, li);  // row_shr:8: lane 15 of each row holds the row's best
      float rv[4];
      int ri[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        rv[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lv), 16 * q + 15));
        ri[q] = __builtin_amdgcn_readlane(li, 16 * q + 15);
      }
      const int r4 = lane >> 4;
      lv = r4 == 0 ? rv[0] : (r4 == 1 ? rv[1] : (r4 == 2 ? rv[2] : rv[3]));
      li = r4 == 0 ? ri[0] : (r4 == 1 ? ri[1] : (r4 == 2 ? ri[2] : ri[3]));
      sel_v[j] = lv;
      sel_i[j] = li;
      if ((li >> 4) == g) taken |= 1u << (li & 15);
    }
  }
  if (live) write_topk(sel_v, sel_i, g, k, row, ids, wts);
}

template <int NV>
static void launch_topk_reduce(const float* part, int S, int T, int E, int EP, int k, const float* bias,
                               float* logits, int32_t* ids, float* wts, dim3 grid, hipStream_t s) {
  if (NV == 4 && EP == 256) {
    // 16 lanes per token: 16 tokens per 256-thread block
    const dim3 g16((unsigned)((T + 15) / 16));
#define MOE_TOPK_REDUCE16(N)                                                                           \
  case N:                                                                                              \
    gate_topk_reduce16_kernel<N><<<g16, 256, 0, s>>>(part, T, E, k, bias, logits, ids, wts); \
    return;
    switch (S) {
      MOE_TOPK_REDUCE16(1)
      MOE_TOPK_REDUCE16(2)
      MOE_TOPK_REDUCE16(3)
      MOE_TOPK_REDUCE16(4)
      MOE_TOPK_REDUCE16(5)
      MOE_TOPK_REDUCE16(6)
      MOE_TOPK_REDUCE16(7)
      MOE_TOPK_REDUCE16(8)
      default:
        return;
    }
#undef MOE_TOPK_REDUCE16
  }
#define MOE_TOPK_REDUCE(N)                                                                               \
  case N:                                                                                                \
    gate_topk_reduce_kernel<NV, N><<<grid, 256, 0, s>>>(part, T, E, EP, k, bias, logits, ids, wts); \
    break;
  switch (S) {
    MOE_TOPK_REDUCE(1)
    MOE_TOPK_REDUCE(2)
    MOE_TOPK_REDUCE(3)
    MOE_TOPK_REDUCE(4)
    MOE_TOPK_REDUCE(5)
    MOE_TOPK_REDUCE(6)
    MOE_TOPK_REDUCE(7)
    MOE_TOPK_REDUCE(8)
    default:
      break;  // S is 1..8 (router_split_factor, router_small_split_factor)
  }
#undef MOE_TOPK_REDUCE
}

// Compute units of the current device (256 if the runtime cannot say).
static int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
  return n;
}

// Batches the split router takes for E = 128: up to kRouterSplitMaxT128
// tokens for rows shorter than 4096 elements; for longer rows every batch
// whose 128-token blocks would fill at most half the CUs, where the one-pass
// kernel leaves CUs idle. Measured with the last-level cache flushed before
// each call, H = 5120: 8192 tokens 56 us split vs 83 one pass, 12000 tokens
// 69 vs 92, 16384 tokens 90 vs 95, but 32768 tokens (256 blocks) 151 vs
// 141; H = 2048: 8192 tokens 46 vs 46, 16384 tokens 69 vs 64. At E = 256 the
// one-pass kernel re-reads all 256 router rows per 64 tokens, so the split
// router takes every batch.
constexpr int kRouterSplitMaxT128 = 4096;
constexpr size_t kRouterSplitMaxBytes = 256ull << 20;  // partial logits at most

// K ranges of the split router for T tokens (0: not used). E = 128 or 256
// (bf16); S fills the CUs with 256-token tiles, each range >= 4 K chunks,
// the partials within kRouterSplitMaxBytes.
static int router_split_factor(int T, int H, int E) {
  if ((E != 128 && E != 256) || T < 1 || H % kGateBK != 0) return 0;
  if (E == 128 && (H >= 4096 ? 2LL * ((T + 127) / 128) > device_cus() : T > kRouterSplitMaxT128)) return 0;
  const long long tiles = (T + 255) / 256;
  const int nK = H / kGateBK;
  long long S = device_cus() / tiles;
  S = S < 1 ? 1 : (S > 8 ? 8 : S);
  while (S > 1 && (nK / S < 4 || (size_t)S * T * E * 4 > kRouterSplitMaxBytes)) --S;
  if ((size_t)S * T * E * 4 > kRouterSplitMaxBytes || nK < (int)S) return 0;
  return (int)S;
}

// Decode-sized batches over at most 128 experts: the small-batch kernel
// (8 waves, one k-step per load group) on S K ranges of H / 16 / S k-steps,
// a multiple of 16 (two per wave and group); 0: not used. Below
// kRouterSmallSplitMinBytes of distinct rows per 32-token block the second
// launch costs more than it saves (one token over 8 experts at H = 4096:
// 11.9 us in one pass, 16.6 us split).
// Larger batches over at most 64 experts whose 32-token blocks would leave
// at least half the CUs idle take the fewest K ranges that give every CU a
// block (same-process A/B, 8 experts at H = 4096, ids the same bits:
// 1024 tokens 21.3 -> 14.6 us, 2048 tokens 21.9 -> 17.4 us; at 4096 tokens,
// 128 blocks, one pass stays faster, 24.9 vs 28.0 us). The 128- and
// 256-expert shapes have the 256-token split router instead.
constexpr int kRouterSmallSplitMaxT = 256;
constexpr long long kRouterSmallSplitMinBytes = 192 << 10;
static int router_small_split_factor(int T, int H, int E) {
  if (E > 128 || T < 1 || H % 16 != 0) return 0;
  const int nks = H / 16;
  if (T <= kRouterSmallSplitMaxT) {
    if ((long long)(std::min(T, 32) + E) * H * 2 < kRouterSmallSplitMinBytes) return 0;
    for (int S = 8; S >= 2; --S)
      if (nks % S == 0 && (nks / S) % 16 == 0) return S;
    return 0;
  }
  const int blocks = (T + 31) / 32, cus = device_cus();
  if (E > 64 || T > kSmallRouterT || 2 * blocks > cus) return 0;
  for (int S = 2; S <= 8; ++S)
    if (nks % S == 0 && (nks / S) % 16 == 0 && (long long)blocks * S >= cus) return S;
  return 0;
}

size_t gate_ws_bytes(int T, int H, int E, bool bf16) {
  if (!bf16 || T < 1) return 0;
  const int Ss = router_small_split_factor(T, H, E);
  if (Ss > 0) return (((size_t)Ss * T * 32 * ((E + 31) / 32) * 4 + 255) / 256) * 256;
  const int S = router_split_factor(T, H, E);
  return S > 0 ? (((size_t)S * T * E * 4 + 255) / 256) * 256 : 0;
}

hipError_t launch_gate_topk(const void* x, const void* wr, const float* bias, int T, int H, int E, int k,
                            bool bf16, float* logits, int32_t* ids, float* wts, void* ws, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (!bf16) {
    gate_topk_f32_kernel<<<(T + 3) / 4, 256, 0, s>>>(static_cast<const float*>(x),
                                                     static_cast<const float*>(wr), bias, T, H, E, k,
                                                     logits, ids, wts);
    return hipGetLastError();
  }
  const int ncb = (E + 31) / 32;
  const bf16_t* xb = static_cast<const bf16_t*>(x);
  const bf16_t* wb = static_cast<const bf16_t*>(wr);
  // Many tokens over 128 or 256 experts, with a workspace: logits by K
  // ranges, then the top-k pass.
  if (ws != nullptr) {
    float* part = static_cast<float*>(ws);
    const dim3 g4((unsigned)((T + 3) / 4));
    const int Ss = router_small_split_factor(T, H, E);
    if (Ss > 0) {
      // decode-sized batch: 32-token blocks x Ss K ranges
      const dim3 g((unsigned)((T + 31) / 32), (unsigned)Ss);
      const int ep = 32 * ncb;
#define MOE_GATE_SMALL_SPLIT(N)                                                                         \
  case N:                                                                                               \
    gate_topk_bf16_small_kernel<N, 8, 1><<<g, 512, 0, s>>>(xb, wb, bias, T, H, E, k, logits, ids, wts, Ss, \
                                                           part);                                       \
    break;
      switch (ncb) {
        MOE_GATE_SMALL_SPLIT(1)
        MOE_GATE_SMALL_SPLIT(2)
        MOE_GATE_SMALL_SPLIT(3)
        MOE_GATE_SMALL_SPLIT(4)
        default:
          return hipErrorInvalidValue;
      }
#undef MOE_GATE_SMALL_SPLIT
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      if (ep <= 64)
        launch_topk_reduce<1>(part, Ss, T, E, ep, k, bias, logits, ids, wts, g4, s);
      else
        launch_topk_reduce<2>(part, Ss, T, E, ep, k, bias, logits, ids, wts, g4, s);
      return hipGetLastError();
    }
    const int S = router_split_factor(T, H, E);
    if (S > 0) {
      hipError_t e = launch_router_logits_split(xb, wb, T, H, E, S, part, s);
      if (e != hipSuccess) return e;
      if (E == 256)
        launch_topk_reduce<4>(part, S, T, E, E, k, bias, logits, ids, wts, g4, s);
      else
        launch_topk_reduce<2>(part, S, T, E, E, k, bias, logits, ids, wts, g4, s);
      return hipGetLastError();
    }
  }
  // Small batches of few experts: 32-token blocks whose waves stream
  // contiguous shares of the K range (NW waves, GK k-steps per load group).
  if (ncb <= 4 && T <= kSmallRouterT) {
    const dim3 g32((T + 31) / 32);
    const int nks = H / 16;
#define MOE_GATE_SMALL(N, NW, GK)                                                                     \
  case N:                                                                                           \
    if (nks % (NW * 2 * GK) != 0) break;                                                            \
    gate_topk_bf16_small_kernel<N, NW, GK><<<g32, NW * 64, 0, s>>>(xb, wb, bias, T, H, E, k, logits, \
                                                                    ids, wts);                       \
    return hipGetLastError();
    switch (ncb) {
      MOE_GATE_SMALL(1, 16, 4)
      MOE_GATE_SMALL(2, 8, 4)
      MOE_GATE_SMALL(3, 8, 2)
      MOE_GATE_SMALL(4, 8, 2)
      default:
        break;
    }
#undef MOE_GATE_SMALL
  }
  // Few experts and fewer than 256 blocks of 128 tokens: 32-token blocks with
  // the K range split over the waves, so more CUs stream x.
  if (ncb <= 4 && (T + 127) / 128 < 256) {
    const dim3 g32((T + 31) / 32);
#define MOE_GATE_KSPLIT(N)                                                                            \
  case N:                                                                                             \
    gate_topk_bf16_ksplit_kernel<N><<<g32, 256, 0, s>>>(xb, wb, bias, T, H, E, k, logits, ids, wts); \
    break;
    switch (ncb) {
      MOE_GATE_KSPLIT(1)
      MOE_GATE_KSPLIT(2)
      MOE_GATE_KSPLIT(3)
      MOE_GATE_KSPLIT(4)
      default:
        return hipErrorInvalidValue;
    }
#undef MOE_GATE_KSPLIT
    return hipGetLastError();
  }
  // More than 32 experts: 8-wave blocks of 64 tokens (E_pad of 128 or 256)
  // when they have each CU load fewer rows than 128-token blocks.
  if (ncb > 1) {
    const int cus = device_cus();
    const int ep = ncb <= 4 ? 128 : 256;
    auto rows_per_cu = [&](int bt) {
      const long long blocks = (T + bt - 1) / bt;
      return ((blocks + cus - 1) / cus) * (long long)(ep + bt);
    };
    if (rows_per_cu(64) < rows_per_cu(128)) {
      const dim3 g((T + 63) / 64);
      if (ncb <= 4)
        gate_topk_bf16_wide_kernel<64, 4><<<g, 512, 0, s>>>(xb, wb, bias, T, H, E, k, logits, ids, wts);
      else
        gate_topk_bf16_wide_kernel<64, 8><<<g, 512, 0, s>>>(xb, wb, bias, T, H, E, k, logits, ids, wts);
      return hipGetLastError();
    }
  }
  const dim3 grid((T + 127) / 128);
#define MOE_GATE_CASE(N)                                                                        \
  case N:                                                                                       \
    gate_topk_bf16_kernel<N><<<grid, 256, 0, s>>>(xb, wb, bias, T, H, E, k, logits, ids, wts); \
    break;
  switch (ncb) {
    MOE_GATE_CASE(1)
    MOE_GATE_CASE(2)
    MOE_GATE_CASE(3)
    MOE_GATE_CASE(4)
    MOE_GATE_CASE(5)
    MOE_GATE_CASE(6)
    MOE_GATE_CASE(7)
    MOE_GATE_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef MOE_GATE_CASE
  return hipGetLastError();
}

size_t hist_ws_bytes(int T, int E, int E_local) {
  const size_t n_blk = (size_t)(T + kTokPerBlk - 1) / kTokPerBlk;
  const size_t table = n_blk * E * sizeof(int32_t);
  const size_t bases = n_blk * E_local * sizeof(int32_t);
  return ((table + 255) / 256) * 256 + ((bases + 255) / 256) * 256 + 256;
}

// Workspace: count table [n_blk][E] | row bases [n_blk][E_local] | local total.
static void hist_ws_split(void* ws, int T, int E, int E_local, int32_t** table, int32_t** bases,
                          int32_t** m_loc) {
  const size_t n_blk = (size_t)(T + kTokPerBlk - 1) / kTokPerBlk;
  const size_t tb = ((n_blk * E * sizeof(int32_t) + 255) / 256) * 256;
  const size_t bb = ((n_blk * E_local * sizeof(int32_t) + 255) / 256) * 256;
  *table = static_cast<int32_t*>(ws);
  *bases = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + tb);
  *m_loc = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + tb + bb);
}

hipError_t launch_hist_scan(const int32_t* ids, int T, int k, const SlotMap& map, int32_t* counts,
                            int32_t* offsets, void* ws, hipStream_t s) {
  const int n_blk = (T + kTokPerBlk - 1) / kTokPerBlk;
  int32_t *table, *bases, *m_loc;
  hist_ws_split(ws, T, map.n_experts, map.n_local, &table, &bases, &m_loc);
  if (n_blk == 1) {
    hist_scan_one_block_kernel<<<1, 256, 0, s>>>(ids, T, k, map, counts, offsets, bases, m_loc);
    return hipGetLastError();
  }
  if (n_blk > 0) {
    hist_kernel<<<n_blk, 256, 0, s>>>(ids, T, k, map.n_experts, table);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if ((long long)n_blk * map.n_experts <= kScanLdsInts)
    scan_lds_kernel<<<1, 256, 0, s>>>(table, n_blk, map, counts, offsets, bases, m_loc);
  else
    scan_kernel<<<1, 256, 0, s>>>(table, n_blk, map, counts, offsets, bases, m_loc);
  return hipGetLastError();
}

hipError_t launch_permute(const void* x, const int32_t* ids, const SlotMap& map, const void* ws, int T, int H,
                          int k, int M_cap, bool bf16, void* x_perm, int32_t* perm_src, int32_t* dest,
                          hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int n_blk = (T + kTokPerBlk - 1) / kTokPerBlk;
  int32_t *table, *bases, *m_loc;
  hist_ws_split(const_cast<void*>(ws), T, map.n_experts, map.n_local, &table, &bases, &m_loc);
  permute_index_kernel<<<n_blk, 256, 0, s>>>(ids, T, k, map, bases, M_cap, perm_src, dest);
  hipError_t e = hipGetLastError();
  // x_perm == nullptr: positions only (the FFN gathers the rows itself)
  if (e != hipSuccess || map.n_local == 0 || M_cap == 0 || x_perm == nullptr) return e;
  const int row_vecs = (H * (bf16 ? 2 : 4)) / 16;
  const int cus = device_cus();
  const long long want = ((long long)M_cap + 3) / 4;
  const unsigned grid = (unsigned)std::min<long long>(want, (long long)cus * 8);
  gather_rows_kernel<<<grid, 256, 0, s>>>(static_cast<const uint4*>(x), row_vecs, T, k, perm_src, m_loc, M_cap,
                                          static_cast<uint4*>(x_perm));
  return hipGetLastError();
}

hipError_t launch_combine(const void* y, const float* w, const int32_t* dest, int T, int k, int H, int M_cap,
                          bool bf16, void* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const dim3 grid((T + 3) / 4);
  if (bf16) {
    combine_bf16_kernel<<<grid, 256, 0, s>>>(static_cast<const uint4*>(y), w, dest, T, k, H / 8, M_cap,
                                             static_cast<uint4*>(out));
  } else {
    combine_f32_kernel<<<grid, 256, 0, s>>>(static_cast<const float4*>(y), w, dest, T, k, H / 4, M_cap,
                                            static_cast<float4*>(out));
  }
  return hipGetLastError();
}

}  // namespace moe
