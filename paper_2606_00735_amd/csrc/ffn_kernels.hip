// Grouped SwiGLU expert FFN (gfx950): the expert computation whose latency
// per token load is ViBE's per-GPU performance model f_g(n) (Section 4.2.1).
//
// Two persistent launches per call:
//   gate/up:  h[R] = bf16( silu(X_R W_gate^T) * (X_R W_up^T) )   (dual GEMM)
//   down:     y[R] = bf16( h[R] W_down^T )
// for each local expert's row range R = [offsets[e], offsets[e+1]), each
// followed by a small reduction that finishes split-K tiles (it returns at
// once when the GEMM split nothing).
//
// Per-expert row counts live only on the device, so each block rebuilds the
// tile list from `offsets` (a scan over at most 256 experts) and walks it
// with a grid stride. Rows are cut into 256-row tiles plus one 64-, 128- or
// 256-row remainder tile (row_tiles, tile_class). Within an expert,
// consecutive tile indices share a weight column block, so blocks running at
// the same time read the same weights.
#include <algorithm>
#include <mutex>

#include "common.hpp"
#include "launch.hpp"
#include "mx.hpp"

namespace moe {

constexpr int kBK = 64;  // K chunk per pipeline stage (128-byte tile rows)

// Blocks of 8 waves (two per SIMD, so one wave's LDS waits are covered by
// the other's MFMAs). Tile classes (see row_tiles):
//   small   64 x 128 tiles, waves 2x4   (weight streaming at small M_e)
//   mid    128 x 128 tiles, waves 2x4
//   large  256 x 128 tiles, waves 4x2   (MFMA bound)
// with 128 output columns per matrix (gate and up both, in the dual GEMM).
// K advances in 64-wide chunks (whole 128-byte cache lines per tile row);
// each class keeps as many chunks in flight as 144 KB of LDS allows
// (Stages below).
constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kSmallM = 64;
constexpr int kDmaRows = kWaves * 1024 / (2 * kBK);  // rows one DMA round of all waves covers

template <int BM, int BN, bool DUAL>
struct Stages {
  static constexpr int NB = DUAL ? 2 : 1;
  static constexpr int AROWS = BM > kDmaRows ? BM : kDmaRows;  // A rows loaded per stage
  static constexpr int ROWS = AROWS + NB * BN;
  static constexpr int ELEMS = ROWS * kBK;
  static constexpr int FIT = (144 * 1024) / (ELEMS * 2);  // stages that fit in 144 KB of LDS
  static constexpr int NS = FIT < 2 ? 2 : (FIT > 8 ? 8 : FIT);
  static constexpr int BYTES = ELEMS * 2 * NS;
  static constexpr int LOADS = ROWS / kDmaRows;  // DMA instructions per wave per chunk
};

struct GemmArgs {
  const bf16_t* A;        // [M_cap, K]
  const bf16_t* B0;       // [E_local, N, K]
  const bf16_t* B1;       // [E_local, N, K] (dual only)
  bf16_t* C;              // [M_cap, N]
  const int32_t* offsets; // [E_local + 1]
  int E_local, M_cap, N, K;
  // Split-K workspace (see the kernel): fp32 partials (part_cap floats) and
  // the plan the reduction reads. part == nullptr disables split-K.
  float* part;
  long long part_cap;
  int32_t* plan;
  int plan_rows;  // rows the plan's row map holds
  // MXFP8 GEMMs (grouped_gemm_mx_kernel): A, B0, B1 hold E4M3 codes (K bytes
  // a row, moved as pairs of bf16 slots), As [K/128][M_cap] and
  // Bs0/Bs1 [E_local][K/128][N] their scale dwords (mx.hpp); the dual GEMM
  // writes E4M3 codes of h to C and their scale dwords to Cs [N/128][M_cap].
  const uint32_t* As;
  const uint32_t* Bs0;
  const uint32_t* Bs1;
  uint32_t* Cs;
  // Per-XCD work counters (8 ints, zero before the launch) or nullptr for
  // the static tile order.
  int32_t* queue;
  // Row gather (bf16 GEMMs): when a_src != nullptr, row m of the A operand
  // is row clamp(a_src[m] / a_div, 0, a_T - 1) of A (A holds a_T rows and
  // a_T * K * 2 < 2^32), so the gate/up GEMM reads the routed tokens of x
  // directly instead of a permuted copy.
  const int32_t* a_src;
  int a_div, a_T;
  // Row stride of B0/B1 in the units of K (elements for bf16, bytes for
  // MXFP8 codes), >= K; expert e's matrix starts at row e * N. A stride off
  // a power of two spreads a tile's rows over more HBM channels.
  int ldb;
  // Counter of finished blocks for the reset of the work counters (zero
  // before the launch; the last block to finish zeroes it and the queue), or
  // nullptr.
  int32_t* done;
  // Decode schedule (bf16; see decode_schedule): with sk != 0 a launch in
  // which every expert has at most sk_rows rows takes it; skpart
  // holds two fp32 slots of NB x sk_rows x 128 floats per block, tcnt one
  // arrival counter per block (zero before the launch; left zero).
  // no_reduce != 0: no reduction launch follows this one.
  int sk;
  int sk_rows;
  float* skpart;
  int32_t* tcnt;
  int no_reduce;
  // Result of the XCD check (see xcd_probe_kernel; 1: block b of a launch
  // runs on XCD b % 8), or nullptr. The decode schedule reads it to choose
  // L2-local partial sums; results do not depend on it.
  const int32_t* xcd_state;
};

// Split-K plan written by block 0 of a grouped GEMM for split_reduce_kernel:
// plan[0] = S (1: nothing was split), plan[1] = R (rows of split experts),
// plan[kPlanHead + j] = row of C that compact row j belongs to.
constexpr int kPlanHead = 64;
constexpr int kMaxSplit = 8;
constexpr int kMinSplitChunks = 8;   // K chunks per split, at least
constexpr int kSplitOverhead = 4;    // per-tile cost of a split tile, in K chunks (fill, epilogue, reduce)
constexpr long long kPartCapFloats = 16ll << 20;  // 64 MB of fp32 partials at most

__device__ __forceinline__ float silu_mul(float g, float u) {
  const float sig = 1.0f / (1.0f + expf(-g));
  return (g * sig) * u;
}

// SiLU(g) * u for the bf16 path: exp2 and reciprocal on the hardware
// transcendental unit (v_exp_f32, v_rcp_f32; about 1 ulp of fp32 each), far
// below the bf16 rounding of h that follows. exp(-g) = exp2(-g * log2 e).
__device__ __forceinline__ float silu_mul_fast(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-g * 1.4426950408889634f);
  const float sig = __builtin_amdgcn_rcpf(1.0f + e);
  return (g * sig) * u;
}

// Split-K epilogue shared by the bf16 and MXFP8 tiles: the fp32 sums of
// output (r, c) of matrix b (r, c within the tile) go to
// pbase[b * pstride + r * ld + col0 + c]; each lane writes its 4 consecutive
// columns per group as one 16-byte store.
// 16-byte stores and loads at agent scope, as two 64-bit relaxed atomic
// accesses (gfx950 gives them the sc1 cache policy): the store writes through
// to the device's point of coherence and the load reads from it, so a block
// on another XCD sees the data within the same launch once the store has
// completed. They are ordinary instructions to the compiler, which tracks
// their completion.
__device__ __forceinline__ void st_coh4(float* p, f32x4_t v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  const uint64_t lo = (uint64_t)__float_as_uint(v[0]) | ((uint64_t)__float_as_uint(v[1]) << 32);
  const uint64_t hi = (uint64_t)__float_as_uint(v[2]) | ((uint64_t)__float_as_uint(v[3]) << 32);
  __hip_atomic_store(q, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ f32x4_t ld_coh4(const float* p) {
  const uint64_t* q = reinterpret_cast<const uint64_t*>(p);
  const uint64_t lo = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t hi = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return f32x4_t{__uint_as_float((uint32_t)lo), __uint_as_float((uint32_t)(lo >> 32)),
                 __uint_as_float((uint32_t)hi), __uint_as_float((uint32_t)(hi >> 32))};
}

// COH: the sums are for another block to read in the same launch (see
// decode_schedule) and the stores have completed on return; coh: stored with
// st_coh4, for a block on another XCD, else with ordinary stores, which a
// block on the same XCD reads from their shared L2.
template <int MI, int NI, int NB, int WM, int WN, bool COH = false>
__device__ __forceinline__ void split_epilogue(const f32x16_t (&acc)[NB][MI][NI], int m0, int m_end, int col0,
                                               int ld, int wm, int wn, int lane, float* pbase, size_t pstride,
                                               bool coh) {
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int r = wm * WM + i * 32 + (lane & 31);  // row within the tile
    if (m0 + r < m_end) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        float* prow = pbase + b * pstride + (size_t)r * ld + col0 + wn * WN + 4 * (lane >> 5);
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float* p = prow + j * 32 + 8 * g;
            if (COH && coh) {
              st_coh4(p, f32x4_t{acc[b][i][j][4 * g], acc[b][i][j][4 * g + 1], acc[b][i][j][4 * g + 2],
                                 acc[b][i][j][4 * g + 3]});
            } else {
              *reinterpret_cast<float4*>(p) = make_float4(acc[b][i][j][4 * g], acc[b][i][j][4 * g + 1],
                                                          acc[b][i][j][4 * g + 2], acc[b][i][j][4 * g + 3]);
            }
          }
      }
    }
  }
  if (COH) wait_vmcnt<0>();
}

// One BM x BN output tile (two of them, gate and up, when DUAL) over the whole
// K range: 8 waves, 32x32x16 bf16 MFMA, operands loaded straight from global
// memory into NS swizzled LDS stages (see pipeline_xk).
// SPLIT: only K chunks [kc0, kc1) are summed and the fp32 sums of output
// (r, c) (r: row within the tile, c: column within the tile) go to
// pbase[b * pstride + r * pld + pcol0 + c] instead of C.
template <int BM, int BN, int WAVES_M, bool DUAL, bool SPLIT = false, bool COH = false>
__device__ __forceinline__ void gemm_tile(const GemmArgs& a, bf16_t* smem, int e, int m0, int m_end, int n0,
                                          int kc0 = 0, int kc1 = -1, float* pbase = nullptr,
                                          size_t pstride = 0, int pld = 0, int pcol0 = 0, bool coh = true) {
  using St = Stages<BM, BN, DUAL>;
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WAVES_N = kWaves / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int MI = WM / 32, NI = WN / 32;
  constexpr int AR = St::AROWS;
  static_assert(MI >= 1 && NI >= 1, "wave tile");

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int K = a.K, N = a.N;
  const bool gather = a.a_src != nullptr;
  const bf16_t* A = gather ? a.A : a.A + (size_t)m0 * K;
  const int a_rows = m_end - m0;
  const int LDB = a.ldb;
  const bf16_t* B0 = a.B0 + ((size_t)e * N + n0) * LDB;
  const bf16_t* B1 = DUAL ? a.B1 + ((size_t)e * N + n0) * LDB : nullptr;

  f32x16_t acc[NB][MI][NI];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[b][i][j] = f32x16_t{};

  // Loop-invariant byte offsets of this lane's 16-byte pieces (dma16s; the
  // chunk's column goes into the wave-uniform base): instruction t of wave w
  // moves rows [8 (t kWaves + w), +8), lane l row l / 8, piece l % 8 of the
  // swizzled row; A rows past the tile re-read its last row. Both weight
  // matrices share offsets. A placeholder load (live == false) reads the
  // first 16 bytes of the chunk in every lane.
  constexpr int RPI = 8, LA = AR / (RPI * kWaves), LB = BN / (RPI * kWaves);
  static_assert(AR % (RPI * kWaves) == 0 && BN % (RPI * kWaves) == 0, "rows per wave");
  uint32_t offA[LA], offB[LB];
#pragma unroll
  for (int t = 0; t < LA; ++t) {
    const int r = (t * kWaves + wave) * RPI + lane / 8;
    int rr = r < a_rows ? r : a_rows - 1;
    if (gather) rr = min(max(a.a_src[m0 + rr] / a.a_div, 0), a.a_T - 1);
    offA[t] = (uint32_t)rr * (uint32_t)(K * 2) + (uint32_t)(swz_chunk<kBK>(r, lane % 8) * 16);
  }
#pragma unroll
  for (int t = 0; t < LB; ++t) {
    const int r = (t * kWaves + wave) * RPI + lane / 8;
    offB[t] = (uint32_t)(r * LDB * 2 + swz_chunk<kBK>(r, lane % 8) * 16);
  }
  if (kc1 < 0) kc1 = K / kBK;
  auto issue = [&](int kc, bool live, bf16_t* st) {
    const size_t col = (size_t)(live ? kc0 + kc : kc0) * kBK;
    const void* pa = uniform_ptr(A + col);
#pragma unroll
    for (int t = 0; t < LA; ++t) dma16s(pa, live ? offA[t] : 0u, st + (t * kWaves + wave) * RPI * kBK);
    const void* pb0 = uniform_ptr(B0 + col);
#pragma unroll
    for (int t = 0; t < LB; ++t) dma16s(pb0, live ? offB[t] : 0u, st + (AR + (t * kWaves + wave) * RPI) * kBK);
    if (DUAL) {
      const void* pb1 = uniform_ptr(B1 + col);
#pragma unroll
      for (int t = 0; t < LB; ++t)
        dma16s(pb1, live ? offB[t] : 0u, st + (AR + BN + (t * kWaves + wave) * RPI) * kBK);
    }
  };
  // Operands of k-step s+1 are read from LDS while the MFMAs of k-step s
  // run (register double buffering), across chunks too (pipeline_xk).
  bf16x8_t af[2][MI], bfr[2][NB][NI];
  auto read = [&](const bf16_t* st, int s, int buf) {
    const int chunk = 2 * s + (lane >> 5);
#pragma unroll
    for (int i = 0; i < MI; ++i) af[buf][i] = lds_frag<kBK>(st, wm * WM + i * 32 + (lane & 31), chunk);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < NI; ++j)
        bfr[buf][b][j] = lds_frag<kBK>(st + (AR + b * BN) * kBK, wn * WN + j * 32 + (lane & 31), chunk);
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int i = 0; i < MI; ++i)
          acc[b][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[buf][b][j], af[buf][i], acc[b][i][j], 0, 0, 0);
  };
  // issue order within a k-step: one MFMA, one LDS read, ...
  auto mix = [&]() {
    constexpr int NREAD = MI + NB * NI, NMFMA = NB * MI * NI;
    constexpr int PAIRS = NREAD < NMFMA ? NREAD : NMFMA;
#pragma unroll
    for (int q = 0; q < PAIRS; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
    if (NMFMA > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, NMFMA - PAIRS, 0);
    if (NREAD > PAIRS) __builtin_amdgcn_sched_group_barrier(0x100, NREAD - PAIRS, 0);
  };
  pipeline_xk<St::NS, St::LOADS, kBK / 16>(kc1 - kc0, smem, St::ELEMS, issue, read, mma, mix);

  // Epilogue. The MFMAs computed transposed 32x32 blocks (weights as the A
  // operand): register v of lane l holds output column 8 * (v / 4) +
  // 4 * (l / 32) + (v % 4) of the block for row (token) l % 32, so each lane
  // owns 4 consecutive columns per group g = v / 4 and stores them as one
  // 8-byte write (or, for a split-K partial, one 16-byte fp32 write).
  if (SPLIT) {
    split_epilogue<MI, NI, NB, WM, WN, COH>(acc, m0, m_end, pcol0, pld, wm, wn, lane, pbase, pstride, coh);
    return;
  }
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int row = m0 + wm * WM + i * 32 + (lane & 31);
    if (row < m_end) {
      bf16_t* crow = a.C + (size_t)row * N + n0 + wn * WN + 4 * (lane >> 5);
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float r[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int v = 4 * g + q;
            r[q] = DUAL ? silu_mul_fast(acc[0][i][j][v], acc[NB - 1][i][j][v]) : acc[0][i][j][v];
          }
          uint2 packed;
          packed.x = pack_bf16x2(r[0], r[1]);
          packed.y = pack_bf16x2(r[2], r[3]);
          *reinterpret_cast<uint2*>(crow + j * 32 + 8 * g) = packed;
        }
    }
  }
}

// MXFP8 stages: the same 128-byte tile rows as the bf16 path (a K chunk is
// 128 E4M3 codes), plus one scale dword per operand row. Every wave loads 64
// scale rows per chunk (one global_load_lds_dword), so a stage holds
// kWaves * 64 = 512 scale rows whatever its operand rows.
template <int BM, int BN, bool DUAL>
struct MxStages {
  static constexpr int NB = DUAL ? 2 : 1;
  static constexpr int AROWS = BM > kDmaRows ? BM : kDmaRows;
  static constexpr int ROWS = AROWS + NB * BN;
  static_assert(ROWS <= kWaves * 64, "one scale dword per operand row");
  static constexpr int SCALE_OFF = ROWS * 2 * kBK;          // bytes
  static constexpr int STAGE = SCALE_OFF + kWaves * 64 * 4;  // bytes
  static constexpr int FIT = (152 * 1024) / STAGE;
  static constexpr int NS = FIT < 2 ? 2 : (FIT > 8 ? 8 : FIT);
  static constexpr int BYTES = STAGE * NS;
  static constexpr int LOADS = ROWS / kDmaRows + 1;  // code rows, then the scale dword
};

__device__ __forceinline__ uint4 lds16(const bf16_t* lds, int row, int chunk) {
  return *reinterpret_cast<const uint4*>(lds + row * kBK + swz_chunk<kBK>(row, chunk) * 8);
}

// One BM x BN MXFP8 tile (two when DUAL) over the whole K range, as
// gemm_tile but with the scaled MFMA v_mfma_scale_f32_32x32x64_f8f6f4: a
// k-step is 64 K, two per chunk. Lane l (row l % 32, h = l / 32) supplies
// K elements [16 h, 16 h + 16) and [32 + 16 h, 48 + 16 h) of the k-step (16-byte
// chunks 4 s + h and 4 s + 2 + h of k-step s) and the scale code of 32-block h,
// i.e. byte 2 s + h of its row's scale dword; the instruction reads the code
// from the low byte of the scale operand.
// DUAL: h = SiLU(gate) * up is quantised per 32 columns (the 32 values of a
// row and block sit in lanes l and l ^ 32) and written as E4M3 codes with their
// scale dwords; otherwise C is written as bf16.
// SPLIT: only K chunks [kc0, kc1) are summed, the fp32 sums written as in
// gemm_tile.
template <int BM, int BN, int WAVES_M, bool DUAL, bool SPLIT = false, bool COH = false>
__device__ __forceinline__ void gemm_tile_mx(const GemmArgs& a, bf16_t* smem, int e, int m0, int m_end, int n0,
                                             int kc0 = 0, int kc1 = -1, float* pbase = nullptr,
                                             size_t pstride = 0, int pld = 0, int pcol0 = 0, bool coh = true) {
  using St = MxStages<BM, BN, DUAL>;
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WAVES_N = kWaves / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int MI = WM / 32, NI = WN / 32;
  constexpr int AR = St::AROWS;
  static_assert(MI >= 1 && NI >= 1, "wave tile");

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int h = lane >> 5, r32 = lane & 31;
  const int K = a.K, N = a.N, nK = K / kMxChunk;  // K: bytes of an operand row
  const int a_rows = m_end - m0;
  const char* A = reinterpret_cast<const char*>(a.A) + (size_t)m0 * K;
  const int LDB = a.ldb;  // bytes
  const char* B0 = reinterpret_cast<const char*>(a.B0) + ((size_t)e * N + n0) * LDB;
  const char* B1 = DUAL ? reinterpret_cast<const char*>(a.B1) + ((size_t)e * N + n0) * LDB : nullptr;

  // Loop-invariant byte offsets of this lane's 16-byte pieces, as in
  // gemm_tile (the rows of a chunk are 128 codes here).
  constexpr int RPI = 8, LA = AR / (RPI * kWaves), LB = BN / (RPI * kWaves);
  uint32_t offA[LA], offB[LB];
#pragma unroll
  for (int t = 0; t < LA; ++t) {
    const int r = (t * kWaves + wave) * RPI + lane / 8;
    const int rr = r < a_rows ? r : a_rows - 1;
    offA[t] = (uint32_t)(rr * K + swz_chunk<kBK>(r, lane % 8) * 16);
  }
#pragma unroll
  for (int t = 0; t < LB; ++t) {
    const int r = (t * kWaves + wave) * RPI + lane / 8;
    offB[t] = (uint32_t)(r * LDB + swz_chunk<kBK>(r, lane % 8) * 16);
  }
  // Scale rows: wave w loads scale rows [64 w, 64 w + 64) of the stage, all
  // in one operand (AR and BN are multiples of 64): A rows (clamped), the
  // gate (or only) weight rows, the up weight rows, or a placeholder that
  // re-reads A's first row.
  const int q0 = wave * 64;
  const char* sb_base;
  size_t s_stride;  // bytes per K chunk
  uint32_t soff;
  if (q0 < AR) {
    sb_base = reinterpret_cast<const char*>(a.As + m0);
    s_stride = (size_t)a.M_cap * 4;
    soff = (uint32_t)(min(q0 + lane, a_rows - 1) * 4);
  } else if (q0 < AR + BN) {
    sb_base = reinterpret_cast<const char*>(a.Bs0 + (size_t)e * nK * N + n0 + (q0 - AR));
    s_stride = (size_t)N * 4;
    soff = (uint32_t)(lane * 4);
  } else if (DUAL && q0 < AR + 2 * BN) {
    sb_base = reinterpret_cast<const char*>(a.Bs1 + (size_t)e * nK * N + n0 + (q0 - AR - BN));
    s_stride = (size_t)N * 4;
    soff = (uint32_t)(lane * 4);
  } else {
    sb_base = reinterpret_cast<const char*>(a.As + m0);
    s_stride = (size_t)a.M_cap * 4;
    soff = 0;
  }

  f32x16_t acc[NB][MI][NI];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[b][i][j] = f32x16_t{};

  // A placeholder load (live == false) re-reads the last chunk, which is in
  // the cache by then, so loads never leave the operands.
  if (kc1 < 0) kc1 = nK;
  auto issue = [&](int kc, bool live, bf16_t* st) {
    const int kcl = live ? kc0 + kc : kc1 - 1;
    char* sl = reinterpret_cast<char*>(st);
    const void* pa = uniform_ptr(A + (size_t)kcl * kMxChunk);
#pragma unroll
    for (int t = 0; t < LA; ++t) dma16s(pa, offA[t], sl + (t * kWaves + wave) * RPI * 128);
    const void* pb0 = uniform_ptr(B0 + (size_t)kcl * kMxChunk);
#pragma unroll
    for (int t = 0; t < LB; ++t) dma16s(pb0, offB[t], sl + (AR + (t * kWaves + wave) * RPI) * 128);
    if (DUAL) {
      const void* pb1 = uniform_ptr(B1 + (size_t)kcl * kMxChunk);
#pragma unroll
      for (int t = 0; t < LB; ++t) dma16s(pb1, offB[t], sl + (AR + BN + (t * kWaves + wave) * RPI) * 128);
    }
    dma4s(uniform_ptr(sb_base + (size_t)kcl * s_stride), soff, sl + St::SCALE_OFF + wave * 256);
  };
  // A fragments (and scales) are double buffered; a weight fragment is
  // refilled for the next k-step once its MI MFMAs of this k-step are issued
  // (pipeline_xk with MMA_FIRST), which keeps the tile within 256 VGPRs.
  int32x8_t af[2][MI], bfr[NB][NI];
  uint32_t sa[2][MI], sb[NB][NI];
  auto frag = [&](const bf16_t* t, int row, int s) {
    const uint4 lo = lds16(t, row, 4 * s + h), hi = lds16(t, row, 4 * s + 2 + h);
    return int32x8_t{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
  };
  auto read = [&](const bf16_t* st, int s, int buf) {
    const uint32_t* sc = reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(st) + St::SCALE_OFF);
    const int sh = 8 * (2 * s + h);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      const int row = wm * WM + i * 32 + r32;
      af[buf][i] = frag(st, row, s);
      sa[buf][i] = sc[row] >> sh;
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int row = wn * WN + j * 32 + r32;
        bfr[b][j] = frag(st + (AR + b * BN) * kBK, row, s);
        sb[b][j] = sc[AR + b * BN + row] >> sh;
      }
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int i = 0; i < MI; ++i)
          acc[b][i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              bfr[b][j], af[buf][i], acc[b][i][j], 0, 0, 0, (int)sb[b][j], 0, (int)sa[buf][i]);
  };
  auto mix = [&]() {
    constexpr int NREAD = 3 * (MI + NB * NI), NMFMA = NB * MI * NI;
    constexpr int PAIRS = NREAD < NMFMA ? NREAD : NMFMA;
#pragma unroll
    for (int p = 0; p < PAIRS; ++p) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
    }
    if (NMFMA > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, NMFMA - PAIRS, 0);
    if (NREAD > PAIRS) __builtin_amdgcn_sched_group_barrier(0x100, NREAD - PAIRS, 0);
  };
  pipeline_xk<St::NS, St::LOADS, kMxChunk / 64, true>(kc1 - kc0, smem, St::STAGE / 2, issue, read, mma, mix);

  if (SPLIT) {
    split_epilogue<MI, NI, NB, WM, WN, COH>(acc, m0, m_end, pcol0, pld, wm, wn, lane, pbase, pstride, coh);
    return;
  }

  // Epilogue: output layout as in gemm_tile (lane l: row l % 32, columns
  // 8 g + 4 h + (0..3) of each 32-column block).
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int row = m0 + wm * WM + i * 32 + r32;
    const bool ok = row < m_end;  // the same for lanes l and l ^ 32
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int col0 = n0 + wn * WN + j * 32;
      if (DUAL) {
        float r[16];
        float amax = 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          r[v] = silu_mul_fast(acc[0][i][j][v], acc[NB - 1][i][j][v]);
          amax = fmaxf(amax, fabsf(r[v]));
        }
        amax = fmaxf(amax, __shfl_xor(amax, 32, kWave));
        const uint32_t code = mx_scale_code(amax);
        const float inv = mx_inv_scale(code);
        if (ok) {
          uint8_t* crow = reinterpret_cast<uint8_t*>(a.C) + (size_t)row * N + col0 + 4 * h;
#pragma unroll
          for (int g = 0; g < 4; ++g)
            *reinterpret_cast<uint32_t*>(crow + 8 * g) =
                e4m3x4(r[4 * g] * inv, r[4 * g + 1] * inv, r[4 * g + 2] * inv, r[4 * g + 3] * inv);
          if (h == 0)
            reinterpret_cast<uint8_t*>(a.Cs + (size_t)(col0 / kMxChunk) * a.M_cap + row)[(col0 / kMxBlock) & 3] =
                static_cast<uint8_t>(code);
        }
      } else if (ok) {
        bf16_t* crow = a.C + (size_t)row * N + col0 + 4 * h;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint2 packed;
          packed.x = pack_bf16x2(acc[0][i][j][4 * g], acc[0][i][j][4 * g + 1]);
          packed.y = pack_bf16x2(acc[0][i][j][4 * g + 2], acc[0][i][j][4 * g + 3]);
          *reinterpret_cast<uint2*>(crow + 8 * g) = packed;
        }
      }
    }
  }
}

template <bool DUAL>
struct GemmShapes {
  // dual: 128 columns per matrix; single: 128 or 256 columns (see the kernel)
  static constexpr int BNW = DUAL ? 128 : 256;
  static constexpr int b0 = Stages<64, BNW, DUAL>::BYTES, b1 = Stages<128, BNW, DUAL>::BYTES;
  static constexpr int b2 = Stages<256, BNW, DUAL>::BYTES, b3 = Stages<256, 128, DUAL>::BYTES;
  static constexpr int m01 = b0 > b1 ? b0 : b1, m23 = b2 > b3 ? b2 : b3;
  static constexpr int kSmem = (m01 > m23 ? m01 : m23) / 2;  // bf16 elements
};

// An expert's rows are cut into 256-row tiles; the last one is a 64-, 128- or
// 256-row tile, whichever is the smallest that holds the remainder (a
// 300-row expert: one 256-row tile and one 64-row tile). A ragged tail then
// wastes at most part of its own class's tile.
__device__ __forceinline__ int row_tiles(int rows) { return (rows + 255) / 256; }
__device__ __forceinline__ int tile_class(int left) { return left > 128 ? 2 : (left > kSmallM ? 1 : 0); }

// Persistent grouped GEMM over every local expert. The grid is a multiple of
// 8 and block b runs on XCD b % 8; in each round of gridDim.x tiles, the
// blocks of one XCD take consecutive logical tiles. The logical order walks
// each expert's row tiles fastest, so the row tiles that share a weight
// column block run at the same time on one XCD: every weight byte comes from
// HBM about once, and the rows (a few hundred MB at most) come from the
// last-level cache.
//
// Split-K. When every expert has at most 64 rows (decode, or one lightly
// loaded expert) the cost is streaming the weights, and a launch with fewer
// tiles than blocks leaves CUs idle (a few experts of a few hundred rows, as
// in the middle of the load sweep). In both cases each tile may be cut into
// S K ranges whose fp32 sums go to the workspace (rows numbered compactly in
// expert order); split_reduce_kernel adds the S partials of each output in a
// fixed order (so results do not depend on timing) and applies the
// epilogue. S in 1..8 minimises rounds(S) * (chunks per split + a fixed
// per-tile cost), each split keeping at least kMinSplitChunks K chunks, and
// only if the partials fit and their bytes stay below the weight bytes the
// launch streams. Every block sees the same offsets, so every block makes
// the same choice.
// Inclusive sum over the lanes of a wave by DPP (a few cycles a step, where
// lane shuffles through LDS take about a hundred): Hillis-Steele within each
// row of 16 lanes (row_shr 1, 2, 4, 8; lanes shifted in from outside the row
// add 0), then lane 15 of rows 0 and 2 added to rows 1 and 3 (row_bcast:15),
// then lane 31 to rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2, 3
  return x;
}

template <int NV>
__device__ __forceinline__ void block_scan(int (&v)[NV], int (&excl)[NV], int (&total)[NV], int (*s_tot)[kWaves]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int inc[NV];
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    inc[q] = wave_incl_scan(v[q]);
    if (lane == 63) s_tot[q][wave] = inc[q];
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NV; ++q) {
    int base = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < wave) base += s_tot[q][w];
      tot += s_tot[q][w];
    }
    excl[q] = base + inc[q] - v[q];
    total[q] = tot;
  }
}

template <bool DUAL>
struct MxShapes {
  static constexpr int BNW = DUAL ? 128 : 256;
  static constexpr int b0 = MxStages<64, BNW, DUAL>::BYTES, b1 = MxStages<128, BNW, DUAL>::BYTES;
  static constexpr int b2 = MxStages<256, BNW, DUAL>::BYTES, b3 = MxStages<256, 128, DUAL>::BYTES;
  static constexpr int b4 = MxStages<64, 128, DUAL>::BYTES, b5 = MxStages<128, 128, DUAL>::BYTES;
  static constexpr int m01 = b0 > b1 ? b0 : b1, m23 = b2 > b3 ? b2 : b3, m45 = b4 > b5 ? b4 : b5;
  static constexpr int m = m01 > m23 ? m01 : m23;
  static constexpr int kSmem = (m > m45 ? m : m45) / 2;  // bf16 slots
};

// One row tile of an unsplit launch: 128 or (single GEMM, wide) 256 columns.
template <bool DUAL, bool MX, bool WIDE>
__device__ __forceinline__ void run_tile(const GemmArgs& a, bf16_t* smem, int cls, int e, int m0, int m_end,
                                         int n0) {
  constexpr int BN = WIDE ? 256 : 128;
  if constexpr (MX) {
    if (cls == 0)
      gemm_tile_mx<64, BN, 2, DUAL>(a, smem, e, m0, m_end, n0);
    else if (cls == 1)
      gemm_tile_mx<128, BN, 2, DUAL>(a, smem, e, m0, m_end, n0);
    else
      gemm_tile_mx<256, BN, 4, DUAL>(a, smem, e, m0, m_end, n0);
  } else {
    if (cls == 0)
      gemm_tile<64, BN, 2, DUAL>(a, smem, e, m0, m_end, n0);
    else if (cls == 1)
      gemm_tile<128, BN, 2, DUAL>(a, smem, e, m0, m_end, n0);
    else
      gemm_tile<256, BN, 4, DUAL>(a, smem, e, m0, m_end, n0);
  }
}

// One split-K tile of BN columns (128, or 256 for a wide single GEMM): K
// chunks [kc0, kc1), fp32 sums to pbase (row stride pld, column base pcol0).
template <bool DUAL, bool MX, int BN, bool COH = false>
__device__ __forceinline__ void run_split_tile(const GemmArgs& a, bf16_t* smem, int cls, int e, int m0, int m_end,
                                               int n0, int kc0, int kc1, float* pbase, size_t ps, int pld,
                                               int pcol0, bool coh = true) {
  if constexpr (MX && COH) {
    // decode schedule: at most kSkRows rows a tile
    if (cls == 0)
      gemm_tile_mx<64, BN, 2, DUAL, true, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0, coh);
    else
      gemm_tile_mx<128, BN, 2, DUAL, true, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0, coh);
  } else if constexpr (MX) {
    if (cls == 0)
      gemm_tile_mx<64, BN, 2, DUAL, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0);
    else if (cls == 1)
      gemm_tile_mx<128, BN, 2, DUAL, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0);
    else
      gemm_tile_mx<256, BN, 4, DUAL, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0);
  } else if constexpr (COH) {
    // decode schedule: at most kSkRows rows a tile
    if (cls == 0)
      gemm_tile<64, BN, 2, DUAL, true, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0, coh);
    else
      gemm_tile<128, BN, 2, DUAL, true, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0, coh);
  } else {
    if (cls == 0)
      gemm_tile<64, BN, 2, DUAL, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0);
    else if (cls == 1)
      gemm_tile<128, BN, 2, DUAL, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0);
    else
      gemm_tile<256, BN, 4, DUAL, true>(a, smem, e, m0, m_end, n0, kc0, kc1, pbase, ps, pld, pcol0);
  }
}

// Tile `tile` of the unsplit schedule (tiles of `cols` columns): its expert,
// rows [m0, m_end) and first column.
struct TileRef {
  int e, m0, m_end, n0, left;
};

// Order of one expert's tiles (n_mt row tiles x n_nt column tiles): bands of
// up to kBand row tiles; in a band the row tiles of a column block are
// consecutive, then the next column block. An XCD runs 32 consecutive tiles
// at a time, which for an expert with many row tiles is then 8 column
// blocks x 4 row tiles (12 operand tiles per K chunk in its L2) instead of,
// e.g., 3 column blocks x 12 row tiles (15).
constexpr int kBand = 4;
__device__ __forceinline__ void tile_rc(int local, int n_mt, int n_nt, int& mt, int& nt) {
  const int full = n_mt / kBand, per_band = kBand * n_nt;
  const int b = local / per_band;
  if (b < full) {
    const int l2 = local - b * per_band;
    nt = l2 / kBand;
    mt = b * kBand + (l2 - nt * kBand);
  } else {
    const int rb = n_mt - full * kBand, l2 = local - full * per_band;
    nt = l2 / rb;
    mt = full * kBand + (l2 - nt * rb);
  }
}

__device__ __forceinline__ TileRef decode_tile(int tile, int E, const int* s_start, const int* s_row0,
                                               const int* s_rows, int cols, int N) {
  // last expert whose first tile is <= tile (experts with no tiles share
  // their start with the next one, so the last match is the owner)
  int lo = 0, hi = E - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_start[mid] <= tile) lo = mid; else hi = mid - 1;
  }
  TileRef t;
  t.e = lo;
  const int local = tile - s_start[lo];
  const int er = s_rows[lo];
  int nt, mt;
  tile_rc(local, row_tiles(er), N / cols, mt, nt);
  t.m0 = s_row0[lo] + mt * 256;
  t.left = er - mt * 256;  // rows from m0 to the expert's end, >= 1
  t.m_end = t.m0 + (t.left < 256 ? t.left : 256);
  t.n0 = nt * cols;
  return t;
}

// Four h values of columns [c, c + 4) of `row`, quantised with the other 28
// of their 32-column block, which the 7 other lanes of this lane's aligned
// group of 8 hold; the group's first lane writes the scale code.
__device__ __forceinline__ void mx_quant_store4(float h0, float h1, float h2, float h3, int row, int c, int N,
                                                int M_cap, uint8_t* C8, uint32_t* Cs) {
  float amax = fmaxf(fmaxf(fabsf(h0), fabsf(h1)), fmaxf(fabsf(h2), fabsf(h3)));
  amax = fmaxf(amax, __shfl_xor(amax, 1, kWave));
  amax = fmaxf(amax, __shfl_xor(amax, 2, kWave));
  amax = fmaxf(amax, __shfl_xor(amax, 4, kWave));
  const uint32_t code = mx_scale_code(amax);
  const float inv = mx_inv_scale(code);
  *reinterpret_cast<uint32_t*>(C8 + (size_t)row * N + c) = e4m3x4(h0 * inv, h1 * inv, h2 * inv, h3 * inv);
  if ((c & (kMxBlock - 1)) == 0)
    reinterpret_cast<uint8_t*>(Cs + (size_t)(c / kMxChunk) * M_cap + row)[(c / kMxBlock) & 3] =
        static_cast<uint8_t>(code);
}

// ---------------------------------------------------------------------------
// Decode schedule (launches in which no expert exceeds sk_rows rows:
// decode-sized batches and lightly loaded experts; bf16 and MXFP8). The work
// is streaming the active experts' weights, and a launch often has fewer
// tiles than CUs or a partly filled last round, so instead of whole tiles
// each block takes an exact, contiguous share of the launch's
// (tile, K chunk) units (stream-K): tile t's chunks are units
// [t nK, t nK + nK), tiles in the order of decode_tile. Blocks are numbered
// XCD by XCD (bo), so consecutive shares sit on one XCD. Two partitions:
//  * per XCD: the tiles are first dealt to the 8 XCDs in contiguous ranges
//    cut at tile boundaries, then each XCD's units to its blocks, so all
//    blocks sharing a tile share one L2;
//  * global: the units of the launch are cut among all blocks.
// The per-XCD partition is used when its largest share is at most one unit
// above the global one's (the tile count divides evenly over the XCDs, or
// the shares are bounded by kSkMinChunks rather than by the blocks).
// A tile whose chunks fall into the shares of several blocks is finished by
// the last of them to arrive: each writes its fp32 sums to a slot of its own,
// waits for the stores to complete, and increments the counter of the tile's
// first block; the block that sees the final count adds the slots in block
// order (a fixed order, so results do not depend on timing), applies the
// epilogue and resets the counter. No block ever waits for another. The
// slots go through the XCD's L2 (ordinary stores and loads) when the
// partition is per XCD and the XCD check confirmed that block b runs on XCD
// b % 8; otherwise through the device's point of coherence (st_coh4 /
// ld_coh4). Which of the two does not change a bit of the results.
// ---------------------------------------------------------------------------
constexpr int kSkMinChunks = 2;  // K chunks per block share, at least (when the launch has as many)
// Largest expert for which the decode schedule is preferred when a
// reduction launch follows anyway (same-process A/B, one to eight
// Mixtral-shaped experts: faster up to 13-16 rows, 3-10 % slower at 29-32).
constexpr int kSkPrefRows = 16;
// floor(n / d) for 0 <= n, 0 < d: 32-bit division when n fits (the GPU has
// no integer divider; a 64-bit division costs several times a 32-bit one)
__device__ __forceinline__ long long sk_div(long long n, long long d) {
  if (((unsigned long long)n | (unsigned long long)d) < (1ULL << 32)) return (long long)((uint32_t)n / (uint32_t)d);
  return n / d;
}
// Units [u0, u0 + U) shared by blocks [b0, b0 + Ga) (share order).
struct SkPart {
  long long U, Ga, u0;
  int b0;
  // first unit of block bo's share
  __device__ long long start(int bo) const { return u0 + sk_div(U * (bo - b0), Ga); }
  // the block whose share holds unit x
  __device__ int block_of(long long x) const { return b0 + (int)(sk_div((x - u0 + 1) * Ga + U - 1, U) - 1); }
};
__device__ __forceinline__ long long sk_blocks(long long U, long long G) {
  return max(1LL, min(G, U / kSkMinChunks));  // every block with work takes >= kSkMinChunks
}

// Sum of the nc contributors' slots of a split tile (rows [m0, m_end) of C,
// columns [n0, n0 + cols): cols = 128 per matrix, or 256 for a single GEMM's
// wide tile) in contributor order, the epilogue, and bf16 (or MXFP8 h)
// stores; every thread of the block takes 4 columns of a row at a time and
// loads the slots of up to kFixBatch contributors before waiting for them.
// coh: the slots were written with st_coh4, else with ordinary stores on
// this block's XCD. A slot holds NB planes of sk_rows x cols floats
// (2 x 128 or 1 x 256 columns: the same size).
constexpr int kFixBatch = 8;
template <bool DUAL, bool MX>
__device__ __forceinline__ void sk_fixup(const GemmArgs& a, int m0, int m_end, int n0, int cols, int bf, int nc,
                                         int j0, bool coh) {
  constexpr int NB = DUAL ? 2 : 1;
  const size_t plane = (size_t)a.sk_rows * cols, slot_f = NB * plane;
  const int c4 = cols / 4;  // items per row
  const int items = (m_end - m0) * c4;
  // the CU's L1 holds no line of these slots from before their stores (each
  // slot is written and read once a launch); invalidate it all the same
  if (!coh) asm volatile("buffer_inv sc0" ::: "memory");
  for (int it = (int)threadIdx.x; it < items; it += kThreads) {
    const int r = it / c4, c = (it - r * c4) * 4;
    const float* p0 = a.skpart + (size_t)r * cols + c;
    f32x4_t g = f32x4_t{}, u = f32x4_t{};
    for (int q0 = 0; q0 < nc; q0 += kFixBatch) {
      f32x4_t vg[kFixBatch], vu[kFixBatch];
#pragma unroll
      for (int j = 0; j < kFixBatch; ++j) {
        const int q = q0 + j < nc ? q0 + j : nc - 1;  // past the last contributor: a repeated, unused load
        const float* p = p0 + ((size_t)(bf + q) * 2 + (q == 0 ? j0 : 0)) * slot_f;
        if (coh) {
          vg[j] = ld_coh4(p);
          if (DUAL) vu[j] = ld_coh4(p + plane);
        } else {
          vg[j] = *reinterpret_cast<const f32x4_t*>(p);
          if (DUAL) vu[j] = *reinterpret_cast<const f32x4_t*>(p + plane);
        }
      }
#pragma unroll
      for (int j = 0; j < kFixBatch; ++j)
        if (q0 + j < nc) {
          g += vg[j];
          if (DUAL) u += vu[j];
        }
    }
    float o[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) o[v] = DUAL ? silu_mul_fast(g[v], u[v]) : g[v];
    if (MX && DUAL) {
      // h as MXFP8: the aligned 8 lanes around this one hold one 32-column
      // block of the row (items come in whole rows of 32 lanes)
      mx_quant_store4(o[0], o[1], o[2], o[3], m0 + r, n0 + c, a.N, a.M_cap, reinterpret_cast<uint8_t*>(a.C), a.Cs);
    } else {
      uint2 packed;
      packed.x = pack_bf16x2(o[0], o[1]);
      packed.y = pack_bf16x2(o[2], o[3]);
      *reinterpret_cast<uint2*>(a.C + (size_t)(m0 + r) * a.N + n0 + c) = packed;
    }
  }
}

// xcd_ok: the XCD check's result (1: block b runs on XCD b % 8). wide: a
// single GEMM in 256-column tiles (T0 and s_start count those tiles), which
// halves the tiles, and so the pipeline fills, of short-K launches.
template <bool DUAL, bool MX>
__device__ __forceinline__ void decode_schedule(const GemmArgs& a, bf16_t* smem, int T0, const int* s_start,
                                                const int* s_row0, const int* s_rows, bool xcd_ok, bool wide) {
  constexpr int NB = DUAL ? 2 : 1;
  const int cols = wide ? 256 : 128;
  __shared__ int s_last;
  const int G = gridDim.x, b = blockIdx.x;
  const bool g8 = (G & 7) == 0;
  const int gx = G >> 3;  // blocks per XCD
  const int bo = g8 ? (b & 7) * gx + (b >> 3) : b;
  const int nK = a.K / (MX ? kMxChunk : kBK);
  // T0 * 8 stays far inside int: T0 <= E_local * N / 128 here
  SkPart P;
  P.U = (long long)T0 * nK;
  P.Ga = sk_blocks(P.U, G);
  P.u0 = 0;
  P.b0 = 0;
  // per XCD when the tiles divide evenly over the XCDs (shares then differ
  // from the global ones by at most a unit), else when the largest share
  // grows by at most one unit (in float: a heuristic, and every block computes
  // the same values, so every block takes the same decision)
  bool per_xcd = g8 && (T0 & 7) == 0;
  if (g8 && !per_xcd) {
    float big = 0.0f;
    for (int x = 0; x < 8; ++x) {
      const long long ux = (long long)((T0 * (x + 1) >> 3) - (T0 * x >> 3)) * nK;
      if (ux > 0) big = fmaxf(big, ceilf((float)ux / (float)sk_blocks(ux, gx)));
    }
    per_xcd = big <= ceilf((float)P.U / (float)P.Ga) + 1.0f;
  }
  if (per_xcd) {
    const int x = b & 7;
    const long long t_lo = T0 * x >> 3, t_hi = T0 * (x + 1) >> 3;
    P.U = (t_hi - t_lo) * nK;
    P.Ga = sk_blocks(P.U, gx);
    P.u0 = t_lo * nK;
    P.b0 = x * gx;
  }
  const bool coh = !(per_xcd && xcd_ok);
  if (P.U == 0 || bo - P.b0 >= P.Ga) return;
  const long long u_beg = P.start(bo), u_end = P.start(bo + 1);
  const size_t plane = (size_t)a.sk_rows * cols, slot_f = NB * plane;
  for (long long u = u_beg; u < u_end;) {
    const int t = (int)sk_div(u, nK);
    const int kc0 = (int)(u - (long long)t * nK);
    const int kc1 = (int)min((long long)nK, kc0 + (u_end - u));
    const TileRef tr = decode_tile(t, a.E_local, s_start, s_row0, s_rows, cols, a.N);
    const int cls = tile_class(tr.left);
    if (kc0 == 0 && kc1 == nK) {
      if constexpr (!DUAL) {
        if (wide)
          run_tile<DUAL, MX, true>(a, smem, cls, tr.e, tr.m0, tr.m_end, tr.n0);
        else
          run_tile<DUAL, MX, false>(a, smem, cls, tr.e, tr.m0, tr.m_end, tr.n0);
      } else {
        run_tile<DUAL, MX, false>(a, smem, cls, tr.e, tr.m0, tr.m_end, tr.n0);
      }
    } else {
      const long long t0 = (long long)t * nK;
      const int bf = P.block_of(t0);
      const int nc = P.block_of(t0 + nK - 1) - bf + 1;
      const int j0 = P.start(bf) == t0 ? 0 : 1;
      float* mine = a.skpart + ((size_t)bo * 2 + (u == u_beg ? 0 : 1)) * slot_f;
      if constexpr (!DUAL) {
        if (wide)
          run_split_tile<DUAL, MX, 256, true>(a, smem, cls, tr.e, tr.m0, tr.m_end, tr.n0, kc0, kc1, mine, plane,
                                              256, 0, coh);
        else
          run_split_tile<DUAL, MX, 128, true>(a, smem, cls, tr.e, tr.m0, tr.m_end, tr.n0, kc0, kc1, mine, plane,
                                              128, 0, coh);
      } else {
        run_split_tile<DUAL, MX, 128, true>(a, smem, cls, tr.e, tr.m0, tr.m_end, tr.n0, kc0, kc1, mine, plane, 128,
                                            0, coh);
      }
      __syncthreads();  // every wave's stores have completed
      if (threadIdx.x == 0) s_last = atomicAdd(a.tcnt + bf, 1) == nc - 1;
      __syncthreads();
      if (s_last) {
        sk_fixup<DUAL, MX>(a, tr.m0, tr.m_end, tr.n0, cols, bf, nc, j0, coh);
        if (threadIdx.x == 0) __hip_atomic_store(a.tcnt + bf, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    u += kc1 - kc0;
  }
}

// Body of the grouped GEMM kernels (bf16 or MXFP8; a K chunk is 64 bf16 or
// 128 E4M3 elements, 128 bytes of a row either way).
template <bool DUAL, bool MX>
__device__ __forceinline__ void grouped_gemm_body(const GemmArgs& a) {
  constexpr int kSmem = MX ? MxShapes<DUAL>::kSmem : GemmShapes<DUAL>::kSmem;
  constexpr int NB = DUAL ? 2 : 1;
  __shared__ __align__(16) bf16_t smem[kSmem];
  __shared__ int s_start[kMaxExperts + 1];
  __shared__ int s_row0[kMaxExperts];
  __shared__ int s_rows[kMaxExperts];
  __shared__ int s_srow0[kMaxExperts];
  __shared__ int s_tot[6][kWaves];

  const int tid = threadIdx.x;
  const int E = a.E_local, G = gridDim.x;
  __shared__ int s_xcd;
  // the XCD check's result, loaded early (its latency overlaps the scan);
  // an ordinary load: the result only ever changes from 0 (none yet, read
  // as "not confirmed") to its final value, so a stale copy is safe
  int xcd = 0;
  if (a.sk && a.xcd_state != nullptr && tid == 0) xcd = *a.xcd_state;

  // Rows of each expert, clamped so no access leaves [0, M_cap).
  int rows = 0;
  if (tid < E) {
    int o0 = a.offsets[tid], o1 = a.offsets[tid + 1];
    o0 = min(max(o0, 0), a.M_cap);
    o1 = min(max(o1, o0), a.M_cap);
    rows = o1 - o0;
    s_row0[tid] = o0;
    s_rows[tid] = rows;
  }
  // tiles at 128 columns, rows, experts above 64 rows, experts with rows,
  // experts above the decode schedule's slot rows and above kSkPrefRows
  int v[6] = {row_tiles(rows) * (a.N / 128), rows, rows > kSmallM ? 1 : 0, rows > 0 ? 1 : 0,
              rows > a.sk_rows ? 1 : 0, rows > kSkPrefRows ? 1 : 0};
  int ex[6], tot[6];
  block_scan<6>(v, ex, tot, s_tot);
  const int T0 = tot[0], R = tot[1], n_big = tot[2], n_active = tot[3];
  // Decode schedule when every expert fits a slot's rows. Otherwise tiles
  // split along K need the reduction launch; when the host launches none
  // (it saw that no expert can exceed the slot rows, so only offsets that
  // break that bound get here) nothing is split.
  const bool can_split = a.part != nullptr && !a.no_reduce;
  // The decode schedule's fix-ups move more partial sums the more rows a
  // split tile holds: above kSkPrefRows rows the round schedule is faster
  // (with split-K and a reduction launch, if one follows), unless the launch
  // is tile-starved (no more tiles than half the blocks, which rounds could
  // only fill by splitting every tile) or, with no reduction launch to
  // follow, no expert exceeds 64 rows. Otherwise a launch with no reduction
  // to follow runs whole tiles in rounds.
  const bool sk_fits = a.sk && tot[4] == 0;
  if (sk_fits && (tot[5] == 0 || 2 * T0 <= G || (a.no_reduce && n_big == 0))) {
    // a single GEMM with at least as many 256-column tiles as blocks takes
    // them (the tile counts at 128 columns are even then): each block then
    // runs whole tiles, half as many pipeline fills (same-process A/B,
    // Qwen3-shaped T = 128, 128 experts of up to 13 rows: FFN 233 -> 220 us).
    // With fewer tiles, wider ones only split more (one expert: up to 70 %
    // slower)
    const bool dwide = !DUAL && (a.N % 256) == 0 && T0 / 2 >= G;
    if (tid < E) s_start[tid] = dwide ? ex[0] / 2 : ex[0];
    if (tid == 0) s_xcd = xcd;
    if (blockIdx.x == 0 && tid == 0 && a.plan != nullptr) {
      a.plan[0] = 1;  // nothing for a reduction launch to do
      a.plan[2] = 1;
    }
    __syncthreads();
    decode_schedule<DUAL, MX>(a, smem, dwide ? T0 / 2 : T0, s_start, s_row0, s_rows, s_xcd == 1, dwide);
    return;
  }

  // Single-output GEMM: 256-column tiles move a third fewer bytes per MFMA
  // than 128-column ones but halve the tile count; use them when every CU
  // still gets at least two of them.
  const bool wide = !DUAL && (a.N % 256 == 0) && (T0 / 2 >= 2 * G);
  constexpr int CK = MX ? kMxChunk : kBK;  // K elements per chunk
  constexpr int EB = MX ? 1 : 2;           // weight bytes per element (MX scales aside)
  const int nK = a.K / CK;
  // K ranges the tail split (below) cuts each tile of the last round of an
  // unsplit launch of `tot` tiles of `tcols` columns into (1: none)
  auto tail_ranges = [&](int tot, int tcols) {
    const int r = tot % G;
    int st = r > 0 ? G / r : 1;
    if (st > kMaxSplit) st = kMaxSplit;
    const long long per = (long long)NB * 256 * tcols;  // floats of one split tile
    while (st > 1 && (st * kMinSplitChunks > nK || (long long)st * r * per > a.part_cap)) --st;
    return (st > 1 && 3 * r <= a.plan_rows) ? st : 1;
  };
  int S = 1;
  if (!wide && T0 > 0 && can_split && R <= a.plan_rows && (n_big == 0 || T0 < G)) {
    long long best = (long long)((T0 + G - 1) / G) * (nK + kSplitOverhead);
    // unsplit with full rounds: the tail split shortens the last round
    const int st1 = T0 >= G ? tail_ranges(T0, 128) : 1;
    if (st1 > 1) best = (long long)(T0 / G) * (nK + kSplitOverhead) + (nK + st1 - 1) / st1 + kSplitOverhead;
    for (int sp = 2; sp <= kMaxSplit && sp * kMinSplitChunks <= nK; ++sp) {
      // partials must fit, and their fp32 write + read must not outweigh the
      // weights the launch streams (large row tiles are compute bound)
      const long long pfl = (long long)NB * sp * R * a.N;
      if (pfl > a.part_cap || pfl * 4 > (long long)NB * a.N * a.K * EB * n_active) break;
      const long long c = (long long)((sp * T0 + G - 1) / G) * ((nK + sp - 1) / sp + kSplitOverhead);
      if (c < best) {
        best = c;
        S = sp;
      }
    }
  }
  const int mul = wide ? 1 : S, div = wide ? 2 : 1;  // tile count per 128-column tile
  const int total = T0 * mul / div;
  const int cols = wide ? 256 : 128;
  // Tail split. An unsplit launch runs its tiles in rounds of G; when the
  // last round is at most half full, its `rem` tiles are each cut into St K
  // ranges (St <= G / rem) spread over the idle CUs, their fp32 sums kept
  // per tile ([tile][b][split][256][cols]) and finished by the reduction
  // launch, which finds each tile's rows and columns in the plan.
  int St = 1, rem = 0;
  if (S == 1 && can_split && total > 0) {
    St = tail_ranges(total, cols);
    rem = St > 1 ? total % G : 0;
  }
  const int full = total - rem;
  const int n_items = full + rem * St;
  if (tid < E) {
    s_start[tid] = ex[0] * mul / div;
    s_srow0[tid] = ex[1];
  }
  __syncthreads();
  if (blockIdx.x == 0 && a.plan != nullptr) {
    if (tid == 0) {
      a.plan[0] = S;
      a.plan[1] = R;
      a.plan[2] = St;
      a.plan[3] = rem;
      a.plan[4] = cols;
    }
    if (S > 1 && tid < E)
      for (int r = 0; r < s_rows[tid]; ++r) a.plan[kPlanHead + s_srow0[tid] + r] = s_row0[tid] + r;
    if (St > 1 && tid < rem) {
      const TileRef t = decode_tile(full + tid, E, s_start, s_row0, s_rows, cols, a.N);
      a.plan[kPlanHead + 3 * tid] = t.m0;
      a.plan[kPlanHead + 3 * tid + 1] = t.m_end;
      a.plan[kPlanHead + 3 * tid + 2] = t.n0;
    }
  }

  // One item: a split-K tile, a split of a tail tile, or a tile.
  auto run_item = [&](int item) {
    if (S > 1) {
      // split tile: S consecutive tiles share a row tile and a column block
      int lo = 0, hi = E - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_start[mid] <= item) lo = mid; else hi = mid - 1;
      }
      const int e = lo;
      const int local = item - s_start[e];
      const int er = s_rows[e];
      const int sp = local % S, rest = local / S;
      int nt, mt;
      tile_rc(rest, row_tiles(er), a.N / 128, mt, nt);
      const int kc0 = sp * nK / S, kc1 = (sp + 1) * nK / S;
      const int m0 = s_row0[e] + mt * 256;
      const int left = er - mt * 256;
      const int m_end = m0 + (left < 256 ? left : 256);
      float* pbase = a.part + ((size_t)sp * R + s_srow0[e] + mt * 256) * a.N;
      const size_t ps = (size_t)S * R * a.N;
      run_split_tile<DUAL, MX, 128>(a, smem, tile_class(left), e, m0, m_end, nt * 128, kc0, kc1, pbase, ps, a.N,
                                    nt * 128);
      return;
    }
    if (item >= full) {
      // a split of a tail tile
      const int u = item - full, pr = u / St, sp = u - pr * St;
      const TileRef t = decode_tile(full + pr, E, s_start, s_row0, s_rows, cols, a.N);
      const int kc0 = sp * nK / St, kc1 = (sp + 1) * nK / St;
      const size_t tsz = (size_t)256 * cols;
      float* pbase = a.part + ((size_t)pr * NB * St + sp) * tsz;
      if constexpr (!DUAL) {
        if (wide) {
          run_split_tile<DUAL, MX, 256>(a, smem, tile_class(t.left), t.e, t.m0, t.m_end, t.n0, kc0, kc1, pbase,
                                        St * tsz, cols, 0);
          return;
        }
      }
      run_split_tile<DUAL, MX, 128>(a, smem, tile_class(t.left), t.e, t.m0, t.m_end, t.n0, kc0, kc1, pbase,
                                    St * tsz, cols, 0);
      return;
    }
    const TileRef t = decode_tile(item, E, s_start, s_row0, s_rows, cols, a.N);
    const int cls = tile_class(t.left);
    if (!DUAL && wide)
      run_tile<DUAL, MX, !DUAL>(a, smem, cls, t.e, t.m0, t.m_end, t.n0);
    else
      run_tile<DUAL, MX, false>(a, smem, cls, t.e, t.m0, t.m_end, t.n0);
  };

  const int per_xcd = G >> 3;
  if (a.queue != nullptr && (G & 7) == 0) {
    // Per-XCD work queues: block b runs on XCD b % 8 and takes items of that
    // XCD's share of every round (the same items the static order below
    // gives it) in order from a counter, so blocks that drew cheap tiles
    // take more. The counter for the next item is requested before a tile
    // and read after it.
    __shared__ int s_item;
    const int xcd = (int)(blockIdx.x & 7);
    auto item_of = [&](int j) { return (j / per_xcd) * G + xcd * per_xcd + j % per_xcd; };
    if (tid == 0) s_item = item_of(atomicAdd(a.queue + xcd, 1));
    __syncthreads();
    int item = s_item;
    while (item < n_items) {
      int j_next = 0;
      if (tid == 0) j_next = atomicAdd(a.queue + xcd, 1);
      run_item(item);
      if (tid == 0) s_item = item_of(j_next);
      __syncthreads();
      item = s_item;
    }
    // The last block to finish (every other block has drawn its last item)
    // zeroes the counters for the next launch.
    if (tid == 0 && a.done != nullptr && atomicAdd(a.done, 1) == G - 1) {
      for (int q = 0; q < 8; ++q) __hip_atomic_store(a.queue + q, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  const int slot = (G & 7) ? (int)blockIdx.x : ((int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3));
  for (int item = slot; item < n_items; item += G) run_item(item);
}

template <bool DUAL>
__global__ __launch_bounds__(kThreads) void grouped_gemm_bf16_kernel(GemmArgs a) {
  grouped_gemm_body<DUAL, false>(a);
}

// MXFP8 grouped GEMM: the same tile schedule (no split-K); the dual GEMM
// writes MXFP8 h, the single one bf16.
template <bool DUAL>
__global__ __launch_bounds__(kThreads) void grouped_gemm_mx_kernel(GemmArgs a) {
  grouped_gemm_body<DUAL, true>(a);
}

// Tail tiles of an unsplit launch (see grouped_gemm_body): item `it` of the
// reduction is (tail tile pr, row rr, 4 columns at c); the tile's rows and
// first column come from the plan. Returns false for rows past the tile's end.
struct TailItem {
  const float* p;  // partials of split 0 of matrix 0
  size_t tsz;      // floats between splits
  int row, col;    // output row and column
};

__device__ __forceinline__ bool tail_item(const float* part, const int32_t* plan, int NB, size_t it,
                                          TailItem& t) {
  const int St = plan[2], cols = plan[4];
  const int c4n = cols / 4;
  const int pr = (int)(it / ((size_t)256 * c4n));
  const int rr = (int)((it / c4n) % 256), c = (int)(it % c4n) * 4;
  const int m0 = plan[kPlanHead + 3 * pr], m_end = plan[kPlanHead + 3 * pr + 1];
  t.tsz = (size_t)256 * cols;
  t.p = part + (size_t)pr * NB * St * t.tsz + (size_t)rr * cols + c;
  t.row = m0 + rr;
  t.col = plan[kPlanHead + 3 * pr + 2] + c;
  return t.row < m_end;
}

__device__ __forceinline__ float4 sum_splits(const float* p, size_t stride, int n) {
  float4 g = *reinterpret_cast<const float4*>(p);
  for (int sp = 1; sp < n; ++sp) {
    const float4 q = *reinterpret_cast<const float4*>(p + sp * stride);
    g.x += q.x, g.y += q.y, g.z += q.z, g.w += q.w;
  }
  return g;
}

// Sums the S split-K partials of every row of a split launch in split order,
// applies the epilogue (SiLU(gate) * up for the dual GEMM) and writes bf16
// rows of C; or, after an unsplit launch with a tail split, the same for the
// tail tiles. Does nothing when the GEMM before it split nothing.
template <bool DUAL>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part,
                                                           const int32_t* __restrict__ plan, int N,
                                                           bf16_t* __restrict__ C) {
  const int S = plan[0];
  if (S <= 1) {
    const int St = plan[2];
    if (St <= 1) return;
    const size_t items = (size_t)plan[3] * 256 * (plan[4] / 4);
    for (size_t it = (size_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (size_t)gridDim.x * 256) {
      TailItem t;
      if (!tail_item(part, plan, DUAL ? 2 : 1, it, t)) continue;
      float4 g = sum_splits(t.p, t.tsz, St);
      if (DUAL) {
        const float4 u = sum_splits(t.p + St * t.tsz, t.tsz, St);
        g = make_float4(silu_mul_fast(g.x, u.x), silu_mul_fast(g.y, u.y), silu_mul_fast(g.z, u.z),
                        silu_mul_fast(g.w, u.w));
      }
      uint2 packed;
      packed.x = pack_bf16x2(g.x, g.y);
      packed.y = pack_bf16x2(g.z, g.w);
      *reinterpret_cast<uint2*>(C + (size_t)t.row * N + t.col) = packed;
    }
    return;
  }
  const int R = plan[1];
  const int n4 = N / 4;
  const size_t items = (size_t)R * n4, sstride = (size_t)R * N, bstride = (size_t)S * R * N;
  for (size_t it = (size_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (size_t)gridDim.x * 256) {
    const int j = (int)(it / n4), c = (int)(it % n4) * 4;
    const float* p = part + (size_t)j * N + c;
    float4 g = *reinterpret_cast<const float4*>(p);
    for (int sp = 1; sp < S; ++sp) {
      const float4 q = *reinterpret_cast<const float4*>(p + sp * sstride);
      g.x += q.x;
      g.y += q.y;
      g.z += q.z;
      g.w += q.w;
    }
    if (DUAL) {
      float4 u = *reinterpret_cast<const float4*>(p + bstride);
      for (int sp = 1; sp < S; ++sp) {
        const float4 q = *reinterpret_cast<const float4*>(p + bstride + sp * sstride);
        u.x += q.x;
        u.y += q.y;
        u.z += q.z;
        u.w += q.w;
      }
      g = make_float4(silu_mul_fast(g.x, u.x), silu_mul_fast(g.y, u.y), silu_mul_fast(g.z, u.z),
                      silu_mul_fast(g.w, u.w));
    }
    uint2 packed;
    packed.x = pack_bf16x2(g.x, g.y);
    packed.y = pack_bf16x2(g.z, g.w);
    *reinterpret_cast<uint2*>(C + (size_t)plan[kPlanHead + j] * N + c) = packed;
  }
}

// The MXFP8 gate/up reduction: sums the S partials of gate and up for 4
// consecutive columns of a row per thread (16-byte loads, consecutive lanes on
// consecutive columns), applies SiLU(gate) * up as the unsplit epilogue does,
// and quantises each 32-column block (the 8 lanes of an aligned lane group:
// block max by three shuffles, the group's first lane writes the scale code).
// N % 32 == 0 keeps every group inside one block and the item count a
// multiple of 8, so a group is wholly in range or wholly out. Does nothing
// when the GEMM before it split nothing.
__global__ __launch_bounds__(256) void split_reduce_mx_kernel(const float* __restrict__ part,
                                                              const int32_t* __restrict__ plan, int N, int M_cap,
                                                              uint8_t* __restrict__ C8, uint32_t* __restrict__ Cs) {
  const int S = plan[0];
  if (S <= 1) {
    // tail tiles of an unsplit launch; a tile's column count is a multiple
    // of 32, so the 8 lanes of a block share the tile and the row
    const int St = plan[2];
    if (St <= 1) return;
    const size_t items = (size_t)plan[3] * 256 * (plan[4] / 4);
    for (size_t it = (size_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (size_t)gridDim.x * 256) {
      TailItem t;
      if (!tail_item(part, plan, 2, it, t)) continue;
      const float4 g = sum_splits(t.p, t.tsz, St), u = sum_splits(t.p + St * t.tsz, t.tsz, St);
      mx_quant_store4(silu_mul_fast(g.x, u.x), silu_mul_fast(g.y, u.y), silu_mul_fast(g.z, u.z),
                      silu_mul_fast(g.w, u.w), t.row, t.col, N, M_cap, C8, Cs);
    }
    return;
  }
  const int R = plan[1];
  const int n4 = N / 4;
  const size_t items = (size_t)R * n4, sstride = (size_t)R * N, bstride = (size_t)S * R * N;
  for (size_t it = (size_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (size_t)gridDim.x * 256) {
    const int j = (int)(it / n4), c = (int)(it % n4) * 4;
    const float* p = part + (size_t)j * N + c;
    float4 g = *reinterpret_cast<const float4*>(p);
    float4 u = *reinterpret_cast<const float4*>(p + bstride);
    for (int sp = 1; sp < S; ++sp) {
      const float4 a = *reinterpret_cast<const float4*>(p + sp * sstride);
      const float4 b = *reinterpret_cast<const float4*>(p + bstride + sp * sstride);
      g.x += a.x, g.y += a.y, g.z += a.z, g.w += a.w;
      u.x += b.x, u.y += b.y, u.z += b.z, u.w += b.w;
    }
    mx_quant_store4(silu_mul_fast(g.x, u.x), silu_mul_fast(g.y, u.y), silu_mul_fast(g.z, u.z),
                    silu_mul_fast(g.w, u.w), plan[kPlanHead + j], c, N, M_cap, C8, Cs);
  }
}

// ---------------------------------------------------------------------------
// fp32 expert FFN: plain VALU dot products, one thread per output element.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_slot(const int32_t* offsets, int E, int M_cap, int row) {
  for (int e = 0; e < E; ++e) {
    const int o0 = min(max(offsets[e], 0), M_cap);
    const int o1 = min(max(offsets[e + 1], o0), M_cap);
    if (row >= o0 && row < o1) return e;
  }
  return -1;
}

__global__ __launch_bounds__(256) void gateup_f32_kernel(const float* __restrict__ X, const float* __restrict__ Wg,
                                                         const float* __restrict__ Wu,
                                                         const int32_t* __restrict__ offsets, int E, int M_cap,
                                                         int H, int I, int ldw, float* __restrict__ h) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)M_cap * I) return;
  const int row = (int)(idx / I), i = (int)(idx % I);
  const int e = find_slot(offsets, E, M_cap, row);
  if (e < 0) return;
  // 16-byte loads (H, ldw multiples of 4, rows 16-byte aligned), the sums
  // still taken in ascending c
  const float4* x = reinterpret_cast<const float4*>(X + (size_t)row * H);
  const float4* wg = reinterpret_cast<const float4*>(Wg + ((size_t)e * I + i) * ldw);
  const float4* wu = reinterpret_cast<const float4*>(Wu + ((size_t)e * I + i) * ldw);
  float g = 0.0f, u = 0.0f;
  for (int c = 0; c < H / 4; ++c) {
    const float4 xv = x[c], gv = wg[c], uv = wu[c];
    g = __builtin_fmaf(xv.x, gv.x, g);
    u = __builtin_fmaf(xv.x, uv.x, u);
    g = __builtin_fmaf(xv.y, gv.y, g);
    u = __builtin_fmaf(xv.y, uv.y, u);
    g = __builtin_fmaf(xv.z, gv.z, g);
    u = __builtin_fmaf(xv.z, uv.z, u);
    g = __builtin_fmaf(xv.w, gv.w, g);
    u = __builtin_fmaf(xv.w, uv.w, u);
  }
  h[(size_t)row * I + i] = silu_mul(g, u);
}

__global__ __launch_bounds__(256) void down_f32_kernel(const float* __restrict__ h, const float* __restrict__ Wd,
                                                       const int32_t* __restrict__ offsets, int E, int M_cap, int H,
                                                       int I, int ldw, float* __restrict__ y) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)M_cap * H) return;
  const int row = (int)(idx / H), c = (int)(idx % H);
  const int e = find_slot(offsets, E, M_cap, row);
  if (e < 0) return;
  const float4* hr = reinterpret_cast<const float4*>(h + (size_t)row * I);
  const float4* wd = reinterpret_cast<const float4*>(Wd + ((size_t)e * H + c) * ldw);
  float s = 0.0f;
  for (int i = 0; i < I / 4; ++i) {
    const float4 hv = hr[i], wv = wd[i];
    s = __builtin_fmaf(hv.x, wv.x, s);
    s = __builtin_fmaf(hv.y, wv.y, s);
    s = __builtin_fmaf(hv.z, wv.z, s);
    s = __builtin_fmaf(hv.w, wv.w, s);
  }
  y[(size_t)row * H + c] = s;
}

// Zeroes the work counters at the start of the scratch of the entry point
// that allocates nothing, at its first use on a device (a kernel, not a
// memset, so that a first call under graph capture records no memset).
__global__ void clear_counters_kernel(int32_t* q, int n) {
  for (int i = (int)threadIdx.x; i < n; i += (int)blockDim.x) q[i] = 0;
}

__global__ void set_offsets_kernel(int32_t* offsets, int m) {
  if (threadIdx.x == 0) {
    offsets[0] = 0;
    offsets[1] = m;
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
static size_t round256(size_t n) { return ((n + 255) / 256) * 256; }

// bf16 workspace: counters (kCntBytes at offset 0, the same place whatever
// the sizes, so a buffer can serve calls of any size) | h [M_cap, I] |
// split-K plan | fp32 partials (split-K, tail split or the decode
// schedule's slots). The counters must be zero before the first call on a
// workspace; every call leaves them zero. A split
// launch has R <= M_cap partial rows for offsets that are a valid scan (and
// R <= 64 E_local when every expert is small), and S <= 8. The kernel splits
// only when R fits the plan's row map and its partials fit in part_cap.
constexpr size_t kCntBytes = 16384;
constexpr int kMaxBlocks = 1024;  // grid limit of a GEMM launch (tcnt entries)
// Rows of a decode-schedule slot: the largest expert the decode schedule
// takes (it finishes split tiles through the XCD's L2). Same-process A/B on
// one expert: 27-36 % faster than split-K with reduction launches at 48-64
// rows, 20-30 % at 80-128 rows; on skewed batches of many experts with up
// to 128 rows it was 20-30 % slower than rounds, so above 64 rows it is
// taken only by tile-starved launches (see grouped_gemm_body). The host
// leaves out the reduction launches when no expert can exceed kSkHostRows
// rows: every launch then either takes the decode schedule or runs whole
// tiles in rounds, which such launches fill without splitting.
constexpr int kSkRows = 128;
constexpr int kSkHostRows = 128;
// int offsets within the counters
constexpr int kQueueGU = 0, kDoneGU = 8, kQueueDN = 16, kDoneDN = 24, kTcntGU = 64, kTcntDN = 64 + kMaxBlocks;
static_assert((kTcntDN + kMaxBlocks) * 4 <= (int)kCntBytes, "counters");

struct FfnWs {
  size_t h, plan, part;  // byte offsets
  long long part_cap;    // floats
  int plan_rows;         // rows of the plan's row map
  bool sk_ok;            // the partial region holds the decode schedule's slots
  size_t bytes;
};

// fp32 partials either split-K (S <= kMaxSplit slices of every row of both
// GEMMs) or the tail split (at most 256 split tiles of 256 x 256 floats, and
// at most kMaxSplit per tile) may need, within kPartCapFloats.
static long long part_cap_floats(int M_cap, int E_local, int H, int I) {
  const long long split_k = (long long)kMaxSplit * M_cap * std::max(2LL * I, (long long)H);
  const long long tiles = ((long long)(M_cap + kSmallM - 1) / kSmallM + E_local) * (std::max(I, H) / 128);
  const long long tail = std::min(256LL, (long long)kMaxSplit * tiles) * 256 * 256;
  return std::min(std::max(split_k, tail), kPartCapFloats);
}

static int device_cu_count();

// the decode schedule's slots: two per block, 2 x kSkRows x 128 floats each
static long long sk_slot_floats() { return 2LL * std::min(device_cu_count(), kMaxBlocks) * 2 * kSkRows * 128; }

// Layout of an FFN workspace of at most `cap` bytes (SIZE_MAX: as large as
// the call can use). A smaller capacity shrinks only the partial region:
// fewer tiles can then split, and below the slots' size the decode schedule
// is off. The fixed part (counters, h, plan) must fit: see ffn_ws_fixed.
static FfnWs ffn_ws_layout(int M_cap, int E_local, int H, int I, bool bf16, size_t cap = SIZE_MAX) {
  FfnWs w{};
  const size_t h = round256((size_t)M_cap * I * (bf16 ? 2 : 4));
  w.h = 0;
  if (!bf16) {
    w.bytes = h + 256;
    return w;
  }
  w.h = kCntBytes;
  w.plan_rows = std::max(M_cap, kSmallM * E_local);
  w.plan = w.h + h;
  w.part = w.plan + round256((size_t)(kPlanHead + (size_t)w.plan_rows) * 4);
  const long long full = std::max(part_cap_floats(M_cap, E_local, H, I), sk_slot_floats());
  size_t part_bytes = round256((size_t)full * 4);
  if (cap != SIZE_MAX) part_bytes = std::min(part_bytes, cap > w.part ? ((cap - w.part) & ~(size_t)255) : 0);
  w.part_cap = std::min(part_cap_floats(M_cap, E_local, H, I), (long long)(part_bytes / 4));
  w.sk_ok = (long long)(part_bytes / 4) >= sk_slot_floats();
  w.bytes = w.part + part_bytes;
  return w;
}

size_t ffn_ws_fixed(int M_cap, int E_local, int H, int I, bool bf16) {
  const FfnWs w = ffn_ws_layout(M_cap, E_local, H, I, bf16, 0);
  return bf16 ? w.part : w.bytes;
}

size_t ffn_ws_bytes(int M_cap, int E_local, int H, int I, bool bf16) {
  return ffn_ws_layout(M_cap, E_local, H, I, bf16).bytes;
}

static int device_cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

// XCD check. The decode schedule keeps partial sums in an XCD's L2 only if
// the blocks that share them run on one XCD, i.e. if workgroup b of a launch
// runs on XCD b % 8 (the hardware deals workgroups to the XCDs round robin).
// This kernel checks that once per device: block b compares the XCC_ID
// hardware register with b % 8; the last block to finish publishes the
// result in st[0] (1: every block matched, 2: some did not; 0 until then).
// st[1] counts mismatches, st[2] finished blocks. It has the GEMMs' block
// size and holds a comparable share of LDS, so blocks are placed as theirs.
static __device__ int32_t xcd_check[4];
__global__ __launch_bounds__(kThreads) void xcd_probe_kernel(int32_t* st) {
  __shared__ int32_t s_pad[32768];
  int x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(x));
  s_pad[threadIdx.x * 64] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    if (s_pad[0] != (int)(blockIdx.x & 7)) atomicAdd(st + 1, 1);
    __threadfence();
    if (atomicAdd(st + 2, 1) == (int)gridDim.x - 1) {
      __threadfence();
      const int bad = __hip_atomic_load(st + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(st, bad == 0 ? 1 : 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// The XCD check's result on the current device for a launch on stream s,
// or nullptr (kernels then keep partial sums at the point of coherence; the
// results are the same). The check is launched on stream s by the first call
// on the device that is not under graph capture. Its result goes to launches
// on that stream (ordered after it) and, once the check has completed, to
// launches on any stream, so that no launch runs while the result changes.
static const int32_t* xcd_state(hipStream_t s) {
  struct Dev {
    int32_t* ptr;
    hipEvent_t done;
    hipStream_t stream;
    bool launched, ready;
  };
  static std::mutex mu;
  static Dev devs[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  Dev& d = devs[dev];
  if (d.ptr == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(xcd_check)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    d.ptr = static_cast<int32_t*>(p);
  }
  // no launch, event record or event query under graph capture (they could
  // end it); the result is then passed on only if it is known
  hipStreamCaptureStatus cs = hipStreamCaptureStatusActive;
  const bool capturing = hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
  if (capturing) (void)hipGetLastError();
  if (!d.launched) {
    if (capturing) return nullptr;
    if (d.done == nullptr && hipEventCreateWithFlags(&d.done, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      d.done = nullptr;
      return nullptr;
    }
    xcd_probe_kernel<<<kMaxBlocks, kThreads, 0, s>>>(d.ptr);
    if (hipGetLastError() != hipSuccess || hipEventRecord(d.done, s) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    d.launched = true;
    d.stream = s;
  }
  if (!d.ready && !capturing) {
    const hipError_t q = hipEventQuery(d.done);
    if (q == hipSuccess)
      d.ready = true;
    else if (q != hipErrorNotReady)
      (void)hipGetLastError();
  }
  return d.ready || s == d.stream ? d.ptr : nullptr;
}

hipError_t launch_ffn(const void* x_perm, const void* w_gate, const void* w_up, const void* w_down,
                      const int32_t* offsets, int E_local, int H, int I, int ld_gu, int ld_dn, int M_cap, bool bf16,
                      void* y_perm, void* ws, hipStream_t s, const int32_t* a_src, int a_div, int a_T,
                      size_t ws_cap) {
  if (E_local == 0 || M_cap == 0) return hipSuccess;
  const FfnWs L = ffn_ws_layout(M_cap, E_local, H, I, bf16, ws_cap);
  char* wsb = static_cast<char*>(ws);
  void* h = wsb + L.h;
  if (!bf16) {
    const size_t n1 = (size_t)M_cap * I, n2 = (size_t)M_cap * H;
    gateup_f32_kernel<<<(unsigned)((n1 + 255) / 256), 256, 0, s>>>(
        static_cast<const float*>(x_perm), static_cast<const float*>(w_gate), static_cast<const float*>(w_up),
        offsets, E_local, M_cap, H, I, ld_gu, static_cast<float*>(h));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    down_f32_kernel<<<(unsigned)((n2 + 255) / 256), 256, 0, s>>>(static_cast<const float*>(h),
                                                                  static_cast<const float*>(w_down), offsets,
                                                                  E_local, M_cap, H, I, ld_dn,
                                                                  static_cast<float*>(y_perm));
    return hipGetLastError();
  }
  const int cus = device_cu_count();
  // Upper bound on unsplit tiles: every expert could need one partial tile
  // plus ceil(rows / 64) full ones. The grid is a multiple of 8 (one share
  // per XCD). A split launch has S times the tiles of a launch with fewer
  // tiles than blocks, so the grid covers at least 8 of those.
  auto grid_for = [&](int N) {
    const long long ub = ((long long)(M_cap + kSmallM - 1) / kSmallM + E_local) * (N / 128) * kMaxSplit;
    long long g = std::min(cus, kMaxBlocks);  // one 8-wave block per CU
    if (ub < g) g = ub;
    if (g >= 8) g &= ~7LL;
    return (unsigned)(g < 1 ? 1 : g);
  };
  float* part = reinterpret_cast<float*>(wsb + L.part);
  int32_t* plan = reinterpret_cast<int32_t*>(wsb + L.plan);
  int32_t* cnt = reinterpret_cast<int32_t*>(wsb);
  // reduce grid: one float4 column group per thread, grid-stride over 4
  // blocks per CU (a split launch has up to max(M_cap, 64 E_local) rows of
  // N columns to finish, a tail split up to G / 2 tiles of 256 x 256)
  auto reduce_grid = [&](int) { return (unsigned)(4 * cus); };
  // The GEMMs take the decode schedule when no expert has more than
  // kSkHostRows rows (or, tile-starved, kSkRows), and finish its split tiles
  // inside their launches. When no expert can have more than kSkHostRows (a
  // token contributes at most one row to an expert, so with the row gather
  // the bound is min(T, M_cap)), the reduction launches are skipped: the
  // call is two launches.
  const int row_bound = a_src != nullptr ? std::min(a_T, M_cap) : M_cap;
  const bool sk = L.sk_ok && row_bound <= kSkHostRows;
  GemmArgs g1{static_cast<const bf16_t*>(x_perm), static_cast<const bf16_t*>(w_gate),
              static_cast<const bf16_t*>(w_up), static_cast<bf16_t*>(h), offsets, E_local, M_cap, I, H,
              part, L.part_cap, plan, L.plan_rows};
  g1.queue = cnt + kQueueGU;
  g1.done = cnt + kDoneGU;
  g1.a_src = a_src;
  g1.a_div = a_div;
  g1.a_T = a_T;
  g1.ldb = ld_gu;
  g1.sk = L.sk_ok ? 1 : 0;
  g1.no_reduce = sk ? 1 : 0;
  g1.sk_rows = kSkRows;
  g1.skpart = part;
  g1.tcnt = cnt + kTcntGU;
  g1.xcd_state = L.sk_ok ? xcd_state(s) : nullptr;
  grouped_gemm_bf16_kernel<true><<<grid_for(I), kThreads, 0, s>>>(g1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // A GEMM can split only if its K range holds two splits of kMinSplitChunks.
  const bool split_gu = H / kBK >= 2 * kMinSplitChunks, split_dn = I / kBK >= 2 * kMinSplitChunks;
  if (split_gu && !sk) {
    split_reduce_kernel<true><<<reduce_grid(I), 256, 0, s>>>(part, plan, I, static_cast<bf16_t*>(h));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  GemmArgs g2{static_cast<const bf16_t*>(h), static_cast<const bf16_t*>(w_down), nullptr,
              static_cast<bf16_t*>(y_perm), offsets, E_local, M_cap, H, I, part, L.part_cap, plan, L.plan_rows};
  g2.queue = cnt + kQueueDN;
  g2.done = cnt + kDoneDN;
  g2.ldb = ld_dn;
  g2.sk = g1.sk;
  g2.no_reduce = g1.no_reduce;
  g2.sk_rows = kSkRows;
  g2.skpart = part;
  g2.tcnt = cnt + kTcntDN;
  g2.xcd_state = g1.xcd_state;
  grouped_gemm_bf16_kernel<false><<<grid_for(H), kThreads, 0, s>>>(g2);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (split_dn && !sk)
    split_reduce_kernel<false><<<reduce_grid(H), 256, 0, s>>>(part, plan, H, static_cast<bf16_t*>(y_perm));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// MXFP8 expert FFN: gate/up (MXFP8 in, MXFP8 h out), then down (bf16 out)
// ---------------------------------------------------------------------------
// MXFP8 FFN workspace: counters (kCntBytes, zero before first use, as for
// bf16) | h codes [M_cap, I] | h scale dwords [I/128][M_cap] | split-K plan |
// fp32 partials (split-K, or the decode schedule's slots).
struct FfnMxWs {
  size_t hq, hs, plan, part;  // byte offsets
  long long part_cap;
  int plan_rows;
  size_t bytes;
};

static FfnMxWs ffn_mx_ws_layout(int M_cap, int E_local, int H, int I) {
  FfnMxWs w{};
  w.hq = kCntBytes;
  w.hs = w.hq + round256((size_t)M_cap * I);
  w.plan = w.hs + round256((size_t)(I / kMxChunk) * M_cap * 4);
  // sized for split-K only, not for the tail split as the bf16 layout is:
  // with room for it, the MXFP8 decode FFN (Mixtral-shaped, T = 32) took the
  // tail split over S = 2 and measured 3 % slower
  const long long need = (long long)kMaxSplit * M_cap * std::max(2LL * I, (long long)H);
  w.part_cap = std::min(need, kPartCapFloats);
  w.plan_rows = std::max(M_cap, kSmallM * E_local);
  w.part = w.plan + round256((size_t)(kPlanHead + (size_t)w.plan_rows) * 4);
  w.bytes = w.part + round256((size_t)std::max(w.part_cap, sk_slot_floats()) * 4);
  return w;
}

size_t ffn_mx_ws_bytes(int M_cap, int E_local, int H, int I) {
  return ffn_mx_ws_layout(M_cap, E_local, H, I).bytes;
}

// One 8-wave block per CU, at most the tile bound (times the largest split
// when split-K is possible), a multiple of 8.
static unsigned mx_grid(int M_cap, int E_local, int N, bool split) {
  const long long ub = ((long long)(M_cap + kSmallM - 1) / kSmallM + E_local) * (N / 128) * (split ? kMaxSplit : 1);
  long long g = std::min(device_cu_count(), kMaxBlocks);
  if (ub < g) g = ub;
  if (g >= 8) g &= ~7LL;
  return (unsigned)(g < 1 ? 1 : g);
}

// as reduce_grid in launch_ffn
static unsigned mx_reduce_grid(int, int) { return (unsigned)(4 * device_cu_count()); }

// Split-K workspace of one MX GEMM launch (plan == nullptr: no split-K).
struct MxSplit {
  float* part;
  long long part_cap;
  int32_t* plan;
  int plan_rows;
  int32_t* queue;  // per-XCD work counters or nullptr
  int32_t* done;   // finished-block counter (the queue's reset) or nullptr
  int32_t* tcnt;   // decode schedule: tile arrival counters, or nullptr (off)
  bool no_reduce;  // no reduction launch follows (nothing may split)
  const int32_t* xcd;  // the XCD check's result (see xcd_state), or nullptr
};

static void mx_split_args(GemmArgs& g, const MxSplit& sp) {
  g.part = sp.part;
  g.part_cap = sp.part_cap;
  g.plan = sp.plan;
  g.plan_rows = sp.plan_rows;
  g.queue = sp.queue;
  g.done = sp.done;
  g.sk = sp.tcnt != nullptr ? 1 : 0;
  g.sk_rows = kSkRows;
  g.skpart = sp.part;
  g.tcnt = sp.tcnt;
  g.no_reduce = sp.no_reduce ? 1 : 0;
  g.xcd_state = sp.xcd;
}

static hipError_t gateup_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                            const uint8_t* wuq, const uint32_t* wus, const int32_t* offsets, int E_local, int H,
                            int I, int ldw, int M_cap, uint8_t* hq, uint32_t* hs, const MxSplit& sp,
                            hipStream_t s) {
  GemmArgs g{};
  g.A = reinterpret_cast<const bf16_t*>(xq);
  g.B0 = reinterpret_cast<const bf16_t*>(wgq);
  g.B1 = reinterpret_cast<const bf16_t*>(wuq);
  g.C = reinterpret_cast<bf16_t*>(hq);
  g.offsets = offsets;
  g.E_local = E_local;
  g.M_cap = M_cap;
  g.N = I;
  g.K = H;
  g.ldb = ldw;
  mx_split_args(g, sp);
  g.As = xs;
  g.Bs0 = wgs;
  g.Bs1 = wus;
  g.Cs = hs;
  const bool split = sp.plan != nullptr && H / kMxChunk >= 2 * kMinSplitChunks;
  grouped_gemm_mx_kernel<true><<<mx_grid(M_cap, E_local, I, split || g.sk), kThreads, 0, s>>>(g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !split || sp.no_reduce) return e;
  split_reduce_mx_kernel<<<mx_reduce_grid(sp.plan_rows, I / 4), 256, 0, s>>>(sp.part, sp.plan, I, M_cap,
                                                                                     hq, hs);
  return hipGetLastError();
}

static hipError_t gemm_mx(const uint8_t* aq, const uint32_t* as, const uint8_t* bq, const uint32_t* bs,
                          const int32_t* offsets, int E_local, int N, int K, int ldb, int M_cap, void* c,
                          const MxSplit& sp, hipStream_t s) {
  GemmArgs g{};
  g.A = reinterpret_cast<const bf16_t*>(aq);
  g.B0 = reinterpret_cast<const bf16_t*>(bq);
  g.C = static_cast<bf16_t*>(c);
  g.offsets = offsets;
  g.E_local = E_local;
  g.M_cap = M_cap;
  g.N = N;
  g.K = K;
  g.ldb = ldb;
  mx_split_args(g, sp);
  g.As = as;
  g.Bs0 = bs;
  const bool split = sp.plan != nullptr && K / kMxChunk >= 2 * kMinSplitChunks;
  grouped_gemm_mx_kernel<false><<<mx_grid(M_cap, E_local, N, split || g.sk), kThreads, 0, s>>>(g);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !split || sp.no_reduce) return e;
  split_reduce_kernel<false><<<mx_reduce_grid(sp.plan_rows, N / 4), 256, 0, s>>>(sp.part, sp.plan, N,
                                                                                  static_cast<bf16_t*>(c));
  return hipGetLastError();
}

hipError_t launch_gateup_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                            const uint8_t* wuq, const uint32_t* wus, const int32_t* offsets, int E_local, int H,
                            int I, int ldw, int M_cap, uint8_t* hq, uint32_t* hs, hipStream_t s) {
  if (E_local == 0 || M_cap == 0) return hipSuccess;
  return gateup_mx(xq, xs, wgq, wgs, wuq, wus, offsets, E_local, H, I, ldw, M_cap, hq, hs, MxSplit{}, s);
}

hipError_t launch_gemm_mx(const uint8_t* aq, const uint32_t* as, const uint8_t* bq, const uint32_t* bs,
                          const int32_t* offsets, int E_local, int N, int K, int ldb, int M_cap, void* c,
                          hipStream_t s) {
  if (E_local == 0 || M_cap == 0) return hipSuccess;
  return gemm_mx(aq, as, bq, bs, offsets, E_local, N, K, ldb, M_cap, c, MxSplit{}, s);
}

hipError_t launch_ffn_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                         const uint8_t* wuq, const uint32_t* wus, const uint8_t* wdq, const uint32_t* wds,
                         const int32_t* offsets, int E_local, int H, int I, int ld_gu, int ld_dn, int M_cap,
                         void* y_perm, void* ws, hipStream_t s) {
  if (E_local == 0 || M_cap == 0) return hipSuccess;
  const FfnMxWs L = ffn_mx_ws_layout(M_cap, E_local, H, I);
  char* w = static_cast<char*>(ws);
  uint8_t* hq = reinterpret_cast<uint8_t*>(w + L.hq);
  uint32_t* hs = reinterpret_cast<uint32_t*>(w + L.hs);
  int32_t* cnt = reinterpret_cast<int32_t*>(w);
  // as in launch_ffn: the decode schedule finishes its split tiles inside the
  // GEMM launches; when no expert can exceed kSkHostRows rows no reduction
  // follows
  const bool no_reduce = M_cap <= kSkHostRows;
  const MxSplit sp1{reinterpret_cast<float*>(w + L.part), L.part_cap, reinterpret_cast<int32_t*>(w + L.plan),
                    L.plan_rows, cnt + kQueueGU, cnt + kDoneGU, cnt + kTcntGU, no_reduce, xcd_state(s)};
  hipError_t e = gateup_mx(xq, xs, wgq, wgs, wuq, wus, offsets, E_local, H, I, ld_gu, M_cap, hq, hs, sp1, s);
  if (e != hipSuccess) return e;
  const MxSplit sp2{sp1.part, sp1.part_cap, sp1.plan, sp1.plan_rows, cnt + kQueueDN, cnt + kDoneDN, cnt + kTcntDN,
                    no_reduce, sp1.xcd};
  return gemm_mx(hq, hs, wdq, wds, offsets, E_local, H, I, ld_dn, M_cap, y_perm, sp2, s);
}

// ---------------------------------------------------------------------------
// Router logits by K ranges (the router GEMM z = x W_r^T for many tokens and
// E = 128 or 256 experts): block (t, s) sums x[256 t, +256) W_r^T over the K
// chunks [s nK / S, (s + 1) nK / S) with the expert FFN's 256-row tile and
// writes the fp32 sums to part[s][row][0, E); gate_topk_reduce_kernel adds the
// S slices in split order. A CU then loads 256 token rows and the E router
// rows of one K range, where a router block that finishes its tokens' top-k
// itself loads all E router rows for every 64 tokens.
// ---------------------------------------------------------------------------
template <int BN>
__global__ __launch_bounds__(kThreads) void router_logits_split_kernel(GemmArgs a, int S, float* __restrict__ part) {
  __shared__ __align__(16) bf16_t smem[Stages<256, BN, false>::BYTES / 2];
  const int T = a.M_cap;
  const int m0 = (int)blockIdx.x * 256;
  const int m_end = min(m0 + 256, T);
  const int nK = a.K / kBK, sp = (int)blockIdx.y;
  const int kc0 = sp * nK / S, kc1 = (sp + 1) * nK / S;
  float* pbase = part + ((size_t)sp * T + m0) * BN;
  gemm_tile<256, BN, 4, false, true>(a, smem, 0, m0, m_end, 0, kc0, kc1, pbase, 0, BN, 0);
}

hipError_t launch_router_logits_split(const void* x, const void* wr, int T, int H, int E, int S, float* part,
                                      hipStream_t s) {
  if (T < 1 || S < 1 || S > 8 || H % kBK != 0 || H / kBK < S) return hipErrorInvalidValue;
  GemmArgs g{};
  g.A = static_cast<const bf16_t*>(x);
  g.B0 = static_cast<const bf16_t*>(wr);
  g.E_local = 1;
  g.M_cap = T;
  g.N = E;
  g.K = H;
  g.ldb = H;
  const dim3 grid((unsigned)((T + 255) / 256), (unsigned)S);
  if (E == 256)
    router_logits_split_kernel<256><<<grid, kThreads, 0, s>>>(g, S, part);
  else if (E == 128)
    router_logits_split_kernel<128><<<grid, kThreads, 0, s>>>(g, S, part);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scratch of the FFN entry point that allocates nothing
// (moe_grouped_swiglu_ffn_noalloc): the workspace of its calls, one copy per
// GPU in the code object's device memory, held until the process ends. In
// host code `scratch` only names the symbol; its address on a device comes
// from hipGetSymbolAddress with that device current, and only that address
// is passed to kernels.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t ffn_scratch(void** out, hipStream_t s) {
  static std::mutex mu;
  static void* ptrs[64] = {nullptr};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    // the counters must start at zero (every call leaves them zero); a
    // kernel rather than a memset, so that a first call under graph capture
    // records no memset node
    clear_counters_kernel<<<1, 1024, 0, s>>>(static_cast<int32_t*>(p), (int)(kCntBytes / 4));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return hipSuccess;
}

hipError_t launch_set_offsets(int32_t* offsets, int m, hipStream_t s) {
  set_offsets_kernel<<<1, 64, 0, s>>>(offsets, m);
  return hipGetLastError();
}

}  // namespace moe
