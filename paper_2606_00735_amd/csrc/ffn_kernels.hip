// Grouped SwiGLU expert FFN (gfx950): the expert computation whose latency
// per token load is ViBE's per-GPU performance model f_g(n) (Section 4.2.1).
//
// Two persistent launches per call:
//   gate/up:  h[R] = bf16( silu(X_R W_gate^T) * (X_R W_up^T) )   (dual GEMM)
//   down:     y[R] = bf16( h[R] W_down^T )
// for each local expert's row range R = [offsets[e], offsets[e+1]).
//
// Per-expert row counts live only on the device, so each block rebuilds the
// tile list from `offsets` (a scan over at most 256 experts) and walks it
// with a grid stride. An expert with M_e <= 32 rows gets 32-row tiles (its
// cost is streaming its weights once); larger experts get 128-row tiles.
// Within an expert, consecutive tile indices share a weight column block, so
// blocks running at the same time read the same weights.
#include "common.hpp"
#include "launch.hpp"

namespace moe {

constexpr int kBK = 64;  // K chunk per pipeline stage

// Blocks of 8 waves (two per SIMD, so one wave's LDS waits are covered by
// the other's MFMAs). Tile classes, chosen per expert from its row count M_e:
//   small  M_e <= 64    64 x 128 tiles, waves 2x4, 3 stages  (weight streaming)
//   mid    M_e <= 192  128 x 128 tiles, waves 2x4, 3 stages
//   large  otherwise   256 x 128 tiles, waves 4x2, 2 stages  (MFMA bound)
// with 128 output columns per matrix (gate and up both, in the dual GEMM).
constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kSmallM = 64;
constexpr int kMidM = 192;

struct GemmArgs {
  const bf16_t* A;        // [M_cap, K]
  const bf16_t* B0;       // [E_local, N, K]
  const bf16_t* B1;       // [E_local, N, K] (dual only)
  bf16_t* C;              // [M_cap, N]
  const int32_t* offsets; // [E_local + 1]
  int E_local, M_cap, N, K;
};

__device__ __forceinline__ float silu_mul(float g, float u) {
  const float sig = 1.0f / (1.0f + expf(-g));
  return (g * sig) * u;
}

// One BM x BN output tile (two of them, gate and up, when DUAL) over the whole
// K range: 4 waves, 32x32x16 bf16 MFMA, operands loaded straight from global
// memory into NS swizzled LDS stages (see pipeline).
template <int BM, int BN, int WAVES_M, int NS, bool DUAL>
__device__ __forceinline__ void gemm_tile(const GemmArgs& a, bf16_t* smem, int e, int m0, int m_end, int n0) {
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WAVES_N = kWaves / WAVES_M;
  constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  constexpr int MI = WM / 32, NI = WN / 32;
  constexpr int LOADS = (BM + NB * BN) / (8 * kWaves);  // DMA instructions per wave per chunk
  constexpr int STAGE = (BM + NB * BN) * 64;        // elements per stage
  static_assert(MI >= 1 && NI >= 1, "wave tile");

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int K = a.K, N = a.N;
  const bf16_t* A = a.A + (size_t)m0 * K;
  const int a_rows = m_end - m0;
  const bf16_t* B0 = a.B0 + ((size_t)e * N + n0) * K;
  const bf16_t* B1 = DUAL ? a.B1 + ((size_t)e * N + n0) * K : nullptr;

  f32x16_t acc[NB][MI][NI];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j) acc[b][i][j] = f32x16_t{};

  auto issue = [&](int kc, bool live, bf16_t* st) {
    dma_rows<BM, kWaves>(A, K, kc * kBK, a_rows, live, st, wave, lane);
    dma_rows<BN, kWaves>(B0, K, kc * kBK, BN, live, st + BM * 64, wave, lane);
    if (DUAL) dma_rows<BN, kWaves>(B1, K, kc * kBK, BN, live, st + (BM + BN) * 64, wave, lane);
  };
  // Fragments of k-step s+1 are read from LDS before the MFMAs of k-step s
  // are issued, so the MFMAs never wait on the read that feeds them.
  auto compute = [&](const bf16_t* st) {
    bf16x8_t af[2][MI], bfr[2][NB][NI];
    auto read = [&](int s, int buf) {
      const int chunk = 2 * s + (lane >> 5);
#pragma unroll
      for (int i = 0; i < MI; ++i) af[buf][i] = lds_frag(st, wm * WM + i * 32 + (lane & 31), chunk);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          bfr[buf][b][j] = lds_frag(st + (BM + b * BN) * 64, wn * WN + j * 32 + (lane & 31), chunk);
    };
    constexpr int NREAD = MI + NB * NI, NMFMA = NB * MI * NI;
    constexpr int PAIRS = NREAD < NMFMA ? NREAD : NMFMA;
    read(0, 0);
#pragma unroll
    for (int s = 0; s < kBK / 16; ++s) {
      const bool next = s + 1 < kBK / 16;
      if (next) read(s + 1, (s + 1) & 1);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < NI; ++j)
#pragma unroll
          for (int i = 0; i < MI; ++i)
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s & 1][i], bfr[s & 1][b][j], acc[b][i][j], 0,
                                                                   0, 0);
      // issue order: one MFMA of this step, one LDS read of the next, ...
      if (next) {
#pragma unroll
        for (int q = 0; q < PAIRS; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        }
        if (NMFMA > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, NMFMA - PAIRS, 0);
        if (NREAD > PAIRS) __builtin_amdgcn_sched_group_barrier(0x100, NREAD - PAIRS, 0);
      }
      __builtin_amdgcn_sched_barrier(0);  // each k-step is its own scheduling region
    }
  };
  pipeline<NS, LOADS>(K / kBK, smem, STAGE, issue, compute);

  // Epilogue. 32x32 accumulator layout: register v of lane l is row
  // 8 * (v / 4) + 4 * (l / 32) + (v % 4), column l % 32 of the MFMA block.
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const int col = n0 + wn * WN + j * 32 + (lane & 31);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m0 + wm * WM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (row < m_end) {
          float r;
          if (DUAL)
            r = silu_mul(acc[0][i][j][v], acc[NB - 1][i][j][v]);
          else
            r = acc[0][i][j][v];
          a.C[(size_t)row * N + col] = f32_to_bf16(r);
        }
      }
    }
}

template <bool DUAL>
struct GemmShapes {
  static constexpr int NB = DUAL ? 2 : 1;
  static constexpr int kSmallStage = (64 + NB * 128) * 64 * 3;
  static constexpr int kMidStage = (128 + NB * 128) * 64 * 3;
  static constexpr int kLargeStage = (256 + NB * 128) * 64 * 2;
  static constexpr int kSmem = kSmallStage > kMidStage ? (kSmallStage > kLargeStage ? kSmallStage : kLargeStage)
                                                       : (kMidStage > kLargeStage ? kMidStage : kLargeStage);
};

__device__ __forceinline__ int tile_class(int rows) { return rows <= kSmallM ? 0 : (rows <= kMidM ? 1 : 2); }
__device__ __forceinline__ int class_rows(int cls) { return cls == 0 ? kSmallM : (cls == 1 ? 128 : 256); }

// Persistent grouped GEMM over every local expert. The grid is a multiple of
// 8 and block b runs on XCD b % 8; in each round of gridDim.x tiles, the
// blocks of one XCD take consecutive logical tiles. The logical order walks
// each expert's row tiles fastest, so the row tiles that share a weight
// column block run at the same time on one XCD: every weight byte comes from
// HBM about once, and the rows (a few hundred MB at most) come from the
// last-level cache.
template <bool DUAL>
__global__ __launch_bounds__(kThreads) void grouped_gemm_bf16_kernel(GemmArgs a) {
  using S = GemmShapes<DUAL>;
  __shared__ __align__(16) bf16_t smem[S::kSmem];
  __shared__ int s_start[kMaxExperts + 1];
  __shared__ int s_row0[kMaxExperts];
  __shared__ int s_rows[kMaxExperts];
  __shared__ int s_tot[kWaves];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int E = a.E_local;

  // Tile list: rows of each expert, clamped so no access leaves [0, M_cap).
  int tiles = 0;
  if (tid < E) {
    int o0 = a.offsets[tid], o1 = a.offsets[tid + 1];
    o0 = min(max(o0, 0), a.M_cap);
    o1 = min(max(o1, o0), a.M_cap);
    const int rows = o1 - o0;
    s_row0[tid] = o0;
    s_rows[tid] = rows;
    const int bm = class_rows(tile_class(rows));
    tiles = ((rows + bm - 1) / bm) * (a.N / 128);
  }
  // exclusive scan of tile counts over experts
  int inc = tiles;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int n = __shfl_up(inc, off, kWave);
    if (lane >= off) inc += n;
  }
  if (lane == 63) s_tot[wave] = inc;
  __syncthreads();
  int base = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    if (w < wave) base += s_tot[w];
    total += s_tot[w];
  }
  if (tid < E) s_start[tid] = base + inc - tiles;
  __syncthreads();

  const int G = gridDim.x;
  const int per_xcd = G >> 3;
  const int slot = (G & 7) ? (int)blockIdx.x : ((int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3));
  for (int tile = slot; tile < total; tile += G) {
    // last expert whose first tile is <= tile (experts with no tiles share
    // their start with the next one, so the last match is the owner)
    int lo = 0, hi = E - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_start[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    const int e = lo;
    const int local = tile - s_start[e];
    const int rows = s_rows[e];
    const int cls = tile_class(rows);
    const int bm = class_rows(cls);
    const int n_mt = (rows + bm - 1) / bm;
    // row tile fastest: all row tiles of a weight column block run together
    const int nt = local / n_mt, mt = local - nt * n_mt;
    const int m0 = s_row0[e] + mt * bm;
    const int m_end = min(m0 + bm, s_row0[e] + rows);
    if (cls == 0)
      gemm_tile<64, 128, 2, 3, DUAL>(a, smem, e, m0, m_end, nt * 128);
    else if (cls == 1)
      gemm_tile<128, 128, 2, 3, DUAL>(a, smem, e, m0, m_end, nt * 128);
    else
      gemm_tile<256, 128, 4, 2, DUAL>(a, smem, e, m0, m_end, nt * 128);
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
                                                         int H, int I, float* __restrict__ h) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)M_cap * I) return;
  const int row = (int)(idx / I), i = (int)(idx % I);
  const int e = find_slot(offsets, E, M_cap, row);
  if (e < 0) return;
  const float* x = X + (size_t)row * H;
  const float* wg = Wg + ((size_t)e * I + i) * H;
  const float* wu = Wu + ((size_t)e * I + i) * H;
  float g = 0.0f, u = 0.0f;
  for (int c = 0; c < H; ++c) {
    g = __builtin_fmaf(x[c], wg[c], g);
    u = __builtin_fmaf(x[c], wu[c], u);
  }
  h[(size_t)row * I + i] = silu_mul(g, u);
}

__global__ __launch_bounds__(256) void down_f32_kernel(const float* __restrict__ h, const float* __restrict__ Wd,
                                                       const int32_t* __restrict__ offsets, int E, int M_cap, int H,
                                                       int I, float* __restrict__ y) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)M_cap * H) return;
  const int row = (int)(idx / H), c = (int)(idx % H);
  const int e = find_slot(offsets, E, M_cap, row);
  if (e < 0) return;
  const float* hr = h + (size_t)row * I;
  const float* wd = Wd + ((size_t)e * H + c) * I;
  float s = 0.0f;
  for (int i = 0; i < I; ++i) s = __builtin_fmaf(hr[i], wd[i], s);
  y[(size_t)row * H + c] = s;
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
size_t ffn_ws_bytes(int M_cap, int I, bool bf16) {
  const size_t h = (size_t)M_cap * I * (bf16 ? 2 : 4);
  return ((h + 255) / 256) * 256 + 256;
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

hipError_t launch_ffn(const void* x_perm, const void* w_gate, const void* w_up, const void* w_down,
                      const int32_t* offsets, int E_local, int H, int I, int M_cap, bool bf16, void* y_perm,
                      void* ws, hipStream_t s) {
  if (E_local == 0 || M_cap == 0) return hipSuccess;
  void* h = ws;
  if (!bf16) {
    const size_t n1 = (size_t)M_cap * I, n2 = (size_t)M_cap * H;
    gateup_f32_kernel<<<(unsigned)((n1 + 255) / 256), 256, 0, s>>>(
        static_cast<const float*>(x_perm), static_cast<const float*>(w_gate), static_cast<const float*>(w_up),
        offsets, E_local, M_cap, H, I, static_cast<float*>(h));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    down_f32_kernel<<<(unsigned)((n2 + 255) / 256), 256, 0, s>>>(static_cast<const float*>(h),
                                                                  static_cast<const float*>(w_down), offsets,
                                                                  E_local, M_cap, H, I,
                                                                  static_cast<float*>(y_perm));
    return hipGetLastError();
  }
  const int cus = device_cu_count();
  // Upper bound on tiles: every expert could need one partial tile plus
  // ceil(rows / 32) full ones. The grid is a multiple of 8 (one share per XCD).
  auto grid_for = [&](int N) {
    const long long ub = ((long long)(M_cap + kSmallM - 1) / kSmallM + E_local) * (N / 128);
    long long g = cus;  // one 8-wave block per CU
    if (ub < g) g = ub;
    if (g >= 8) g &= ~7LL;
    return (unsigned)(g < 1 ? 1 : g);
  };
  GemmArgs g1{static_cast<const bf16_t*>(x_perm), static_cast<const bf16_t*>(w_gate),
              static_cast<const bf16_t*>(w_up), static_cast<bf16_t*>(h), offsets, E_local, M_cap, I, H};
  grouped_gemm_bf16_kernel<true><<<grid_for(I), kThreads, 0, s>>>(g1);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  GemmArgs g2{static_cast<const bf16_t*>(h), static_cast<const bf16_t*>(w_down), nullptr,
              static_cast<bf16_t*>(y_perm), offsets, E_local, M_cap, H, I};
  grouped_gemm_bf16_kernel<false><<<grid_for(H), kThreads, 0, s>>>(g2);
  return hipGetLastError();
}

hipError_t launch_set_offsets(int32_t* offsets, int m, hipStream_t s) {
  set_offsets_kernel<<<1, 64, 0, s>>>(offsets, m);
  return hipGetLastError();
}

}  // namespace moe
