// ViBE's placement control path on the GPU (Section 4.2; Algorithms 1 and 2):
// the per-GPU latency model f_g, the latency-aware greedy placement, the
// incremental swap solver and the cosine-distance drift detector, one block
// per MoE layer. The inputs (per-layer expert loads) are produced on the GPU
// by the expert histogram, so the control path needs no host round trip.
//
// All decisions are taken in fp64 with every operation rounded on its own
// (contraction off) and every sum in a fixed order, so results do not depend
// on scheduling.
#include "common.hpp"
#include "launch.hpp"

#pragma clang fp contract(off)

namespace moe {

constexpr int kPlaceThreads = 256;
constexpr int kPlaceMaxE = 1024;  // experts per layer
constexpr int kPlaceMaxG = 64;    // GPUs (one wave holds them)

// f(n) of one GPU's model: knots (kn[k], kt[k]), k < nk, kn strictly
// increasing and positive. f = 0 for n <= 0, kt[0] up to kn[0], linear
// between knots, the last segment's slope beyond the last knot (with one
// knot: kt[0] n / kn[0]).
__device__ double latency_at(const double* kn, const double* kt, int nk, double n) {
  if (n <= 0.0) return 0.0;
  if (n <= kn[0]) return kt[0];
  if (nk == 1) return kt[0] * (n / kn[0]);
  for (int k = 0; k + 1 < nk; ++k)
    if (n <= kn[k + 1]) return kt[k] + (kt[k + 1] - kt[k]) * ((n - kn[k]) / (kn[k + 1] - kn[k]));
  const double lo_n = kn[nk - 2], hi_n = kn[nk - 1], lo_t = kt[nk - 2], hi_t = kt[nk - 1];
  return hi_t + (hi_t - lo_t) * ((n - hi_n) / (hi_n - lo_n));
}

__device__ __forceinline__ double shfl_f64(double v, int src) {
  const int2 p = __builtin_bit_cast(int2, v);
  return __builtin_bit_cast(double, make_int2(__shfl(p.x, src, kWave), __shfl(p.y, src, kWave)));
}

// (value, index) arg-max over one wave: larger value, then lower index.
__device__ __forceinline__ void wave_argmax(double& v, int& i) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const int src = (threadIdx.x & 63) ^ off;
    const double ov = shfl_f64(v, src);
    const int oi = __shfl(i, src, kWave);
    if (ov > v || (ov == v && oi < i)) {
      v = ov;
      i = oi;
    }
  }
}

// ---------------------------------------------------------------------------
// Algorithm 1, Phase 2: speed-proportional targets and descending-load greedy.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kPlaceThreads) void place_greedy_kernel(const double* __restrict__ W, int E,
                                                                     const double* __restrict__ knots_n,
                                                                     const double* __restrict__ knots_t, int G,
                                                                     int nk, int cap, int32_t* __restrict__ assign,
                                                                     double* __restrict__ loads,
                                                                     double* __restrict__ targets) {
  __shared__ double s_w[kPlaceMaxE];
  __shared__ double s_key[kPlaceMaxE];  // sort keys: load, descending
  __shared__ int s_id[kPlaceMaxE];      // expert ids, ascending among equal loads
  __shared__ double s_speed[kPlaceMaxG];
  __shared__ double s_N, s_S;
  const int l = blockIdx.x, tid = threadIdx.x;
  const double* w = W + (size_t)l * E;

  int P = 1;
  while (P < E) P <<= 1;
  for (int i = tid; i < P; i += kPlaceThreads) {
    if (i < E) {
      s_w[i] = w[i];
      s_key[i] = w[i];
      s_id[i] = i;
    } else {
      s_key[i] = -__builtin_inf();
      s_id[i] = 0x7fffffff;
    }
  }
  __syncthreads();
  if (tid == 0) {  // N = sum_e w_e in ascending e
    double N = 0.0;
    for (int e = 0; e < E; ++e) N += s_w[e];
    s_N = N;
  }
  __syncthreads();
  const double N = s_N;
  if (tid < G) {
    const double* kn = knots_n + (size_t)tid * nk;
    const double* kt = knots_t + (size_t)tid * nk;
    s_speed[tid] = N > 0.0 ? 1.0 / latency_at(kn, kt, nk, N / E) : 1.0;
  }
  __syncthreads();
  if (tid == 0) {
    double S = 0.0;
    for (int g = 0; g < G; ++g) S += s_speed[g];
    s_S = S;
  }
  // bitonic sort of (key desc, id asc) over P entries
  for (int k = 2; k <= P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      __syncthreads();
      for (int i = tid; i < P; i += kPlaceThreads) {
        const int p = i ^ j;
        if (p > i) {
          const bool up = (i & k) == 0;  // this run sorts "before" first
          const double ka = s_key[i], kb = s_key[p];
          const int ia = s_id[i], ib = s_id[p];
          const bool b_first = kb > ka || (kb == ka && ib < ia);  // b belongs before a
          if (b_first == up) {
            s_key[i] = kb;
            s_key[p] = ka;
            s_id[i] = ib;
            s_id[p] = ia;
          }
        }
      }
    }
  __syncthreads();
  if (tid >= kWave) return;
  // greedy: lane g holds tau_g, n_g and its expert count
  const int g = tid;
  const double tau = g < G ? N * s_speed[g] / s_S : 0.0;
  double n = 0.0;
  int cnt = 0;
  for (int r = 0; r < E; ++r) {
    const int e = s_id[r];
    double gap = (g < G && (cap == 0 || cnt < cap)) ? tau - n : -__builtin_inf();
    int best = g < G ? g : 0x7fffffff;
    wave_argmax(gap, best);
    if (g == best) {
      n += s_w[e];
      ++cnt;
    }
    if (g == 0) assign[(size_t)l * E + e] = best;
  }
  if (g < G) {
    if (loads) loads[(size_t)l * G + g] = n;
    if (targets) targets[(size_t)l * G + g] = tau;
  }
}

// ---------------------------------------------------------------------------
// Algorithm 2: swaps between the slowest and the fastest GPU.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kPlaceThreads) void place_incremental_kernel(
    const double* __restrict__ W, int E, const double* __restrict__ knots_n, const double* __restrict__ knots_t,
    int G, int nk, double eps, int max_swaps, int32_t* __restrict__ assign, int32_t* __restrict__ n_swaps) {
  __shared__ double s_w[kPlaceMaxE];
  __shared__ int s_a[kPlaceMaxE];
  __shared__ int s_hi_list[kPlaceMaxE], s_lo_list[kPlaceMaxE];
  __shared__ double s_n[kPlaceMaxG], s_lat[kPlaceMaxG];
  __shared__ int s_hi, s_lo, s_nhi, s_nlo, s_stop;
  __shared__ double s_red_v[kPlaceThreads / kWave];
  __shared__ int s_red_i[kPlaceThreads / kWave];
  const int l = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const double* w = W + (size_t)l * E;
  int32_t* a = assign + (size_t)l * E;
  for (int e = tid; e < E; e += kPlaceThreads) {
    s_w[e] = w[e];
    const int g = a[e];
    s_a[e] = (g >= 0 && g < G) ? g : 0;  // placements out of range are read as GPU 0
  }
  __syncthreads();
  if (tid == 0) {  // n_g in ascending expert id
    for (int g = 0; g < G; ++g) s_n[g] = 0.0;
    for (int e = 0; e < E; ++e) s_n[s_a[e]] += s_w[e];
  }
  __syncthreads();
  auto lat_of = [&](int g, double n) {
    return latency_at(knots_n + (size_t)g * nk, knots_t + (size_t)g * nk, nk, n);
  };
  int swaps = 0;
  for (;;) {
    if (tid < G) s_lat[tid] = lat_of(tid, s_n[tid]);
    __syncthreads();
    if (tid == 0) {
      double tot = 0.0;
      for (int g = 0; g < G; ++g) tot += s_lat[g];
      const double fbar = tot / G;
      int hi = 0, lo = 0;
      for (int g = 1; g < G; ++g) {
        if (s_lat[g] > s_lat[hi]) hi = g;
        if (s_lat[g] < s_lat[lo]) lo = g;
      }
      s_hi = hi;
      s_lo = lo;
      s_stop = (swaps >= max_swaps || s_lat[hi] <= (1.0 + eps) * fbar || hi == lo) ? 1 : 0;
    }
    __syncthreads();
    if (s_stop) break;
    const int hi = s_hi, lo = s_lo;
    // experts of hi and lo in ascending id (wave 0 compacts with ballots)
    if (wave == 0) {
      int nh = 0, nl = 0;
      for (int base = 0; base < E; base += kWave) {
        const int e = base + lane;
        const bool in_h = e < E && s_a[e] == hi, in_l = e < E && s_a[e] == lo;
        const uint64_t bh = __ballot(in_h), bl = __ballot(in_l);
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        if (in_h) s_hi_list[nh + __popcll(bh & below)] = e;
        if (in_l) s_lo_list[nl + __popcll(bl & below)] = e;
        nh += __popcll(bh);
        nl += __popcll(bl);
      }
      if (lane == 0) {
        s_nhi = nh;
        s_nlo = nl;
      }
    }
    __syncthreads();
    const int nh = s_nhi, nl = s_nlo;
    const double lat_hi = s_lat[hi], n_hi = s_n[hi], n_lo = s_n[lo];
    // best swap: largest gain, then lowest (position in hi list, position in lo list)
    double best = 0.0;
    int best_p = 0x7fffffff;
    const int pairs = nh * nl;
    for (int p = tid; p < pairs; p += kPlaceThreads) {
      const int ei = s_hi_list[p / nl], ej = s_lo_list[p % nl];
      const double nhi = n_hi - s_w[ei] + s_w[ej];
      const double nlo = n_lo - s_w[ej] + s_w[ei];
      const double lh = lat_of(hi, nhi), ll = lat_of(lo, nlo);
      const double gain = lat_hi - (lh > ll ? lh : ll);
      if (gain > best) {  // p increases within a thread: the first maximum is kept
        best = gain;
        best_p = p;
      }
    }
    // block arg-max over (gain, -p)
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const double ov = shfl_f64(best, lane ^ off);
      const int op = __shfl(best_p, lane ^ off, kWave);
      if (ov > best || (ov == best && op < best_p)) {
        best = ov;
        best_p = op;
      }
    }
    if (lane == 0) {
      s_red_v[wave] = best;
      s_red_i[wave] = best_p;
    }
    __syncthreads();
    if (tid == 0) {
      double bv = 0.0;
      int bp = 0x7fffffff;
      for (int q = 0; q < kPlaceThreads / kWave; ++q)
        if (s_red_v[q] > bv || (s_red_v[q] == bv && s_red_i[q] < bp)) {
          bv = s_red_v[q];
          bp = s_red_i[q];
        }
      if (bp == 0x7fffffff) {
        s_stop = 1;  // no swap lowers the pair's latency
      } else {
        const int ei = s_hi_list[bp / nl], ej = s_lo_list[bp % nl];
        const double nhi = n_hi - s_w[ei] + s_w[ej];
        const double nlo = n_lo - s_w[ej] + s_w[ei];
        s_a[ei] = lo;
        s_a[ej] = hi;
        s_n[hi] = nhi;
        s_n[lo] = nlo;
      }
    }
    __syncthreads();
    if (s_stop) break;
    ++swaps;
  }
  for (int e = tid; e < E; e += kPlaceThreads) a[e] = s_a[e];
  if (tid == 0 && n_swaps) n_swaps[l] = swaps;
}

// ---------------------------------------------------------------------------
// Predicted cost of a placement (Section 4.2.3): per layer and GPU, the load
// n_g = sum_{e in S_g} w_e (ascending e), f_g(n_g), and the grouped reading
// sum_{e in S_g} f_g(w_e). The layer latency is the maximum over GPUs.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kWave) void placement_cost_kernel(const double* __restrict__ W,
                                                               const int32_t* __restrict__ assign, int E,
                                                               const double* __restrict__ knots_n,
                                                               const double* __restrict__ knots_t, int G, int nk,
                                                               double* __restrict__ loads,
                                                               double* __restrict__ lat,
                                                               double* __restrict__ lat_grouped) {
  const int l = blockIdx.x, g = threadIdx.x;
  if (g >= G) return;
  const double* w = W + (size_t)l * E;
  const int32_t* a = assign + (size_t)l * E;
  const double* kn = knots_n + (size_t)g * nk;
  const double* kt = knots_t + (size_t)g * nk;
  double n = 0.0, grouped = 0.0;
  for (int e = 0; e < E; ++e)
    if (a[e] == g) {
      n += w[e];
      grouped += latency_at(kn, kt, nk, w[e]);
    }
  if (loads) loads[(size_t)l * G + g] = n;
  lat[(size_t)l * G + g] = latency_at(kn, kt, nk, n);
  if (lat_grouped) lat_grouped[(size_t)l * G + g] = grouped;
}

// ---------------------------------------------------------------------------
// Drift detector (Section 4.2.4): window sums and cosine distance per layer.
// ---------------------------------------------------------------------------
__global__ void window_push_kernel(const int32_t* __restrict__ counts, int32_t* __restrict__ ring_slot,
                                   double* __restrict__ sums, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int32_t c = counts[i];
  sums[i] = sums[i] + (double)c - (double)ring_slot[i];
  ring_slot[i] = c;
}

// One block: thread t handles layers t, t + 256, ...; the trigger is the OR
// of d > delta over all layers, written by thread 0 (no atomics, no memset).
__global__ __launch_bounds__(256) void drift_distance_kernel(const double* __restrict__ w_cur,
                                                             const double* __restrict__ w_ref, int L, int E,
                                                             double delta, double* __restrict__ d,
                                                             int32_t* __restrict__ trigger) {
  bool over = false;
  for (int l = threadIdx.x; l < L; l += 256) {
    const double* u = w_cur + (size_t)l * E;
    const double* v = w_ref + (size_t)l * E;
    double dot = 0.0, na = 0.0, nb = 0.0;
    for (int e = 0; e < E; ++e) {
      dot += u[e] * v[e];
      na += u[e] * u[e];
      nb += v[e] * v[e];
    }
    double dist;
    if (na == 0.0 || nb == 0.0)
      dist = (na == nb) ? 0.0 : 1.0;
    else
      dist = 1.0 - dot / (__builtin_sqrt(na) * __builtin_sqrt(nb));
    d[l] = dist;
    over = over || dist > delta;
  }
  const int any = __syncthreads_or(over ? 1 : 0);
  if (threadIdx.x == 0 && trigger) *trigger = any ? 1 : 0;
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
hipError_t launch_place_greedy(const double* W, int L, int E, const double* kn, const double* kt, int G, int nk,
                               int cap, int32_t* assign, double* loads, double* targets, hipStream_t s) {
  if (L == 0) return hipSuccess;
  place_greedy_kernel<<<L, kPlaceThreads, 0, s>>>(W, E, kn, kt, G, nk, cap, assign, loads, targets);
  return hipGetLastError();
}

hipError_t launch_place_incremental(const double* W, int L, int E, const double* kn, const double* kt, int G,
                                    int nk, double eps, int max_swaps, int32_t* assign, int32_t* n_swaps,
                                    hipStream_t s) {
  if (L == 0) return hipSuccess;
  place_incremental_kernel<<<L, kPlaceThreads, 0, s>>>(W, E, kn, kt, G, nk, eps, max_swaps, assign, n_swaps);
  return hipGetLastError();
}

hipError_t launch_placement_cost(const double* W, const int32_t* assign, int L, int E, const double* kn,
                                 const double* kt, int G, int nk, double* loads, double* lat, double* lat_grouped,
                                 hipStream_t s) {
  if (L == 0) return hipSuccess;
  placement_cost_kernel<<<L, kWave, 0, s>>>(W, assign, E, kn, kt, G, nk, loads, lat, lat_grouped);
  return hipGetLastError();
}

hipError_t launch_window_push(const int32_t* counts, int32_t* ring, double* sums, int L, int E, int slot,
                              hipStream_t s) {
  const size_t n = (size_t)L * E;
  if (n == 0) return hipSuccess;
  window_push_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(counts, ring + (size_t)slot * n, sums, n);
  return hipGetLastError();
}

hipError_t launch_drift_distance(const double* w_cur, const double* w_ref, int L, int E, double delta, double* d,
                                 int32_t* trigger, hipStream_t s) {
  drift_distance_kernel<<<1, 256, 0, s>>>(w_cur, w_ref, L, E, delta, d, trigger);
  return hipGetLastError();
}

}  // namespace moe
