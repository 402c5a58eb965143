// C ABI of libmoe (declared in include/moe.h): argument validation on the
// host, then stream-ordered kernel launches. Nothing here allocates device
// memory; the load sweep creates HIP events only.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "../../include/moe.h"
#include "common.hpp"
#include "launch.hpp"

namespace {

using moe::SlotMap;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
bool valid_dtype(moe_dtype dt) { return dt == MOE_F32 || dt == MOE_BF16; }

moe_status hip_status(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_ERR_HIP; }

// Validates a host expert map: entries in [-1, E_local), slots 0..E_local-1
// each used exactly once.
moe_status build_slot_map(const int32_t* expert_map, int E, int E_local, SlotMap* m) {
  if (expert_map == nullptr) return MOE_ERR_INVALID_ARG;
  if (E < 1 || E > MOE_MAX_EXPERTS || E_local < 0 || E_local > E) return MOE_ERR_INVALID_ARG;
  m->n_experts = E;
  m->n_local = E_local;
  for (int i = 0; i < moe::kMaxExperts; ++i) {
    m->slot_of[i] = -1;
    m->expert_of[i] = -1;
  }
  for (int e = 0; e < E; ++e) {
    const int s = expert_map[e];
    if (s < -1 || s >= E_local) return MOE_ERR_INVALID_ARG;
    if (s >= 0) {
      if (m->expert_of[s] != -1) return MOE_ERR_INVALID_ARG;  // slot used twice
      m->expert_of[s] = static_cast<int16_t>(e);
      m->slot_of[e] = static_cast<int16_t>(s);
    }
  }
  for (int s = 0; s < E_local; ++s)
    if (m->expert_of[s] == -1) return MOE_ERR_INVALID_ARG;  // slot unused
  return MOE_OK;
}

moe_status check_tk(int T, int k, int E) {
  if (T < 0 || E < 1 || E > MOE_MAX_EXPERTS) return MOE_ERR_INVALID_ARG;
  if (k < 1 || k > E || k > MOE_MAX_TOPK) return MOE_ERR_INVALID_ARG;
  if ((long long)T * k > INT_MAX) return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

moe_status ffn_shape_ok(int E_local, int H, int I, int M_cap, moe_dtype dt) {
  if (!valid_dtype(dt) || E_local < 0 || H < 1 || I < 1 || M_cap < 0) return MOE_ERR_INVALID_ARG;
  if (E_local > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
  if (dt == MOE_BF16 && (H % 128 != 0 || I % 128 != 0)) return MOE_ERR_UNSUPPORTED;
  if (dt == MOE_F32 && (H % 4 != 0 || I % 4 != 0)) return MOE_ERR_UNSUPPORTED;
  // the fp32 kernels use one thread per output element
  if (dt == MOE_F32 && (long long)M_cap * std::max(H, I) > (long long)INT_MAX) return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

// Row stride of an expert weight matrix whose rows hold K elements: 0 means
// K (dense); otherwise at least K, a whole number of 16-byte pieces and small
// enough that 256 rows span less than 2^31 bytes (32-bit lane offsets).
moe_status resolve_ld(int ld, int K, moe_dtype dt, int* out) {
  if (ld == 0) ld = K;
  const int per16 = dt == MOE_BF16 ? 8 : 4;
  if (ld < K || ld % per16 != 0 || ld > (1 << 20)) return MOE_ERR_INVALID_ARG;
  *out = ld;
  return MOE_OK;
}

// Row stride in bytes of MXFP8 weight codes with K codes a row: 0 means K;
// otherwise at least K, a multiple of 16 and at most 2^20.
moe_status resolve_ld_mx(int ld, int K, int* out) {
  if (ld == 0) ld = K;
  if (ld < K || ld % 16 != 0 || ld > (1 << 20)) return MOE_ERR_INVALID_ARG;
  *out = ld;
  return MOE_OK;
}

// The timing loop shared by the load sweeps: for each M of Ms, sets
// offsets = [0, M], then runs `run(rot, M)` warmup + iters times rotating
// through n_rot weight copies, each timed run bracketed by HIP events.
template <class Run>
moe_status sweep_loop(const int32_t* Ms, int nM, int warmup, int iters, int n_rot, int32_t* offsets,
                      float* us_out, float* us_all, hipStream_t stream, Run&& run) {
  std::vector<hipEvent_t> ev(2 * (size_t)iters, nullptr);
  for (auto& e : ev)
    if (hipEventCreate(&e) != hipSuccess) {
      for (auto& d : ev)
        if (d) (void)hipEventDestroy(d);
      return MOE_ERR_HIP;
    }
  std::vector<float> t(iters);
  moe_status result = MOE_OK;
  int rot = 0;
  for (int mi = 0; mi < nM && result == MOE_OK; ++mi) {
    const int m = Ms[mi];
    if (moe::launch_set_offsets(offsets, m, stream) != hipSuccess) {
      result = MOE_ERR_HIP;
      break;
    }
    for (int it = 0; it < warmup + iters; ++it) {
      const int r = rot;
      rot = (rot + 1) % n_rot;
      const int ti = it - warmup;
      if (ti >= 0 && hipEventRecord(ev[2 * ti], stream) != hipSuccess) {
        result = MOE_ERR_HIP;
        break;
      }
      if (run(r, m) != hipSuccess) {
        result = MOE_ERR_HIP;
        break;
      }
      if (ti >= 0 && hipEventRecord(ev[2 * ti + 1], stream) != hipSuccess) {
        result = MOE_ERR_HIP;
        break;
      }
    }
    if (result != MOE_OK) break;
    if (hipEventSynchronize(ev[2 * iters - 1]) != hipSuccess) {
      result = MOE_ERR_HIP;
      break;
    }
    for (int i = 0; i < iters; ++i) {
      float ms = 0.0f;
      if (hipEventElapsedTime(&ms, ev[2 * i], ev[2 * i + 1]) != hipSuccess) {
        result = MOE_ERR_HIP;
        break;
      }
      t[i] = ms * 1000.0f;
      if (us_all) us_all[(size_t)mi * iters + i] = t[i];
    }
    std::vector<float> sorted(t);
    std::sort(sorted.begin(), sorted.end());
    us_out[mi] = (iters % 2) ? sorted[iters / 2] : 0.5f * (sorted[iters / 2 - 1] + sorted[iters / 2]);
  }
  if (result != MOE_OK) (void)hipStreamSynchronize(stream);
  for (auto& e : ev) (void)hipEventDestroy(e);
  return result;
}

// Shape limits of the MXFP8 GEMMs: every K and N a multiple of the 128-wide
// scale chunk, row and byte counts within int / size_t range.
moe_status mx_gemm_shape_ok(int E_local, int N, int K, int M_cap) {
  if (E_local < 0 || N < 1 || K < 1 || M_cap < 0) return MOE_ERR_INVALID_ARG;
  if (E_local > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
  if (N % 128 != 0 || K % 128 != 0) return MOE_ERR_UNSUPPORTED;
  // tile offsets (256 rows of K bytes) are 32-bit in the kernels
  if (N > (1 << 20) || K > (1 << 20)) return MOE_ERR_UNSUPPORTED;
  if ((long long)M_cap * std::max(N, K) > (1LL << 40)) return MOE_ERR_UNSUPPORTED;
  return MOE_OK;
}

bool mx_operand_ok(const void* codes, const void* scales) {
  return codes && scales && aligned16(codes) && aligned4(scales);
}

}  // namespace

extern "C" {

const char* moe_status_string(moe_status s) {
  switch (s) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported shape or option";
    case MOE_ERR_WORKSPACE: return "workspace too small";
    case MOE_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

int moe_abi_version(void) { return MOE_ABI_VERSION; }

moe_status moe_gate_topk(const void* x, const void* w_router, const float* bias, int T, int H, int E, int k,
                         moe_dtype dt, float* logits_out, int32_t* topk_ids, float* topk_w, void* ws,
                         size_t* ws_bytes, hipStream_t stream) {
  moe_status st = check_tk(T, k, E);
  if (st != MOE_OK) return st;
  if (!valid_dtype(dt) || H < 1 || H % 8 != 0) return MOE_ERR_INVALID_ARG;
  if (dt == MOE_BF16 && H % 64 != 0) return MOE_ERR_UNSUPPORTED;
  const size_t need = moe::gate_ws_bytes(T, H, E, dt == MOE_BF16);
  if (ws == nullptr && ws_bytes != nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (ws != nullptr && (ws_bytes == nullptr || !aligned16(ws))) return MOE_ERR_INVALID_ARG;
  if (ws != nullptr && *ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (T == 0) return MOE_OK;
  if (!x || !w_router || !topk_ids || !topk_w) return MOE_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(w_router) || !aligned4(topk_ids) || !aligned4(topk_w) ||
      (bias && !aligned4(bias)) || (logits_out && !aligned4(logits_out)))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_gate_topk(x, w_router, bias, T, H, E, k, dt == MOE_BF16, logits_out, topk_ids,
                                          topk_w, need > 0 ? ws : nullptr, stream));
}

moe_status moe_expert_histogram_scan(const int32_t* topk_ids, int T, int k, int E, const int32_t* expert_map,
                                     int E_local, int32_t* counts, int32_t* offsets, void* ws,
                                     size_t* ws_bytes, hipStream_t stream) {
  moe_status st = check_tk(T, k, E);
  if (st != MOE_OK) return st;
  if (E_local < 0 || E_local > E || ws_bytes == nullptr) return MOE_ERR_INVALID_ARG;
  const size_t need = moe::hist_ws_bytes(T, E, E_local);
  if (ws == nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (*ws_bytes < need) return MOE_ERR_WORKSPACE;
  SlotMap map;
  st = build_slot_map(expert_map, E, E_local, &map);
  if (st != MOE_OK) return st;
  if (!counts || !offsets || (T > 0 && !topk_ids)) return MOE_ERR_INVALID_ARG;
  if (!aligned4(counts) || !aligned4(offsets) || !aligned16(ws) || (topk_ids && !aligned4(topk_ids)))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_hist_scan(topk_ids, T, k, map, counts, offsets, ws, stream));
}

moe_status moe_permute(const void* x, const int32_t* topk_ids, const int32_t* expert_map, const void* ws,
                       size_t ws_bytes, int T, int H, int k, int E, int E_local, int M_cap, moe_dtype dt,
                       void* x_perm, int32_t* perm_src, int32_t* dest, hipStream_t stream) {
  moe_status st = check_tk(T, k, E);
  if (st != MOE_OK) return st;
  if (!valid_dtype(dt) || H < 1 || H % 8 != 0 || E_local < 0 || E_local > E) return MOE_ERR_INVALID_ARG;
  if (M_cap < 0 || (long long)M_cap < (long long)T * k) return MOE_ERR_INVALID_ARG;
  SlotMap map;
  st = build_slot_map(expert_map, E, E_local, &map);
  if (st != MOE_OK) return st;
  if (ws == nullptr) return MOE_ERR_INVALID_ARG;
  if (ws_bytes < moe::hist_ws_bytes(T, E, E_local)) return MOE_ERR_WORKSPACE;
  if (T == 0) return MOE_OK;
  if (!x || !topk_ids || !dest || (M_cap > 0 && !perm_src)) return MOE_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(ws) || (x_perm && !aligned16(x_perm)) || !aligned4(topk_ids) ||
      !aligned4(dest) || (perm_src && !aligned4(perm_src)))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_permute(x, topk_ids, map, ws, T, H, k, M_cap, dt == MOE_BF16, x_perm, perm_src,
                                        dest, stream));
}

moe_status moe_grouped_swiglu_ffn(const void* x_perm, const void* w_gate, const void* w_up, const void* w_down,
                                  const int32_t* offsets, int E_local, int H, int I, int ldw_gu, int ldw_dn,
                                  int M_cap, moe_dtype dt, void* y_perm, void* ws, size_t* ws_bytes,
                                  hipStream_t stream) {
  moe_status st = ffn_shape_ok(E_local, H, I, M_cap, dt);
  if (st != MOE_OK) return st;
  int ld_gu = 0, ld_dn = 0;
  if ((st = resolve_ld(ldw_gu, H, dt, &ld_gu)) != MOE_OK || (st = resolve_ld(ldw_dn, I, dt, &ld_dn)) != MOE_OK)
    return st;
  if (ws_bytes == nullptr) return MOE_ERR_INVALID_ARG;
  const size_t need = moe::ffn_ws_bytes(M_cap, E_local, H, I, dt == MOE_BF16);
  if (ws == nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (*ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (E_local == 0 || M_cap == 0) return MOE_OK;
  if (!x_perm || !w_gate || !w_up || !w_down || !offsets || !y_perm) return MOE_ERR_INVALID_ARG;
  if (!aligned16(x_perm) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) || !aligned16(y_perm) ||
      !aligned16(ws) || !aligned4(offsets))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_ffn(x_perm, w_gate, w_up, w_down, offsets, E_local, H, I, ld_gu, ld_dn, M_cap,
                                    dt == MOE_BF16, y_perm, ws, stream));
}

moe_status moe_grouped_swiglu_ffn_noalloc(const void* x_perm, const void* w_gate, const void* w_up,
                                          const void* w_down, const int32_t* offsets, int E_local, int H, int I,
                                          int ldw_gu, int ldw_dn, int M_cap, moe_dtype dt, void* y_perm,
                                          hipStream_t stream) {
  moe_status st = ffn_shape_ok(E_local, H, I, M_cap, dt);
  if (st != MOE_OK) return st;
  int ld_gu = 0, ld_dn = 0;
  if ((st = resolve_ld(ldw_gu, H, dt, &ld_gu)) != MOE_OK || (st = resolve_ld(ldw_dn, I, dt, &ld_dn)) != MOE_OK)
    return st;
  // the part of the workspace that cannot shrink must fit the scratch
  if (moe::ffn_ws_fixed(M_cap, E_local, H, I, dt == MOE_BF16) > moe::kScratchBytes) return MOE_ERR_WORKSPACE;
  if (E_local == 0 || M_cap == 0) return MOE_OK;
  if (!x_perm || !w_gate || !w_up || !w_down || !offsets || !y_perm) return MOE_ERR_INVALID_ARG;
  if (!aligned16(x_perm) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) || !aligned16(y_perm) ||
      !aligned4(offsets))
    return MOE_ERR_INVALID_ARG;
  void* ws = nullptr;
  if (moe::ffn_scratch(&ws, stream) != hipSuccess) return MOE_ERR_HIP;
  return hip_status(moe::launch_ffn(x_perm, w_gate, w_up, w_down, offsets, E_local, H, I, ld_gu, ld_dn, M_cap,
                                    dt == MOE_BF16, y_perm, ws, stream, nullptr, 1, 0, moe::kScratchBytes));
}

size_t moe_ffn_scratch_bytes(void) { return moe::kScratchBytes; }

moe_status moe_grouped_swiglu_ffn_gather(const void* x, const int32_t* perm_src, int T, int k, const void* w_gate,
                                         const void* w_up, const void* w_down, const int32_t* offsets, int E_local,
                                         int H, int I, int ldw_gu, int ldw_dn, int M_cap, moe_dtype dt,
                                         void* y_perm, void* ws, size_t* ws_bytes, hipStream_t stream) {
  moe_status st = ffn_shape_ok(E_local, H, I, M_cap, dt);
  if (st != MOE_OK) return st;
  int ld_gu = 0, ld_dn = 0;
  if ((st = resolve_ld(ldw_gu, H, dt, &ld_gu)) != MOE_OK || (st = resolve_ld(ldw_dn, I, dt, &ld_dn)) != MOE_OK)
    return st;
  if (ws_bytes == nullptr || T < 1 || k < 1 || k > MOE_MAX_TOPK) return MOE_ERR_INVALID_ARG;
  if (dt != MOE_BF16) return MOE_ERR_UNSUPPORTED;
  // row offsets into x are 32-bit byte offsets
  if ((unsigned long long)T * (unsigned long long)H * 2ull > 0xFFFFFFFFull) return MOE_ERR_UNSUPPORTED;
  const size_t need = moe::ffn_ws_bytes(M_cap, E_local, H, I, true);
  if (ws == nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (*ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (E_local == 0 || M_cap == 0) return MOE_OK;
  if (!x || !perm_src || !w_gate || !w_up || !w_down || !offsets || !y_perm) return MOE_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) || !aligned16(y_perm) ||
      !aligned16(ws) || !aligned4(offsets) || !aligned4(perm_src))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_ffn(x, w_gate, w_up, w_down, offsets, E_local, H, I, ld_gu, ld_dn, M_cap, true,
                                    y_perm, ws, stream, perm_src, k, T));
}

moe_status moe_unpermute_combine(const void* y_perm, const float* topk_w, const int32_t* dest, int T, int k,
                                 int H, int M_cap, moe_dtype dt, void* out, hipStream_t stream) {
  if (T < 0 || k < 1 || k > MOE_MAX_TOPK || H < 1 || M_cap < 0 || !valid_dtype(dt)) return MOE_ERR_INVALID_ARG;
  if ((long long)T * k > INT_MAX) return MOE_ERR_UNSUPPORTED;
  if (H % (dt == MOE_BF16 ? 8 : 4) != 0) return MOE_ERR_INVALID_ARG;
  if (T == 0) return MOE_OK;
  if (!topk_w || !dest || !out || (M_cap > 0 && !y_perm)) return MOE_ERR_INVALID_ARG;
  if (!aligned16(out) || (y_perm && !aligned16(y_perm)) || !aligned4(topk_w) || !aligned4(dest))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_combine(y_perm, topk_w, dest, T, k, H, M_cap, dt == MOE_BF16, out, stream));
}

moe_status moe_load_sweep(const void* x, const void* w_gate, const void* w_up, const void* w_down, int n_rot,
                          int H, int I, int ldw_gu, int ldw_dn, moe_dtype dt, const int32_t* Ms, int nM,
                          int warmup, int iters,
                          void* y_scratch, void* ws, size_t* ws_bytes, float* us_out, float* us_all,
                          hipStream_t stream) {
  if (Ms == nullptr || nM < 1 || nM > 64 || warmup < 0 || iters < 1 || iters > 10000 || n_rot < 1 ||
      ws_bytes == nullptr)
    return MOE_ERR_INVALID_ARG;
  int max_m = 0;
  for (int i = 0; i < nM; ++i) {
    if (Ms[i] < 1 || Ms[i] > (1 << 20)) return MOE_ERR_INVALID_ARG;
    max_m = std::max(max_m, Ms[i]);
  }
  moe_status st = ffn_shape_ok(1, H, I, max_m, dt);
  if (st != MOE_OK) return st;
  int ld_gu = 0, ld_dn = 0;
  if ((st = resolve_ld(ldw_gu, H, dt, &ld_gu)) != MOE_OK || (st = resolve_ld(ldw_dn, I, dt, &ld_dn)) != MOE_OK)
    return st;
  const bool bf16 = dt == MOE_BF16;
  const size_t ffn_ws = moe::ffn_ws_bytes(max_m, 1, H, I, bf16);
  const size_t need = ffn_ws + 256;
  if (ws == nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (*ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (!x || !w_gate || !w_up || !w_down || !y_scratch || !us_out) return MOE_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) || !aligned16(y_scratch) ||
      !aligned16(ws))
    return MOE_ERR_INVALID_ARG;

  const size_t es = bf16 ? 2 : 4;
  const size_t wgu = (size_t)I * ld_gu * es, wdn = (size_t)H * ld_dn * es;  // bytes of one copy
  int32_t* offsets = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + ffn_ws);
  return sweep_loop(Ms, nM, warmup, iters, n_rot, offsets, us_out, us_all, stream, [&](int rot, int m) {
    const char* g = static_cast<const char*>(w_gate) + (size_t)rot * wgu;
    const char* u = static_cast<const char*>(w_up) + (size_t)rot * wgu;
    const char* d = static_cast<const char*>(w_down) + (size_t)rot * wdn;
    return moe::launch_ffn(x, g, u, d, offsets, 1, H, I, ld_gu, ld_dn, m, bf16, y_scratch, ws, stream);
  });
}

moe_status moe_load_sweep_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                             const uint8_t* wuq, const uint32_t* wus, const uint8_t* wdq, const uint32_t* wds,
                             int n_rot, int H, int I, int ldw_gu, int ldw_dn, const int32_t* Ms, int nM, int warmup,
                             int iters,
                             void* y_scratch, void* ws, size_t* ws_bytes, float* us_out, float* us_all,
                             hipStream_t stream) {
  if (Ms == nullptr || nM < 1 || nM > 64 || warmup < 0 || iters < 1 || iters > 10000 || n_rot < 1 ||
      ws_bytes == nullptr)
    return MOE_ERR_INVALID_ARG;
  int max_m = 0;
  for (int i = 0; i < nM; ++i) {
    if (Ms[i] < 1 || Ms[i] > (1 << 20)) return MOE_ERR_INVALID_ARG;
    max_m = std::max(max_m, Ms[i]);
  }
  moe_status st = mx_gemm_shape_ok(1, I, H, max_m);
  if (st != MOE_OK) return st;
  int ld_gu = 0, ld_dn = 0;
  if ((st = resolve_ld_mx(ldw_gu, H, &ld_gu)) != MOE_OK || (st = resolve_ld_mx(ldw_dn, I, &ld_dn)) != MOE_OK)
    return st;
  // x and its scales are laid out for max_m rows, so every run uses
  // M_cap = max_m with offsets [0, M]
  const size_t ffn_ws = moe::ffn_mx_ws_bytes(max_m, 1, H, I);
  const size_t need = ffn_ws + 256;
  if (ws == nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (*ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (!mx_operand_ok(xq, xs) || !mx_operand_ok(wgq, wgs) || !mx_operand_ok(wuq, wus) ||
      !mx_operand_ok(wdq, wds) || !y_scratch || !aligned16(y_scratch) || !aligned16(ws) || !us_out)
    return MOE_ERR_INVALID_ARG;
  const size_t wgu = (size_t)I * ld_gu, wdn = (size_t)H * ld_dn;  // code bytes of one copy
  const size_t smat = (size_t)(H / 128) * I;           // scale dwords of W_gate / W_up
  const size_t sdown = (size_t)(I / 128) * H;          // scale dwords of W_down
  int32_t* offsets = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + ffn_ws);
  return sweep_loop(Ms, nM, warmup, iters, n_rot, offsets, us_out, us_all, stream, [&](int rot, int m) {
    return moe::launch_ffn_mx(xq, xs, wgq + rot * wgu, wgs + rot * smat, wuq + rot * wgu, wus + rot * smat,
                              wdq + rot * wdn, wds + rot * sdown, offsets, 1, H, I, ld_gu, ld_dn, max_m, y_scratch,
                              ws, stream);
  });
}

}  // extern "C"

// ---------------------------------------------------------------------------
// MXFP8 expert FFN
// ---------------------------------------------------------------------------
extern "C" {

moe_status moe_mx_quantize(const void* x, moe_dtype dt, int batch, int rows, int K, int ld_codes,
                           const int32_t* row_count, uint8_t* codes, uint32_t* scales, hipStream_t stream) {
  if (!valid_dtype(dt) || batch < 0 || rows < 0 || K < 1) return MOE_ERR_INVALID_ARG;
  if (K % 128 != 0) return MOE_ERR_UNSUPPORTED;
  int ldc = 0;
  if (resolve_ld_mx(ld_codes, K, &ldc) != MOE_OK) return MOE_ERR_INVALID_ARG;
  if ((long long)batch * rows * K > (1LL << 40)) return MOE_ERR_UNSUPPORTED;
  if (row_count != nullptr && (batch > 1 || !aligned4(row_count))) return MOE_ERR_INVALID_ARG;
  if (batch == 0 || rows == 0) return MOE_OK;
  if (!x || !aligned16(x) || !mx_operand_ok(codes, scales)) return MOE_ERR_INVALID_ARG;
  return hip_status(
      moe::launch_mx_quantize(x, dt == MOE_F32, batch, rows, K, ldc, row_count, codes, scales, stream));
}

moe_status moe_grouped_swiglu_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                                 const uint8_t* wuq, const uint32_t* wus, const int32_t* offsets, int E_local,
                                 int H, int I, int ldw, int M_cap, uint8_t* hq, uint32_t* hs, hipStream_t stream) {
  moe_status st = mx_gemm_shape_ok(E_local, I, H, M_cap);
  if (st != MOE_OK) return st;
  int ld = 0;
  if ((st = resolve_ld_mx(ldw, H, &ld)) != MOE_OK) return st;
  if (E_local == 0 || M_cap == 0) return MOE_OK;
  if (!mx_operand_ok(xq, xs) || !mx_operand_ok(wgq, wgs) || !mx_operand_ok(wuq, wus) || !mx_operand_ok(hq, hs) ||
      !offsets || !aligned4(offsets))
    return MOE_ERR_INVALID_ARG;
  return hip_status(
      moe::launch_gateup_mx(xq, xs, wgq, wgs, wuq, wus, offsets, E_local, H, I, ld, M_cap, hq, hs, stream));
}

moe_status moe_grouped_gemm_mx(const uint8_t* aq, const uint32_t* as, const uint8_t* bq, const uint32_t* bs,
                               const int32_t* offsets, int E_local, int N, int K, int ldb, int M_cap, void* c,
                               hipStream_t stream) {
  moe_status st = mx_gemm_shape_ok(E_local, N, K, M_cap);
  if (st != MOE_OK) return st;
  int ld = 0;
  if ((st = resolve_ld_mx(ldb, K, &ld)) != MOE_OK) return st;
  if (E_local == 0 || M_cap == 0) return MOE_OK;
  if (!mx_operand_ok(aq, as) || !mx_operand_ok(bq, bs) || !c || !aligned16(c) || !offsets || !aligned4(offsets))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_gemm_mx(aq, as, bq, bs, offsets, E_local, N, K, ld, M_cap, c, stream));
}

moe_status moe_grouped_swiglu_ffn_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                                     const uint8_t* wuq, const uint32_t* wus, const uint8_t* wdq,
                                     const uint32_t* wds, const int32_t* offsets, int E_local, int H, int I,
                                     int ldw_gu, int ldw_dn, int M_cap, void* y_perm, void* ws, size_t* ws_bytes,
                                     hipStream_t stream) {
  moe_status st = mx_gemm_shape_ok(E_local, I, H, M_cap);
  if (st != MOE_OK) return st;
  int ld_gu = 0, ld_dn = 0;
  if ((st = resolve_ld_mx(ldw_gu, H, &ld_gu)) != MOE_OK || (st = resolve_ld_mx(ldw_dn, I, &ld_dn)) != MOE_OK)
    return st;
  if (ws_bytes == nullptr) return MOE_ERR_INVALID_ARG;
  const size_t need = moe::ffn_mx_ws_bytes(M_cap, E_local, H, I);
  if (ws == nullptr) {
    *ws_bytes = need;
    return MOE_OK;
  }
  if (*ws_bytes < need) return MOE_ERR_WORKSPACE;
  if (E_local == 0 || M_cap == 0) return MOE_OK;
  if (!mx_operand_ok(xq, xs) || !mx_operand_ok(wgq, wgs) || !mx_operand_ok(wuq, wus) ||
      !mx_operand_ok(wdq, wds) || !y_perm || !aligned16(y_perm) || !aligned16(ws) || !offsets || !aligned4(offsets))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_ffn_mx(xq, xs, wgq, wgs, wuq, wus, wdq, wds, offsets, E_local, H, I, ld_gu, ld_dn,
                                       M_cap, y_perm, ws, stream));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Placement control path
// ---------------------------------------------------------------------------
namespace {

bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }

moe_status place_shape_ok(const double* w, int L, int E, const double* kn, const double* kt, int G, int nk) {
  if (L < 0 || E < 1 || G < 1 || nk < 1) return MOE_ERR_INVALID_ARG;
  if (E > 1024 || G > 64 || nk > 64) return MOE_ERR_UNSUPPORTED;
  if (L == 0) return MOE_OK;
  if (!w || !kn || !kt) return MOE_ERR_INVALID_ARG;
  if (!aligned8(w) || !aligned8(kn) || !aligned8(kt)) return MOE_ERR_INVALID_ARG;
  return MOE_OK;
}

}  // namespace

extern "C" {

moe_status moe_fit_latency_model(const int32_t* loads, const float* latencies, int n, double* knots_n,
                                 double* knots_t) {
  if (!loads || !latencies || !knots_n || !knots_t || n < 1 || n > 64) return MOE_ERR_INVALID_ARG;
  std::vector<int> order(n);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int a, int b) { return loads[a] < loads[b]; });
  double run = -INFINITY;
  for (int i = 0; i < n; ++i) {
    const int j = order[i];
    if (loads[j] <= 0 || !std::isfinite(latencies[j])) return MOE_ERR_INVALID_ARG;
    if (i > 0 && loads[j] == loads[order[i - 1]]) return MOE_ERR_INVALID_ARG;
    run = std::max(run, static_cast<double>(latencies[j]));
    knots_n[i] = static_cast<double>(loads[j]);
    knots_t[i] = run;
  }
  return MOE_OK;
}

moe_status moe_place_greedy(const double* w, int L, int E, const double* knots_n, const double* knots_t, int G,
                            int nk, int cap, int32_t* assign, double* loads, double* targets,
                            hipStream_t stream) {
  moe_status st = place_shape_ok(w, L, E, knots_n, knots_t, G, nk);
  if (st != MOE_OK) return st;
  if (cap < 0 || (cap > 0 && (long long)cap * G < E)) return MOE_ERR_INVALID_ARG;
  if (L == 0) return MOE_OK;
  if (!assign || !aligned4(assign) || (loads && !aligned8(loads)) || (targets && !aligned8(targets)))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_place_greedy(w, L, E, knots_n, knots_t, G, nk, cap, assign, loads, targets, stream));
}

moe_status moe_place_incremental(const double* w, int L, int E, const double* knots_n, const double* knots_t,
                                 int G, int nk, double eps, int max_swaps, int32_t* assign, int32_t* n_swaps,
                                 hipStream_t stream) {
  moe_status st = place_shape_ok(w, L, E, knots_n, knots_t, G, nk);
  if (st != MOE_OK) return st;
  if (!std::isfinite(eps) || eps < 0.0 || max_swaps < 0 || max_swaps > (1 << 20)) return MOE_ERR_INVALID_ARG;
  if (L == 0) return MOE_OK;
  if (!assign || !aligned4(assign) || (n_swaps && !aligned4(n_swaps))) return MOE_ERR_INVALID_ARG;
  return hip_status(
      moe::launch_place_incremental(w, L, E, knots_n, knots_t, G, nk, eps, max_swaps, assign, n_swaps, stream));
}

moe_status moe_placement_cost(const double* w, const int32_t* assign, int L, int E, const double* knots_n,
                              const double* knots_t, int G, int nk, double* loads, double* lat, double* lat_grouped,
                              hipStream_t stream) {
  moe_status st = place_shape_ok(w, L, E, knots_n, knots_t, G, nk);
  if (st != MOE_OK) return st;
  if (L == 0) return MOE_OK;
  if (!assign || !lat || !aligned4(assign) || !aligned8(lat) || (loads && !aligned8(loads)) ||
      (lat_grouped && !aligned8(lat_grouped)))
    return MOE_ERR_INVALID_ARG;
  return hip_status(
      moe::launch_placement_cost(w, assign, L, E, knots_n, knots_t, G, nk, loads, lat, lat_grouped, stream));
}

moe_status moe_window_push(const int32_t* counts, int32_t* ring, double* sums, int L, int E, int window, int slot,
                           hipStream_t stream) {
  if (L < 0 || E < 1 || window < 1 || slot < 0 || slot >= window) return MOE_ERR_INVALID_ARG;
  if (L == 0) return MOE_OK;
  if (!counts || !ring || !sums || !aligned4(counts) || !aligned4(ring) || !aligned8(sums))
    return MOE_ERR_INVALID_ARG;
  return hip_status(moe::launch_window_push(counts, ring, sums, L, E, slot, stream));
}

moe_status moe_drift_distance(const double* w_cur, const double* w_ref, int L, int E, double delta, double* d,
                              int32_t* trigger, hipStream_t stream) {
  if (L < 0 || L > 65536 || E < 1 || !std::isfinite(delta)) return MOE_ERR_INVALID_ARG;
  if (L > 0 && (!w_cur || !w_ref || !d || !aligned8(w_cur) || !aligned8(w_ref) || !aligned8(d)))
    return MOE_ERR_INVALID_ARG;
  if (trigger && !aligned4(trigger)) return MOE_ERR_INVALID_ARG;
  if (L == 0 && !trigger) return MOE_OK;
  return hip_status(moe::launch_drift_distance(w_cur, w_ref, L, E, delta, d, trigger, stream));
}

}  // extern "C"
