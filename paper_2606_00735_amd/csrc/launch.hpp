// Host-side launchers of the libmoe kernels. Arguments are validated by the
// C ABI (moe_abi.cpp) before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.hpp"

namespace moe {

// ws (optional, gate_ws_bytes): fp32 partial logits of the K-split router.
size_t gate_ws_bytes(int T, int H, int E, bool bf16);
hipError_t launch_gate_topk(const void* x, const void* wr, const float* bias, int T, int H, int E, int k,
                            bool bf16, float* logits, int32_t* ids, float* wts, void* ws, hipStream_t s);
hipError_t launch_router_logits_split(const void* x, const void* wr, int T, int H, int E, int S, float* part,
                                      hipStream_t s);

size_t hist_ws_bytes(int T, int E, int E_local);
hipError_t launch_hist_scan(const int32_t* ids, int T, int k, const SlotMap& map, int32_t* counts,
                            int32_t* offsets, void* ws, hipStream_t s);
hipError_t launch_permute(const void* x, const int32_t* ids, const SlotMap& map, const void* ws, int T, int H,
                          int k, int M_cap, bool bf16, void* x_perm, int32_t* perm_src, int32_t* dest,
                          hipStream_t s);
hipError_t launch_combine(const void* y, const float* w, const int32_t* dest, int T, int k, int H, int M_cap,
                          bool bf16, void* out, hipStream_t s);

size_t ffn_ws_bytes(int M_cap, int E_local, int H, int I, bool bf16);
// bytes of a workspace that cannot shrink (counters, h, plan); a workspace of
// at least this many bytes serves a call, with less room to split tiles
size_t ffn_ws_fixed(int M_cap, int E_local, int H, int I, bool bf16);
// a_src != nullptr (bf16 only): the gate/up GEMM's row m is row
// a_src[m] / a_div of x_perm, which then holds a_T rows (see GemmArgs).
// ws_cap: bytes of ws when smaller than ffn_ws_bytes (>= ffn_ws_fixed).
hipError_t launch_ffn(const void* x_perm, const void* w_gate, const void* w_up, const void* w_down,
                      const int32_t* offsets, int E_local, int H, int I, int ld_gu, int ld_dn, int M_cap, bool bf16,
                      void* y_perm, void* ws, hipStream_t s, const int32_t* a_src = nullptr, int a_div = 1,
                      int a_T = 0, size_t ws_cap = SIZE_MAX);
// The FFN scratch of this process on the current device (kScratchBytes),
// resolved on first use; its counters are cleared on stream s then.
constexpr size_t kScratchBytes = (size_t)128 << 20;
hipError_t ffn_scratch(void** out, hipStream_t s);
hipError_t launch_set_offsets(int32_t* offsets, int m, hipStream_t s);

// MXFP8: code rows of weight operands (and of quantiser outputs) are
// ldw / ldb / ldc bytes apart; activation codes are dense.
hipError_t launch_mx_quantize(const void* x, bool f32, int batch, int rows, int K, int ldc,
                              const int32_t* row_count, uint8_t* codes, uint32_t* scales, hipStream_t s);
hipError_t launch_gateup_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                            const uint8_t* wuq, const uint32_t* wus, const int32_t* offsets, int E_local, int H,
                            int I, int ldw, int M_cap, uint8_t* hq, uint32_t* hs, hipStream_t s);
hipError_t launch_gemm_mx(const uint8_t* aq, const uint32_t* as, const uint8_t* bq, const uint32_t* bs,
                          const int32_t* offsets, int E_local, int N, int K, int ldb, int M_cap, void* c,
                          hipStream_t s);
size_t ffn_mx_ws_bytes(int M_cap, int E_local, int H, int I);
hipError_t launch_ffn_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq, const uint32_t* wgs,
                         const uint8_t* wuq, const uint32_t* wus, const uint8_t* wdq, const uint32_t* wds,
                         const int32_t* offsets, int E_local, int H, int I, int ld_gu, int ld_dn, int M_cap,
                         void* y_perm, void* ws, hipStream_t s);

hipError_t launch_place_greedy(const double* W, int L, int E, const double* kn, const double* kt, int G, int nk,
                               int cap, int32_t* assign, double* loads, double* targets, hipStream_t s);
hipError_t launch_place_incremental(const double* W, int L, int E, const double* kn, const double* kt, int G,
                                    int nk, double eps, int max_swaps, int32_t* assign, int32_t* n_swaps,
                                    hipStream_t s);
hipError_t launch_placement_cost(const double* W, const int32_t* assign, int L, int E, const double* kn,
                                 const double* kt, int G, int nk, double* loads, double* lat, double* lat_grouped,
                                 hipStream_t s);
hipError_t launch_window_push(const int32_t* counts, int32_t* ring, double* sums, int L, int E, int slot,
                              hipStream_t s);
hipError_t launch_drift_distance(const double* w_cur, const double* w_ref, int L, int E, double delta, double* d,
                                 int32_t* trigger, hipStream_t s);

}  // namespace moe
