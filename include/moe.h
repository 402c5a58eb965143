/*
 * moe.h - C ABI of libmoe: one GPU's share of an expert-parallel MoE layer on
 * AMD Instinct MI355X (gfx950).
 *
 * ViBE (arXiv 2606.00735) balances per-GPU execution time of expert-parallel
 * MoE layers. What it balances is the work of this library: each GPU gates its
 * tokens, builds the per-expert token histogram (one row of the activation
 * matrix W, Section 4.2.2), runs its local experts on the tokens routed to them
 * (its token load n_g = sum of w_e over its experts S_g, Section 4.2.3) and
 * combines the results; the latency of that expert computation as a function
 * of the token load is the per-GPU performance model f_g(n) (Section 4.2.1,
 * Algorithm 1 Phase 1).
 *
 * Conventions shared by every entry point:
 *  - Array arguments are caller-owned DEVICE pointers unless marked "host".
 *    The library allocates no device memory and keeps no device state.
 *  - Matrices are row-major and dense. Weight matrices are stored
 *    out-features by in-features (the nn.Linear layout): row n of a matrix
 *    holds the input weights of output n, so every contraction reads its
 *    operands along contiguous rows.
 *  - bf16 data is IEEE bfloat16 (2 bytes); MOE_F32 data is IEEE binary32.
 *    Gate logits and weights are always fp32.
 *  - Calls are stream-ordered and asynchronous (except moe_load_sweep) and
 *    launch only on `stream`. Pointers must be 16-byte aligned.
 *  - Workspace: call with ws == NULL to receive the byte count in *ws_bytes
 *    (returns MOE_OK, launches nothing). With ws != NULL, *ws_bytes must be at
 *    least that count, else MOE_ERR_WORKSPACE.
 *  - Errors: every call returns a moe_status and never aborts. Arguments are
 *    validated on the host before anything is launched; launch failures are
 *    reported as MOE_ERR_HIP (hipGetLastError after each launch). Device
 *    data the host cannot see (ids, offsets, dest) is clamped inside the
 *    kernels so that no access leaves its buffer.
 *  - Thread safety: calls with distinct workspaces and streams are
 *    independent.
 */
#ifndef MOE_SHARD_MOE_H
#define MOE_SHARD_MOE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_ABI_VERSION 3
#define MOE_MAX_EXPERTS 256 /* E and E_local limit */
#define MOE_MAX_TOPK 16

typedef enum moe_status {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = 1, /* NULL pointer, negative size, k > E, misaligned */
  MOE_ERR_UNSUPPORTED = 2, /* valid but outside what the kernels handle */
  MOE_ERR_WORKSPACE = 3,   /* workspace smaller than the queried size */
  MOE_ERR_HIP = 4          /* a HIP launch or runtime call failed */
} moe_status;

typedef enum moe_dtype { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

/* Short text for a status code (static storage, never NULL). */
const char* moe_status_string(moe_status s);

/* MOE_ABI_VERSION of the built library. */
int moe_abi_version(void);

/*
 * moe_gate_topk - router logits, top-k selection and renormalised gate weights.
 *
 * Section 2 (Mixture-of-Experts and Expert Parallelism): each token is routed
 * to a subset of experts. For token t:
 *   z[t,e]  = fl32( fl32(sum_h x[t,h] * w_router[e,h]) + bias[e] )
 *   ids[t,:] = the k experts with the largest z, ordered by (z descending,
 *              expert id ascending): equal logits go to the lower expert id
 *   w[t,j]  = exp(z_j - z_0) / sum_{j'<k} exp(z_j' - z_0)  (fp32, j ascending)
 *
 * x          [T, H]  dt          token activations
 * w_router   [E, H]  dt          row e = routing vector of expert e
 * bias       [E]     fp32        per-expert logit bias (may be NULL = 0)
 * logits_out [T, E]  fp32        optional (NULL to skip): z
 * topk_ids   [T, k]  int32       selected expert ids
 * topk_w     [T, k]  fp32        gate weights
 * Limits: 1 <= E <= 256, 1 <= k <= min(E, 16), H % 8 == 0 (bf16: H % 64 == 0).
 * ws         optional workspace: with ws == NULL and ws_bytes != NULL the
 *            call stores the byte count in *ws_bytes and launches nothing;
 *            with ws and ws_bytes both NULL the router runs in one pass
 *            without it. Given one (16-byte aligned, *ws_bytes at least the
 *            count, else MOE_ERR_WORKSPACE), bf16 routers compute the logits
 *            as fp32 partial sums over K ranges there and add them in a
 *            fixed order before the top-k:
 *              - batches of at most 256 tokens over at most 128 experts
 *                (when a 32-token block's distinct x and router rows reach
 *                192 KB), and batches over at most 64 experts whose
 *                32-token blocks would fill at most half the CUs: 32-token
 *                blocks times up to 8 K ranges;
 *              - 256 experts (any batch) or 128 experts (up to 4096 tokens;
 *                when H >= 4096, every batch whose 128-token blocks would
 *                fill at most half the CUs): 256-token tiles times K
 *                ranges, so a CU loads 256 tokens' rows and a K range of
 *                the router rows instead of every router row for each 64
 *                or 128 tokens.
 *            The count is 0 where no workspace is used (fp32 and every other
 *            case). It depends on the device's compute-unit count: query it
 *            with the device the call will run on current.
 * T == 0 is a no-op. The kernel accumulates in fp32; inputs whose products
 * and partial sums are exact in fp32 give order-independent logits (and the
 * same logits with or without the workspace).
 */
moe_status moe_gate_topk(const void* x, const void* w_router, const float* bias,
                         int T, int H, int E, int k, moe_dtype dt,
                         float* logits_out, int32_t* topk_ids, float* topk_w,
                         void* ws, size_t* ws_bytes, hipStream_t stream);

/*
 * moe_expert_histogram_scan - the activation profile and local offsets.
 *
 * counts[e] = #{(t,j) : topk_ids[t,j] == e} for all E experts (one row of the
 * activation matrix W of Section 4.2.2). expert_map (HOST array [E]) gives
 * the local slot of each expert on this GPU, or -1 for a remote expert; the
 * local slots must be exactly 0..E_local-1, each used once (the placement
 * S_g of Section 4.2.3). offsets[0] = 0 and offsets[l+1] = offsets[l] +
 * counts[expert in slot l]; offsets[E_local] is the GPU's token load.
 *
 * counts  [E]          int32 (device, written)
 * offsets [E_local+1]  int32 (device, written)
 * ws      per-block count table and per-block row bases; pass it unchanged
 *         to moe_permute. Size depends on T, E and E_local only.
 * Limits: 1 <= E <= 256, 0 <= E_local <= E, 1 <= k <= min(E, 16). Expert ids
 * outside [0, E) in topk_ids are ignored.
 */
moe_status moe_expert_histogram_scan(const int32_t* topk_ids, int T, int k, int E,
                                     const int32_t* expert_map, int E_local,
                                     int32_t* counts, int32_t* offsets,
                                     void* ws, size_t* ws_bytes, hipStream_t stream);

/*
 * moe_permute - dispatch: a stable counting sort of assignments by local slot.
 *
 * For flat assignment i = t*k + j in ascending order, if its expert is local
 * (slot l), it gets row pos = offsets[l] + (number of earlier assignments to
 * slot l): perm_src[pos] = i, dest[i] = pos and x_perm[pos,:] = x[t,:].
 * Remote assignments get dest[i] = -1. Under expert parallelism x_perm is the
 * send buffer of the dispatch all-to-all (Section 2).
 *
 * ws, ws_bytes  the workspace filled by moe_expert_histogram_scan (same T, k,
 *               E, E_local); expert_map is the same HOST array.
 * x_perm   [M_cap, H] dt   rows [0, offsets[E_local]) written; may be NULL,
 *          then only perm_src and dest are written (for
 *          moe_grouped_swiglu_ffn_gather, which reads the rows from x)
 * perm_src [M_cap]    int32 entries [0, offsets[E_local]) written
 * dest     [T*k]      int32 all written
 * Requires M_cap >= T*k (the worst case, so no host sync is needed).
 */
moe_status moe_permute(const void* x, const int32_t* topk_ids, const int32_t* expert_map,
                       const void* ws, size_t ws_bytes, int T, int H, int k, int E,
                       int E_local, int M_cap, moe_dtype dt, void* x_perm,
                       int32_t* perm_src, int32_t* dest, hipStream_t stream);

/*
 * moe_grouped_swiglu_ffn - every local expert on its rows of x_perm.
 *
 * For local slot l and rows R = [offsets[l], offsets[l+1]):
 *   G = x_perm[R] W_gate[l]^T, U = x_perm[R] W_up[l]^T   (fp32 accumulation)
 *   h = round_dt( silu(G) * U ),  silu(g) = g / (1 + exp(-g))   (fp32)
 *   y_perm[R] = round_dt( h W_down[l]^T )                  (fp32 accumulation)
 * This is the expert computation whose latency per token load is f_g(n)
 * (Section 4.2.1). Experts with no rows cost nothing and are not read.
 *
 * w_gate, w_up [E_local, I, H] dt with row stride ldw_gu elements (expert
 *              l's matrix starts at row l * I); w_down [E_local, H, I] dt with
 *              row stride ldw_dn (expert l at row l * H). A stride of 0 means
 *              dense (H, resp. I); otherwise it must be >= that, a multiple
 *              of 16 bytes and <= 2^20 (else MOE_ERR_INVALID_ARG). Padding
 *              the rows off a power of two (e.g. H + 64 for H = 4096) spreads
 *              a weight tile's rows over more HBM channels; padding elements
 *              are never read.
 * offsets      [E_local+1] int32 (device, from moe_expert_histogram_scan);
 *              clamped to [0, M_cap] inside the kernels
 * y_perm       [M_cap, H] dt, rows [0, offsets[E_local]) written
 * ws           holds h [M_cap, I] dt; for bf16 also work counters, the
 *              fp32 partial sums of tiles split along K (summed in a fixed
 *              order, so results are deterministic) and a split plan.
 *              bf16: the workspace's first 16 KiB are counters that must be
 *              zero before the first call that uses the workspace (allocate
 *              it zero-filled); every call leaves them zero again. Calls on
 *              one workspace must not overlap.
 *              Schedule (bf16): when no expert has more than 16 rows, or
 *              64 when no reduction launch follows (see below), or 128 in a
 *              GEMM launch with no more 128-column tiles than half its
 *              blocks, each GEMM's (tile, K chunk) units are dealt to the
 *              CUs in equal shares and tiles split between CUs are finished
 *              inside the GEMM launch; otherwise whole tiles run in rounds,
 *              with split-K for tile-starved launches and a split of a
 *              partly filled last round, whose partials a launch after each
 *              GEMM sums. When no expert can have more than 128 rows
 *              (M_cap <= 128; for the _gather variant min(T, M_cap) <= 128,
 *              since a token adds at most one row to an expert) those
 *              launches are left out (two kernel launches in all) and
 *              nothing is split outside the decode schedule. The first call on a device
 *              that is not under graph capture also launches a small
 *              one-time check of the GPU's workgroup-to-XCD assignment.
 * Limits: 0 <= E_local <= 256 (0 is a no-op); bf16: H % 128 == 0 and
 * I % 128 == 0; fp32: H % 4 == 0 and I % 4 == 0.
 */
moe_status moe_grouped_swiglu_ffn(const void* x_perm, const void* w_gate, const void* w_up,
                                  const void* w_down, const int32_t* offsets, int E_local,
                                  int H, int I, int ldw_gu, int ldw_dn, int M_cap, moe_dtype dt,
                                  void* y_perm, void* ws, size_t* ws_bytes, hipStream_t stream);

/*
 * moe_grouped_swiglu_ffn_gather - moe_grouped_swiglu_ffn with the dispatch
 * gather folded into the gate/up GEMM's operand loads.
 *
 * Computes what moe_permute followed by moe_grouped_swiglu_ffn computes
 * (bitwise the same y_perm and h whenever both take the same schedule; with
 * T <= 128 this one may finish split tiles in its GEMM launches where the
 * permuted call, bounded only by M_cap, splits differently, and results then
 * agree within the FFN's tolerance), but row r of the expert input is
 * read as x[perm_src[r] / k] (the token of flat assignment perm_src[r],
 * Section 2's dispatch) instead of from a permuted copy, so the x_perm write
 * and re-read are skipped: call moe_permute with x_perm = NULL for perm_src.
 *
 * x        [T, H] bf16 (the layer's input tokens); T >= 1, T*H*2 < 2^32
 * perm_src [M_cap] int32 from moe_permute; entries of rows outside
 *          [offsets[0], offsets[E_local]) are not read, the others are
 *          clamped to a token of x
 * k        the top-k of the routing (1..MOE_MAX_TOPK)
 * other arguments, workspace and limits: as moe_grouped_swiglu_ffn (bf16
 * only; fp32 returns MOE_ERR_UNSUPPORTED).
 */
moe_status moe_grouped_swiglu_ffn_gather(const void* x, const int32_t* perm_src, int T, int k,
                                         const void* w_gate, const void* w_up, const void* w_down,
                                         const int32_t* offsets, int E_local, int H, int I,
                                         int ldw_gu, int ldw_dn, int M_cap, moe_dtype dt,
                                         void* y_perm, void* ws, size_t* ws_bytes, hipStream_t stream);

/*
 * moe_grouped_swiglu_ffn_noalloc - moe_grouped_swiglu_ffn for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).
 *
 * Same arguments, results and limits as moe_grouped_swiglu_ffn, without the
 * workspace: the call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine) and uses instead this library's scratch, a
 * device array of moe_ffn_scratch_bytes() bytes (128 MiB) in each GPU's copy
 * of the code object, held until the process ends. Its counters are cleared
 * on `stream` by the first call on a device; every call leaves them zero.
 * The scratch must hold the workspace's fixed part, the counters (16 KiB),
 * h [M_cap, I] and the split plan, i.e. roughly M_cap * I * sizeof(dt) +
 * 4 * max(M_cap, 64 E_local) + 16 KiB bytes (decode-sized batches: e.g.
 * M_cap <= 500 rows at I = 14336 in bf16); larger calls return
 * MOE_ERR_WORKSPACE and launch nothing. The rest of the scratch holds
 * partial sums of split tiles; where it is smaller than the workspace
 * moe_grouped_swiglu_ffn would use, fewer tiles are split (results stay
 * within the same tolerances, but need not be bitwise those of
 * moe_grouped_swiglu_ffn). All calls on one GPU share its scratch, whatever
 * their stream: calls that overlap in time on one GPU race, so serialise
 * them (one stream, or events).
 */
moe_status moe_grouped_swiglu_ffn_noalloc(const void* x_perm, const void* w_gate, const void* w_up,
                                          const void* w_down, const int32_t* offsets, int E_local,
                                          int H, int I, int ldw_gu, int ldw_dn, int M_cap, moe_dtype dt,
                                          void* y_perm, hipStream_t stream);

/* Bytes of the scratch that moe_grouped_swiglu_ffn_noalloc uses on each GPU. */
size_t moe_ffn_scratch_bytes(void);

/*
 * moe_unpermute_combine - gather and weighted sum back to token order.
 *
 * out[t,:] = round_dt( sum over j ascending with dest[t*k+j] >= 0 of
 *            topk_w[t,j] * y_perm[dest[t*k+j],:] ), fp32 accumulator.
 * Tokens with no local assignment get an exactly zero row, so summing the
 * partial outputs of all GPUs of an expert-parallel group gives the layer
 * output (the combine all-to-all of Section 2). dest entries outside
 * [0, M_cap) are treated as -1.
 *
 * out [T, H] dt (written completely).
 */
moe_status moe_unpermute_combine(const void* y_perm, const float* topk_w, const int32_t* dest,
                                 int T, int k, int H, int M_cap, moe_dtype dt, void* out,
                                 hipStream_t stream);

/*
 * MXFP8 expert FFN (FP8 experts).
 *
 * The paper serves its models in FP8 (Table 2a) without naming a scaling
 * scheme. These entry points use OCP Microscaling FP8 (MXFP8), the block
 * scaling gfx950's scaled MFMA consumes directly: elements are FP8 E4M3 (OCP
 * encoding: bias 7, no infinities, S.1111.111 NaN, largest finite 448), and
 * every 32 consecutive elements along the reduction dimension share one E8M0
 * scale code c, the power of two 2^(c - 127).
 *
 * Quantisation of a 32-element block v (OCP MX conversion): shared exponent
 * s = floor(log2(max |v_i|)) - 8 clamped to [-127, 127] (an all-zero block
 * takes -127), code c = s + 127, element q_i = E4M3 of v_i / 2^s clamped to
 * +-448 and rounded to nearest, ties to even (a value that rounds to zero
 * keeps its sign).
 *
 * Layout of an MXFP8 matrix with R rows and reduction length K (K % 128 == 0):
 *   codes  [R, K]        uint8, row-major (16-byte aligned)
 *   scales [K/128, R]    uint32, chunk-major: dword (k, r) holds the codes of
 *                        row r for elements [128 k, 128 k + 128), byte b
 *                        (little-endian) for elements [128 k + 32 b, +32)
 * A batch of B such matrices (expert weights) is codes [B, R, K] and scales
 * [B, K/128, R]. Weight codes may have padded rows: row r of matrix b at
 * byte (b * R + r) * ld, with ld >= K a multiple of 16 and <= 2^20 (0 means
 * ld = K); padding bytes are never read. Rows a multiple of 4 KiB long
 * (K = 4096) stream faster from HBM with 128 bytes of padding.
 * Activation codes (x, h, a) are always dense.
 */

/*
 * moe_mx_quantize - MXFP8 quantisation of `batch` matrices of `rows` x K.
 *
 * x         [batch, rows, K] dt (bf16 or fp32)
 * row_count DEVICE int32 or NULL (batch 1 only): quantise rows
 *           [0, min(rows, *row_count)) only, e.g. the routed rows of x_perm
 *           with row_count = offsets + E_local, without a host sync; the
 *           other rows' codes and scales are left untouched
 * codes     [batch, rows, K] uint8, rows ld_codes bytes apart (0: dense;
 *           otherwise as padded weight rows above, else MOE_ERR_INVALID_ARG)
 * scales    [batch, K/128, rows] uint32
 * Limits: K % 128 == 0; batch * rows * K <= 2^40.
 */
moe_status moe_mx_quantize(const void* x, moe_dtype dt, int batch, int rows, int K,
                           int ld_codes, const int32_t* row_count, uint8_t* codes,
                           uint32_t* scales, hipStream_t stream);

/*
 * moe_grouped_swiglu_mx - the gate/up half of the MXFP8 expert FFN.
 *
 * For local slot l and rows R = [offsets[l], offsets[l+1]) (clamped to
 * [0, M_cap]):
 *   G = X[R] Wg[l]^T, U = X[R] Wu[l]^T  from the MXFP8 operands (scaled MFMA,
 *                                        fp32 accumulation)
 *   h = silu(G) * U                      (fp32)
 *   (hq, hs)[R] = MXFP8 quantisation of h along I (rules above)
 * xq [M_cap, H], xs [H/128, M_cap]; wgq, wuq [E_local, I, H] (code rows ldw
 * bytes apart, 0: dense), wgs, wus [E_local, H/128, I]; hq [M_cap, I],
 * hs [I/128, M_cap]: rows R of every local expert written, the rest
 * untouched.
 * Limits: 0 <= E_local <= 256; H % 128 == 0, I % 128 == 0; H, I <= 2^20.
 */
moe_status moe_grouped_swiglu_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq,
                                 const uint32_t* wgs, const uint8_t* wuq, const uint32_t* wus,
                                 const int32_t* offsets, int E_local, int H, int I, int ldw,
                                 int M_cap, uint8_t* hq, uint32_t* hs, hipStream_t stream);

/*
 * moe_grouped_gemm_mx - grouped MXFP8 GEMM with bf16 output: for local slot l,
 * c[R] = bf16( A[R] B[l]^T ) (fp32 accumulation), R as above.
 * aq [M_cap, K], as [K/128, M_cap]; bq [E_local, N, K] (code rows ldb bytes
 * apart, 0: dense), bs [E_local, K/128, N]; c [M_cap, N] bf16, rows R
 * written. The down projection of the MXFP8 FFN.
 * Limits: 0 <= E_local <= 256; N % 128 == 0, K % 128 == 0; N, K <= 2^20.
 */
moe_status moe_grouped_gemm_mx(const uint8_t* aq, const uint32_t* as, const uint8_t* bq,
                               const uint32_t* bs, const int32_t* offsets, int E_local, int N,
                               int K, int ldb, int M_cap, void* c, hipStream_t stream);

/*
 * moe_grouped_swiglu_ffn_mx - the MXFP8 expert FFN (the FP8 counterpart of
 * moe_grouped_swiglu_ffn): moe_grouped_swiglu_mx into the workspace, then
 * moe_grouped_gemm_mx with W_down (wdq [E_local, H, I], wds
 * [E_local, I/128, H]) into y_perm [M_cap, H] bf16. Weight code rows are
 * ldw_gu (W_gate, W_up) and ldw_dn (W_down) bytes apart (0: dense).
 * ws starts with 16 KiB of counters that must be zero before the first call
 * on the workspace (every call leaves them zero), then h codes [M_cap, I]
 * and, 256-byte aligned after them, their scales [I/128, M_cap], then the
 * split plan and the fp32 partial sums of tiles split along K (summed in a
 * fixed order, so results are deterministic). The schedules and launches
 * are those of moe_grouped_swiglu_ffn, with M_cap as the bound on an
 * expert's rows. Calls that share a workspace must not overlap.
 */
moe_status moe_grouped_swiglu_ffn_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq,
                                     const uint32_t* wgs, const uint8_t* wuq, const uint32_t* wus,
                                     const uint8_t* wdq, const uint32_t* wds,
                                     const int32_t* offsets, int E_local, int H, int I,
                                     int ldw_gu, int ldw_dn, int M_cap, void* y_perm, void* ws,
                                     size_t* ws_bytes, hipStream_t stream);

/*
 * moe_load_sweep - per-expert latency versus token load.
 *
 * Algorithm 1 Phase 1 / Section 4.2.1: profile the expert computation over a
 * range of token counts to obtain f_g(n). For each M = Ms[i] (HOST array),
 * runs moe_grouped_swiglu_ffn on one expert with offsets [0, M]: `warmup`
 * untimed runs, then `iters` runs each bracketed by HIP events on `stream`.
 * Successive runs rotate through n_rot copies of the expert's weights so
 * that the 256 MB last-level cache does not hold them between runs.
 *
 * x        [maxM, H] dt        input rows (maxM = max of Ms)
 * w_gate, w_up [n_rot, I, H]; w_down [n_rot, H, I]   dt, rows strided by
 *          ldw_gu and ldw_dn as in moe_grouped_swiglu_ffn (0: dense)
 * y_scratch [maxM, H] dt       output rows (contents unspecified afterwards)
 * ws       workspace for maxM (query with ws == NULL); bf16: zero-filled
 *          before its first use, as for moe_grouped_swiglu_ffn
 * us_out   HOST [nM]: median microseconds per run
 * us_all   HOST [nM * iters] or NULL: every timed run, in order
 * Blocks the calling thread until the sweep is done. Limits: 1 <= nM <= 64,
 * 1 <= Ms[i] <= 1 << 20, 0 <= warmup, 1 <= iters <= 10000, n_rot >= 1.
 */
moe_status moe_load_sweep(const void* x, const void* w_gate, const void* w_up,
                          const void* w_down, int n_rot, int H, int I, int ldw_gu,
                          int ldw_dn, moe_dtype dt,
                          const int32_t* Ms, int nM, int warmup, int iters,
                          void* y_scratch, void* ws, size_t* ws_bytes,
                          float* us_out, float* us_all, hipStream_t stream);

/*
 * moe_load_sweep_mx - moe_load_sweep for the MXFP8 expert FFN (the FP8
 * kernel the paper's models run, Table 2a): f_g(n) profiled on
 * moe_grouped_swiglu_ffn_mx with one expert and offsets [0, M].
 *
 * xq [maxM, H], xs [H/128, maxM]   MXFP8 input rows (maxM = max of Ms)
 * wgq, wuq [n_rot, I, H], wgs, wus [n_rot, H/128, I];
 * wdq [n_rot, H, I], wds [n_rot, I/128, H]   MXFP8 weight copies, code rows
 *          ldw_gu / ldw_dn bytes apart (0: dense)
 * y_scratch [maxM, H] bf16; ws, us_out, us_all and limits as moe_load_sweep;
 * H % 128 == 0, I % 128 == 0.
 */
moe_status moe_load_sweep_mx(const uint8_t* xq, const uint32_t* xs, const uint8_t* wgq,
                             const uint32_t* wgs, const uint8_t* wuq, const uint32_t* wus,
                             const uint8_t* wdq, const uint32_t* wds, int n_rot, int H, int I,
                             int ldw_gu, int ldw_dn, const int32_t* Ms, int nM, int warmup, int iters, void* y_scratch,
                             void* ws, size_t* ws_bytes, float* us_out, float* us_all,
                             hipStream_t stream);

/* ------------------------------------------------------------------------
 * Placement control path (Section 4.2, Algorithms 1 and 2): the per-GPU
 * latency model f_g, the latency-aware greedy placement, the drift detector
 * and the incremental swap solver, for L MoE layers of E experts on G GPUs.
 *
 * Latency models: G models of nk knots each, knots_n [G, nk] and knots_t
 * [G, nk] fp64 (DEVICE arrays), knots_n strictly increasing and positive,
 * knots_t non-decreasing (moe_fit_latency_model builds them). f(n) = 0 for
 * n <= 0, knots_t[0] for 0 < n <= knots_n[0], linear between knots, and the
 * last segment's slope beyond the last knot (knots_t[0] n / knots_n[0] with
 * one knot). Knots that break these rules give unspecified placements but no
 * out-of-bounds access.
 *
 * Determinism: every decision is taken in fp64 with separately rounded
 * operations and sums in ascending index order; ties go to the lower GPU
 * index and, among experts, to the lower expert id. Limits: 1 <= E <= 1024,
 * 1 <= G <= 64, 1 <= nk <= 64, L >= 0 (0 is a no-op).
 * ---------------------------------------------------------------------- */

/*
 * moe_fit_latency_model - knots of f_g from measured points (HOST only,
 * launches nothing).
 *
 * Section 4.2.1: f_g(n) maps token load to kernel latency. loads [n] (HOST,
 * distinct, positive) and latencies [n] (HOST, finite) are the measured
 * points, e.g. one moe_load_sweep; the knots are the loads in ascending
 * order and the running maximum of the latencies in that order, so f is
 * monotone. knots_n, knots_t: HOST [n] outputs. 1 <= n <= 64.
 */
moe_status moe_fit_latency_model(const int32_t* loads, const float* latencies, int n,
                                 double* knots_n, double* knots_t);

/*
 * moe_place_greedy - initial latency-aware placement (Algorithm 1, Phase 2).
 *
 * Per layer l: N = sum_e w[l,e]; speeds s_g = 1 / f_g(N / E) (1 when N = 0);
 * token targets tau_g = N s_g / sum_h s_h; experts in descending load order
 * (ascending id among equal loads) each go to the GPU with the largest
 * tau_g - n_g among those holding fewer than `cap` experts (cap = 0: no
 * limit), whose load n_g then grows by the expert's load.
 *
 * w        [L, E] fp64 per-expert loads (DEVICE)
 * assign   [L, E] int32 (DEVICE): the GPU of each expert
 * loads    [L, G] fp64 (DEVICE) or NULL: final n_g
 * targets  [L, G] fp64 (DEVICE) or NULL: tau_g
 * cap: 0, or cap * G >= E.
 */
moe_status moe_place_greedy(const double* w, int L, int E, const double* knots_n,
                            const double* knots_t, int G, int nk, int cap, int32_t* assign,
                            double* loads, double* targets, hipStream_t stream);

/*
 * moe_place_incremental - incremental placement update (Algorithm 2).
 *
 * Per layer, starting from `assign` (DEVICE [L, E] int32, in/out; entries
 * outside [0, G) are read as GPU 0): while the largest f_g(n_g) exceeds
 * (1 + eps) times the mean of f_g(n_g) over the G GPUs, take the slowest GPU
 * g+ and the fastest g- and apply the swap of one expert of g+ with one of
 * g- that lowers max(f_g+(n_g+), f_g-(n_g-)) the most (first in ascending
 * expert ids on ties); stop when none lowers it or after max_swaps swaps.
 * Expert counts per GPU are kept.
 *
 * w        [L, E] fp64 loads (DEVICE)
 * n_swaps  [L] int32 (DEVICE) or NULL: swaps applied per layer
 * eps >= 0 finite; 0 <= max_swaps <= 1 << 20.
 */
moe_status moe_place_incremental(const double* w, int L, int E, const double* knots_n,
                                 const double* knots_t, int G, int nk, double eps, int max_swaps,
                                 int32_t* assign, int32_t* n_swaps, hipStream_t stream);

/*
 * moe_placement_cost - predicted cost of a placement (Section 4.2.3).
 *
 * Per layer l and GPU g: loads[l,g] = n_g = sum of w[l,e] over the experts
 * with assign[l,e] == g (ascending e), lat[l,g] = f_g(n_g), and
 * lat_grouped[l,g] = sum of f_g(w[l,e]) over the same experts (the reading
 * in which each expert runs as its own group). The layer latency the paper
 * minimises is max_g lat[l,g]. Experts with assign outside [0, G) count
 * nowhere.
 *
 * w [L, E] fp64, assign [L, E] int32, loads / lat_grouped [L, G] fp64 or
 * NULL, lat [L, G] fp64 (all DEVICE).
 */
moe_status moe_placement_cost(const double* w, const int32_t* assign, int L, int E,
                              const double* knots_n, const double* knots_t, int G, int nk,
                              double* loads, double* lat, double* lat_grouped, hipStream_t stream);

/*
 * moe_window_push - add one forward pass's per-layer expert counts to a
 * sliding window (Section 4.2.4: load vectors averaged over a window of
 * samples).
 *
 * ring [window, L, E] int32 and sums [L, E] fp64 (DEVICE) are the caller's
 * state, zeroed by the caller before the first push; slot = the ring entry
 * this pass replaces (the caller cycles it 0, 1, ..., window - 1, 0, ...).
 * sums += counts - ring[slot]; ring[slot] = counts. Exact for counts below
 * 2^53 / window. counts [L, E] int32 (DEVICE), e.g. the histogram's counts
 * of each layer. 1 <= window, 0 <= slot < window.
 */
moe_status moe_window_push(const int32_t* counts, int32_t* ring, double* sums, int L, int E,
                           int window, int slot, hipStream_t stream);

/*
 * moe_drift_distance - drift test (Section 4.2.4).
 *
 * d[l] = 1 - w_cur[l].w_ref[l] / (|w_cur[l]| |w_ref[l]|) (0 if both vectors
 * are zero, 1 if exactly one is), sums in ascending expert id; *trigger =
 * 1 if any d[l] > delta, else 0.
 *
 * w_cur, w_ref [L, E] fp64 (DEVICE; window sums or means: the distance does
 * not depend on scale); d [L] fp64 (DEVICE); trigger [1] int32 (DEVICE) or
 * NULL. delta finite. L <= 65536.
 */
moe_status moe_drift_distance(const double* w_cur, const double* w_ref, int L, int E, double delta,
                              double* d, int32_t* trigger, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_SHARD_MOE_H */
