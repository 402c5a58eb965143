// Device-side types and helpers shared by the libmoe kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef uint16_t bf16_t;  // raw IEEE bfloat16 bits

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kWave = 64;
constexpr int kMaxExperts = 256;
constexpr int kMaxTopk = 16;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to bf16 (nearest, ties to even) in one
// v_cvt_pk_bf16_f32; `lo` lands in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

// ---------------------------------------------------------------------------
// Swizzled LDS tiles filled by direct global->LDS loads.
//
// A tile row holds BK bf16 (BK = 64: 128 B = 8 chunks of 16 B; BK = 32: 64 B
// = 4 chunks). The LDS serves a 128-bit read 16 lanes at a time across 64
// banks (256 B), and an MFMA operand load has 16 lanes read 16 consecutive
// rows at the same logical chunk. Chunk c of row r is stored at position
//   BK = 64: c ^ ((r >> 1) & 7)   (even rows in banks 0-31, odd in 32-63)
//   BK = 32: c ^ ((r >> 2) & 3)   (row r in bank quarter r % 4)
// so those 16 lanes always touch 16 different 16-byte bank slots. Each
// wave's load instruction fills 1 KB of LDS contiguously, as
// global_load_lds_dwordx4 requires (lane i writes bytes [16 i, 16 i + 16)
// past the wave-uniform LDS address); the swizzle is its own inverse, so the
// lane that fills position p of row r fetches chunk swz_chunk<BK>(r, p).
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

template <int BK>
__device__ __forceinline__ int swz_chunk(int row, int chunk) {
  static_assert(BK == 64 || BK == 32, "chunk width");
  return BK == 64 ? (chunk ^ ((row >> 1) & 7)) : (chunk ^ ((row >> 2) & 3));
}

// The load is issued through inline assembly, so the compiler does not track
// it: every consumer waits for it explicitly (wait_vmcnt + lds_barrier).
// Tracked, the compiler would add a vmcnt(0) before LDS reads it cannot prove
// disjoint from a load still in flight, which serialises the pipeline. Its
// own vmcnt waits stay correct: loads complete in issue order, so untracked
// younger loads only make those waits more conservative. Nothing else in
// these kernels uses M0.
__device__ __forceinline__ void dma16(const void* gaddr, const bf16_t* lds) {
  const uint32_t m0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gaddr), "s"(m0)
               : "memory");
}

// The same loads with a wave-uniform 64-bit base in SGPRs and a 32-bit
// per-lane byte offset (global address = base + offset): one VGPR per load
// instead of two. dma16s moves 16 bytes per lane, dma4s 4 bytes (lane i
// writes LDS bytes [4 i, 4 i + 4) past `lds`).
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
  return reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo);
}

__device__ __forceinline__ void dma16s(const void* sbase, uint32_t voff, const void* lds) {
  const uint32_t m0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(m0)
               : "memory");
}

__device__ __forceinline__ void dma4s(const void* sbase, uint32_t voff, const void* lds) {
  const uint32_t m0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_void_t*)lds));
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(m0)
               : "memory");
}

// Loads rows [0, R) (BK bf16 each, starting at column `col0`) of a row-major
// matrix with row stride `ld` into a swizzled LDS tile. Rows at or beyond
// `row_limit` re-read row `row_limit - 1` (their results are never stored),
// so no load leaves the matrix. With live == false every lane reads the
// first 16 bytes of the matrix instead (one cache line per instruction): the
// pipelines below issue such a load where no chunk is left, so the number of
// loads in flight never depends on a branch. NW waves share the rows; one
// instruction covers 1 KB = 1024 / (2 BK) rows; R must be a multiple of
// NW times that.
template <int R, int NW, int BK>
__device__ __forceinline__ void dma_rows(const bf16_t* __restrict__ src, size_t ld, int col0, int row_limit,
                                         bool live, bf16_t* lds, int wave, int lane) {
  constexpr int CPR = BK / 8;           // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;         // rows per instruction
  static_assert(R % (RPI * NW) == 0, "rows per wave");
#pragma unroll
  for (int i = 0; i < R / (RPI * NW); ++i) {
    const int r0 = (i * NW + wave) * RPI;
    const int r = r0 + lane / CPR;
    const int c = swz_chunk<BK>(r, lane % CPR);
    const int rr = r < row_limit ? r : row_limit - 1;
    const size_t off = live ? (size_t)rr * ld + col0 + c * 8 : 0;
    dma16(src + off, lds + r0 * BK);
  }
}

// 16-byte operand fragment: elements [8 * chunk, 8 * chunk + 8) of tile row `row`.
template <int BK>
__device__ __forceinline__ bf16x8_t lds_frag(const bf16_t* lds, int row, int chunk) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(lds + row * BK + swz_chunk<BK>(row, chunk) * 8));
}

// s_waitcnt vmcnt(N) (gfx9 encoding; expcnt and lgkmcnt left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt lgkmcnt(0) (vmcnt and expcnt left unconstrained): every LDS
// read of this wave has returned its data.
__device__ __forceinline__ void wait_lgkmcnt0() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x0 << 8) | (0x3 << 14));
}

// Workgroup barrier for the LDS pipelines. __syncthreads() adds a release
// fence, which makes the compiler drain every outstanding global load
// (vmcnt(0)) before the barrier, prefetches included. The pipelines instead
// wait explicitly (wait_vmcnt) for the stage they are about to read, so the
// barrier itself only needs to keep the compiler from moving memory
// operations across it (signal fences emit no instructions).
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// NS-stage K pipeline over K chunks held in one LDS array (stage i at
// smem + i * stage_elems). issue(kc, live, stage) loads chunk kc into a stage
// with exactly LOADS load instructions per wave (live == false: a placeholder
// load, see dma_rows); compute(stage) consumes one stage. Chunk c+NS-1 is
// requested while the MFMAs work on chunk c, so NS-1 chunks are in flight.
// The loads are invisible to the compiler (dma16), so it adds no waits of its
// own; each wave writes only its own 1 KB slices of a stage. On return no
// load is in flight and every wave is done with the stages, so the caller
// may reuse the LDS for anything.
template <int NS, int LOADS, class Issue, class Compute>
__device__ __forceinline__ void pipeline(int nK, bf16_t* smem, int stage_elems, Issue&& issue,
                                         Compute&& compute) {
  static_assert(NS >= 2 && NS <= 8, "stages");
  wait_vmcnt<0>();  // nothing older (e.g. a previous tile's stores) is left in the count
#pragma unroll
  for (int i = 0; i < NS - 1; ++i) issue(i, i < nK, smem + i * stage_elems);
  int cur = 0;
  for (int c = 0; c < nK; ++c) {
    wait_vmcnt<LOADS * (NS - 2)>();  // chunk c landed; the NS-2 newer ones may still be in flight
    lds_barrier();                   // every wave's chunk c landed; every wave is done with chunk c-1
    const int pf = (cur == 0 ? NS : cur) - 1;  // stage of chunk c-1 == stage of chunk c+NS-1
    issue(c + NS - 1, c + NS - 1 < nK, smem + pf * stage_elems);
    __builtin_amdgcn_sched_barrier(0);
    compute(smem + cur * stage_elems);
    cur = (cur + 1 == NS) ? 0 : cur + 1;
  }
  // The last steps issued placeholder loads into stages nobody reads; they
  // must land before the caller reuses the LDS (or refills the stages).
  wait_vmcnt<0>();
  lds_barrier();  // all waves are done reading and no load is in flight
}

// The same pipeline for consumers that read their operands from LDS one
// k-step ahead of the MFMAs that use them, across chunk boundaries too. A
// chunk holds KS k-steps (KS even); read(stage, s, buf) loads the fragments of
// k-step s into register buffer buf, mma(buf) issues one k-step's MFMAs from
// buffer buf (k-step s always uses buffer s % 2), and mix() orders the LDS
// reads and MFMAs of one k-step (sched_group_barrier hints).
//
// The wait for chunk c+1 and the barrier come before the last k-step of
// chunk c, whose operands are already in registers: after the barrier the
// wave issues the next load, the first reads of chunk c+1 and the MFMAs of
// that last k-step together, so the MFMAs never wait for a read issued after
// a barrier. Before the barrier each wave waits for its own reads of chunk c
// (lgkmcnt), so the load issued into that stage right after it cannot
// overwrite data still being read. NS-1 chunks are in flight during each
// chunk's MFMAs, as in pipeline(). On return no load is in flight and every
// wave is done with the stages.
//
// MMA_FIRST puts each k-step's MFMAs before the reads of the next k-step in
// program order (the issue order is still set by mix()). A consumer can then
// refill an operand register right after its last MFMA of the k-step instead
// of keeping a second buffer for it.
template <int NS, int LOADS, int KS, bool MMA_FIRST = false, class Issue, class Read, class Mma, class Mix>
__device__ __forceinline__ void pipeline_xk(int nK, bf16_t* smem, int stage_elems, Issue&& issue, Read&& read,
                                            Mma&& mma, Mix&& mix) {
  static_assert(NS >= 2 && NS <= 8, "stages");
  static_assert(KS >= 2 && KS % 2 == 0, "k-steps per chunk");
  wait_vmcnt<0>();  // nothing older (e.g. a previous tile's stores) is left in the count
#pragma unroll
  for (int i = 0; i < NS - 1; ++i) issue(i, i < nK, smem + i * stage_elems);
  wait_vmcnt<LOADS * (NS - 2)>();  // chunk 0 landed
  lds_barrier();
  issue(NS - 1, NS - 1 < nK, smem + (NS - 1) * stage_elems);  // stage NS-1 holds nothing yet
  read(smem, 0, 0);
  int cur = 0;
  for (int c = 0; c < nK; ++c) {
    const bf16_t* st = smem + cur * stage_elems;
    const int nxt = (cur + 1 == NS) ? 0 : cur + 1;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s + 1 < KS; ++s) {
      if (MMA_FIRST) {
        mma(s & 1);
        read(st, s + 1, (s + 1) & 1);
      } else {
        read(st, s + 1, (s + 1) & 1);
        mma(s & 1);
      }
      mix();
      __builtin_amdgcn_sched_barrier(0);
    }
    // chunks c+1 .. c+NS-1 are in flight
    wait_lgkmcnt0();                 // this wave's reads of chunk c returned
    wait_vmcnt<LOADS * (NS - 2)>();  // chunk c+1 landed
    lds_barrier();                   // every wave: chunk c+1 landed, chunk c read
    issue(c + NS, c + NS < nK, smem + cur * stage_elems);
    __builtin_amdgcn_sched_barrier(0);
    // first fragments of chunk c+1 (after the last chunk: an unused read of a
    // stage that holds a placeholder load; LDS reads cannot fault)
    if (MMA_FIRST) {
      mma((KS - 1) & 1);
      read(smem + nxt * stage_elems, 0, 0);
    } else {
      read(smem + nxt * stage_elems, 0, 0);
      mma((KS - 1) & 1);
    }
    mix();
    __builtin_amdgcn_sched_barrier(0);
    cur = nxt;
  }
  wait_vmcnt<0>();
  lds_barrier();  // all waves are done reading and no load is in flight
}

// (value, index) ordering of the router: larger value first, then lower index.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// Slot map of a shard, passed to kernels by value (kernel argument segment).
struct SlotMap {
  int32_t n_experts;                 // E
  int32_t n_local;                   // E_local
  int16_t slot_of[kMaxExperts];      // expert -> local slot or -1
  int16_t expert_of[kMaxExperts];    // local slot -> expert
};

}  // namespace moe
