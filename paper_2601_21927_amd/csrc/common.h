// Shared device-side definitions of the SONIC HIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/sonic.h"

namespace sonic {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;          // MI355X: 8 accelerator complex dies, one L2 each

// Roles (one byte per token), as in sonic.h.
constexpr int kSystem = SONIC_ROLE_SYSTEM;
constexpr int kText = SONIC_ROLE_HISTORY_TEXT;
constexpr int kNexus = SONIC_ROLE_NEXUS;
constexpr int kCurrent = SONIC_ROLE_CURRENT;

__device__ __forceinline__ void raise_status(int32_t *status, int32_t code) {
  atomicCAS(status, 0, code);
}

// Read the status word once per workgroup so that every wave takes the same
// early-exit decision (waves must not diverge around a later barrier).
__device__ __forceinline__ bool block_status_clear(const int32_t *status, int *lds_flag) {
  if (threadIdx.x == 0) *lds_flag = (__atomic_load_n(status, __ATOMIC_RELAXED) == 0) ? 1 : 0;
  __syncthreads();
  return *lds_flag != 0;
}

// s_waitcnt vmcnt(N), the other counters left at their maximum (gfx9 encoding):
// wait until at most N of this wave's vector-memory operations are outstanding.
// They complete in issue order, so this waits for all but the N most recent.
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier for the LDS pipeline.  __syncthreads() would also wait for
// every outstanding vector-memory operation (its release fence covers the
// direct-to-LDS loads still in flight), which would drain the prefetch; here the
// loads a step needs are waited for explicitly with wait_vm, this wave's LDS
// reads are completed (lgkmcnt(0)) before it arrives, and the signal fences keep
// the compiler from moving memory operations across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));   // lgkmcnt(0)
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// One direct-to-LDS load: every lane fetches 16 bytes from its global address
// and the wave writes them to LDS at dst + 16 * lane (dst is wave-uniform, passed
// in M0).  Written as inline assembly so that the compiler does not track it as a
// pending LDS write: it would otherwise wait for every such load, including the
// prefetches into the other buffers, before each LDS read.  Completion is waited
// for explicitly (wait_vm) before the data is read.
__device__ __forceinline__ void dma_row16(const char *src, const uint16_t *dst) {
  // the low 32 bits of a generic pointer into LDS are its LDS address
  const uint32_t lds = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(dst)));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(lds) : "memory", "m0");
}

// A wave-uniform pointer moved into SGPRs (values loaded through ordinary global
// loads live in VGPRs even when every lane holds the same one).
__device__ __forceinline__ const char *uniform_ptr(const char *p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
  return reinterpret_cast<const char *>((static_cast<uint64_t>(hi) << 32) | lo);
}

// The same load with a wave-uniform 64-bit base (in SGPRs) and a 32-bit per-lane
// byte offset: no per-lane 64-bit address arithmetic.
// The LDS destination is given as its 32-bit LDS address.
__device__ __forceinline__ void dma_row16_s(const char *base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(off), "s"(uniform_ptr(base)),
               "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory", "m0");
}

// Combine a value with the one of lane ^ 32 (or lane ^ 16) without an LDS round
// trip: v_permlane32_swap (v_permlane16_swap) hands every lane the pair
// {lane, lane ^ 32} ({lane, lane ^ 16}), the lower lane's value first, so both
// lanes of a pair combine the same two values in the same order.
__device__ __forceinline__ float pair32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair32_add(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair16_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair16_add(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sum of the bf16 values of a packed operand, in fp32: v_dot2c_f32_bf16 against (1, 1)
// adds one pair per instruction, four independent chains.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
template <int N>
__device__ __forceinline__ float rounded_sum(const bf16x8 (&p)[N]) {
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < N; ++i) {
    acc[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p[i], p[i], 0, 1), ones, acc[0], false);
    acc[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p[i], p[i], 2, 3), ones, acc[1], false);
    acc[2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p[i], p[i], 4, 5), ones, acc[2], false);
    acc[3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(p[i], p[i], 6, 7), ones, acc[3], false);
  }
  return (acc[0] + acc[1]) + (acc[2] + acc[3]);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Prefill work descriptor of one block of up to 32 query rows that share one
// visible-key list.  Every list is two contiguous pieces:
//   prefix rows [0, npre)            of the request's prefix copy (system prompt,
//                                    then its Nexus tokens in order); every row sees them
//   positions [seg_start, seg_start + seg_len)
//                                    of the request itself; every row sees the first
//                                    seg_len - ndiag, and the last ndiag are the block's
//                                    own rows, causal (key j seen by row >= j)
// Positions are request-local.
struct TileDesc {
  int32_t req;
  int32_t p0;
  int32_t nrows;
  int32_t npre;
  int32_t seg_start;
  int32_t seg_len;
  int32_t ndiag;
  int32_t pad;
};
static_assert(sizeof(TileDesc) == 32, "descriptor is eight words");

constexpr int kTileRows = 32;       // query rows per descriptor (one MFMA N block)
constexpr int kKeyChunk = 64;       // keys per inner-loop step

__host__ __device__ __forceinline__ int tile_key_count(const TileDesc &t) { return t.npre + t.seg_len; }
__host__ __device__ __forceinline__ int tile_cost(const TileDesc &t) {
  return (tile_key_count(t) + kKeyChunk - 1) / kKeyChunk;
}

// Per-request summary written by the planner.
struct ReqInfo {
  int32_t ntiles;
  int32_t system;
  int32_t nexus_total;
  int32_t nruns;       // runs of the request (the next-turn plan: tail rows after the segment body)
  int64_t cost;        // sum of tile_cost over the request's descriptors
  int64_t pad;
};

// Where the rows of an attention call live.  Request b's query rows (and output
// rows) start at row seg_row0[b] of q/out, its own key rows at row seg_row0[b] of
// seg_k/seg_v, and its prefix rows at row pre_row0[b] of pre_k/pre_v (row
// seg_row0[b] when pre_row0 is null).  Rows are [H, D] records.  The statistics
// outputs, [rows][Hq] like out without D, are written by the statistics variant
// of the prefill kernel only: the attention mass on prefix keys past the
// request's system rows (its Nexus keys) and the row's log2-domain softmax
// normaliser.
struct AttnRows {
  const int32_t *seg_row0;
  const int64_t *pre_row0;
  const uint16_t *q;
  const uint16_t *seg_k;
  const uint16_t *seg_v;
  const uint16_t *pre_k;
  const uint16_t *pre_v;
  float *out;
  float *nexus_mass;
  float *lse;
};

// Device workspace of the prefill, carved from one caller buffer.
struct PrefillWs {
  ReqInfo *req;        // [B]
  int32_t *prefix_pos; // [T]  request b's prefix rows (system, then Nexus) at offset cu[b]: positions
  int2 *runs;          // [T]  (run start, Nexus count before it) at offset cu[b]
  TileDesc *tiles;     // [T]  request b's descriptors at offset cu[b]
  int32_t *order;      // [T]  descriptor slots: requests by decreasing cost, inside a request by
                       //      decreasing tile cost
  uint16_t *k_pre;     // [T, Hkv, D] prefix copies of K and V, request b's rows at offset cu[b]
  uint16_t *v_pre;
  int32_t *ctrl;       // [16] ctrl[0] = number of descriptors, ctrl[1] = number of key blocks of
                       //      the key-weight pass, ctrl[8 + x] = queue head of XCD x
  // attention statistics (used only when they are asked for)
  float *lse;          // [T, Hq] log2-domain softmax normaliser of every row and q-head
  float *wpart;        // [Hkv, T] key weight of every kept key, one partial per kv-head
  int2 *kblocks;       // [T / 64 + B] (request, block of 64 kept keys) of the key-weight pass
  int32_t *ncur;       // [B] current-query rows of request b
};

// Device workspace of the decode; the counters are zero between calls.
struct DecodeWs {
  int32_t *done;      // [B]      kv-heads of request b whose splits have all counted in this call
  int32_t *arrive;    // [B*Hkv]  splits of a (request, kv-head) finished in this call
  float *part;        // [B*Hkv][nsplit][G*(D+2)] partial (m[G], l[G], acc[G][D]) per split
};

// The decode's fixed-layout scratch (the entry point that allocates nothing): counters
// for up to kScratchMaxRequests requests and kScratchMaxPairs (request, kv-head) pairs,
// then the partial records, kScratchBytes in all.
constexpr int kScratchMaxRequests = 4096;
constexpr int kScratchMaxPairs = 12288;
constexpr size_t kScratchCounterBytes = (kScratchMaxRequests + kScratchMaxPairs) * sizeof(int32_t);   // 64 KiB
constexpr size_t kScratchBytes = size_t(8) << 20;

// Instruction order of one product block of NMFMA MFMAs whose operands each take
// READS LDS reads: the reads of the first AHEAD products, then one MFMA and the reads
// of one more product at a time, then the last AHEAD MFMAs.  The reads so run AHEAD
// products ahead of the MFMA that consumes them, hiding the LDS latency behind the
// matrix cores (the compiler, left alone, keeps one read ahead to save registers).
// Placed after the block's code, in the same basic block.
template <int NMFMA, int READS, int AHEAD>
__device__ __forceinline__ void order_reads_ahead() {
  static_assert(AHEAD >= 1 && AHEAD <= NMFMA, "lookahead within the block");
  __builtin_amdgcn_sched_group_barrier(0x100, READS * AHEAD, 0);   // DS reads
#pragma unroll
  for (int i = 0; i < NMFMA - AHEAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);              // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, READS, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, AHEAD, 0);
}

}  // namespace sonic
