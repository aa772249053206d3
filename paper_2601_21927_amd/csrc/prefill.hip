// Masked prefill attention (Sec. 3.2) on gfx950 matrix cores.
//
// Work item = (descriptor, kv-head).  A workgroup holds G waves, one per q-head
// of the kv-head's group, so every K/V block staged in LDS serves G heads.
// Each wave owns the 32 query rows of its descriptor for one q-head and walks
// the descriptor's visible keys in steps of 64:
//
//   S^T (64 keys x 32 rows)   = K . Q^T   v_mfma_f32_32x32x16_bf16, fp32 accumulate
//   online softmax over keys  (fp32, exp2 with log2(e) folded into the scale)
//   O^T (d x 32 rows)        += V^T . P^T  v_mfma_f32_32x32x16_bf16, P rounded to bf16;
//                              the softmax sum adds the rounded values
//
// Computing the transposed products leaves each lane with one query row
// (lane % 32) in every accumulator, so row maxima and sums need a single
// cross-lane exchange (lane ^ 32) and rescaling needs no exchange at all.
//
// Only the last one or two 64-key steps of a descriptor can hold masked
// entries (the ragged end of the key list and the causal diagonal); all
// earlier steps are fully visible and skip the predicate.
//
// LDS is double-buffered: while step c is computed, the K and V rows of step
// c+1 stream straight into the other buffer (global_load_lds_dwordx4, no
// registers); one barrier per step.  V stays row-major in LDS and the V^T
// operand of the second product is read with ds_read_b64_tr_b16, which
// transposes 16-bit elements across each group of 16 lanes.  The running
// max is updated lazily: O and the sum are rescaled only when the max grows by
// more than 2^8, so most steps skip the rescale (p stays below 2^8).
//
// Keys come from two contiguous pieces (see TileDesc): the request's prefix copy
// (system prompt, then its Nexus tokens, copied by the planner) and one range of
// the request itself, so every load address is arithmetic on the descriptor.
//
// The grid is persistent: workgroup w serves the queue of XCD (w mod 8); item i
// (descriptor slot i / Hkv, kv-head i mod Hkv) belongs to queue i mod 8.  Slots
// run request by request, so the workgroups of one XCD work on one request at a
// time and the K/V rows its blocks share stay in that XCD's L2.
#include "common.h"

namespace sonic {

// MFMA row m of a 32-key block holds key perm32(m) (bits 2 and 3 swapped), so
// that accumulator element v of lane half g maps to key 8g+v (v < 8) and
// 16+8g+(v-8) (v >= 8): eight consecutive keys per half, which is exactly the
// K-operand layout the P.V product needs.  The permutation is an involution.
__device__ __forceinline__ int perm32(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

// Key of accumulator element v, less the lane half's 8g.  It is a compile-time
// constant once the element loop is unrolled, so a bound compared with it is shifted
// by 8g once, instead of 32 per-lane key indices being held in registers for the
// whole kernel.
__device__ __forceinline__ constexpr int acc_key0(int v) { return v < 8 ? v : 8 + v; }

// LDS reads run ahead of the MFMAs (order_reads_ahead): K-operand reads of the S
// product, V-operand products of the P.V product
constexpr int kAheadS = 4;
constexpr int kAheadPV = 3;


typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void global_void_t;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;

// LDS bank swizzles (XOR on the 16-byte chunk index of a row), chosen so that the
// reads below are conflict-free whether a pass covers 16 lanes of 32 banks or
// 32 lanes of 64 banks.
//   K rows are read with ds_read_b128, 16 rows at one chunk per pass;
//   V rows are read with ds_read_b64_tr_b16, 4 rows x 4 chunks per pass.
template <int D> __device__ __forceinline__ int swz_k(int m) {
  return D == 128 ? (m & 15) : ((m & 7) ^ ((m >> 3) & 1));
}
template <int D> __device__ __forceinline__ int swz_v(int r) {
  return D == 128 ? ((4 * (r & 3)) ^ (2 * ((r >> 1) & 1))) : (2 * (r & 3));
}

// One 64-key step of one tensor into LDS, straight from global memory (no
// registers), one 16-byte chunk per lane: the lane that fills (row m, slot s)
// fetches chunk s ^ swizzle(m).  K row m holds key perm32(m) (MFMA row order);
// V row r holds key r.  Virtual key vk < npre is row vk of the prefix copy, any
// other is request position vk + seg_shift.  Keys past the list end repeat its
// first key: their scores are masked, so they contribute exactly zero (a step
// wholly past the end loads key 0 throughout and is never read).  Wave w issues
// instructions w, w + G, ... of the INSTS the step needs.
//
// Byte offset of a lane's chunk within a step, for instruction ii:
//   row(ii, lane) * row_bytes + 16 * chunk(ii, lane)
//     = urow(ii) * row_bytes + (lane_off ^ 16 * xu(ii))
// with urow and xu wave-uniform and lane_off fixed per lane (the low bits that
// the chunk XOR touches are below D * 2, where row offsets are zero).  A step
// whose 64 keys lie in one piece of the list therefore needs no per-lane address
// arithmetic beyond one XOR: its base row goes into SGPRs.
template <int D, bool IS_V> __device__ __forceinline__ uint32_t dma_lane_off(int lane, uint32_t row_bytes) {
  constexpr int DC = D / 8;
  const int l = lane / DC;     // row within the instruction's rows
  const int lc = lane % DC;    // chunk slot
  int lrow = l, lchunk = lc ^ l;
  if (IS_V) lchunk = lc ^ swz_v<D>(l);
  else if (D == 64) lrow = (l & 3) + 8 * (l >> 2);
  return static_cast<uint32_t>(lrow) * row_bytes + 16u * static_cast<uint32_t>(lchunk);
}
template <int D, bool IS_V> __device__ __forceinline__ int dma_urow(int ii) {
  constexpr int ROWS_PER_INST = kWave / (D / 8);
  if (IS_V) return ii * ROWS_PER_INST;
  if (D == 128) return 4 * ((ii & ~3) | ((ii & 1) << 1) | ((ii >> 1) & 1));
  return 4 * (ii & 1) + 16 * (ii >> 1);
}
template <int D, bool IS_V> __device__ __forceinline__ uint32_t dma_xu(int ii) {
  if (IS_V) return 0u;
  return D == 128 ? 64u * static_cast<uint32_t>(ii & 3) : 16u * static_cast<uint32_t>(ii & 1);
}

template <int D, int G, bool IS_V>
__device__ __forceinline__ void stage_tensor(uint16_t *lds_buf, const char *pre_base, const char *req_base,
                                             uint32_t row_bytes, uint32_t lane_off, int wave, int lane, int c,
                                             int nv, int npre, int seg_shift) {
  constexpr int DC = D / 8;
  constexpr int ROWS_PER_INST = kWave / DC;
  constexpr int INSTS = kKeyChunk / ROWS_PER_INST;
  constexpr int NJ = (INSTS + G - 1) / G;
  const int vk0 = c * kKeyChunk;
  // Every wave issues exactly NJ instructions (so that its wait counts are
  // static); where G does not divide INSTS, the surplus ones repeat the last
  // instruction, writing the same bytes to the same LDS rows.
  if (vk0 + kKeyChunk <= npre || (vk0 >= npre && vk0 + kKeyChunk <= nv)) {
    // the whole step in one piece: SGPR base row, fixed per-lane offsets
    const char *sb = vk0 < npre ? pre_base + static_cast<size_t>(vk0) * row_bytes
                                : req_base + static_cast<size_t>(vk0 + seg_shift) * row_bytes;
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds_buf));
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
      const int ii = min(wave + jj * G, INSTS - 1);
      // Opaque copies: each instruction's row offset and LDS address are formed
      // here with two scalar operations instead of being hoisted out of the key
      // loop into SGPRs (one pair per instruction and buffer would not fit).
      uint32_t rb = __builtin_amdgcn_readfirstlane(row_bytes), la = __builtin_amdgcn_readfirstlane(lds0);
      asm volatile("" : "+s"(rb), "+s"(la));
      dma_row16_s(sb + static_cast<size_t>(static_cast<uint32_t>(dma_urow<D, IS_V>(ii)) * rb),
                  lane_off ^ dma_xu<D, IS_V>(ii), la + static_cast<uint32_t>(ii * ROWS_PER_INST * D * 2));
    }
    return;
  }
#pragma unroll
  for (int jj = 0; jj < NJ; ++jj) {
    const int ii = min(wave + jj * G, INSTS - 1);
    {
      const int m = ii * ROWS_PER_INST + lane / DC;
      const int r = IS_V ? m : ((m & 32) | perm32(m & 31));
      int vk = vk0 + r;
      if (vk >= nv) vk = 0;
      const bool pre = vk < npre;
      const uint32_t chunk_bytes = static_cast<uint32_t>(((lane % DC) ^ (IS_V ? swz_v<D>(m) : swz_k<D>(m))) * 16);
      const uint32_t off = static_cast<uint32_t>(pre ? vk : vk + seg_shift) * row_bytes + chunk_bytes;
      dma_row16(pre ? pre_base + off : req_base + off, lds_buf + ii * ROWS_PER_INST * D);
    }
  }
}

// STATS: also write, per row and q-head, the attention mass on the request's
// Nexus keys (prefix keys at or past its system rows) and the log2-domain softmax
// normaliser, for the key-weight pass.
// KS = 2 (G <= 4; for launches with fewer work items than twice the CUs, such as
// the next-turn Nexus step): the workgroup holds two groups of G waves that take the
// first and the second half of the item's key steps, each with its own LDS
// buffers, in lock step (the same number of steps; a step past the end of the
// list is fully masked).  The second group then hands its (max, sum, O) to the
// first through LDS, which merges them by log-sum-exp and stores the rows: one
// resident workgroup per CU with twice the waves, instead of half the CUs idle.
template <int D, int G, bool STATS, int KS>
__global__ __launch_bounds__(G * kWave * KS, 3 - KS) void prefill_kernel(AttnRows rows, PrefillWs ws, int Hkv,
                                                                        float scale_log2) {
  static_assert(KS == 1 || (KS == 2 && !STATS), "the key split serves the attention output only");
  const uint16_t *__restrict__ q = rows.q;
  float *__restrict__ out = rows.out;
  constexpr int DC = D / 8;              // 16-byte chunks per K/V row
  constexpr int DS = D / 16;             // d steps of the S product
  constexpr int DB = D / 32;             // 32-wide d blocks of the output
  constexpr float kLazy = 8.f;           // rescale only when the running max grows by > 2^8
  // Two buffers per tensor, as distinct arrays: the compiler then knows that the
  // direct-to-LDS loads into one buffer cannot alias reads of the other and does
  // not wait for them before those reads.
  __shared__ __align__(16) uint16_t k_lds0[KS][kKeyChunk * D];   // [64 keys][D], MFMA row order
  __shared__ __align__(16) uint16_t k_lds1[KS][kKeyChunk * D];
  __shared__ __align__(16) uint16_t v_lds0[KS][kKeyChunk * D];   // [64 keys][D], key order
  __shared__ __align__(16) uint16_t v_lds1[KS][kKeyChunk * D];
  // KS = 2: the second group's running max and sum per wave and lane (its O goes
  // to the K/V buffers, one buffer of 64 x D bf16 = 32 x D floats per wave)
  __shared__ float ml_lds[KS == 2 ? 2 * G * kWave : 1];
  // KS = 2 keeps two waves per SIMD (G <= 4), so the registers of the single-group
  // variant still fit; each of the first eight buffers holds one wave's O
  static_assert(KS == 1 || (G <= 4 && (D / 32) * 16 * kWave <= kKeyChunk * D / 2), "key split shape");
  __shared__ int s_item;

  const int Hq = Hkv * G;
  const int wave_id = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);   // uniform: lets waves branch on it
  const int grp = KS == 1 ? 0 : wave_id / G;          // key half (KS = 2)
  const int wave = KS == 1 ? wave_id : wave_id % G;   // q-head within the kv-head's group
  uint16_t *const kbuf0 = k_lds0[grp];
  uint16_t *const kbuf1 = k_lds1[grp];
  uint16_t *const vbuf0 = v_lds0[grp];
  uint16_t *const vbuf1 = v_lds1[grp];
  const int lane = threadIdx.x % kWave;
  const int n = lane & 31;
  const int g = lane >> 5;
  const int xcd = blockIdx.x % kNumXcd;
  const int nitems = ws.ctrl[0] * Hkv;

  // Transposed-read geometry of the P.V operand (fixed per lane): 16-lane group q,
  // index i.  Lane i of a group receives d = base + i for keys kbase + 4h + e.
  const int tq = lane >> 4;
  const int ti = lane & 15;
  const int v_row_off = 8 * (tq >> 1) + (ti >> 2);      // + 16*ks + 4*h
  const int v_d_off = 16 * (tq & 1) + 4 * (ti & 3);     // + 32*db
  const uint32_t row_bytes = static_cast<uint32_t>(Hkv) * D * 2;
  const uint32_t koff_lane = dma_lane_off<D, false>(lane, row_bytes);
  const uint32_t voff_lane = dma_lane_off<D, true>(lane, row_bytes);

  for (;;) {
    if (threadIdx.x == 0) s_item = atomicAdd(&ws.ctrl[8 + xcd], 1) * kNumXcd + xcd;
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(s_item);
    __syncthreads();
    if (item >= nitems) break;
    const int slot = ws.order[item / Hkv];
    const int kvh = item % Hkv;
    TileDesc t = ws.tiles[slot];
    t.req = __builtin_amdgcn_readfirstlane(t.req);       // uniform: scalar branches and bases
    t.p0 = __builtin_amdgcn_readfirstlane(t.p0);
    t.nrows = __builtin_amdgcn_readfirstlane(t.nrows);
    t.npre = __builtin_amdgcn_readfirstlane(t.npre);
    t.seg_start = __builtin_amdgcn_readfirstlane(t.seg_start);
    t.seg_len = __builtin_amdgcn_readfirstlane(t.seg_len);
    t.ndiag = __builtin_amdgcn_readfirstlane(t.ndiag);
    const int base = rows.seg_row0[t.req];
    const int64_t pbase = rows.pre_row0 != nullptr ? rows.pre_row0[t.req] : static_cast<int64_t>(base);
    const int h = kvh * G + wave;
    const int nv = tile_key_count(t);
    const int nF = nv - t.ndiag;
    const int npre = t.npre;
    const int seg_shift = t.seg_start - npre;    // request position of virtual key vk >= npre
    const size_t tok_stride = static_cast<size_t>(Hkv) * D;
    const size_t head0 = static_cast<size_t>(base) * tok_stride + static_cast<size_t>(kvh) * D;
    const size_t phead0 = static_cast<size_t>(pbase) * tok_stride + static_cast<size_t>(kvh) * D;
    // row 0 of the request (and of its prefix rows) for this kv-head; rows are
    // row_bytes apart, and every row of a request lies below 4 GiB from its row 0
    const char *kreq = uniform_ptr(reinterpret_cast<const char *>(rows.seg_k + head0));
    const char *vreq = uniform_ptr(reinterpret_cast<const char *>(rows.seg_v + head0));
    const char *kpre = uniform_ptr(reinterpret_cast<const char *>(rows.pre_k + phead0));
    const char *vpre = uniform_ptr(reinterpret_cast<const char *>(rows.pre_v + phead0));

    const int nchunks = (nv + kKeyChunk - 1) / kKeyChunk;
    // this group's steps: [c_first, c_first + nloc); loads for steps past them
    // (the pipeline runs two ahead) fetch a step past the list end instead
    const int nloc = KS == 1 ? nchunks : (nchunks + 1) / 2;
    const int c_first = grp * nloc;
    const int c_stop = c_first + nloc;
    auto stage_step = [&](int c) { return (KS == 1 || c < c_stop) ? c : max(c, nchunks); };
    auto stage_k = [&](int c, uint16_t *buf) {
      stage_tensor<D, G, false>(buf, kpre, kreq, row_bytes, koff_lane, wave, lane, stage_step(c), nv, npre,
                                seg_shift);
    };
    auto stage_v = [&](int c, uint16_t *buf) {
      stage_tensor<D, G, true>(buf, vpre, vreq, row_bytes, voff_lane, wave, lane, stage_step(c), nv, npre,
                               seg_shift);
    };

    // Q^T fragments (B operand of S): lane (row n, half g) holds d = 16*ds + 8*g .. +7.
    bf16x8 qf[DS];
    {
      const bool ok = n < t.nrows;
      const uint16_t *qrow = q + (static_cast<size_t>(base + t.p0 + n) * Hq + h) * D;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (ok) w = *reinterpret_cast<const u32x4 *>(qrow + 16 * ds + 8 * g);
        qf[ds] = __builtin_bit_cast(bf16x8, w);
      }
    }

    f32x16 oacc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) oacc[i] = f32x16{};
    float m_run = -INFINITY;   // running max in the log2 domain (lags by at most kLazy)
    float l_run = 0.f;         // sum of the bf16-rounded probabilities the P.V product uses
    float l_ex = 0.f;          // STATS: the same sum before rounding (normaliser, Nexus mass)
    float l_nex = 0.f;         // STATS: the part of l_ex from Nexus keys
    // STATS: Nexus keys are the virtual keys [nex_lo, npre) (the prefix past the system rows)
    const int nex_lo = STATS ? min(ws.req[t.req].system, npre) : npre;

    // One 64-key step: compute on (kc_lds, vc_lds) while step c + 1 streams into
    // (kn_lds, vn_lds).
    // Pipeline, per wave: K of step c + 2 is requested as soon as every wave has
    // finished S(c), V of step c + 1 as soon as every wave has finished P.V(c - 1).
    // Each wave issues exactly NJ direct-to-LDS instructions per tensor and step,
    // in the order K(0) V(0) K(1) | V(1) K(2) | V(2) K(3) | ..., also for steps past
    // the end of the key list (those load key 0 and are never read).  So at the start
    // of step c the loads newer than K(c) are V(c) and K(c+1), and in its middle the
    // loads newer than V(c) are K(c+1) and V(c+1): both waits are "all but the 2 * NJ
    // most recent", the same at every step.
    constexpr int NJ = ((kKeyChunk / (kWave / (D / 8))) + G - 1) / G;
    static_assert(2 * NJ < 64, "the wait count fits vmcnt");
    __builtin_assume(wave < G);
    auto step = [&](int c, uint16_t *kc_lds, const uint16_t *vc_lds, uint16_t *vn_lds) {
      wait_vm<2 * NJ>();
      lds_barrier();                                   // K(c) in LDS; every wave is past P.V(c - 1)
      stage_v(c + 1, vn_lds);
      const int vk0 = c * kKeyChunk;

      // ---- S^T = K . Q^T for two 32-key blocks ----
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        sacc[kb] = f32x16{};
        const int m = kb * 32 + n;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8 *>(&kc_lds[(m * DC + ((2 * ds + g) ^ swz_k<D>(m))) * 8]);
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ds], sacc[kb], 0, 0, 0);
        }
      }
      order_reads_ahead<2 * DS, 1, kAheadS>();

      wait_vm<2 * NJ>();
      lds_barrier();                                   // V(c) in LDS; every wave is past S(c)
      stage_k(c + 2, kc_lds);
      // ---- mask (ragged end / causal diagonal only), online softmax ----
      if (vk0 + kKeyChunk > nF) {
        // Row n sees every key before the diagonal block and diagonal keys j <= n:
        // virtual key vk is visible iff vk < min(nv, nF + n + 1).  One compare and a
        // select per element, no divergent branches.
        const int lim_g = min(nv, nF + n + 1) - vk0 - 8 * g;   // bound on acc_key0
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            sacc[kb][e] = (kb * 32 + acc_key0(e) < lim_g) ? sacc[kb][e] : -INFINITY;
      }
      float mloc = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mloc = fmaxf(mloc, sacc[kb][e]);
      mloc = pair32_max(mloc) * scale_log2;
      if (__any(mloc > m_run + kLazy)) {
        const float m_new = fmaxf(m_run, mloc);
        const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= corr;
        if (STATS) {
          l_ex *= corr;
          l_nex *= corr;
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] *= corr;
      }
      // STATS: this step's Nexus keys are step-local keys [nx0, nx1)
      const int nx0 = max(nex_lo - vk0, 0), nx1 = min(npre - vk0, kKeyChunk);
      const bool nex_all = STATS && nx0 == 0 && nx1 == kKeyChunk;
      const bool nex_some = STATS && nx0 < nx1 && !nex_all;
      const int nx0_g = nx0 - 8 * g, nx1_g = nx1 - 8 * g;   // the same range on acc_key0
      float lsum = 0.f, nsum = 0.f;
      bf16x8 pb[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x8 lo, hi;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          lo[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], scale_log2, -m_run));
          hi[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][8 + e], scale_log2, -m_run));
          if (STATS) lsum += lo[e] + hi[e];
          if (nex_some) {
            const int klo = kb * 32 + acc_key0(e), khi = kb * 32 + acc_key0(8 + e);
            nsum += ((klo >= nx0_g && klo < nx1_g) ? lo[e] : 0.f) + ((khi >= nx0_g && khi < nx1_g) ? hi[e] : 0.f);
          }
        }
        pb[2 * kb] = __builtin_convertvector(lo, bf16x8);
        pb[2 * kb + 1] = __builtin_convertvector(hi, bf16x8);
      }
      // The output is normalised by the sum of the rounded probabilities themselves, so
      // that it stays a convex combination of the V rows: a row dominated by one key then
      // loses nothing to the rounding of that key's probability (which the lagging max
      // leaves anywhere in [1, 2^8), not exactly 1).  v_dot2c_f32_bf16 against (1, 1)
      // adds a packed pair of them in one instruction.
      l_run += rounded_sum(pb);
      if (STATS) l_ex += lsum;
      if (nex_all) l_nex += lsum;
      if (nex_some) l_nex += nsum;

      // ---- O^T += V^T . P^T, V^T operands read transposed from row-major V ----
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int dd = db * 32 + v_d_off;     // this lane's 4 d-values, a 4-aligned start
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          v4i16 part[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int r = 16 * ks + 4 * hh + v_row_off;
            const int chunk = (dd >> 3) ^ swz_v<D>(r);
            const uint16_t *pa = &vc_lds[r * D + chunk * 8 + (dd & 4)];
            part[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)pa);
          }
          const u32x4 w = {__builtin_bit_cast(uint2, part[0]).x, __builtin_bit_cast(uint2, part[0]).y,
                           __builtin_bit_cast(uint2, part[1]).x, __builtin_bit_cast(uint2, part[1]).y};
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w), pb[ks], oacc[db], 0,
                                                             0, 0);
        }
      }
      order_reads_ahead<4 * DB, 2, kAheadPV>();
    };

    stage_k(c_first, kbuf0);
    stage_v(c_first, vbuf0);
    stage_k(c_first + 1, kbuf1);
    step(c_first, kbuf0, vbuf0, vbuf1);
    for (int c = 1; c < nloc; c += 2) {
      step(c_first + c, kbuf1, vbuf1, vbuf0);
      if (c + 1 >= nloc) break;
      step(c_first + c + 1, kbuf0, vbuf0, vbuf1);
    }

    if constexpr (KS == 2) {
      // the second group hands its partial to the first: wave w's O into buffer w
      // (lane-minor, so both sides touch consecutive words), max and sum into ml_lds
      wait_vm<0>();
      __syncthreads();                 // every wave past its last step's LDS reads and loads
      uint16_t *const ob = wave < 4 ? (wave < 2 ? k_lds0[wave & 1] : k_lds1[wave & 1])
                                    : (wave < 6 ? v_lds0[wave & 1] : v_lds1[wave & 1]);
      float *const xo = reinterpret_cast<float *>(ob);
      if (grp == 1) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int e = 0; e < 16; ++e) xo[(db * 16 + e) * kWave + lane] = oacc[db][e];
        ml_lds[(2 * wave) * kWave + lane] = m_run;
        ml_lds[(2 * wave + 1) * kWave + lane] = l_run;
      }
      __syncthreads();
      if (grp == 1) continue;          // the loop head's barrier waits for the first group
      const float m1 = ml_lds[(2 * wave) * kWave + lane];
      const float l1 = ml_lds[(2 * wave + 1) * kWave + lane];
      // A group that saw no key of this row (its steps were past the list end) kept
      // the max at -inf, and its sum and O are NaN (-inf - -inf in the exponent):
      // select them away rather than scale them by zero.
      const bool has0 = m_run != -INFINITY, has1 = m1 != -INFINITY;
      const float mm = fmaxf(m_run, m1);
      const float c0 = has0 ? __builtin_amdgcn_exp2f(m_run - mm) : 0.f;
      const float c1 = has1 ? __builtin_amdgcn_exp2f(m1 - mm) : 0.f;
      l_run = (has0 ? l_run * c0 : 0.f) + (has1 ? l1 * c1 : 0.f);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float x = xo[(db * 16 + e) * kWave + lane];
          oacc[db][e] = (has0 ? oacc[db][e] * c0 : 0.f) + (has1 ? x * c1 : 0.f);
        }
    }

    // ---- normalise and store: lane (n, g) holds d = 32*db + 8*i + 4*g + (0..3) ----
    const float l_tot = pair32_add(l_run);
    const float inv = 1.f / l_tot;
    if (STATS) {
      const float n_tot = pair32_add(l_nex);
      const float x_tot = pair32_add(l_ex);
      if (n < t.nrows && g == 0) {
        const size_t idx = static_cast<size_t>(base + t.p0 + n) * Hq + h;
        if (rows.nexus_mass != nullptr) rows.nexus_mass[idx] = n_tot / x_tot;
        rows.lse[idx] = m_run + __builtin_amdgcn_logf(x_tot);
      }
    }
    if (n < t.nrows) {
      float *orow = out + (static_cast<size_t>(base + t.p0 + n) * Hq + h) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f32x4 o = {oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv, oacc[db][4 * i + 2] * inv,
                     oacc[db][4 * i + 3] * inv};
          *reinterpret_cast<f32x4 *>(orow + db * 32 + 8 * i + 4 * g) = o;
        }
      }
    }
  }
}

// Ping-pong variant for G > 4 (one key group, one head per wave, no statistics).
// The waves form two groups, waves [0, 4) and [4, G), one wave of each on a SIMD
// (a workgroup's waves go to the SIMDs in turn), and the groups run half a step
// apart, so that in every phase one group runs matrix work while the other runs
// its softmax and each SIMD overlaps one wave's MFMAs with the other's VALU work:
//   phase 2c:     group 0: P.V(c-1), S(c)     group 1: softmax(c-1)
//   phase 2c+1:   group 0: softmax(c)         group 1: P.V(c-1), S(c)
// (In the single-group kernel the two waves of a SIMD belong to one workgroup and
// are held in step by its barriers, so their MFMA and VALU phases coincide.)
// LDS slot c % 2 holds K(c) and V(c-1) through phases 2c and 2c+1.  The first group
// issues the loads of K(c+1) and V(c) into the other slot at the start of phase 2c,
// behind the barrier that ends the last use of that slot, and waits for them at the
// start of phase 2c+2.  Every phase begins with a barrier: two per 64-key step, as
// in the single-group kernel.  The arithmetic of a row and head is the same as
// there, in the same order, so the outputs are identical.
template <int D, int G>
__global__ __launch_bounds__(G * kWave, 2) void prefill_pp_kernel(AttnRows rows, PrefillWs ws, int Hkv,
                                                                  float scale_log2) {
  static_assert(G > 4 && G <= 8, "two groups of waves, the second of G - 4");
  const uint16_t *__restrict__ q = rows.q;
  float *__restrict__ out = rows.out;
  constexpr int DC = D / 8;              // 16-byte chunks per K/V row
  constexpr int DS = D / 16;             // d steps of the S product
  constexpr int DB = D / 32;             // 32-wide d blocks of the output
  constexpr float kLazy = 8.f;           // rescale only when the running max grows by > 2^8
  __shared__ __align__(16) uint16_t k_lds0[kKeyChunk * D];   // [64 keys][D], MFMA row order
  __shared__ __align__(16) uint16_t k_lds1[kKeyChunk * D];
  __shared__ __align__(16) uint16_t v_lds0[kKeyChunk * D];   // [64 keys][D], key order
  __shared__ __align__(16) uint16_t v_lds1[kKeyChunk * D];
  __shared__ int s_item;

  const int Hq = Hkv * G;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int grp = wave < 4 ? 0 : 1;
  const int lane = threadIdx.x % kWave;
  const int n = lane & 31;
  const int g = lane >> 5;
  const int xcd = blockIdx.x % kNumXcd;
  const int nitems = ws.ctrl[0] * Hkv;
  const int tq = lane >> 4;
  const int ti = lane & 15;
  const int v_row_off = 8 * (tq >> 1) + (ti >> 2);
  const int v_d_off = 16 * (tq & 1) + 4 * (ti & 3);
  const uint32_t row_bytes = static_cast<uint32_t>(Hkv) * D * 2;
  const uint32_t koff_lane = dma_lane_off<D, false>(lane, row_bytes);
  const uint32_t voff_lane = dma_lane_off<D, true>(lane, row_bytes);
  __builtin_assume(wave < G);

  for (;;) {
    if (threadIdx.x == 0) s_item = atomicAdd(&ws.ctrl[8 + xcd], 1) * kNumXcd + xcd;
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(s_item);
    __syncthreads();
    if (item >= nitems) break;
    const int slot = ws.order[item / Hkv];
    const int kvh = item % Hkv;
    TileDesc t = ws.tiles[slot];
    t.req = __builtin_amdgcn_readfirstlane(t.req);
    t.p0 = __builtin_amdgcn_readfirstlane(t.p0);
    t.nrows = __builtin_amdgcn_readfirstlane(t.nrows);
    t.npre = __builtin_amdgcn_readfirstlane(t.npre);
    t.seg_start = __builtin_amdgcn_readfirstlane(t.seg_start);
    t.seg_len = __builtin_amdgcn_readfirstlane(t.seg_len);
    t.ndiag = __builtin_amdgcn_readfirstlane(t.ndiag);
    const int base = rows.seg_row0[t.req];
    const int64_t pbase = rows.pre_row0 != nullptr ? rows.pre_row0[t.req] : static_cast<int64_t>(base);
    const int h = kvh * G + wave;
    const int nv = tile_key_count(t);
    const int nF = nv - t.ndiag;
    const int npre = t.npre;
    const int seg_shift = t.seg_start - npre;
    const size_t tok_stride = static_cast<size_t>(Hkv) * D;
    const size_t head0 = static_cast<size_t>(base) * tok_stride + static_cast<size_t>(kvh) * D;
    const size_t phead0 = static_cast<size_t>(pbase) * tok_stride + static_cast<size_t>(kvh) * D;
    const char *kreq = uniform_ptr(reinterpret_cast<const char *>(rows.seg_k + head0));
    const char *vreq = uniform_ptr(reinterpret_cast<const char *>(rows.seg_v + head0));
    const char *kpre = uniform_ptr(reinterpret_cast<const char *>(rows.pre_k + phead0));
    const char *vpre = uniform_ptr(reinterpret_cast<const char *>(rows.pre_v + phead0));
    const int nch = (nv + kKeyChunk - 1) / kKeyChunk;

    bf16x8 qf[DS];
    {
      const bool ok = n < t.nrows;
      const uint16_t *qrow = q + (static_cast<size_t>(base + t.p0 + n) * Hq + h) * D;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (ok) w = *reinterpret_cast<const u32x4 *>(qrow + 16 * ds + 8 * g);
        qf[ds] = __builtin_bit_cast(bf16x8, w);
      }
    }
    f32x16 oacc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) oacc[i] = f32x16{};
    float m_run = -INFINITY;
    float l_run = 0.f;
    f32x16 sacc[2];       // S(c), from the matrix phase to the softmax phase
    bf16x8 pb[4];         // P(c) in bf16, from the softmax phase to the next matrix phase
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) sacc[kb] = f32x16{};
#pragma unroll
    for (int i = 0; i < 4; ++i) pb[i] = bf16x8{};

    // matrix phase c: O += V(c-1)^T . P(c-1)^T, then S(c) = K(c) . Q^T (both from slot c % 2)
    auto matrix_phase = [&](int c, const uint16_t *kc_lds, const uint16_t *vc_lds) {
      if (c >= 1) {
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int dd = db * 32 + v_d_off;
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
            v4i16 part[2];
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
              const int r = 16 * ks + 4 * hh + v_row_off;
              const int chunk = (dd >> 3) ^ swz_v<D>(r);
              const uint16_t *pa = &vc_lds[r * D + chunk * 8 + (dd & 4)];
              part[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)pa);
            }
            const u32x4 w = {__builtin_bit_cast(uint2, part[0]).x, __builtin_bit_cast(uint2, part[0]).y,
                             __builtin_bit_cast(uint2, part[1]).x, __builtin_bit_cast(uint2, part[1]).y};
            oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w), pb[ks], oacc[db], 0,
                                                               0, 0);
          }
        }
        order_reads_ahead<4 * DB, 2, kAheadPV>();
      }
      if (c < nch) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          sacc[kb] = f32x16{};
          const int m = kb * 32 + n;
#pragma unroll
          for (int ds = 0; ds < DS; ++ds) {
            const bf16x8 a =
                *reinterpret_cast<const bf16x8 *>(&kc_lds[(m * DC + ((2 * ds + g) ^ swz_k<D>(m))) * 8]);
            sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ds], sacc[kb], 0, 0, 0);
          }
        }
        order_reads_ahead<2 * DS, 1, kAheadS>();
      }
    };
    // softmax phase c: mask, lazy max, P(c) in bf16 and the sum of its rounded values
    auto softmax_phase = [&](int c) {
      const int vk0 = c * kKeyChunk;
      if (vk0 + kKeyChunk > nF) {
        const int lim_g = min(nv, nF + n + 1) - vk0 - 8 * g;   // bound on acc_key0
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e) sacc[kb][e] = (kb * 32 + acc_key0(e) < lim_g) ? sacc[kb][e] : -INFINITY;
      }
      float mloc = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mloc = fmaxf(mloc, sacc[kb][e]);
      mloc = pair32_max(mloc) * scale_log2;
      if (__any(mloc > m_run + kLazy)) {
        const float m_new = fmaxf(m_run, mloc);
        const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
        m_run = m_new;
        l_run *= corr;
#pragma unroll
        for (int db = 0; db < DB; ++db) oacc[db] *= corr;
      }
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x8 lo, hi;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          lo[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][e], scale_log2, -m_run));
          hi[e] = __builtin_amdgcn_exp2f(fmaf(sacc[kb][8 + e], scale_log2, -m_run));
        }
        pb[2 * kb] = __builtin_convertvector(lo, bf16x8);
        pb[2 * kb + 1] = __builtin_convertvector(hi, bf16x8);
      }
      l_run += rounded_sum(pb);
    };
    // Step c of a group: its matrix phase, a barrier, its softmax phase.  Both groups run
    // the same code; the second enters one barrier later (and the first leaves one
    // barrier later), so its step c falls on phases 2c+1 and 2c+2.  Slot c % 2 =
    // (k_cur, v_cur) holds K(c) and V(c-1).  Only the first group loads: at the start of
    // its step c it waits for its loads of slot c % 2, passes the barrier, then requests
    // K(c+1) and V(c) into the other slot, whose last reader (the second group's step
    // c-1 matrix phase) has passed that barrier too.  Steps run to c = nch, whose
    // matrix phase only adds P(nch-1).
    auto pp_step = [&](int c, const uint16_t *k_cur, const uint16_t *v_cur, uint16_t *k_nxt, uint16_t *v_nxt) {
      wait_vm<0>();
      lds_barrier();
      if (grp == 0) {
        if (c + 1 < nch)
          stage_tensor<D, 4, false>(k_nxt, kpre, kreq, row_bytes, koff_lane, wave, lane, c + 1, nv, npre, seg_shift);
        if (c < nch)
          stage_tensor<D, 4, true>(v_nxt, vpre, vreq, row_bytes, voff_lane, wave, lane, c, nv, npre, seg_shift);
      }
      matrix_phase(c, k_cur, v_cur);
      lds_barrier();
      if (c < nch) softmax_phase(c);
    };

    if (grp == 0)
      stage_tensor<D, 4, false>(k_lds0, kpre, kreq, row_bytes, koff_lane, wave, lane, 0, nv, npre, seg_shift);
    else
      lds_barrier();
    for (int c = 0; c <= nch; c += 2) {
      pp_step(c, k_lds0, v_lds0, k_lds1, v_lds1);
      if (c + 1 > nch) break;
      pp_step(c + 1, k_lds1, v_lds1, k_lds0, v_lds0);
    }
    if (grp == 0) lds_barrier();

    const float l_tot = pair32_add(l_run);
    const float inv = 1.f / l_tot;
    if (n < t.nrows) {
      float *orow = out + (static_cast<size_t>(base + t.p0 + n) * Hq + h) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f32x4 o = {oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv, oacc[db][4 * i + 2] * inv,
                     oacc[db][4 * i + 3] * inv};
          *reinterpret_cast<f32x4 *>(orow + db * 32 + 8 * i + 4 * g) = o;
        }
      }
    }
  }
}

template <int D, int G>
static hipError_t launch_prefill_dg(int grid, bool stats, int ks, AttnRows rows, PrefillWs ws, int Hkv,
                                    float scale_log2, hipStream_t stream) {
  if (stats)
    prefill_kernel<D, G, true, 1><<<dim3(grid), dim3(G * kWave), 0, stream>>>(rows, ws, Hkv, scale_log2);
  else if (ks == 2) {
    if constexpr (G <= 4)
      prefill_kernel<D, G, false, 2><<<dim3(grid), dim3(2 * G * kWave), 0, stream>>>(rows, ws, Hkv, scale_log2);
    else
      return hipErrorInvalidValue;
  } else if constexpr (G > 4)
    prefill_pp_kernel<D, G><<<dim3(grid), dim3(G * kWave), 0, stream>>>(rows, ws, Hkv, scale_log2);
  else
    prefill_kernel<D, G, false, 1><<<dim3(grid), dim3(G * kWave), 0, stream>>>(rows, ws, Hkv, scale_log2);
  return hipGetLastError();
}

template <int D, int G>
static hipError_t occupancy_dg(bool stats, int ks, int *blocks) {
  if (stats)
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, prefill_kernel<D, G, true, 1>, G * kWave, 0);
  if (ks == 2) {
    if constexpr (G <= 4)
      return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, prefill_kernel<D, G, false, 2>, 2 * G * kWave, 0);
    else
      return hipErrorInvalidValue;
  }
  if constexpr (G > 4)
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, prefill_pp_kernel<D, G>, G * kWave, 0);
  else
    return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, prefill_kernel<D, G, false, 1>, G * kWave, 0);
}

#define SONIC_FOR_G(D, X) \
  switch (G) {            \
    case 1: X(D, 1); break; \
    case 2: X(D, 2); break; \
    case 3: X(D, 3); break; \
    case 4: X(D, 4); break; \
    case 5: X(D, 5); break; \
    case 6: X(D, 6); break; \
    case 7: X(D, 7); break; \
    case 8: X(D, 8); break; \
    default: return hipErrorInvalidValue; \
  }

hipError_t prefill_occupancy(int D, int G, bool stats, int ks, int *blocks) {
#define OCC(DD, GG) return occupancy_dg<DD, GG>(stats, ks, blocks)
  if (D == 64) {
    SONIC_FOR_G(64, OCC)
  } else if (D == 128) {
    SONIC_FOR_G(128, OCC)
  }
#undef OCC
  return hipErrorInvalidValue;
}

hipError_t launch_prefill(int D, int G, int grid, bool stats, int ks, AttnRows rows, PrefillWs ws, int Hkv,
                          float scale_log2, hipStream_t stream) {
#define LAUNCH(DD, GG) return launch_prefill_dg<DD, GG>(grid, stats, ks, rows, ws, Hkv, scale_log2, stream)
  if (D == 64) {
    SONIC_FOR_G(64, LAUNCH)
  } else if (D == 128) {
    SONIC_FOR_G(128, LAUNCH)
  }
#undef LAUNCH
  return hipErrorInvalidValue;
}

}  // namespace sonic
