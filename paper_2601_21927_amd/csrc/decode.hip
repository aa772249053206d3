// Decode over the retained context {I_sys, N, Q_n} (problem statement).
//
// decode_kernel: grid (split, kv-head, request), 8 waves.  A split owns a
// contiguous range of the request's context rows 0..len (row len is the token
// being generated: it is read from k_new/v_new, and split 0 of each kv-head also
// appends it to the cache).  The range is cut into 16-row groups, dealt to the
// waves round-robin; per group a wave computes
//   scores   S^T (16 rows x 16 cols) = K . Q^T   v_mfma_f32_16x16x32_bf16;
//            column c < G is q-head kvh*G + c;
//   softmax  per q-head, online, fp32, exp2 with log2(e) folded into the scale;
//            a column's statistics live in the four lanes that hold it;
//   values   O^T (d x 16 cols) += V^T . P^T   v_mfma_f32_16x16x16_bf16, V read
//            back transposed (ds_read_b64_tr_b16); P^T is the score accumulator
//            itself, rounded to bf16 (its lane layout is the operand layout), and
//            the softmax sum adds those rounded values.
// K and V rows go straight from global memory to a two-slot LDS ring of the
// wave's own (direct-to-LDS loads), so a wave keeps its next group in flight
// while it computes one.  The waves then merge through LDS.
//
// With one split the workgroup writes the output.  With several, each split
// stores its partial (max, sum, acc) and counts itself done with an atomic; the
// split that arrives last merges the partials by log-sum-exp and writes the
// output.  The eight XCDs' L2 caches are not coherent with each other, so the
// hand-off does not go through them: the partials are stored write-through at
// system scope and read back with loads that bypass the caches, which needs no
// L2 writeback or invalidate (either would evict the K/V other workgroups are
// streaming).  Every split of a pair counts itself once per call, splits
// without rows included, so the last to count knows that every workgroup of
// the pair has read cache_len; it counts the pair for its request while it
// loads the partials, and the last pair of a request advances cache_len.
#include "common.h"

namespace sonic {

constexpr int kDecWaves = 8;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kGroupRows = 16;
constexpr int kMergeBatch = 16;   // partials loaded per memory round trip of the merge

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// The K/V loads of the pipeline go straight to LDS and are written as inline
// assembly, so the compiler does not count them (it would otherwise wait for the
// prefetched group as well before reading the current one); their completion is
// waited for explicitly (wait_vm).
// 16 bytes per lane into LDS at dst + 16 * lane (dst wave-uniform, passed in M0)
__device__ __forceinline__ void dma16(const void *src, const uint16_t *dst) {
  // C-style cast: converting the LDS pointer to its 32-bit address
  const uint32_t lds = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) uint16_t *)dst)));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(lds) : "memory", "m0");
}
// A load that bypasses the (non-coherent) caches, for partials another XCD stored
// write-through; completion is waited for explicitly.
__device__ __forceinline__ float load_sys(const float *p) {
  float v;
  asm volatile("global_load_dword %0, %1, off sc0 sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// atomic add of 1 returning the old value; the result register is written when the
// atomic returns, so it is read only after an explicit wait_vm<0>
__device__ __forceinline__ int atomic_inc_pending(int32_t *p) {
  int old;
  asm volatile("global_atomic_add %0, %1, %2, off sc0" : "=v"(old) : "v"(p), "v"(1) : "memory");
  return old;
}

template <int D, int G, bool MASKED>
__global__ __launch_bounds__(kDecThreads, 1) void decode_kernel(
    uint16_t *__restrict__ kc, uint16_t *__restrict__ vc, const int64_t *__restrict__ row_off,
    const int32_t *__restrict__ row_cap, int32_t *__restrict__ cache_len, const uint8_t *__restrict__ row_role,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new,
    float *__restrict__ out, DecodeWs ws, int32_t *status, int Hkv, int nsplit_max, int max_ctx,
    float scale_log2) {
  constexpr int KS = D / 32;                   // k steps of the 16x16x32 score product
  constexpr int DB = D / 16;                   // 16-wide d blocks of the value product
  constexpr int DC = D / 8;                    // 16-byte chunks per row
  constexpr int NI = kGroupRows * DC / kWave;  // direct-to-LDS instructions per tensor and group
  constexpr int NG = 2 * NI;                   // loads per lane per group
  constexpr int REC = G * (D + 2);             // floats of one partial record
  constexpr int SLOT = kGroupRows * D;         // elements of one tensor's slot
  constexpr int KSWZ = DC - 1;                 // K: 16-byte chunk p of row r at p ^ (r & KSWZ)
  constexpr int VSWZ = DC / 2 - 1;             // V: 32-byte segment s of row r at s ^ (r & VSWZ)
  static_assert(NI * kWave == kGroupRows * DC, "a group's rows are whole DMA instructions");
  // ring: [wave][slot 0/1][K, V][16 rows][D] with the swizzles above (K for the
  // row-fragment reads of the scores, V for the transposing reads); reused for the
  // merge of the waves at the end
  __shared__ __align__(16) uint16_t ring[kDecWaves * 2 * 2 * SLOT];
  // each wave's copy of the G query rows (direct-to-LDS, so that no load the
  // compiler counts precedes the pipeline's)
  constexpr int NQ = (G * D * 2 + 1023) / 1024;   // direct-to-LDS instructions for Q
  __shared__ __align__(16) uint16_t q_lds[kDecWaves][NQ * 512];
  // split 0: the new token's k and v rows, fetched at the start and appended at the end
  __shared__ __align__(16) uint16_t app_lds[kWave * 8];
  static_assert(2 * DC <= kWave, "one direct-to-LDS instruction holds the new k and v rows");
  __shared__ float m_lds[kDecWaves][16];
  __shared__ float l_lds[kDecWaves][16];
  __shared__ int s_last;
  static_assert(sizeof(float) * kDecWaves * G * D <= sizeof(uint16_t) * kDecWaves * 4 * SLOT,
                "the merge fits in the ring");

  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int Hq = Hkv * G;
  // the status word, the length and the request's first cache row are requested
  // together (one round trip for all three)
  const int32_t pending = __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int len = cache_len[b];
  const int cap = row_cap[b];
  const int64_t base = row_off[b];
  asm volatile("" ::"s"(base));
  // A pending error other than a capacity error (a layout error of an earlier call)
  // stops the whole call: nothing is appended, written or advanced.  Only capacity
  // errors can appear during the call (raised below, per request), so every
  // workgroup of the call takes the same decision and no counter is touched.
  if (pending != 0 && pending != SONIC_ERR_CAPACITY) return;
  const int n_ctx = len + 1;
  if (n_ctx > cap || n_ctx > max_ctx) {   // uniform over the request: no append, no output
    if (split == 0 && kvh == 0 && threadIdx.x == 0) raise_status(status, SONIC_ERR_CAPACITY);
    return;
  }
  // split ranges: R rows each, a multiple of the group size
  const int R = ((n_ctx + nsplit_max - 1) / nsplit_max + kGroupRows - 1) / kGroupRows * kGroupRows;
  const int nsp = (n_ctx + R - 1) / R;   // splits that hold rows; the others have nothing to do
  const int nsplit = gridDim.x;
  const int pair = b * Hkv + kvh;
  float *orow = out + (static_cast<size_t>(b) * Hq + kvh * G) * D;

  // Every split counts itself once, after its partial (if any) is stored.  The last
  // to count merges the partials of the nsp splits with rows by log-sum-exp, a batch
  // of kMergeBatch per memory round trip, writes the output, and counts the pair for its
  // request while the partials load; the last pair of a request advances the length.
  auto finish_pair = [&]() {
    if (threadIdx.x == 0) s_last = (atomicAdd(&ws.arrive[pair], 1) == nsplit - 1);
    __syncthreads();
    if (!s_last) return;
    int old_done = 0;
    if (threadIdx.x == 0) old_done = atomic_inc_pending(&ws.done[b]);
    const float *recs = ws.part + static_cast<size_t>(pair) * nsplit_max * REC;
    for (int idx = threadIdx.x; idx < G * D; idx += kDecThreads) {
      const int hh = idx / D, dd = idx % D;
      float M = -INFINITY, L = 0.f, A = 0.f;
      for (int sp0 = 0; sp0 < nsp; sp0 += kMergeBatch) {
        float m[kMergeBatch], l[kMergeBatch], a[kMergeBatch];
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
          const float *r = recs + static_cast<size_t>(min(sp0 + u, nsp - 1)) * REC + hh * (D + 2);
          m[u] = load_sys(r);
          l[u] = load_sys(r + 1);
          a[u] = load_sys(r + 2 + dd);
        }
        wait_vm<0>();
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) asm volatile("" : "+v"(m[u]), "+v"(l[u]), "+v"(a[u]));
        float Mb = M;
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u)
          if (sp0 + u < nsp) Mb = fmaxf(Mb, m[u]);
        const float c = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mb);
        L *= c;
        A *= c;
#pragma unroll
        for (int u = 0; u < kMergeBatch; ++u) {
          const float w = (sp0 + u < nsp && m[u] != -INFINITY) ? __builtin_amdgcn_exp2f(m[u] - Mb) : 0.f;
          L = fmaf(w, l[u], L);
          A = fmaf(w, a[u], A);
        }
        M = Mb;
      }
      orow[idx] = A / L;
    }
    wait_vm<0>();
    if (threadIdx.x == 0) {
      asm volatile("" : "+v"(old_done));
      ws.arrive[pair] = 0;
      if (old_done == Hkv - 1) {
        cache_len[b] = n_ctx;
        ws.done[b] = 0;
      }
    }
  };
  if (split >= nsp) {   // no rows (only when nsplit > 1)
    finish_pair();
    return;
  }
  const int r_begin = split * R;
  const int r_end = min(n_ctx, r_begin + R);
  const int ngroups = (r_end - r_begin + kGroupRows - 1) / kGroupRows;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int col = lane & 15;       // score column (q-head) / value-product column
  const int quarter = lane >> 4;   // score rows 4*quarter .. +3
  const size_t row_stride = static_cast<size_t>(Hkv) * D;
  const uint16_t *knew = k_new + (static_cast<size_t>(b) * Hkv + kvh) * D;
  const uint16_t *vnew = v_new + (static_cast<size_t>(b) * Hkv + kvh) * D;
  uint16_t *kbase = kc + static_cast<size_t>(base) * row_stride + static_cast<size_t>(kvh) * D;
  uint16_t *vbase = vc + static_cast<size_t>(base) * row_stride + static_cast<size_t>(kvh) * D;

  // Split 0 appends the new token at row len.  Its rows go to LDS ahead of every other
  // load of wave 0 (so the first wait covers them, and no wave waits for a load of its
  // own before the pipeline starts); the stores happen after the streaming.  Rows of
  // this call read the new token from k_new / v_new, so nothing here depends on them.
  const bool appender = split == 0 && wave == 0;
  if (appender) {
    const int c = lane < 2 * DC ? lane % DC : 0;
    dma16((lane >= DC && lane < 2 * DC ? vnew : knew) + c * 8, app_lds);
  }

  // The wave's Q rows go to q_lds (lanes past the G rows fetch row 0 again); the
  // Q^T fragments (B operand of the scores) are read from there once the first wait
  // has passed: lane (col, quarter) takes d = 32*ks + 8*quarter .. +7 of q-head
  // kvh*G + col (columns col >= G take head kvh*G and are never read back).
  {
    const uint16_t *q0 = q + (static_cast<size_t>(b) * Hq + kvh * G) * D;
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      const int e = (i * kWave + lane) * 8;   // element of the [G][D] block
      dma16(q0 + (e < G * D ? e : e % D), &q_lds[wave][i * 512]);
    }
  }
  bf16x8 qf[KS];
  auto read_q = [&]() {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[ks] = *reinterpret_cast<const bf16x8 *>(&q_lds[wave][(col < G ? col : 0) * D + 32 * ks + 8 * quarter]);
  };

  // Row r of the context: the cache below len, the new token at len.  Rows past the
  // split's end load row r_begin instead (and are masked), so every group issues the
  // same loads and the waits can be counted.
  auto row_of = [&](int r) { return r < r_end ? r : r_begin; };
  auto kptr = [&](int r) { return r < len ? kbase + static_cast<size_t>(r) * row_stride : knew; };
  auto vptr = [&](int r) { return r < len ? vbase + static_cast<size_t>(r) * row_stride : vnew; };
  uint16_t *my_ring = ring + wave * 4 * SLOT;

  // Group g of the split covers rows r_begin + 16 g ...; wave w takes groups w, w + 8,
  // w + 16, ... (a fixed order, so the result does not depend on timing).
  auto group_row0 = [&](int g) { return r_begin + kGroupRows * g; };
  // issue the loads of group g into ring slot s: lane -> (row, 16-byte position) of
  // each instruction's rows; the position holds the row's swizzled chunk
  auto issue = [&](int g, int s) {
    const int r0 = group_row0(g);
    uint16_t *kslot = my_ring + s * 2 * SLOT;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int rl = (i * kWave + lane) / DC;
      const int pos = (i * kWave + lane) % DC;
      const int r = row_of(r0 + rl);
      dma16(kptr(r) + (pos ^ (rl & KSWZ)) * 8, kslot + i * kWave * 8);
      dma16(vptr(r) + (pos ^ (2 * (rl & VSWZ))) * 8, kslot + SLOT + i * kWave * 8);
    }
  };
  // masked full-cache mode: the role bytes of this lane's four score rows
  auto load_roles = [&](int r0) {
    uint32_t roles = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // the clamped index keeps the load inside the request's rows; rows at or past
      // len are the new token, whose role is CURRENT (see the mask below)
      const int r = r0 + 4 * quarter + i;
      roles |= static_cast<uint32_t>(row_role[base + max(0, min(r, len - 1))]) << (8 * i);
    }
    return roles;
  };

  f32x4 oacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) oacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;   // running max (log2 domain) of column col, lagging by at most 8
  float l_run = 0.f;         // this lane's share of the column's sum

  // score fragments: lane (col, quarter) reads row col, d = 32*ks + 8*quarter (chunk 4*ks + quarter)
  const int k_off = col * D;
  // transposed-read geometry (value product): 16-lane group kq reads rows 4*kq + (t >> 2)
  // at d = 16*db + 4*(t & 3), t = lane % 16; lane t then holds V[4*kq .. +3][16*db + t]
  const int tr_row = 4 * quarter + (col >> 2);
  const int tr_off = tr_row * D + 4 * (col & 3);
  const int tr_swz = tr_row & VSWZ;

  auto process = [&](int g, int s) {
    const int r0 = group_row0(g);
    const uint16_t *kslot = my_ring + s * 2 * SLOT;
    const uint32_t roles = MASKED ? load_roles(r0) : 0u;
    f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kslot + k_off + (((4 * ks + quarter) ^ (col & KSWZ)) * 8));
      sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[ks], sacc, 0, 0, 0);
    }
    // lane (col, quarter) holds rows r0 + 4*quarter + i of column col
    float x[4];
    float mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = r0 + 4 * quarter + i;
      bool vis = r < r_end;
      if (MASKED) vis = vis && (r >= len || ((roles >> (8 * i)) & 0xFF) != kText);
      x[i] = vis ? sacc[i] * scale_log2 : -INFINITY;
      mloc = fmaxf(mloc, x[i]);
    }
    mloc = pair32_max(pair16_max(mloc));
    if (__any(mloc > m_run + 8.f)) {   // rescale only when the max grows by more than 2^8
      const float m_new = fmaxf(m_run, mloc);
      const float corr = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= corr;
#pragma unroll
      for (int i = 0; i < DB; ++i) oacc[i] *= corr;
    }
    f32x4 p;
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = (x[i] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(x[i] - m_run);
    const bf16x4 pr = __builtin_convertvector(p, bf16x4);
    const v4i16 pb = __builtin_bit_cast(v4i16, pr);
    // the sum is taken over the rounded probabilities the value product uses, so the
    // output stays a convex combination of the V rows (see the prefill)
    {
      const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);
      l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pr, pr, 0, 1), ones, l_run, false);
      l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pr, pr, 2, 3), ones, l_run, false);
    }
    const uint16_t *vslot = kslot + SLOT;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint16_t *pa = vslot + tr_off + ((db ^ tr_swz) * 16);
      // C-style cast: the transposing read takes an LDS-qualified pointer
      const v4i16 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)pa);
      oacc[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, pb, oacc[db], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));   // lgkmcnt(0): slot s may be refilled
  };

  // two-deep pipeline: a slot is refilled as soon as its group has been processed
  int ga = wave, gb = wave + kDecWaves;   // the groups in ring slots 0 and 1
  issue(ga, 0);
  issue(gb, 1);
  wait_vm<NG>();                          // Q and slot 0 have landed (slot 1 may not have)
  read_q();
  while (ga < ngroups) {
    process(ga, 0);
    ga += 2 * kDecWaves;
    issue(ga, 0);
    wait_vm<NG>();                        // slot 1 has landed (slot 0 may not have)
    if (gb >= ngroups) break;
    process(gb, 1);
    gb += 2 * kDecWaves;
    issue(gb, 1);
    wait_vm<NG>();
  }
  wait_vm<0>();   // the trailing (unused) loads, before the ring is reused
  if (appender && lane < 2 * DC) {
    const size_t dst = static_cast<size_t>(len) * row_stride + (lane % DC) * 8;
    *reinterpret_cast<u32x4 *>((lane < DC ? kbase : vbase) + dst) = *reinterpret_cast<const u32x4 *>(&app_lds[lane * 8]);
  }

  // ---- merge: columns across the four quarters, then the waves through LDS ----
  l_run = pair32_add(pair16_add(l_run));
  if (quarter == 0) {
    m_lds[wave][col] = m_run;
    l_lds[wave][col] = l_run;
  }
  __syncthreads();   // every wave is done with the ring
  float *acc_lds = reinterpret_cast<float *>(ring);   // [wave][G][D]
  if (col < G) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc_lds[(wave * G + col) * D + 16 * db + 4 * quarter + i] = oacc[db][i];
  }
  __syncthreads();

  float *rec = ws.part + (static_cast<size_t>(pair) * nsplit_max + split) * REC;
  for (int idx = threadIdx.x; idx < G * D; idx += kDecThreads) {
    const int hh = idx / D, dd = idx % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, m_lds[w][hh]);
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float sc = (m_lds[w][hh] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_lds[w][hh] - M);
      L = fmaf(sc, l_lds[w][hh], L);
      A = fmaf(sc, acc_lds[(w * G + hh) * D + dd], A);
    }
    if (nsplit == 1) {
      orow[idx] = A / L;
    } else {   // write-through at system scope (see the top of the file)
      if (dd == 0) {
        __hip_atomic_store(rec + hh * (D + 2), M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(rec + hh * (D + 2) + 1, L, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
      }
      __hip_atomic_store(rec + hh * (D + 2) + 2 + dd, A, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
  }
  if (nsplit > 1) {
    wait_vm<0>();      // this thread's partial is stored
    __syncthreads();   // ... and every thread's
    finish_pair();
  } else if (threadIdx.x == 0 && atomicAdd(&ws.done[b], 1) == Hkv - 1) {
    cache_len[b] = n_ctx;
    ws.done[b] = 0;
  }
}

// Splits per (request, kv-head).  A workgroup fills a CU (one per CU), so with fewer
// than 256 pairs the grid takes as many splits as keep every workgroup resident at
// once (a 257th would wait for a whole workgroup to finish: on the 8B-shaped batch,
// 64 pairs, 4 splits take 13.7 us per call and 5 take 18.3), each of at least 256
// rows, and at most 16 (the merging split loads sixteen partials per memory round
// trip; on the long-dialogue shape, 16 pairs of ~8k rows, 8 splits take 19.0 us per
// call and 16 take 18.5, 22.6 against 24.6 us with the caches cold).  With 256 pairs
// or more, one split, or three when the longest context reaches 2048 rows, so that
// the longest pairs do not outlast the rest of the call when lengths are uneven
// (dynamic-budget batch: 1 split 127.7 us, 2 117.1, 3 111.4, 4 121.3 per call).
int decode_splits(int batch, int Hkv, int max_ctx) {
  const long pairs = static_cast<long>(batch) * Hkv;
  if (pairs >= 256) return max_ctx >= 2048 ? 3 : 1;
  long s = 256 / pairs;
  const long by_rows = (static_cast<long>(max_ctx) + 255) / 256;
  if (s > by_rows) s = by_rows;
  if (s > kMergeBatch) s = kMergeBatch;
  return static_cast<int>(s < 1 ? 1 : s);
}

// Fixed layout of a scratch array shared by calls of different shapes: the counters
// sit at the same offsets for every call (each call leaves them at zero), the partial
// records after them.  Returns the bytes a call needs, or 0 when its requests or
// (request, kv-head) pairs exceed the fixed counter regions.
size_t decode_scratch_layout(int batch, int Hkv, int G, int D, int nsplit, DecodeWs *ws, char *base) {
  if (batch > kScratchMaxRequests || static_cast<long>(batch) * Hkv > kScratchMaxPairs) return 0;
  const size_t pbytes = nsplit > 1 ? static_cast<size_t>(batch) * Hkv * nsplit * G * (D + 2) * sizeof(float) : 0;
  if (ws) {
    ws->done = reinterpret_cast<int32_t *>(base);
    ws->arrive = reinterpret_cast<int32_t *>(base + kScratchMaxRequests * sizeof(int32_t));
    ws->part = reinterpret_cast<float *>(base + kScratchCounterBytes);
  }
  return kScratchCounterBytes + pbytes;
}

size_t decode_ws_layout(int batch, int Hkv, int G, int D, int nsplit, DecodeWs *ws, char *base) {
  const size_t dbytes = (static_cast<size_t>(batch) * sizeof(int32_t) + 255) / 256 * 256;
  const size_t abytes = (static_cast<size_t>(batch) * Hkv * sizeof(int32_t) + 255) / 256 * 256;
  const size_t pbytes = nsplit > 1 ? static_cast<size_t>(batch) * Hkv * nsplit * G * (D + 2) * sizeof(float) : 0;
  if (ws) {
    ws->done = reinterpret_cast<int32_t *>(base);
    ws->arrive = reinterpret_cast<int32_t *>(base + dbytes);
    ws->part = reinterpret_cast<float *>(base + dbytes + abytes);
  }
  return dbytes + abytes + pbytes;
}

template <int D, int G>
static void launch_decode_dg(dim3 grid, int batch, int Hkv, int max_ctx, int nsplit, uint16_t *kc, uint16_t *vc,
                             const int64_t *row_off, const int32_t *row_cap, int32_t *cache_len,
                             const uint8_t *row_role, const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                             float scale_log2, float *out, DecodeWs ws, int32_t *status, hipStream_t stream) {
  if (row_role != nullptr)
    decode_kernel<D, G, true><<<grid, dim3(kDecThreads), 0, stream>>>(kc, vc, row_off, row_cap, cache_len, row_role,
                                                                      q, k_new, v_new, out, ws, status, Hkv, nsplit,
                                                                      max_ctx, scale_log2);
  else
    decode_kernel<D, G, false><<<grid, dim3(kDecThreads), 0, stream>>>(kc, vc, row_off, row_cap, cache_len,
                                                                       row_role, q, k_new, v_new, out, ws, status,
                                                                       Hkv, nsplit, max_ctx, scale_log2);
}

hipError_t launch_decode(int batch, int Hq, int Hkv, int D, int max_ctx, int nsplit, uint16_t *kc, uint16_t *vc,
                         const int64_t *row_off, const int32_t *row_cap, int32_t *cache_len, const uint8_t *row_role,
                         const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new, float scale_log2,
                         float *out, const DecodeWs &ws, int32_t *status, hipStream_t stream) {
  const int G = Hq / Hkv;
  dim3 grid(nsplit, Hkv, batch);
#define DEC(DD, GG)                                                                                               \
  case GG:                                                                                                        \
    launch_decode_dg<DD, GG>(grid, batch, Hkv, max_ctx, nsplit, kc, vc, row_off, row_cap, cache_len, row_role, q, \
                             k_new, v_new, scale_log2, out, ws, status, stream);                                  \
    break;
#define DEC_ALL_G(DD)                     \
  switch (G) {                            \
    DEC(DD, 1)                            \
    DEC(DD, 2)                            \
    DEC(DD, 3)                            \
    DEC(DD, 4)                            \
    DEC(DD, 5)                            \
    DEC(DD, 6)                            \
    DEC(DD, 7)                            \
    DEC(DD, 8)                            \
    default: return hipErrorInvalidValue; \
  }
  if (D == 64) {
    DEC_ALL_G(64)
  } else if (D == 128) {
    DEC_ALL_G(128)
  } else {
    return hipErrorInvalidValue;
  }
#undef DEC_ALL_G
#undef DEC
  return hipGetLastError();
}

}  // namespace sonic
