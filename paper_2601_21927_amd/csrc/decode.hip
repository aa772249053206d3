// Decode over the retained context {I_sys, N, Q_n} (App. C, Eq.(15)).
//
// decode_kernel: grid (split, kv-head, request), 4 waves.  A
// split owns rows [split*R, split*R + R) of the request's context rows 0..len
// (row len is the token being generated: it is read from k_new/v_new, and split 0
// of each kv-head also appends it to the cache).  A split is processed in rounds
// of 256 rows; each wave issues the loads of all four of its 16-row groups of a
// round before working through them:
//   scores    S^T (16 rows x 16 cols) = K . Q^T with v_mfma_f32_16x16x32_bf16;
//             column c < G is q-head kvh*G + c, the other columns are zero;
//   softmax   per q-head, online, fp32, exp2 with log2(e) folded into the scale;
//   values    P . V on the vector ALUs in fp32: lane (d chunk, row slot)
//             accumulates 8 d-values of every q-head of the group.
// The four waves merge through LDS.  With one split the workgroup writes the
// output; otherwise it stores its partial (max, sum, acc) for decode_combine.
//
// decode_combine_kernel: grid (kv-head, request) merges the splits with the
// log-sum-exp rule and (kv-head 0) advances cache_len.  Cross-workgroup merging
// is left to a second kernel on purpose: the L2 caches of the eight XCDs are
// not coherent with each other, so an in-kernel hand-off needs device-scope
// fences that write back and invalidate a whole L2, evicting the K/V that
// other workgroups are streaming; the kernel boundary gives the same
// visibility for free.
#include "common.h"

namespace sonic {

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kDecRowsPerGroup = 16;
constexpr int kGroups = 4;                                           // groups per wave per round
constexpr int kRoundRows = kGroups * kDecWaves * kDecRowsPerGroup;  // 256 rows per round

struct DecodeWs {
  float *part;        // [B*Hkv][nsplit][G*(D+2)] partial (m[G], l[G], acc[G][D]) per split
  int32_t *nsplit;    // [B] splits used by request b in this step (0: request skipped)
};

template <int D, int G>
__global__ __launch_bounds__(kDecThreads, 2) void decode_kernel(
    uint16_t *__restrict__ kc, uint16_t *__restrict__ vc, const int64_t *__restrict__ row_off,
    const int32_t *__restrict__ row_cap, int32_t *__restrict__ cache_len, const uint8_t *__restrict__ row_role,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new,
    float *__restrict__ out, DecodeWs ws, int32_t *status, int Hkv, int rows_per_split, int nsplit_max, int max_ctx,
    float scale_log2) {
  constexpr int KS = D / 32;            // k steps of the 16x16x32 product
  constexpr int DCH = D / 8;            // 8-value d chunks per row
  constexpr int ROWQ = kWave / DCH;     // row slots of the value phase
  constexpr int VPL = kDecRowsPerGroup / ROWQ;   // V rows per lane per group
  constexpr int REC = G * (D + 2);      // floats of one partial record
  __shared__ float p_lds[kDecWaves][kDecRowsPerGroup][8];
  __shared__ float corr_lds[kDecWaves][8];
  __shared__ float m_lds[kDecWaves][8];
  __shared__ float l_lds[kDecWaves][8];
  __shared__ float acc_lds[kDecWaves][G][D];

  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int Hq = Hkv * G;
  const int len = cache_len[b];
  const int n_ctx = len + 1;
  if (n_ctx > row_cap[b] || n_ctx > max_ctx) {   // uniform over the request: no append, no output
    if (split == 0 && kvh == 0 && threadIdx.x == 0) {
      raise_status(status, SONIC_ERR_CAPACITY);
      ws.nsplit[b] = 0;
    }
    return;
  }
  const int nsp = (n_ctx + rows_per_split - 1) / rows_per_split;
  if (split == 0 && kvh == 0 && threadIdx.x == 0) ws.nsplit[b] = nsp;
  if (split >= nsp) {
    // an unused split leaves an empty record (max -inf, sum 0, acc 0) so that the merge can
    // read every record without first waiting for the split count
    if (nsp > 1) {
      float *rec = ws.part + (static_cast<size_t>(b * Hkv + kvh) * nsplit_max + split) * REC;
      for (int idx = threadIdx.x; idx < REC; idx += kDecThreads) rec[idx] = (idx % (D + 2) == 0) ? -INFINITY : 0.f;
    }
    return;
  }
  const int r_begin = split * rows_per_split;
  const int r_end = min(n_ctx, r_begin + rows_per_split);
  const int64_t base = row_off[b];
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const size_t row_stride = static_cast<size_t>(Hkv) * D;
  const uint16_t *knew = k_new + (static_cast<size_t>(b) * Hkv + kvh) * D;
  const uint16_t *vnew = v_new + (static_cast<size_t>(b) * Hkv + kvh) * D;
  uint16_t *kbase = kc + static_cast<size_t>(base) * row_stride + static_cast<size_t>(kvh) * D;
  uint16_t *vbase = vc + static_cast<size_t>(base) * row_stride + static_cast<size_t>(kvh) * D;

  if (split == 0 && threadIdx.x < DCH) {   // append the new token at row len
    const size_t dst = static_cast<size_t>(len) * row_stride + threadIdx.x * 8;
    *reinterpret_cast<u32x4 *>(kbase + dst) = reinterpret_cast<const u32x4 *>(knew)[threadIdx.x];
    *reinterpret_cast<u32x4 *>(vbase + dst) = reinterpret_cast<const u32x4 *>(vnew)[threadIdx.x];
  }

  // Q^T fragments (B operand): lane (col = lane%16, quarter = lane/16) holds
  // d = 32*ks + 8*quarter .. +7 of q-head kvh*G + col (zero for col >= G).
  const int col = lane & 15;
  const int quarter = lane >> 4;
  bf16x8 qf[KS];
  {
    const uint16_t *qrow = q + (static_cast<size_t>(b) * Hq + kvh * G + col) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (col < G) w = *reinterpret_cast<const u32x4 *>(qrow + 32 * ks + 8 * quarter);
      qf[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }
  const int dc = lane % DCH;   // value phase: d chunk
  const int rq = lane / DCH;   // value phase: row slot

  // Rows below len come from the cache; row len is the new token (its inputs, not the
  // cache, so no split depends on split 0's append).  Loads are unconditional: a row
  // past the split's end reads row r_begin instead and is masked out of the softmax,
  // so the compiler can wait for each group's loads alone (a conditional load would
  // make it wait for all of them).
  auto row_ptr = [&](int r, const uint16_t *cache_base, const uint16_t *fresh) {
    const int rr = r < r_end ? r : r_begin;
    return rr < len ? cache_base + static_cast<size_t>(rr) * row_stride : fresh;
  };
  auto load_k = [&](int r0, u32x4 (&kr)[KS]) {
    const uint16_t *krow = row_ptr(r0 + (lane & 15), kbase, knew);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kr[ks] = *reinterpret_cast<const u32x4 *>(krow + 32 * ks + 8 * quarter);
  };
  auto load_v = [&](int r0, u32x4 (&vr)[VPL]) {
#pragma unroll
    for (int i = 0; i < VPL; ++i) {
      const uint16_t *vrow = row_ptr(r0 + rq + i * ROWQ, vbase, vnew);
      vr[i] = *reinterpret_cast<const u32x4 *>(vrow + 8 * dc);
    }
  };
  // masked full-cache mode: the role bytes of this lane's four score rows r0 + 4*quarter + i
  auto load_roles = [&](int r0) {
    uint32_t roles = 0;
    if (row_role != nullptr) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = r0 + 4 * quarter + i;
        // rows at or past len are the new token (role CURRENT); the clamped index keeps
        // the load inside the request's rows
        const uint32_t rb = row_role[base + max(0, min(r, len - 1))];
        roles |= (r >= len ? static_cast<uint32_t>(kCurrent) : rb) << (8 * i);
      }
    }
    return roles;
  };

  float acc[G][8];
#pragma unroll
  for (int hh = 0; hh < G; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[hh][e] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;

  // A round covers kRoundRows rows: wave w takes 16-row groups j*4 + w, j < kGroups.  All
  // of a round's loads are issued before any of its groups is processed, so a wave keeps
  // kGroups x (K + V) rows in flight instead of waiting one memory round trip per group.
  for (int rb = r_begin; rb < r_end; rb += kRoundRows) {
    u32x4 kr[kGroups][KS], vr[kGroups][VPL];
    uint32_t roles[kGroups];
#pragma unroll
    for (int j = 0; j < kGroups; ++j) {
      const int r0 = rb + (j * kDecWaves + wave) * kDecRowsPerGroup;
      load_k(r0, kr[j]);
      load_v(r0, vr[j]);
      roles[j] = load_roles(r0);
    }
#pragma unroll
    for (int j = 0; j < kGroups; ++j) {
      const int r0 = rb + (j * kDecWaves + wave) * kDecRowsPerGroup;
      if (r0 >= r_end) break;   // uniform across the wave
      f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[j][ks]), qf[ks], sacc, 0, 0, 0);
      // lane (col, quarter) holds rows r0 + 4*quarter + i, i = 0..3, of head col
      float x[4];
      float mloc = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = r0 + 4 * quarter + i;
        const bool vis = r < r_end && ((roles[j] >> (8 * i)) & 0xFF) != kText;
        x[i] = vis ? sacc[i] * scale_log2 : -INFINITY;
        mloc = fmaxf(mloc, x[i]);
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run, mloc);
      const float corr = (m_new == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      float psum = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = (m_new == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(x[i] - m_new);
        psum += p;
        if (col < 8) p_lds[wave][4 * quarter + i][col] = p;
      }
      m_run = m_new;
      l_run = l_run * corr + psum;
      if (quarter == 0 && col < 8) corr_lds[wave][col] = corr;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

#pragma unroll
      for (int hh = 0; hh < G; ++hh) {
        const float c = corr_lds[wave][hh];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[hh][e] *= c;
      }
#pragma unroll
      for (int i = 0; i < VPL; ++i) {
        const int rr = rq + i * ROWQ;
        float vv[8];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          vv[2 * w] = bf16_lo(vr[j][i][w]);
          vv[2 * w + 1] = bf16_hi(vr[j][i][w]);
        }
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
          const float p = p_lds[wave][rr][hh];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[hh][e] = fmaf(p, vv[e], acc[hh][e]);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }

  // ---- merge row slots inside the wave, then the four waves through LDS ----
#pragma unroll
  for (int hh = 0; hh < G; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float a = acc[hh][e];
#pragma unroll
      for (int o = DCH; o < kWave; o <<= 1) a += __shfl_xor(a, o);
      acc[hh][e] = a;
    }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (lane < DCH) {
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc_lds[wave][hh][8 * dc + e] = acc[hh][e];
  }
  if (quarter == 0 && col < 8) {
    m_lds[wave][col] = m_run;
    l_lds[wave][col] = l_run;
  }
  __syncthreads();

  const int pair = b * Hkv + kvh;
  float *orow = out + (static_cast<size_t>(b) * Hq + kvh * G) * D;
  if (nsp == 1) {
    for (int idx = threadIdx.x; idx < G * D; idx += kDecThreads) {
      const int hh = idx / D, dd = idx % D;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, m_lds[w][hh]);
      float L = 0.f, A = 0.f;
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) {
        const float sc = (m_lds[w][hh] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_lds[w][hh] - M);
        L += sc * l_lds[w][hh];
        A += sc * acc_lds[w][hh][dd];
      }
      orow[idx] = A / L;
    }
    return;
  }
  float *rec = ws.part + (static_cast<size_t>(pair) * nsplit_max + split) * REC;
  for (int idx = threadIdx.x; idx < REC; idx += kDecThreads) {
    const int hh = idx / (D + 2), f = idx % (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, m_lds[w][hh]);
    float val = M;
    if (f > 0) {
      val = 0.f;
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) {
        const float sc = (m_lds[w][hh] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_lds[w][hh] - M);
        val += sc * (f == 1 ? l_lds[w][hh] : acc_lds[w][hh][f - 2]);
      }
    }
    rec[idx] = val;
  }
}

// Merge the split partials of one (kv-head, request); kv-head 0 advances the length.
// Every thread owns output elements (q-head, d) and loads, for a batch of up to
// eight splits at once, the split's max, sum and accumulator of its element, so a
// batch costs one memory round trip; batches are merged online.
template <int D, int G>
__global__ __launch_bounds__(kDecThreads) void decode_combine_kernel(int32_t *__restrict__ cache_len,
                                                                     float *__restrict__ out, DecodeWs ws, int Hkv,
                                                                     int nsplit_max) {
  constexpr int REC = G * (D + 2);
  constexpr int BATCH = 8;
  const int kvh = blockIdx.x;
  const int b = blockIdx.y;
  const int pair = b * Hkv + kvh;
  const float *recs = ws.part + static_cast<size_t>(pair) * nsplit_max * REC;
  // every record of the launch is valid (unused splits wrote empty ones), so the split
  // count and the records are fetched together
  const int nsp = ws.nsplit[b];
  float *orow = out + (static_cast<size_t>(b) * Hkv * G + kvh * G) * D;
  for (int idx = threadIdx.x; idx < G * D; idx += kDecThreads) {
    const int hh = idx / D, dd = idx % D;
    float M = -INFINITY, L = 0.f, A = 0.f;
    for (int sp0 = 0; sp0 < nsplit_max; sp0 += BATCH) {
      float m[BATCH], l[BATCH], a[BATCH];
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const int sp = min(sp0 + u, nsplit_max - 1);   // a repeated record is weighted 0 below
        const float *r = recs + static_cast<size_t>(sp) * REC + hh * (D + 2);
        m[u] = r[0];
        l[u] = r[1];
        a[u] = r[2 + dd];
      }
      float Mb = M;
#pragma unroll
      for (int u = 0; u < BATCH; ++u)
        if (sp0 + u < nsplit_max) Mb = fmaxf(Mb, m[u]);
      if (Mb == -INFINITY) continue;
      const float c = (M == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(M - Mb);
      L *= c;
      A *= c;
#pragma unroll
      for (int u = 0; u < BATCH; ++u) {
        const float w = (sp0 + u < nsplit_max && m[u] != -INFINITY) ? __builtin_amdgcn_exp2f(m[u] - Mb) : 0.f;
        L = fmaf(w, l[u], L);
        A = fmaf(w, a[u], A);
      }
      M = Mb;
    }
    if (nsp > 1) orow[idx] = A / L;   // nsp == 1: the split kernel wrote the output itself
  }
  // nsp == 0: the request could not append this step and keeps its length
  if (nsp > 0 && kvh == 0 && threadIdx.x == 0) cache_len[b] += 1;   // nothing else reads it here
}

int decode_num_splits(int max_ctx, int rows_per_split) { return (max_ctx + rows_per_split - 1) / rows_per_split; }

size_t decode_ws_layout(int batch, int Hkv, int G, int D, int nsplit, DecodeWs *ws, char *base) {
  const size_t nbytes = (static_cast<size_t>(batch) * sizeof(int32_t) + 255) / 256 * 256;
  const size_t pbytes = static_cast<size_t>(batch) * Hkv * nsplit * G * (D + 2) * sizeof(float);
  if (ws) {
    ws->nsplit = reinterpret_cast<int32_t *>(base);
    ws->part = reinterpret_cast<float *>(base + nbytes);
  }
  return nbytes + pbytes;
}

template <int D, int G>
static void launch_decode_dg(dim3 grid, int batch, int Hkv, int max_ctx, int rows_per_split, int nsplit,
                             uint16_t *kc, uint16_t *vc, const int64_t *row_off, const int32_t *row_cap,
                             int32_t *cache_len, const uint8_t *row_role, const uint16_t *q, const uint16_t *k_new,
                             const uint16_t *v_new, float scale_log2, float *out, DecodeWs ws, int32_t *status,
                             hipStream_t stream) {
  decode_kernel<D, G><<<grid, dim3(kDecThreads), 0, stream>>>(kc, vc, row_off, row_cap, cache_len, row_role, q, k_new,
                                                              v_new, out, ws, status, Hkv, rows_per_split, nsplit,
                                                              max_ctx, scale_log2);
  decode_combine_kernel<D, G><<<dim3(Hkv, batch), dim3(kDecThreads), 0, stream>>>(cache_len, out, ws, Hkv, nsplit);
}

hipError_t launch_decode(int batch, int Hq, int Hkv, int D, int max_ctx, int rows_per_split, uint16_t *kc,
                         uint16_t *vc, const int64_t *row_off, const int32_t *row_cap, int32_t *cache_len,
                         const uint8_t *row_role, const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                         float scale_log2, float *out, void *ws_base, int32_t *status, hipStream_t stream) {
  const int G = Hq / Hkv;
  const int nsplit = decode_num_splits(max_ctx, rows_per_split);
  DecodeWs ws;
  decode_ws_layout(batch, Hkv, G, D, nsplit, &ws, static_cast<char *>(ws_base));
  dim3 grid(nsplit, Hkv, batch);
#define DEC(DD, GG)                                                                                               \
  case GG:                                                                                                        \
    launch_decode_dg<DD, GG>(grid, batch, Hkv, max_ctx, rows_per_split, nsplit, kc, vc, row_off, row_cap,        \
                             cache_len, row_role, q, k_new, v_new, scale_log2, out, ws, status, stream);          \
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
