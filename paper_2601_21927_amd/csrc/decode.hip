// Decode over the retained context {I_sys, N, Q_n} (App. C, Eq.(15)).
//
// decode_split_kernel: grid (split, kv-head, request), 4 waves.  A split owns
// rows [split*R, split*R + R) of the request's context rows 0..len (row len is
// the token being generated: it is read from k_new/v_new, and split 0 of each
// kv-head also writes it into the cache).  Each wave takes 16 rows at a time:
//   scores    S^T (16 rows x 16 cols) = K . Q^T with v_mfma_f32_16x16x32_bf16;
//             column c < G is q-head kvh*G + c, the other columns are zero;
//   softmax   per q-head, online, fp32, exp2 with log2(e) folded in;
//   values    P . V on the vector ALUs in fp32: lane (d chunk, row quarter)
//             accumulates 8 d-values of every q-head of the group.
// The four waves' partial (max, sum, acc) are merged through LDS and one
// partial per (request, q-head, split) goes to the workspace.
//
// decode_combine_kernel: one workgroup per request merges the splits with the
// log-sum-exp rule, writes out[b] and then increments cache_len[b].
#include "common.h"

namespace sonic {

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kDecRowsPerGroup = 16;

template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_split_kernel(
    uint16_t *__restrict__ kc, uint16_t *__restrict__ vc, const int64_t *__restrict__ row_off,
    const int32_t *__restrict__ row_cap, const int32_t *__restrict__ cache_len, const uint8_t *__restrict__ row_role,
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new,
    float *__restrict__ ws, int32_t *status, int Hq, int Hkv, int rows_per_split, int nsplit_max, int max_ctx,
    float scale_log2) {
  constexpr int KS = D / 32;      // k steps of the 16x16x32 product
  constexpr int DCH = D / 8;      // 8-value d chunks (16 lanes cover D = 128; 8 cover D = 64)
  constexpr int ROWQ = kWave / DCH;   // rows handled per value-load instruction
  __shared__ float p_lds[kDecWaves][kDecRowsPerGroup][8];
  __shared__ float corr_lds[kDecWaves][8];
  __shared__ float m_lds[kDecWaves][8];
  __shared__ float l_lds[kDecWaves][8];
  __shared__ float acc_lds[kDecWaves][8][D];
  __shared__ int s_ok;

  if (!block_status_clear(status, &s_ok)) return;
  const int split = blockIdx.x;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int G = Hq / Hkv;
  const int len = cache_len[b];
  const int n_ctx = len + 1;
  if (n_ctx > row_cap[b] || n_ctx > max_ctx) {
    if (split == 0 && kvh == 0 && threadIdx.x == 0) raise_status(status, SONIC_ERR_CAPACITY);
    return;
  }
  const int r_begin = split * rows_per_split;
  if (r_begin >= n_ctx) return;
  const int r_end = min(n_ctx, r_begin + rows_per_split);
  const int64_t base = row_off[b];
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const size_t row_stride = static_cast<size_t>(Hkv) * D;   // elements per cache row
  const uint16_t *knew = k_new + (static_cast<size_t>(b) * Hkv + kvh) * D;
  const uint16_t *vnew = v_new + (static_cast<size_t>(b) * Hkv + kvh) * D;

  // split 0 appends the new token's k/v at row len of this kv-head
  if (split == 0 && threadIdx.x < DCH) {
    const size_t dst = (static_cast<size_t>(base + len)) * row_stride + static_cast<size_t>(kvh) * D + threadIdx.x * 8;
    *reinterpret_cast<u32x4 *>(kc + dst) = reinterpret_cast<const u32x4 *>(knew)[threadIdx.x];
    *reinterpret_cast<u32x4 *>(vc + dst) = reinterpret_cast<const u32x4 *>(vnew)[threadIdx.x];
  }

  // Q^T fragments (B operand of 16x16x32): lane (col = lane%16, quarter = lane/16) holds
  // d = 32*ks + 8*quarter .. +7 of q-head kvh*G + col (zero for col >= G).
  const int col = lane & 15;
  const int quarter = lane >> 4;
  bf16x8 qf[KS];
  {
    const bool ok = col < G;
    const uint16_t *qrow = q + (static_cast<size_t>(b) * Hq + kvh * G + col) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (ok) w = *reinterpret_cast<const u32x4 *>(qrow + 32 * ks + 8 * quarter);
      qf[ks] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // value-phase lane roles: d chunk dc (8 values), row slot rq within a 16-row group
  const int dc = lane % DCH;
  const int rq = lane / DCH;
  float acc[8][8];
#pragma unroll
  for (int hh = 0; hh < 8; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[hh][e] = 0.f;
  float m_run = -INFINITY;   // running max of head `col` (score lanes)
  float l_run = 0.f;         // this lane's share of the running sum of head `col`

  for (int r0 = r_begin + wave * kDecRowsPerGroup; r0 < r_end; r0 += kDecWaves * kDecRowsPerGroup) {
    // ---- scores: A operand lane (row = lane%16, quarter) holds d = 32*ks + 8*quarter .. +7 ----
    f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
    {
      const int r = r0 + (lane & 15);
      const uint16_t *krow = nullptr;
      if (r < len) krow = kc + static_cast<size_t>(base + r) * row_stride + static_cast<size_t>(kvh) * D;
      else if (r == len) krow = knew;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (krow) w = *reinterpret_cast<const u32x4 *>(krow + 32 * ks + 8 * quarter);
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w), qf[ks], sacc, 0, 0, 0);
      }
    }
    // lane (col, quarter) now holds rows r0 + 4*quarter + i, i = 0..3, of head col
    float x[4];
    float mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = r0 + 4 * quarter + i;
      bool vis = r < r_end;
      if (vis && row_role != nullptr && r < len) vis = row_role[base + r] != kText;
      x[i] = vis ? sacc[i] * scale_log2 : -INFINITY;
      mloc = fmaxf(mloc, x[i]);
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    // a group may be fully masked for this head: keep the old max then
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
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");

    // ---- values: lane (dc, rq) takes rows rq, rq + ROWQ, ... of the group ----
    float cr[8];
#pragma unroll
    for (int hh = 0; hh < 8; ++hh) cr[hh] = corr_lds[wave][hh];
#pragma unroll
    for (int hh = 0; hh < 8; ++hh)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[hh][e] *= cr[hh];
#pragma unroll
    for (int rr = rq; rr < kDecRowsPerGroup; rr += ROWQ) {
      const int r = r0 + rr;
      if (r >= r_end) break;
      const uint16_t *vrow = (r < len) ? vc + static_cast<size_t>(base + r) * row_stride + static_cast<size_t>(kvh) * D
                                       : vnew;
      const u32x4 w = *reinterpret_cast<const u32x4 *>(vrow + 8 * dc);
      float vv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        vv[2 * i] = bf16_lo(w[i]);
        vv[2 * i + 1] = bf16_hi(w[i]);
      }
#pragma unroll
      for (int hh = 0; hh < 8; ++hh) {
        if (hh < G) {
          const float p = p_lds[wave][rr][hh];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[hh][e] = fmaf(p, vv[e], acc[hh][e]);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  }

  // ---- merge row slots within the wave (lanes with equal dc), then waves through LDS ----
#pragma unroll
  for (int hh = 0; hh < 8; ++hh)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float a = acc[hh][e];
      for (int o = DCH; o < kWave; o <<= 1) a += __shfl_xor(a, o);
      acc[hh][e] = a;
    }
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  if (lane < DCH) {
#pragma unroll
    for (int hh = 0; hh < 8; ++hh)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc_lds[wave][hh][8 * dc + e] = acc[hh][e];
  }
  if (quarter == 0 && col < 8) {
    m_lds[wave][col] = m_run;
    l_lds[wave][col] = l_run;
  }
  __syncthreads();
  const int nsplit = nsplit_max;
  for (int idx = threadIdx.x; idx < G * (D + 2); idx += kDecThreads) {
    const int hh = idx / (D + 2);
    const int f = idx % (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, m_lds[w][hh]);
    float val = 0.f;
    if (f == 0) {
      val = M;
    } else {
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) {
        const float sc = (m_lds[w][hh] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_lds[w][hh] - M);
        val += sc * (f == 1 ? l_lds[w][hh] : acc_lds[w][hh][f - 2]);
      }
    }
    const int h = kvh * G + hh;
    ws[((static_cast<size_t>(b) * Hq + h) * nsplit + split) * (D + 2) + f] = val;
  }
}

template <int D>
__global__ __launch_bounds__(kDecThreads) void decode_combine_kernel(int32_t *__restrict__ cache_len,
                                                                     const float *__restrict__ ws,
                                                                     float *__restrict__ out, int32_t *status, int Hq,
                                                                     int rows_per_split, int nsplit_max) {
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int b = blockIdx.x;
  const int len = cache_len[b];
  const int nsp = (len + 1 + rows_per_split - 1) / rows_per_split;
  for (int idx = threadIdx.x; idx < Hq * D; idx += kDecThreads) {
    const int h = idx / D;
    const int d = idx % D;
    const float *part = ws + (static_cast<size_t>(b) * Hq + h) * nsplit_max * (D + 2);
    float M = -INFINITY;
    for (int sp = 0; sp < nsp; ++sp) M = fmaxf(M, part[sp * (D + 2)]);
    float L = 0.f, A = 0.f;
    for (int sp = 0; sp < nsp; ++sp) {
      const float ms = part[sp * (D + 2)];
      const float sc = (ms == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(ms - M);
      L += sc * part[sp * (D + 2) + 1];
      A += sc * part[sp * (D + 2) + 2 + d];
    }
    out[(static_cast<size_t>(b) * Hq + h) * D + d] = A / L;
  }
  __syncthreads();
  if (threadIdx.x == 0) cache_len[b] = len + 1;
}

template <int D>
static void launch_decode_d(dim3 grid, int batch, int Hq, int Hkv, int max_ctx, int rows_per_split, int nsplit,
                            uint16_t *kc, uint16_t *vc, const int64_t *row_off, const int32_t *row_cap,
                            int32_t *cache_len, const uint8_t *row_role, const uint16_t *q, const uint16_t *k_new,
                            const uint16_t *v_new, float scale_log2, float *out, float *ws, int32_t *status,
                            hipStream_t stream) {
  decode_split_kernel<D><<<grid, dim3(kDecThreads), 0, stream>>>(kc, vc, row_off, row_cap, cache_len, row_role, q,
                                                                 k_new, v_new, ws, status, Hq, Hkv, rows_per_split,
                                                                 nsplit, max_ctx, scale_log2);
  decode_combine_kernel<D><<<dim3(batch), dim3(kDecThreads), 0, stream>>>(cache_len, ws, out, status, Hq,
                                                                          rows_per_split, nsplit);
}

int decode_num_splits(int max_ctx, int rows_per_split) { return (max_ctx + rows_per_split - 1) / rows_per_split; }

hipError_t launch_decode(int batch, int Hq, int Hkv, int D, int max_ctx, int rows_per_split, uint16_t *kc,
                         uint16_t *vc, const int64_t *row_off, const int32_t *row_cap, int32_t *cache_len,
                         const uint8_t *row_role, const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                         float scale_log2, float *out, float *ws, int32_t *status, hipStream_t stream) {
  const int nsplit = decode_num_splits(max_ctx, rows_per_split);
  dim3 grid(nsplit, Hkv, batch);
  if (D == 64)
    launch_decode_d<64>(grid, batch, Hq, Hkv, max_ctx, rows_per_split, nsplit, kc, vc, row_off, row_cap, cache_len,
                        row_role, q, k_new, v_new, scale_log2, out, ws, status, stream);
  else if (D == 128)
    launch_decode_d<128>(grid, batch, Hq, Hkv, max_ctx, rows_per_split, nsplit, kc, vc, row_off, row_cap, cache_len,
                         row_role, q, k_new, v_new, scale_log2, out, ws, status, stream);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sonic
