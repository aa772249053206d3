// Key weights of the attention statistics: w(x), the attention key x receives
// from the current rows of its request, summed over the current rows and
// averaged over the q-heads (the importance score of the attention-guided
// distillation objective, Sec. 4).
//
// A current row sees the system prompt, every Nexus token and the current rows
// up to itself (Sec. 3.2; the bodies are removed, Eq.(4)), so only those "kept"
// keys get weight: the request's prefix copy (system, then Nexus, as the
// planner laid it out) followed by its current rows.  The pass is key-major
// and runs after the statistics variant of the prefill, which leaves each row's
// log2-domain softmax normaliser lse:
//   work item = (request, block of 64 kept keys, kv-head), G waves, one per
//   q-head of the kv-head; each wave walks the current rows 32 at a time,
//   computes S^T = K . Q^T with v_mfma_f32_32x32x16_bf16, p = exp2(s - lse) on
//   the visible pairs, and adds p into per-lane key sums (a lane keeps the same
//   keys for every row block).  The sums are reduced over rows, then over the
//   waves in a fixed order, and stored per kv-head; a last kernel adds the
//   kv-heads in order.  No atomics on the sums, so the result is reproducible.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kStatThreads = 1024;
constexpr int kWBlock = 64;   // kept keys per work item

// One workgroup: the current-row count of every request and the list of work
// blocks (request, first kept key / 64).
__global__ __launch_bounds__(kStatThreads) void stats_plan_kernel(int batch, const int32_t *__restrict__ cu,
                                                                  const uint8_t *__restrict__ role, PrefillWs ws,
                                                                  const int32_t *status) {
  __shared__ int lds[kStatThreads / kWave + 1];
  __shared__ int s_ok;
  const bool ok = block_status_clear(status, &s_ok);
  int carry = 0;
  for (int base = 0; base < batch; base += kStatThreads) {
    const int b = base + threadIdx.x;
    int nblk = 0, c = 0, s0 = 0;
    if (ok && b < batch) {
      s0 = cu[b];
      const int L = cu[b + 1] - s0;
      const ReqInfo ri = ws.req[b];
      if (ri.nruns > 0) {   // the current query is the request's last run, if any
        const int start = ws.runs[s0 + ri.nruns - 1].x;
        if (role[s0 + start] == kCurrent) c = L - start;
      }
      ws.ncur[b] = c;
      nblk = (ri.system + ri.nexus_total + c + kWBlock - 1) / kWBlock;
    }
    int tot;
    const int off = block_int_scan<kStatThreads>(nblk, &tot, lds);
    for (int j = 0; j < nblk; ++j) ws.kblocks[carry + off + j] = make_int2(b, j);
    carry += tot;
  }
  if (threadIdx.x == 0) ws.ctrl[1] = carry;
}

template <int D> __device__ __forceinline__ int swz_w(int m) { return m & (D / 8 - 1); }

template <int D, int G>
__global__ __launch_bounds__(G * kWave) void key_weight_kernel(const int32_t *__restrict__ cu,
                                                               const uint16_t *__restrict__ q,
                                                               const uint16_t *__restrict__ k, PrefillWs ws,
                                                               int Hkv, int T, float scale_log2) {
  constexpr int DC = D / 8;    // 16-byte chunks per row
  constexpr int DS = D / 16;   // d steps of the S product
  __shared__ __align__(16) uint16_t k_lds[kWBlock * D];   // [64 keys][D], chunk-swizzled
  __shared__ float red[G][kWBlock];
  const int Hq = Hkv * G;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  const int n = lane & 31;     // query row of the block (column of S^T)
  const int g = lane >> 5;
  const int nitems = ws.ctrl[1] * Hkv;
  for (int item = blockIdx.x; item < nitems; item += gridDim.x) {
    const int2 kbk = ws.kblocks[item / Hkv];
    const int kvh = item % Hkv;
    const int b = kbk.x;
    const int s0 = cu[b];
    const int L = cu[b + 1] - s0;
    const ReqInfo ri = ws.req[b];
    const int npre = ri.system + ri.nexus_total;   // kept keys [0, npre) are the prefix copy
    const int C = ws.ncur[b];
    const int nkeep = npre + C;
    const int j0 = kbk.y * kWBlock;
    // request-local position of kept key j
    auto key_pos = [&](int j) { return j < npre ? ws.prefix_pos[s0 + j] : L - C + (j - npre); };

    // stage the 64 keys of this kv-head (keys past the end read as zero)
    for (int u = threadIdx.x; u < kWBlock * DC; u += G * kWave) {
      const int m = u / DC, c = u % DC;
      const int j = j0 + m;
      u32x4 w = {0u, 0u, 0u, 0u};
      if (j < nkeep) {
        const uint16_t *src = j < npre ? ws.k_pre + (static_cast<size_t>(s0 + j) * Hkv + kvh) * D
                                       : k + (static_cast<size_t>(s0 + L - C + (j - npre)) * Hkv + kvh) * D;
        w = reinterpret_cast<const u32x4 *>(src)[c];
      }
      *reinterpret_cast<u32x4 *>(&k_lds[(m * DC + (c ^ swz_w<D>(m))) * 8]) = w;
    }
    __syncthreads();

    const int h = kvh * G + wave;
    f32x16 wacc[2] = {f32x16{}, f32x16{}};
    for (int r0 = 0; r0 < C; r0 += 32) {
      const int r = r0 + n;   // current-query row of this lane's column
      const bool valid = r < C;
      const size_t qidx = static_cast<size_t>(s0 + L - C + (valid ? r : 0)) * Hq + h;
      bf16x8 qf[DS];
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (valid) w = *reinterpret_cast<const u32x4 *>(q + qidx * D + 16 * ds + 8 * g);
        qf[ds] = __builtin_bit_cast(bf16x8, w);
      }
      const float lse = valid ? ws.lse[qidx] : INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16 s = f32x16{};
        const int m = kb * 32 + n;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
          const bf16x8 a = *reinterpret_cast<const bf16x8 *>(&k_lds[(m * DC + ((2 * ds + g) ^ swz_w<D>(m))) * 8]);
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ds], s, 0, 0, 0);
        }
        // element e holds key 8 * (e / 4) + 4 * g + e % 4 of the 32-key block, row r
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int j = j0 + kb * 32 + 8 * (e >> 2) + 4 * g + (e & 3);
          const bool vis = valid && j < nkeep && (j < npre || j - npre <= r);
          wacc[kb][e] += vis ? __builtin_amdgcn_exp2f(fmaf(s[e], scale_log2, -lse)) : 0.f;
        }
      }
    }
    // Sum over the 32 rows (lanes with the same half g), then over the waves.  The 32
    // values E = 16 kb + e of a lane are summed over its 32 lanes by halving: at the
    // stage of lane bit m, a lane keeps the half of its values whose E bit matches its
    // own bit m and adds the partner's copy of that half, so after five stages lane n
    // holds the sum for E = n (31 exchanges instead of 160).  The first stage (bit 4)
    // is one v_permlane16_swap per pair (E, E + 16): it leaves every lane its pair's
    // kept value and the partner's in two registers.
    float v16[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(wacc[0][e]), __float_as_uint(wacc[1][e]),
                                                      false, false);
      v16[e] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    }
    auto halve = [&](auto &src, auto &dst, int half, int m) {
      const bool hi = (n & m) != 0;
#pragma unroll
      for (int i = 0; i < half; ++i) {
        const float keep = hi ? src[i + half] : src[i];
        const float send = hi ? src[i] : src[i + half];
        dst[i] = keep + __shfl_xor(send, m);
      }
    };
    float v8[8], v4[4], v2[2], v1[1];
    halve(v16, v8, 8, 8);
    halve(v8, v4, 4, 4);
    halve(v4, v2, 2, 2);
    halve(v2, v1, 1, 1);
    {
      const int E = n, kb = E >> 4, e = E & 15;
      red[wave][kb * 32 + 8 * (e >> 2) + 4 * g + (e & 3)] = v1[0];
    }
    __syncthreads();
    if (threadIdx.x < kWBlock) {
      const int j = j0 + threadIdx.x;
      if (j < nkeep) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < G; ++w) v += red[w][threadIdx.x];
        ws.wpart[static_cast<size_t>(kvh) * T + s0 + key_pos(j)] = v;
      }
    }
    __syncthreads();   // k_lds and red are reused by the next item
  }
}

// w[x] = (sum over kv-heads of the partials) / Hq for kept keys, 0 for body keys.
__global__ __launch_bounds__(256) void key_weight_sum_kernel(const uint8_t *__restrict__ role, PrefillWs ws,
                                                             int Hkv, int Hq, int T, float *__restrict__ w,
                                                             const int32_t *status) {
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  for (int x = blockIdx.x * 256 + threadIdx.x; x < T; x += gridDim.x * 256) {
    float v = 0.f;
    if (role[x] != kText)
      for (int kvh = 0; kvh < Hkv; ++kvh) v += ws.wpart[static_cast<size_t>(kvh) * T + x];
    w[x] = v / static_cast<float>(Hq);
  }
}

template <int D, int G>
static void launch_kw_dg(int grid, const int32_t *cu, const uint16_t *q, const uint16_t *k, PrefillWs ws, int Hkv,
                         int T, float scale_log2, hipStream_t stream) {
  key_weight_kernel<D, G><<<dim3(grid), dim3(G * kWave), 0, stream>>>(cu, q, k, ws, Hkv, T, scale_log2);
}

hipError_t launch_key_weight(int batch, int T, int Hq, int Hkv, int D, int num_cus, const int32_t *cu,
                             const uint8_t *role, const uint16_t *q, const uint16_t *k, PrefillWs ws,
                             float scale_log2, float *w, int32_t *status, hipStream_t stream) {
  stats_plan_kernel<<<dim3(1), dim3(kStatThreads), 0, stream>>>(batch, cu, role, ws, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int G = Hq / Hkv;
  const int grid = num_cus * 4;
#define KW(DD, GG)                                                          \
  case GG:                                                                  \
    launch_kw_dg<DD, GG>(grid, cu, q, k, ws, Hkv, T, scale_log2, stream); \
    break;
#define KW_ALL_G(DD)                      \
  switch (G) {                            \
    KW(DD, 1)                             \
    KW(DD, 2)                             \
    KW(DD, 3)                             \
    KW(DD, 4)                             \
    KW(DD, 5)                             \
    KW(DD, 6)                             \
    KW(DD, 7)                             \
    KW(DD, 8)                             \
    default: return hipErrorInvalidValue; \
  }
  if (D == 64) {
    KW_ALL_G(64)
  } else if (D == 128) {
    KW_ALL_G(128)
  } else {
    return hipErrorInvalidValue;
  }
#undef KW_ALL_G
#undef KW
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  long blocks = (static_cast<long>(T) + 255) / 256;
  if (blocks > 4L * num_cus) blocks = 4L * num_cus;
  if (blocks < 1) blocks = 1;
  key_weight_sum_kernel<<<dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream>>>(role, ws, Hkv, Hq, T, w,
                                                                                        status);
  return hipGetLastError();
}

}  // namespace sonic
