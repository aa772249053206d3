// Reconstruction targets of the information bottleneck (Sec. 4): the body of
// each history segment is cut into one sub-interval per Nexus token of the
// segment (interval j of a b-token body for K Nexus tokens is
// [floor(j b / K), max(floor((j + 1) b / K), floor(j b / K) + 1)): near-equal
// pieces, or single tokens when b < K), and the j-th Nexus token's target is
//     target = sum over x of alpha(x) h(x),   alpha = softmax over x of cos(h(N_j), h(x)),
// reported with cos(h(N_j), target) and the weights' entropy over log |interval|
// (1 for a one-token interval).  A zero vector has cosine 0 with anything.
//
// The segment structure comes from the prefill planner's run table; one small
// kernel numbers the Nexus tokens of the batch (position order) and lists, per
// Nexus token, its position and its interval.  The pooling is HBM-bound:
// one workgroup per Nexus token (persistent grid) reads the Nexus row and its
// interval's rows once, four or six rows per step (fewer for wide rows), the first step
// requested together with the Nexus row: each thread holds 8-element chunks
// of the rows, the dot products and squared norms are reduced across the
// workgroup in a fixed order (reproducible), and since a cosine lies in
// [-1, 1] the softmax needs no running maximum: the weighted sum, the
// normaliser Z and sum(e^c c) (for the entropy, H = ln Z - sum(e^c c) / Z)
// accumulate in one pass.
#include "common.h"
#include "scan.h"

#include <type_traits>

namespace sonic {

constexpr int kReconThreads = 256;
constexpr int kReconWaves = kReconThreads / kWave;
constexpr int kReconMaxRows = 6;   // body rows per step (fewer for wide rows)

hipError_t launch_plan_runs(int batch, int total_tokens, const int32_t *cu, const uint8_t *role, const int32_t *turn,
                            PrefillWs ws, int32_t *status, hipStream_t stream);

// Per request: one item per Nexus token, (position, first interval row, end row), rows
// as batch positions.  The workgroup first sums the Nexus counts of the requests
// before its own (its first output row) and of the whole batch; workgroup 0 stores
// the total in ctrl[0] (0 when it exceeds the caller's rows, which it reports), and
// nothing is listed then.  The run table is read 256 runs at a time into LDS; then
// the workgroup walks those runs and its threads fill a Nexus run's items in parallel.
__global__ __launch_bounds__(256) void recon_items_kernel(int batch, int max_rows, const int32_t *__restrict__ cu,
                                                          const uint8_t *__restrict__ role, PrefillWs ws,
                                                          int4 *__restrict__ items, int32_t *status) {
  __shared__ int s_x[256 + 2];    // starts of runs c0 - 1 .. c0 + 256 (the last: the next run or L)
  __shared__ int s_y[256];        // prefix rows (system + Nexus) before each run
  __shared__ int s_nx[256];       // run is a Nexus run
  __shared__ int s_red[2][256 / kWave];
  __shared__ int s_ok;
  const bool clear = block_status_clear(status, &s_ok);
  const int b = blockIdx.x;
  int before = 0, total = 0;
  for (int i = threadIdx.x; i < batch; i += 256) {
    const int n = ws.req[i].nexus_total;
    total += n;
    before += i < b ? n : 0;
  }
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) {
    total += __shfl_xor(total, o);
    before += __shfl_xor(before, o);
  }
  if (threadIdx.x % kWave == 0) {
    s_red[0][threadIdx.x / kWave] = total;
    s_red[1][threadIdx.x / kWave] = before;
  }
  __syncthreads();
  total = 0;
  before = 0;
#pragma unroll
  for (int w = 0; w < 256 / kWave; ++w) {
    total += s_red[0][w];
    before += s_red[1][w];
  }
  const bool fits = total <= max_rows;
  if (b == 0 && threadIdx.x == 0) {
    if (clear && !fits) raise_status(status, SONIC_ERR_CAPACITY);
    ws.ctrl[0] = (clear && fits) ? total : 0;
  }
  if (!clear || !fits) return;
  const int s0 = cu[b];
  const int L = cu[b + 1] - s0;
  const ReqInfo ri = ws.req[b];
  const int base = before - ri.system;
  for (int c0 = 0; c0 < ri.nruns; c0 += 256) {
    const int cnt = min(256, ri.nruns - c0);
    if (threadIdx.x < cnt) {
      const int2 run = ws.runs[s0 + c0 + threadIdx.x];
      s_x[threadIdx.x + 1] = run.x;
      s_y[threadIdx.x] = run.y;
      s_nx[threadIdx.x] = role[s0 + run.x] == kNexus;
    }
    if (threadIdx.x == 0) s_x[0] = c0 > 0 ? ws.runs[s0 + c0 - 1].x : 0;
    if (threadIdx.x == 1) s_x[cnt + 1] = c0 + cnt < ri.nruns ? ws.runs[s0 + c0 + cnt].x : L;
    __syncthreads();
    for (int i = 0; i < cnt; ++i) {
      if (!s_nx[i]) continue;                 // a Nexus run follows its body run (the grammar)
      const int body = s_x[i], start = s_x[i + 1], end = s_x[i + 2];
      const int blen = start - body, K = end - start;
      const int first = base + s_y[i];        // Nexus tokens of the request before this run
      for (int j = threadIdx.x; j < K; j += 256) {
        const int s = static_cast<int>(static_cast<int64_t>(j) * blen / K);
        const int e = max(static_cast<int>(static_cast<int64_t>(j + 1) * blen / K), s + 1);
        items[first + j] = make_int4(s0 + start + j, s0 + body + s, s0 + body + e, 0);
      }
    }
    __syncthreads();
  }
}

// Sum R values over the workgroup, the same order every time; two LDS buffers in turn,
// so one barrier per call suffices.
template <int R>
__device__ __forceinline__ void block_sum(float (&v)[R], float (*red)[kReconWaves][2 * kReconMaxRows + 1], int &par) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
#pragma unroll
  for (int k = 0; k < R; ++k) {
    v[k] = pair16_add(pair32_add(v[k]));
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) v[k] += __shfl_xor(v[k], o);
  }
  if (lane == 0)
#pragma unroll
    for (int k = 0; k < R; ++k) red[par][wave][k] = v[k];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < R; ++k) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kReconWaves; ++w) s += red[par][w][k];
    v[k] = s;
  }
  par ^= 1;
}

__device__ __forceinline__ void widen8(const u32x4 &w, float (&f)[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = bf16_lo(w[i]);
    f[2 * i + 1] = bf16_hi(w[i]);
  }
}

// CPT: 8-element chunks per thread (hidden size up to CPT * 8 * 256); RW: rows per step
template <int CPT, int RW>
__global__ __launch_bounds__(kReconThreads) void recon_kernel(const uint16_t *__restrict__ h, int Dm,
                                                              const int4 *__restrict__ items, PrefillWs ws,
                                                              float *__restrict__ target,
                                                              float *__restrict__ cos_out,
                                                              float *__restrict__ ratio_out) {
  static_assert(RW <= kReconMaxRows, "reduction buffer size");
  __shared__ float red[2][kReconWaves][2 * kReconMaxRows + 1];
  const int n_items = ws.ctrl[0];
  const int nch = Dm / 8;
  int par = 0;
  for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
    const int4 it = items[item];
    const int s = it.y, e = it.z;
    float hn[CPT][8];
    u32x4 hraw[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + i * kReconThreads;
      hraw[i] = u32x4{0u, 0u, 0u, 0u};
      if (c < nch) hraw[i] = *reinterpret_cast<const u32x4 *>(h + static_cast<size_t>(it.x) * Dm + 8 * c);
    }
    float acc[CPT][8];
#pragma unroll
    for (int i = 0; i < CPT; ++i)
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[i][k] = 0.f;
    float Z = 0.f, S1 = 0.f, nn = 0.f;
    // One step: RW rows from x0.  The first step (an interval has at least one row)
    // requests its rows before the Nexus row is used, so both arrive in one round
    // trip, and it also reduces |h(N)|^2.
    auto step = [&](int x0, auto first_tag) {
      constexpr bool kFirst = decltype(first_tag)::value;
      u32x4 raw[RW][CPT];
      float dq[kFirst ? 2 * RW + 1 : 2 * RW];   // dot with h(N), then squared norm, per row; |h(N)|^2 last
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        const bool ok = x0 + r < e;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
          const int c = threadIdx.x + i * kReconThreads;
          raw[r][i] = u32x4{0u, 0u, 0u, 0u};
          if (ok && c < nch) raw[r][i] = *reinterpret_cast<const u32x4 *>(h + static_cast<size_t>(x0 + r) * Dm + 8 * c);
        }
      }
      if constexpr (kFirst) {
        dq[2 * RW] = 0.f;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
          widen8(hraw[i], hn[i]);
#pragma unroll
          for (int k = 0; k < 8; ++k) dq[2 * RW] = fmaf(hn[i][k], hn[i][k], dq[2 * RW]);
        }
      }
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        dq[r] = 0.f;
        dq[RW + r] = 0.f;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
          float f[8];
          widen8(raw[r][i], f);
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            dq[r] = fmaf(f[k], hn[i][k], dq[r]);
            dq[RW + r] = fmaf(f[k], f[k], dq[RW + r]);
          }
        }
      }
      block_sum(dq, red, par);
      if constexpr (kFirst) nn = dq[2 * RW];
      // widen the rows again below rather than keep their fp32 copies live
#pragma unroll
      for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int i = 0; i < CPT; ++i) asm volatile("" : "+v"(raw[r][i]));
#pragma unroll
      for (int r = 0; r < RW; ++r) {
        if (x0 + r < e) {
          const float den = nn * dq[RW + r];
          const float c = den > 0.f ? dq[r] / sqrtf(den) : 0.f;
          const float wgt = expf(c);
          Z += wgt;
          S1 = fmaf(wgt, c, S1);
#pragma unroll
          for (int i = 0; i < CPT; ++i) {
            float f[8];
            widen8(raw[r][i], f);
#pragma unroll
            for (int k = 0; k < 8; ++k) acc[i][k] = fmaf(wgt, f[k], acc[i][k]);
          }
        }
      }
    };
    step(s, std::true_type{});
    for (int x0 = s + RW; x0 < e; x0 += RW) step(x0, std::false_type{});
    const float invz = 1.f / Z;
    float tt[2] = {0.f, 0.f};   // target . h(N), |target|^2
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + i * kReconThreads;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        acc[i][k] *= invz;
        tt[0] = fmaf(acc[i][k], hn[i][k], tt[0]);
        tt[1] = fmaf(acc[i][k], acc[i][k], tt[1]);
      }
      if (c < nch) {
        float *dst = target + static_cast<size_t>(item) * Dm + 8 * c;
        *reinterpret_cast<f32x4 *>(dst) = f32x4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]};
        *reinterpret_cast<f32x4 *>(dst + 4) = f32x4{acc[i][4], acc[i][5], acc[i][6], acc[i][7]};
      }
    }
    block_sum<2>(tt, red, par);
    if (threadIdx.x == 0) {
      const float den = nn * tt[1];
      cos_out[item] = den > 0.f ? tt[0] / sqrtf(den) : 0.f;
      const int n = e - s;
      ratio_out[item] = n > 1 ? (logf(Z) - S1 * invz) / logf(static_cast<float>(n)) : 1.f;
    }
  }
}

hipError_t launch_recon(int batch, int total_tokens, int Dm, int max_rows, int num_cus, const int32_t *cu,
                        const uint8_t *role, const int32_t *turn, const uint16_t *h, PrefillWs ws,
                        int4 *items, float *target, float *cos_out, float *ratio_out,
                        int32_t *status, hipStream_t stream) {
  hipError_t e = launch_plan_runs(batch, total_tokens, cu, role, turn, ws, status, stream);
  if (e != hipSuccess) return e;
  recon_items_kernel<<<dim3(batch), dim3(256), 0, stream>>>(batch, max_rows, cu, role, ws, items, status);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int chunks = (Dm / 8 + kReconThreads - 1) / kReconThreads;
  const dim3 grid(num_cus * 8), block(kReconThreads);
  if (chunks <= 1)
    recon_kernel<1, 4><<<grid, block, 0, stream>>>(h, Dm, items, ws, target, cos_out, ratio_out);
  else if (chunks <= 2)
    recon_kernel<2, 6><<<grid, block, 0, stream>>>(h, Dm, items, ws, target, cos_out, ratio_out);
  else if (chunks <= 4)
    recon_kernel<4, 2><<<grid, block, 0, stream>>>(h, Dm, items, ws, target, cos_out, ratio_out);
  else
    recon_kernel<8, 1><<<grid, block, 0, stream>>>(h, Dm, items, ws, target, cos_out, ratio_out);
  return hipGetLastError();
}

}  // namespace sonic
