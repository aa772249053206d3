// Role-routed linear layer (Sec. 3.1: Nexus tokens get their own projection
// matrices W_Q^N, W_K^N, W_V^N, W_O^N and their own MLP branches; every other
// token keeps the model's standard ones):
//     y[t] = W_N x[t]   for Nexus rows,   y[t] = W x[t]   for all other rows,
// x [T][K] bf16, W and W_N [N][K] bf16 (a linear layer's output-by-input
// layout), y [T][N] fp32.
//
// Routing: three small kernels lay the rows out as one permutation: the
// non-Nexus rows in order, then the Nexus rows in order.  The GEMM then runs
// over 128-row tiles of that permutation (a tile never mixes the two groups, so
// each tile reads one weight set), gathering its x rows through the
// permutation and scattering its y rows back.
//
// GEMM: 128 x 256 output tile per workgroup of eight waves, each wave a 64 x 64
// part as 2 x 2 blocks of v_mfma_f32_32x32x16_bf16, K in steps of 64.  Both
// operands are K-contiguous rows (x rows and weight rows), staged straight from
// global memory into LDS (direct-to-LDS loads), double-buffered: step s + 1
// streams in while step s is multiplied.  LDS rows are 128 bytes with an XOR
// swizzle on the 16-byte chunk index, so the fragment reads (32 rows at one
// chunk) are bank-conflict free.  Each fragment read feeds two MFMAs, and the
// reads are scheduled two K sub-steps ahead of the MFMAs that consume them.
// Tiles are laid out so that the workgroups of one XCD share a band of output
// columns and walk the row tiles in order: the x rows a tile needs are also
// needed by the tiles of the other columns of the band, resident on the same
// XCD at the same time, and so is each weight chunk, which keeps both in its L2.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kRouteThreads = 1024;
// 128 x 256 tiles, eight waves as 2 (rows) x 4 (columns), each 64 x 64.  Measured on
// the 8B-shaped QKV product (T = 43392, K = 4096, N = 6144): 128 x 128 with four waves
// 0.80-0.88 PFLOP/s, 256 x 128 0.91, 128 x 256 0.93; 256 x 256 tiles need more than
// 256 registers per lane and spill.
constexpr int kPM = 128, kPN = 256, kPK = 64;    // tile rows, tile columns, K step
constexpr int kPWavesM = 2, kPWavesN = 4;        // waves along rows and columns
constexpr int kPThreads = kPWavesM * kPWavesN * kWave;
constexpr int kPBM = kPM / kPWavesM / 32, kPBN = kPN / kPWavesN / 32;   // 32x32 blocks per wave
constexpr int kPRowChunks = kPK / 8;            // 16-byte chunks per staged row

// Pass 1: Nexus rows per block of 1024 rows.
__global__ __launch_bounds__(kRouteThreads) void route_count_kernel(const uint8_t *__restrict__ role, int T,
                                                                    int32_t *__restrict__ blk_nexus,
                                                                    const int32_t *status) {
  __shared__ int lds[kRouteThreads / kWave + 1];
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int i = blockIdx.x * kRouteThreads + threadIdx.x;
  int tot;
  block_flag_scan<kRouteThreads>(i < T && role[i] == kNexus, &tot, lds);
  if (threadIdx.x == 0) blk_nexus[blockIdx.x] = tot;
}

// Pass 2 (one workgroup): Nexus rows before each block, in place; counts = (non-Nexus, Nexus).
__global__ __launch_bounds__(kRouteThreads) void route_scan_kernel(int nblk, int T, int32_t *__restrict__ blk_nexus,
                                                                   int32_t *__restrict__ counts,
                                                                   const int32_t *status) {
  __shared__ int lds[kRouteThreads / kWave + 1];
  __shared__ int s_ok;
  const bool ok = block_status_clear(status, &s_ok);
  int carry = 0;
  for (int base = 0; base < nblk; base += kRouteThreads) {
    const int i = base + threadIdx.x;
    const int v = (ok && i < nblk) ? blk_nexus[i] : 0;
    int tot;
    const int off = block_int_scan<kRouteThreads>(v, &tot, lds);
    if (ok && i < nblk) blk_nexus[i] = carry + off;
    carry += tot;
  }
  if (threadIdx.x == 0) {   // no rows at all when the status is set: every GEMM tile exits
    counts[0] = ok ? T - carry : 0;
    counts[1] = ok ? carry : 0;
  }
}

// Pass 3: row i to its slot of the permutation.
__global__ __launch_bounds__(kRouteThreads) void route_fill_kernel(const uint8_t *__restrict__ role, int T,
                                                                   const int32_t *__restrict__ blk_nexus,
                                                                   const int32_t *__restrict__ counts,
                                                                   int32_t *__restrict__ perm,
                                                                   const int32_t *status) {
  __shared__ int lds[kRouteThreads / kWave + 1];
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int i = blockIdx.x * kRouteThreads + threadIdx.x;
  const bool in = i < T;
  const bool nx = in && role[i] == kNexus;
  int tot;
  const int r = block_flag_scan<kRouteThreads>(nx, &tot, lds);
  const int nexus_before = blk_nexus[blockIdx.x] + r;   // Nexus rows before row i
  if (in) perm[nx ? counts[0] + nexus_before : i - nexus_before] = i;
}

// chunk position of chunk c in staged row r (16 rows hit 16 distinct 4-bank groups)
__device__ __forceinline__ int swz_p(int r) { return (r & 7) ^ ((r >> 3) & 1); }

__global__ __launch_bounds__(kPThreads) void routed_gemm_kernel(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ w_text, const uint16_t *__restrict__ w_nexus,
    float *__restrict__ y, const int32_t *__restrict__ perm, const int32_t *__restrict__ counts, int K, int N,
    int n_tiles, int band) {
  __shared__ __align__(16) uint16_t a_lds0[kPM * kPK];
  __shared__ __align__(16) uint16_t a_lds1[kPM * kPK];
  __shared__ __align__(16) uint16_t b_lds0[kPN * kPK];
  __shared__ __align__(16) uint16_t b_lds1[kPN * kPK];
  __shared__ int rows_lds[kPM];

  // tile of this workgroup: XCD x takes column tiles [x * band, (x + 1) * band), row tiles in order
  const int xcd = blockIdx.x % kNumXcd;
  const int loc = blockIdx.x / kNumXcd;
  const int m_tile = loc / band;
  const int n_tile = xcd * band + loc % band;
  const int n_text = counts[0], n_nexus = counts[1];
  const int mt_text = (n_text + kPM - 1) / kPM;
  const int mt_all = mt_text + (n_nexus + kPM - 1) / kPM;
  if (n_tile >= n_tiles || m_tile >= mt_all) return;
  const bool nexus = m_tile >= mt_text;
  const int g0 = nexus ? n_text : 0;                           // first slot of the group
  const int row0 = (nexus ? m_tile - mt_text : m_tile) * kPM;  // first row of the tile in the group
  const int nrows = min(kPM, (nexus ? n_nexus : n_text) - row0);
  const int n0 = n_tile * kPN;
  const uint16_t *__restrict__ w = nexus ? w_nexus : w_text;

  for (int r = threadIdx.x; r < kPM; r += kPThreads) rows_lds[r] = perm[g0 + row0 + min(r, nrows - 1)];
  __syncthreads();

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int lane = threadIdx.x % kWave;
  // staging: instruction i of a tile fills rows 8i .. 8i + 7 (lane L: row 8i + L / 8 at
  // chunk position L % 8); wave w issues instructions w * IA .. of A and w * IB .. of B
  constexpr int kNW = kPThreads / kWave;
  constexpr int IA = kPM / 8 / kNW, IB = kPN / 8 / kNW;   // per wave and step
  static_assert(IA * kNW * 8 == kPM && IB * kNW * 8 == kPN, "whole instructions per wave");
  // per-lane byte offsets from the operand bases (the host checks that both operands
  // lie below 4 GiB), with the K step added to the wave-uniform base
  uint32_t a_off[IA], b_off[IB];
#pragma unroll
  for (int q = 0; q < IA; ++q) {
    const int r = 8 * (wave * IA + q) + lane / 8;
    const int c = (lane % 8) ^ swz_p(r);
    a_off[q] = static_cast<uint32_t>(rows_lds[r]) * static_cast<uint32_t>(K) * 2u + 16u * static_cast<uint32_t>(c);
  }
#pragma unroll
  for (int q = 0; q < IB; ++q) {
    const int r = 8 * (wave * IB + q) + lane / 8;
    const int c = (lane % 8) ^ swz_p(r);
    b_off[q] = static_cast<uint32_t>(min(n0 + r, N - 1)) * static_cast<uint32_t>(K) * 2u +
               16u * static_cast<uint32_t>(c);
  }
  const char *xb = uniform_ptr(reinterpret_cast<const char *>(x));
  const char *wb = uniform_ptr(reinterpret_cast<const char *>(w));
  auto stage = [&](int s, uint16_t *a_buf, uint16_t *b_buf) {
    const size_t koff = static_cast<size_t>(s) * kPK * 2;   // bytes
    const uint32_t la = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(a_buf));
    const uint32_t lb = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(b_buf));
#pragma unroll
    for (int q = 0; q < IA; ++q) dma_row16_s(xb + koff, a_off[q], la + (wave * IA + q) * kWave * 16);
#pragma unroll
    for (int q = 0; q < IB; ++q) dma_row16_s(wb + koff, b_off[q], lb + (wave * IB + q) * kWave * 16);
  };

  // this wave's (32 kPBM) x (32 kPBN) part of the tile
  const int wm = 32 * kPBM * (wave % kPWavesM), wn = 32 * kPBN * (wave / kPWavesM);
  const int li = lane & 31, lg = lane >> 5;
  f32x16 acc[kPBM][kPBN];
#pragma unroll
  for (int bi = 0; bi < kPBM; ++bi)
#pragma unroll
    for (int bj = 0; bj < kPBN; ++bj) acc[bi][bj] = f32x16{};

  // each A fragment feeds kPBN MFMAs, each B fragment kPBM
  auto mult = [&](const uint16_t *a_buf, const uint16_t *b_buf) {
#pragma unroll
    for (int kk = 0; kk < kPK / 16; ++kk) {
      const int c = 2 * kk + lg;
      bf16x8 af[kPBM], bf[kPBN];
#pragma unroll
      for (int t = 0; t < kPBM; ++t) {
        const int ra = wm + 32 * t + li;
        af[t] = *reinterpret_cast<const bf16x8 *>(&a_buf[(ra * kPRowChunks + (c ^ swz_p(ra))) * 8]);
      }
#pragma unroll
      for (int t = 0; t < kPBN; ++t) {
        const int rb = wn + 32 * t + li;
        bf[t] = *reinterpret_cast<const bf16x8 *>(&b_buf[(rb * kPRowChunks + (c ^ swz_p(rb))) * 8]);
      }
#pragma unroll
      for (int bi = 0; bi < kPBM; ++bi)
#pragma unroll
        for (int bj = 0; bj < kPBN; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[bi], bf[bj], acc[bi][bj], 0, 0, 0);
    }
    // the fragment reads run two K sub-steps (eight reads) ahead of the MFMAs
    order_reads_ahead<(kPK / 16) * kPBM * kPBN, 1, 2 * (kPBM + kPBN)>();
  };

  // double buffer: each wave issues IA + IB loads per step, so "step s has landed"
  // is "all but the IA + IB most recent" while step s + 1 streams
  const int steps = K / kPK;
  stage(0, a_lds0, b_lds0);
  for (int s = 0; s < steps; s += 2) {
    if (s + 1 < steps) {
      stage(s + 1, a_lds1, b_lds1);
      wait_vm<IA + IB>();
    } else {
      wait_vm<0>();
    }
    lds_barrier();            // step s is in buffer 0 for every wave
    mult(a_lds0, b_lds0);
    lds_barrier();            // every wave is done with buffer 0
    if (s + 1 >= steps) break;
    if (s + 2 < steps) {
      stage(s + 2, a_lds0, b_lds0);
      wait_vm<IA + IB>();
    } else {
      wait_vm<0>();
    }
    lds_barrier();            // step s + 1 is in buffer 1
    mult(a_lds1, b_lds1);
    lds_barrier();            // every wave is done with buffer 1
  }

  // lane (j = li, half lg) holds rows 8 (e / 4) + 4 lg + e % 4 of column j of each block
#pragma unroll
  for (int bi = 0; bi < kPBM; ++bi)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int r = wm + 32 * bi + 8 * (e >> 2) + 4 * lg + (e & 3);
      if (r < nrows) {
        float *yrow = y + static_cast<size_t>(rows_lds[r]) * N;
#pragma unroll
        for (int bj = 0; bj < kPBN; ++bj) {
          const int n = n0 + wn + 32 * bj + li;
          if (n < N) yrow[n] = acc[bi][bj][e];
        }
      }
    }
}

int routed_gemm_blocks(int T, int N) {
  const int m_tiles = (T + kPM - 1) / kPM + 1;   // the two groups can each end in a partial tile
  const int n_tiles = (N + kPN - 1) / kPN;
  const int band = (n_tiles + kNumXcd - 1) / kNumXcd;
  return kNumXcd * band * m_tiles;
}

hipError_t launch_routed_gemm(int T, int K, int N, const uint8_t *role, const uint16_t *x, const uint16_t *w_text,
                              const uint16_t *w_nexus, float *y, int32_t *blk_nexus, int32_t *counts, int32_t *perm,
                              int32_t *status, hipStream_t stream) {
  const int nblk = (T + kRouteThreads - 1) / kRouteThreads;
  route_count_kernel<<<dim3(nblk), dim3(kRouteThreads), 0, stream>>>(role, T, blk_nexus, status);
  route_scan_kernel<<<dim3(1), dim3(kRouteThreads), 0, stream>>>(nblk, T, blk_nexus, counts, status);
  route_fill_kernel<<<dim3(nblk), dim3(kRouteThreads), 0, stream>>>(role, T, blk_nexus, counts, perm, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n_tiles = (N + kPN - 1) / kPN;
  const int band = (n_tiles + kNumXcd - 1) / kNumXcd;
  routed_gemm_kernel<<<dim3(routed_gemm_blocks(T, N)), dim3(kPThreads), 0, stream>>>(
      x, w_text, w_nexus, y, perm, counts, K, N, n_tiles, band);
  return hipGetLastError();
}

}  // namespace sonic
