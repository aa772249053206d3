// Workgroup-wide prefix sums built from wave ballots (flags) and wave shuffles (integers).
#pragma once

#include "common.h"

namespace sonic {

// Number of lanes below this one whose predicate is set.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0));
}

// Exclusive prefix count of a 0/1 flag over an NT-thread workgroup.
// `lds` must hold NT/64 + 1 ints; the workgroup total is returned in *total.
template <int NT>
__device__ __forceinline__ int block_flag_scan(bool flag, int *total, int *lds) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const uint64_t m = __ballot(flag);
  const int below = lanes_below(m);
  if (lane == 0) lds[w] = __popcll(m);
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < NW; ++i) {
      const int c = lds[i];
      lds[i] = run;
      run += c;
    }
    lds[NW] = run;
  }
  __syncthreads();
  const int res = lds[w] + below;
  *total = lds[NW];
  __syncthreads();
  return res;
}

// Exclusive prefix sums of NV ints at once over an NT-thread workgroup: below[f] =
// the sum of x[f] over lower threads, total[f] = the workgroup's sum.  Two barriers.
template <int NT, int NV>
__device__ __forceinline__ void block_int_scan_n(const int (&x)[NV], int (&below)[NV], int (&total)[NV],
                                                 int *lds) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  int v[NV];
#pragma unroll
  for (int f = 0; f < NV; ++f) v[f] = x[f];
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
#pragma unroll
    for (int f = 0; f < NV; ++f) {
      const int y = __shfl_up(v[f], o);
      if (lane >= o) v[f] += y;
    }
  }
  if (lane == kWave - 1)
#pragma unroll
    for (int f = 0; f < NV; ++f) lds[f * NW + w] = v[f];
  lds_barrier();
#pragma unroll
  for (int f = 0; f < NV; ++f) {
    int before = 0, tot = 0;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      const int c = lds[f * NW + k];
      before += k < w ? c : 0;
      tot += c;
    }
    below[f] = v[f] - x[f] + before;
    total[f] = tot;
  }
  lds_barrier();
}

// Exclusive prefix sum of a non-negative int over an NT-thread workgroup.
template <int NT>
__device__ __forceinline__ int block_int_scan(int x, int *total, int *lds) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  int v = x;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(v, o);
    if (lane >= o) v += y;
  }
  if (lane == kWave - 1) lds[w] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < NW; ++i) {
      const int c = lds[i];
      lds[i] = run;
      run += c;
    }
    lds[NW] = run;
  }
  __syncthreads();
  const int res = lds[w] + v - x;
  *total = lds[NW];
  __syncthreads();
  return res;
}

}  // namespace sonic
