// Prefill planner: layout grammar, segment table and visible-key descriptors.
//
// The mask of Sec. 3.2 depends only on (role, segment) runs, so the planner
// works run by run instead of materialising an L x L mask:
//   * a system row sees the system rows before it (Eq.(3));
//   * a body row of segment i sees the system prompt, every Nexus token of the
//     earlier segments (causal; A1), and its own body up to itself; earlier
//     bodies are removed because the row lies after their segment (Eq.(4));
//   * a Nexus row of segment i sees the system prompt, its own body (it is not
//     after max(N_i)) and every Nexus token of the request (Eq.(5));
//   * a current-query row sees the system prompt, every Nexus token and the
//     current query up to itself; all bodies are removed (Eq.(4)).
// Every block of at most 32 rows of one run therefore sees the same key list
// apart from its own causal diagonal, and that list is "one contiguous range,
// a prefix of the request's Nexus positions, one more contiguous range".  One
// TileDesc per block encodes it; masked key blocks are never enumerated.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kPlanThreads = 1024;
constexpr int kCostBuckets = 1024;

// One step of the grammar SYSTEM* (TEXT+ NEXUS*)* CURRENT* of Eq.(1): may a token
// with role r and segment id t follow one with role rp and id tp (rp = -1 at the
// first token of a request)?  Segment ids are constant within a segment and
// strictly increase between segments.
__device__ __forceinline__ bool legal_step(int rp, int tp, int r, int t) {
  if (r < kSystem || r > kCurrent) return false;
  switch (rp) {
    case -1:
    case kSystem:
      return r != kNexus;
    case kText:
      if (r == kText) return t >= tp;
      if (r == kNexus) return t == tp;
      return r == kCurrent;
    case kNexus:
      if (r == kNexus) return t == tp;
      if (r == kText) return t > tp;
      return r == kCurrent;
    case kCurrent:
      return r == kCurrent;
    default:
      return false;
  }
}

// One workgroup per request: validate, list the Nexus positions and the runs,
// then emit one descriptor per block of up to 32 rows of a run.
__global__ __launch_bounds__(kPlanThreads) void plan_runs_kernel(const int32_t *__restrict__ cu,
                                                                 const uint8_t *__restrict__ role,
                                                                 const int32_t *__restrict__ turn, PrefillWs ws,
                                                                 int total_tokens, int32_t *status) {
  __shared__ int lds[kPlanThreads / kWave + 1];
  __shared__ int s_bad;
  const int b = blockIdx.x;
  const int s = cu[b];
  const int e = cu[b + 1];
  if (s < 0 || e < s || e > total_tokens) {   // cu_seqlens itself is malformed
    if (threadIdx.x == 0) {
      raise_status(status, SONIC_ERR_BAD_LAYOUT);
      ws.req[b] = ReqInfo{0, 0, 0, 0};
    }
    return;
  }
  const int L = e - s;
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();

  // Pass 1: grammar, Nexus positions, run starts (with the Nexus count before each).
  int nexus_carry = 0, run_carry = 0;
  for (int base = 0; base < L; base += kPlanThreads) {
    const int i = base + threadIdx.x;
    const bool in = i < L;
    int r = -1, t = 0, rp = -1, tp = 0;
    if (in) {
      r = role[s + i];
      t = turn[s + i];
      if (i > 0) {
        rp = role[s + i - 1];
        tp = turn[s + i - 1];
      }
    }
    if (in && !legal_step(rp, tp, r, t)) s_bad = 1;
    const bool is_nexus = in && r == kNexus;
    const bool run_start = in && (i == 0 || r != rp || (r == kText && t != tp));
    int ntot, rtot;
    const int nrank = block_flag_scan<kPlanThreads>(is_nexus, &ntot, lds);
    const int rrank = block_flag_scan<kPlanThreads>(run_start, &rtot, lds);
    if (is_nexus) ws.nexus_pos[s + nexus_carry + nrank] = i;
    if (run_start) ws.runs[s + run_carry + rrank] = make_int2(i, nexus_carry + nrank);
    nexus_carry += ntot;
    run_carry += rtot;
  }
  __syncthreads();
  if (s_bad) {
    if (threadIdx.x == 0) {
      raise_status(status, SONIC_ERR_BAD_LAYOUT);
      ws.req[b] = ReqInfo{0, 0, 0, 0};
    }
    return;
  }
  const int nruns = run_carry;
  const int k_tot = nexus_carry;
  int S = 0;
  if (L > 0 && role[s] == kSystem) S = nruns > 1 ? ws.runs[s + 1].x : L;

  // Pass 2: descriptors, run by run.
  int tile_carry = 0;
  for (int rb = 0; rb < nruns; rb += kPlanThreads) {
    const int r = rb + threadIdx.x;
    const bool in = r < nruns;
    int start = 0, end = 0, nt = 0;
    if (in) {
      start = ws.runs[s + r].x;
      end = (r + 1 < nruns) ? ws.runs[s + r + 1].x : L;
      nt = (end - start + kTileRows - 1) / kTileRows;
    }
    int ttot;
    const int toff = block_int_scan<kPlanThreads>(nt, &ttot, lds);
    if (in) {
      const int kind = role[s + start];
      const int nexus_before = ws.runs[s + r].y;
      int body_start = 0, body_len = 0;
      if (kind == kNexus) {  // the grammar puts the owning body run right before
        body_start = ws.runs[s + r - 1].x;
        body_len = start - body_start;
      }
      for (int j = 0; j < nt; ++j) {
        TileDesc d;
        d.req = b;
        d.p0 = start + j * kTileRows;
        d.nrows = min(kTileRows, end - d.p0);
        if (kind == kSystem) {
          d.r0_end = d.p0;
          d.nx = 0;
          d.r1_start = 0;
          d.r1_len = 0;
          d.ndiag = d.nrows;
        } else if (kind == kText) {
          d.r0_end = S;
          d.nx = nexus_before;
          d.r1_start = start;
          d.r1_len = d.p0 - start;
          d.ndiag = d.nrows;
        } else if (kind == kNexus) {
          d.r0_end = S;
          d.nx = k_tot;
          d.r1_start = body_start;
          d.r1_len = body_len;
          d.ndiag = 0;
        } else {
          d.r0_end = S;
          d.nx = k_tot;
          d.r1_start = start;
          d.r1_len = d.p0 - start;
          d.ndiag = d.nrows;
        }
        ws.tiles[s + tile_carry + toff + j] = d;
      }
    }
    tile_carry += ttot;
  }
  if (threadIdx.x == 0) ws.req[b] = ReqInfo{tile_carry, S, k_tot, nruns};
}

// One workgroup: order all descriptors by cost (number of 64-key steps),
// most expensive first, and reset the per-XCD work queues.
__global__ __launch_bounds__(kPlanThreads) void plan_order_kernel(int batch, const int32_t *__restrict__ cu,
                                                                  PrefillWs ws, const int32_t *status) {
  __shared__ int hist[kCostBuckets];
  __shared__ int lds[kPlanThreads / kWave + 1];
  __shared__ int s_ok;
  static_assert(kCostBuckets == kPlanThreads, "one histogram bucket per thread");
  hist[threadIdx.x] = 0;
  const bool ok = block_status_clear(status, &s_ok);
  if (ok) {
    for (int b = 0; b < batch; ++b) {
      const int nt = ws.req[b].ntiles;
      const int base = cu[b];
      for (int j = threadIdx.x; j < nt; j += kPlanThreads) {
        const int c = min(tile_cost(ws.tiles[base + j]), kCostBuckets - 1);
        atomicAdd(&hist[kCostBuckets - 1 - c], 1);
      }
    }
  }
  __syncthreads();
  int total;
  const int off = block_int_scan<kPlanThreads>(hist[threadIdx.x], &total, lds);
  hist[threadIdx.x] = off;
  __syncthreads();
  if (ok) {
    for (int b = 0; b < batch; ++b) {
      const int nt = ws.req[b].ntiles;
      const int base = cu[b];
      for (int j = threadIdx.x; j < nt; j += kPlanThreads) {
        const int c = min(tile_cost(ws.tiles[base + j]), kCostBuckets - 1);
        const int pos = atomicAdd(&hist[kCostBuckets - 1 - c], 1);
        ws.order[pos] = base + j;
      }
    }
  }
  if (threadIdx.x == 0) ws.ctrl[0] = ok ? total : 0;
  if (threadIdx.x < kNumXcd) ws.ctrl[8 + threadIdx.x] = 0;
}

hipError_t launch_plan(int batch, int total_tokens, const int32_t *cu, const uint8_t *role, const int32_t *turn,
                       PrefillWs ws, int32_t *status, hipStream_t stream) {
  plan_runs_kernel<<<dim3(batch), dim3(kPlanThreads), 0, stream>>>(cu, role, turn, ws, total_tokens, status);
  plan_order_kernel<<<dim3(1), dim3(kPlanThreads), 0, stream>>>(batch, cu, ws, status);
  return hipGetLastError();
}

}  // namespace sonic
