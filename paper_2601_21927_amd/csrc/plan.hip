// Prefill planner: layout grammar, segment table and visible-key descriptors.
//
// The mask of Sec. 3.2 depends only on (role, segment) runs, so the planner
// works run by run instead of materialising an L x L mask:
//   * a system row sees the system rows before it (Eq.(3));
//   * a body row of segment i sees the system prompt, every Nexus token of the
//     earlier segments (causal; A1), and its own body up to itself; earlier
//     bodies are removed because the row lies after their segment (Eq.(4));
//   * a Nexus row of segment i sees the system prompt, its own body (it is not
//     after max(N_i)) and every Nexus token of the request (Eq.(5)), or, with the
//     narrower Nexus scope, those of segments 1..i only: a shorter leading part
//     of the same prefix;
//   * a current-query row sees the system prompt, every Nexus token and the
//     current query up to itself; all bodies are removed (Eq.(4)).
// Every block of at most 32 rows of one run therefore sees the same key list
// apart from its own causal diagonal.  With the request's system and Nexus rows
// copied, in order, into one contiguous "prefix" (system prompt first, then the
// Nexus tokens segment by segment), that list is "a leading part of the prefix,
// then one contiguous range of the request ending in the block's own rows".
// One TileDesc per block encodes it; masked key blocks are never enumerated.
//
// Work order: requests by decreasing total cost, and inside a request its blocks
// by decreasing cost.  Blocks of one request run close together in time, so the
// K/V rows they share (system prompt, Nexus tokens, bodies) stay in the L2 of
// the XCD that serves them.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kPlanThreads = 1024;
constexpr int kPlanTok = 8;        // tokens per thread in the run kernel's pass 1
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
                                                                 int total_tokens, int nexus_scope,
                                                                 int32_t *status) {
  __shared__ int lds[kPlanThreads / kWave + 1];
  __shared__ int lds4[4 * (kPlanThreads / kWave)];
  __shared__ unsigned long long s_cost;
  const int b = blockIdx.x;
  const int s = cu[b];
  const int e = cu[b + 1];
  if (s < 0 || e < s || e > total_tokens) {   // cu_seqlens itself is malformed
    if (threadIdx.x == 0) {
      raise_status(status, SONIC_ERR_BAD_LAYOUT);
      ws.req[b] = ReqInfo{0, 0, 0, 0, 0, 0};
    }
    return;
  }
  const int L = e - s;

  // Pass 1: grammar, prefix rows (system and Nexus positions, in order), run starts
  // with the number of prefix rows before each.  In a well-formed request the
  // system rows come first, so the prefix is the system prompt followed by the
  // Nexus tokens.  Each thread takes kPlanTok consecutive tokens (one chunk of
  // kPlanThreads * kPlanTok tokens covers most requests): it counts them, one
  // block scan places its entries, and a second walk over its registers writes
  // them.  A token's predecessor is the thread's previous token, or the lower
  // lane's last one (lane 0 loads its own).
  int pre_carry = 0, run_carry = 0, nexus_count = 0, bad_count = 0;
  const int lane = threadIdx.x % kWave;
  for (int base = 0; base < L; base += kPlanThreads * kPlanTok) {
    const int i0 = base + threadIdx.x * kPlanTok;
    int r[kPlanTok], t[kPlanTok];
#pragma unroll
    for (int j = 0; j < kPlanTok; ++j) {
      r[j] = -1;
      t[j] = 0;
      if (i0 + j < L) {
        r[j] = role[s + i0 + j];
        t[j] = turn[s + i0 + j];
      }
    }
    int rp0 = __shfl_up(r[kPlanTok - 1], 1), tp0 = __shfl_up(t[kPlanTok - 1], 1);
    if (lane == 0) {
      rp0 = -1;
      tp0 = 0;
      if (i0 > 0 && i0 <= L) {
        rp0 = role[s + i0 - 1];
        tp0 = turn[s + i0 - 1];
      }
    }
    int cnt[4] = {0, 0, 0, 0};   // prefix rows, run starts, Nexus tokens, illegal steps
    {
      int rp = rp0, tp = tp0;
#pragma unroll
      for (int j = 0; j < kPlanTok; ++j) {
        if (i0 + j < L) {
          cnt[0] += (r[j] == kSystem || r[j] == kNexus) ? 1 : 0;
          cnt[1] += (i0 + j == 0 || r[j] != rp || (r[j] == kText && t[j] != tp)) ? 1 : 0;
          cnt[2] += r[j] == kNexus ? 1 : 0;
          cnt[3] += legal_step(rp, tp, r[j], t[j]) ? 0 : 1;
        }
        rp = r[j];
        tp = t[j];
      }
    }
    int below[4], tot[4];
    block_int_scan_n<kPlanThreads, 4>(cnt, below, tot, lds4);
    {
      int rp = rp0, tp = tp0;
      int pc = pre_carry + below[0], rc = run_carry + below[1];
#pragma unroll
      for (int j = 0; j < kPlanTok; ++j) {
        const int i = i0 + j;
        if (i < L) {
          if (i == 0 || r[j] != rp || (r[j] == kText && t[j] != tp)) ws.runs[s + rc++] = make_int2(i, pc);
          if (r[j] == kSystem || r[j] == kNexus) ws.prefix_pos[s + pc++] = i;
        }
        rp = r[j];
        tp = t[j];
      }
    }
    pre_carry += tot[0];
    run_carry += tot[1];
    nexus_count += tot[2];
    bad_count += tot[3];
  }
  __syncthreads();
  if (bad_count) {
    if (threadIdx.x == 0) {
      raise_status(status, SONIC_ERR_BAD_LAYOUT);
      ws.req[b] = ReqInfo{0, 0, 0, 0, 0, 0};
    }
    return;
  }
  const int nruns = run_carry;
  const int k_tot = nexus_count;
  int S = 0;
  if (L > 0 && role[s] == kSystem) S = nruns > 1 ? ws.runs[s + 1].x : L;
  const int npre_all = S + k_tot;
  if (threadIdx.x == 0) s_cost = 0ull;

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
      const int pre_before = ws.runs[s + r].y;
      int body_start = 0, body_len = 0;
      if (kind == kNexus) {  // the grammar puts the owning body run right before
        body_start = ws.runs[s + r - 1].x;
        body_len = start - body_start;
      }
      unsigned long long my_cost = 0;
      for (int j = 0; j < nt; ++j) {
        TileDesc d;
        d.req = b;
        d.p0 = start + j * kTileRows;
        d.nrows = min(kTileRows, end - d.p0);
        d.pad = 0;
        if (kind == kSystem) {          // system rows before the block, then the block
          d.npre = d.p0;
          d.seg_start = d.p0;
          d.seg_len = d.nrows;
          d.ndiag = d.nrows;
        } else if (kind == kText) {     // system + earlier Nexus, own body up to the block
          d.npre = pre_before;
          d.seg_start = start;
          d.seg_len = d.p0 + d.nrows - start;
          d.ndiag = d.nrows;
        } else if (kind == kNexus) {    // system + every Nexus (or up to its own), the owning body
          d.npre = nexus_scope == SONIC_NEXUS_ALL ? npre_all : pre_before + (end - start);
          d.seg_start = body_start;
          d.seg_len = body_len;
          d.ndiag = 0;
        } else {                        // system + every Nexus, current query up to the block
          d.npre = npre_all;
          d.seg_start = start;
          d.seg_len = d.p0 + d.nrows - start;
          d.ndiag = d.nrows;
        }
        ws.tiles[s + tile_carry + toff + j] = d;
        my_cost += static_cast<unsigned long long>(tile_cost(d));
      }
      if (my_cost) atomicAdd(&s_cost, my_cost);
    }
    tile_carry += ttot;
  }
  __syncthreads();
  if (threadIdx.x == 0) ws.req[b] = ReqInfo{tile_carry, S, k_tot, nruns, static_cast<int64_t>(s_cost), 0};
}

// One workgroup per request: its descriptors by decreasing cost (a histogram
// sort over kCostBuckets cost values, larger costs share the last bucket), from
// its first slot in `order`.  Requests run by decreasing total cost (ties by
// index), so that first slot is the number of descriptors of the requests ranked
// before it: a workgroup sum over the batch, no global sort.  Workgroup 0 also
// writes the descriptor count and resets the queues.
__global__ __launch_bounds__(kPlanThreads) void plan_order_kernel(int batch, const int32_t *__restrict__ cu,
                                                                  PrefillWs ws, const int32_t *status) {
  __shared__ int hist[kCostBuckets];
  __shared__ int lds[kPlanThreads / kWave + 1];
  __shared__ int s_ok;
  static_assert(kCostBuckets == kPlanThreads, "one histogram bucket per thread");
  const int b = blockIdx.x;
  hist[threadIdx.x] = 0;
  const bool ok = block_status_clear(status, &s_ok);
  if (b == 0 && threadIdx.x < kNumXcd) ws.ctrl[8 + threadIdx.x] = 0;
  if (!ok) {
    if (b == 0 && threadIdx.x == 0) ws.ctrl[0] = 0;
    return;
  }
  const int64_t cb = ws.req[b].cost;
  int before = 0, all = 0;
  for (int j0 = 0; j0 < batch; j0 += kPlanThreads) {
    const int j = j0 + threadIdx.x;
    int nt_j = 0, nb = 0;
    if (j < batch) {
      const ReqInfo rj = ws.req[j];
      nt_j = rj.ntiles;
      nb = (rj.cost > cb || (rj.cost == cb && j < b)) ? nt_j : 0;
    }
    int t0, t1;
    block_int_scan<kPlanThreads>(nb, &t0, lds);
    block_int_scan<kPlanThreads>(nt_j, &t1, lds);
    before += t0;
    all += t1;
  }
  if (b == 0 && threadIdx.x == 0) ws.ctrl[0] = all;
  const int nt = ws.req[b].ntiles;
  const int base = cu[b];
  const int dst = before;
  for (int j = threadIdx.x; j < nt; j += kPlanThreads) {
    const int c = min(tile_cost(ws.tiles[base + j]), kCostBuckets - 1);
    atomicAdd(&hist[kCostBuckets - 1 - c], 1);
  }
  __syncthreads();
  int total;
  const int off = block_int_scan<kPlanThreads>(hist[threadIdx.x], &total, lds);
  hist[threadIdx.x] = off;
  __syncthreads();
  for (int j = threadIdx.x; j < nt; j += kPlanThreads) {
    const int c = min(tile_cost(ws.tiles[base + j]), kCostBuckets - 1);
    const int pos = atomicAdd(&hist[kCostBuckets - 1 - c], 1);
    ws.order[dst + pos] = base + j;
  }
}

// Prefix copies: row j < S + K_tot of request b's prefix gets the K and V rows
// of position prefix_pos[cu[b] + j].  Workgroups gx*b .. gx*b + gx-1 copy request
// b's prefix, one wave per kGatherRows consecutive rows, waves striding over the
// prefix.  The wave's first lanes read the rows' positions, then every
// lane has all of its 16-byte pieces of those rows in flight before it stores
// (kGatherPieces per row and tensor at a time).
constexpr int kGatherThreads = 256;
constexpr int kGatherWaves = kGatherThreads / kWave;
constexpr int kGatherRows = 4;
constexpr int kGatherPieces = 2;

__global__ __launch_bounds__(kGatherThreads) void gather_prefix_kernel(const int32_t *__restrict__ cu,
                                                                      const uint16_t *__restrict__ k,
                                                                      const uint16_t *__restrict__ v, PrefillWs ws,
                                                                      int row_pieces, int gx,
                                                                      const int32_t *status) {
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int b = blockIdx.x / gx;
  const int bx = blockIdx.x % gx;
  const int s0 = cu[b];
  const ReqInfo ri = ws.req[b];
  const int npre = ri.system + ri.nexus_total;
  const int lane = threadIdx.x % kWave;
  const int wave = threadIdx.x / kWave;
  const u32x4 *__restrict__ k4 = reinterpret_cast<const u32x4 *>(k);
  const u32x4 *__restrict__ v4 = reinterpret_cast<const u32x4 *>(v);
  u32x4 *__restrict__ kd = reinterpret_cast<u32x4 *>(ws.k_pre);
  u32x4 *__restrict__ vd = reinterpret_cast<u32x4 *>(ws.v_pre);
  const int stride = gx * kGatherWaves * kGatherRows;
  for (int j0 = (bx * kGatherWaves + wave) * kGatherRows; j0 < npre; j0 += stride) {
    int src = -1;   // lane u < kGatherRows: source row of copy row j0 + u, or -1 past the prefix
    if (lane < kGatherRows && j0 + lane < npre) src = s0 + ws.prefix_pos[s0 + j0 + lane];
    int sr[kGatherRows];
#pragma unroll
    for (int u = 0; u < kGatherRows; ++u) sr[u] = __builtin_amdgcn_readlane(src, u);
    for (int c0 = 0; c0 < row_pieces; c0 += kGatherPieces * kWave) {
      u32x4 kr[kGatherRows][kGatherPieces], vr[kGatherRows][kGatherPieces];
#pragma unroll
      for (int u = 0; u < kGatherRows; ++u)
#pragma unroll
        for (int p = 0; p < kGatherPieces; ++p) {
          const int c = c0 + p * kWave + lane;
          if (sr[u] >= 0 && c < row_pieces) {
            kr[u][p] = k4[static_cast<size_t>(sr[u]) * row_pieces + c];
            vr[u][p] = v4[static_cast<size_t>(sr[u]) * row_pieces + c];
          }
        }
#pragma unroll
      for (int u = 0; u < kGatherRows; ++u)
#pragma unroll
        for (int p = 0; p < kGatherPieces; ++p) {
          const int c = c0 + p * kWave + lane;
          if (sr[u] >= 0 && c < row_pieces) {
            const size_t dst = static_cast<size_t>(s0 + j0 + u) * row_pieces + c;
            kd[dst] = kr[u][p];
            vd[dst] = vr[u][p];
          }
        }
    }
  }
}

// Work order of the prefill's descriptors (request b's at offset cu[b] of ws.tiles)
// and reset queues.
hipError_t launch_plan_order(int batch, const int32_t *cu, PrefillWs ws, int32_t *status, hipStream_t stream) {
  plan_order_kernel<<<dim3(batch), dim3(kPlanThreads), 0, stream>>>(batch, cu, ws, status);
  return hipGetLastError();
}

// Grammar check and run table only (ws.req, ws.prefix_pos, ws.runs; ws.tiles is
// written as scratch), for callers that need the segment structure but no prefill.
hipError_t launch_plan_runs(int batch, int total_tokens, const int32_t *cu, const uint8_t *role, const int32_t *turn,
                            PrefillWs ws, int32_t *status, hipStream_t stream) {
  plan_runs_kernel<<<dim3(batch), dim3(kPlanThreads), 0, stream>>>(cu, role, turn, ws, total_tokens,
                                                                    SONIC_NEXUS_ALL, status);
  return hipGetLastError();
}

hipError_t launch_plan(int batch, int total_tokens, int Hkv, int D, int nexus_scope, const int32_t *cu,
                       const uint8_t *role, const int32_t *turn, const uint16_t *k, const uint16_t *v, PrefillWs ws,
                       int32_t *status, hipStream_t stream) {
  plan_runs_kernel<<<dim3(batch), dim3(kPlanThreads), 0, stream>>>(cu, role, turn, ws, total_tokens, nexus_scope,
                                                                    status);
  hipError_t e = launch_plan_order(batch, cu, ws, status, stream);
  if (e != hipSuccess) return e;
  const int row_pieces = Hkv * D / 8;
  // about 2048 workgroups over the batch, none with nothing but rows past every prefix
  constexpr int rows_per_block = kGatherWaves * kGatherRows;
  const int by_rows = (total_tokens + rows_per_block - 1) / rows_per_block;
  const int gx = max(1, min((2048 + batch - 1) / batch, by_rows));
  gather_prefix_kernel<<<dim3(gx * batch), dim3(kGatherThreads), 0, stream>>>(cu, k, v, ws, row_pieces, gx,
                                                                              status);
  return hipGetLastError();
}

}  // namespace sonic
