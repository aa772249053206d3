// Next-turn Nexus step over the compact cache.
//
// When a turn ends, its rows (query and response) sit at the end of the
// request's compact cache.  Each of its segments (the user utterance, the
// assistant response: Sec. 3.1) becomes the body of a history segment followed
// by its Nexus tokens.  One call computes one segment's Nexus tokens: the
// segment's body is the first body_len tail rows (all of them without body_len).
// A Nexus row of that segment sees every kept cache row (the system prompt and
// the earlier segments' Nexus tokens), its own body (Eqs.(3)-(4) of Sec. 3.2) and
// every Nexus row of its own segment (Eq.(5)); tail rows after the body come
// later in the sequence (Eq.(3)).  So each 32-row block of new Nexus rows has
// the two-piece key list the prefill kernel walks: the request's cache rows
// 0 .. keep_len + body_len, then its new Nexus rows, all visible.  The attention
// runs on the prefill kernels; afterwards the new Nexus K/V replace the body in
// the cache (rows keep_len ..), since no later row may see the body (Eq.(4)), and
// the tail rows after the body (staged in the workspace beforehand, the regions
// may overlap) follow them.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kExtendThreads = 256;

// Lengths of request j, checked: its new-row count kn, the tail rows after its
// segment's body (rest), its block count and cost (every block costs the same:
// all keep + body + kn keys).  Returns 0, SONIC_ERR_BAD_LAYOUT or SONIC_ERR_CAPACITY.
struct ExtendReq {
  int kn, rest, nt;
  int64_t cost;
};
__device__ __forceinline__ int extend_check(int j, const int32_t *__restrict__ nexus_cu,
                                            const int32_t *__restrict__ keep_len, const int32_t *__restrict__ body_len,
                                            const int32_t *__restrict__ cache_len, const int32_t *__restrict__ row_cap,
                                            int max_rows, int total_new, ExtendReq *r) {
  const int s = nexus_cu[j];
  const int e = nexus_cu[j + 1];
  const int len = cache_len[j];
  const int keep = keep_len[j];
  const int cap = row_cap[j];
  const int body = body_len != nullptr ? body_len[j] : len - keep;
  const bool bad = s < 0 || e < s || e > total_new || keep < 0 || keep > len || len > cap || len > max_rows ||
                   body < 0 || body > len - keep;
  *r = ExtendReq{0, 0, 0, 0};
  if (bad) return SONIC_ERR_BAD_LAYOUT;
  const int kn = e - s;
  const int rest = len - keep - body;
  if (keep + kn + rest > cap) return SONIC_ERR_CAPACITY;
  const int nt = (kn + kTileRows - 1) / kTileRows;
  *r = ExtendReq{kn, rest, nt, static_cast<int64_t>(nt) * ((keep + body + kn + kKeyChunk - 1) / kKeyChunk)};
  return 0;
}

// One workgroup per request b, the whole plan in one launch.  The lengths of every
// request are inputs, so each workgroup checks all of them and knows the batch's
// block counts and costs: blocks run requests by decreasing cost (ties by index),
// and request b's first slot in the work order is the number of blocks of the
// requests ranked before it.  A bad request, or an error left on the status word by
// an earlier call, makes the whole call write nothing (no work items).  Then one
// descriptor per block of up to 32 new Nexus rows; ReqInfo.nruns carries the
// number of tail rows after the body to the cache update.
__global__ __launch_bounds__(kExtendThreads) void plan_extend_kernel(
    int batch, const int32_t *__restrict__ nexus_cu, const int32_t *__restrict__ keep_len,
    const int32_t *__restrict__ body_len, const int32_t *__restrict__ cache_len, const int32_t *__restrict__ row_cap,
    int max_rows, int total_new, PrefillWs ws, int32_t *status) {
  __shared__ int lds[kExtendThreads / kWave + 1];
  __shared__ int s_ok;
  const int b = blockIdx.x;
  if (b == 0 && threadIdx.x < kNumXcd) ws.ctrl[8 + threadIdx.x] = 0;   // the work queues
  const bool clear = block_status_clear(status, &s_ok);
  ExtendReq own;
  const int own_code = extend_check(b, nexus_cu, keep_len, body_len, cache_len, row_cap, max_rows, total_new, &own);
  int before = 0, all = 0, nbad = 0;
  for (int j0 = 0; j0 < batch; j0 += kExtendThreads) {
    const int j = j0 + threadIdx.x;
    ExtendReq r{0, 0, 0, 0};
    int code = 0;
    if (j < batch) code = extend_check(j, nexus_cu, keep_len, body_len, cache_len, row_cap, max_rows, total_new, &r);
    const int nb = (r.cost > own.cost || (r.cost == own.cost && j < b)) ? r.nt : 0;
    int t0, t1, t2;
    block_int_scan<kExtendThreads>(nb, &t0, lds);
    block_int_scan<kExtendThreads>(r.nt, &t1, lds);
    block_int_scan<kExtendThreads>(code != 0 ? 1 : 0, &t2, lds);
    before += t0;
    all += t1;
    nbad += t2;
  }
  if (own_code != 0 && clear && threadIdx.x == 0) raise_status(status, own_code);
  if (!clear || nbad > 0) {
    if (threadIdx.x == 0) {
      if (b == 0) ws.ctrl[0] = 0;
      ws.req[b] = ReqInfo{0, 0, 0, 0, 0, 0};
    }
    return;
  }
  if (b == 0 && threadIdx.x == 0) ws.ctrl[0] = all;
  const int s = nexus_cu[b];
  const int keep = keep_len[b];
  const int body = cache_len[b] - keep - own.rest;
  for (int j = threadIdx.x; j < own.nt; j += kExtendThreads) {
    TileDesc d;
    d.req = b;
    d.p0 = j * kTileRows;
    d.nrows = min(kTileRows, own.kn - d.p0);
    d.npre = keep + body;  // the kept cache rows and the segment's body
    d.seg_start = 0;       // then every new Nexus row, no causal part
    d.seg_len = own.kn;
    d.ndiag = 0;
    d.pad = 0;
    ws.tiles[s + j] = d;
    ws.order[before + j] = s + j;   // a request's blocks all cost the same: index order
  }
  if (threadIdx.x == 0) ws.req[b] = ReqInfo{own.nt, 0, own.kn, own.rest, own.cost, 0};
}

// Before the cache update: the tail rows after the body, rows keep + body .. len of
// request b, to the workspace (rows b * max_rows ..).  Grid (chunks of rows,
// requests); one thread per 16-byte piece of a row.
__global__ __launch_bounds__(kExtendThreads) void extend_stage_kernel(
    const int32_t *__restrict__ keep_len, const int32_t *__restrict__ body_len, const uint16_t *__restrict__ kc,
    const uint16_t *__restrict__ vc, const int64_t *__restrict__ row_off, PrefillWs ws, uint16_t *__restrict__ k_stage,
    uint16_t *__restrict__ v_stage, int max_rows, int row_pieces, const int32_t *status) {
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int b = blockIdx.y;
  const int rest = ws.req[b].nruns;
  const size_t src0 = static_cast<size_t>(row_off[b] + keep_len[b] + body_len[b]) * row_pieces;
  const size_t dst0 = static_cast<size_t>(b) * max_rows * row_pieces;
  const long total = static_cast<long>(rest) * row_pieces;
  for (long u = static_cast<long>(blockIdx.x) * kExtendThreads + threadIdx.x; u < total;
       u += static_cast<long>(gridDim.x) * kExtendThreads) {
    reinterpret_cast<u32x4 *>(k_stage)[dst0 + u] = reinterpret_cast<const u32x4 *>(kc)[src0 + u];
    reinterpret_cast<u32x4 *>(v_stage)[dst0 + u] = reinterpret_cast<const u32x4 *>(vc)[src0 + u];
  }
}

// After the attention: request b's new Nexus rows go to cache rows keep_len[b] ..,
// over the body, the staged tail rows after them, and the length becomes
// keep_len[b] + (its Nexus count) + (the staged rows).  Grid (chunks of rows,
// requests); one thread per 16-byte piece of a row.
__global__ __launch_bounds__(kExtendThreads) void extend_append_kernel(
    const int32_t *__restrict__ nexus_cu, const int32_t *__restrict__ keep_len, uint16_t *__restrict__ kc,
    uint16_t *__restrict__ vc, const int64_t *__restrict__ row_off, int32_t *__restrict__ cache_len,
    const uint16_t *__restrict__ k_new, const uint16_t *__restrict__ v_new, PrefillWs ws,
    const uint16_t *__restrict__ k_stage, const uint16_t *__restrict__ v_stage, int max_rows, int row_pieces,
    const int32_t *status) {
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int b = blockIdx.y;
  const int s = nexus_cu[b];
  const int kn = nexus_cu[b + 1] - s;
  const int keep = keep_len[b];
  const int rest = ws.req[b].nruns;
  const size_t dst0 = static_cast<size_t>(row_off[b] + keep) * row_pieces;
  const size_t src0 = static_cast<size_t>(s) * row_pieces;
  const size_t stage0 = static_cast<size_t>(b) * max_rows * row_pieces;
  const long nnew = static_cast<long>(kn) * row_pieces;
  const long total = nnew + static_cast<long>(rest) * row_pieces;
  for (long u = static_cast<long>(blockIdx.x) * kExtendThreads + threadIdx.x; u < total;
       u += static_cast<long>(gridDim.x) * kExtendThreads) {
    if (u < nnew) {
      reinterpret_cast<u32x4 *>(kc)[dst0 + u] = reinterpret_cast<const u32x4 *>(k_new)[src0 + u];
      reinterpret_cast<u32x4 *>(vc)[dst0 + u] = reinterpret_cast<const u32x4 *>(v_new)[src0 + u];
    } else {
      reinterpret_cast<u32x4 *>(kc)[dst0 + u] = reinterpret_cast<const u32x4 *>(k_stage)[stage0 + u - nnew];
      reinterpret_cast<u32x4 *>(vc)[dst0 + u] = reinterpret_cast<const u32x4 *>(v_stage)[stage0 + u - nnew];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) cache_len[b] = keep + kn + rest;   // nothing else reads it here
}

hipError_t launch_plan_extend(int batch, int total_new, int max_rows, const int32_t *nexus_cu,
                              const int32_t *keep_len, const int32_t *body_len, const int32_t *cache_len,
                              const int32_t *row_cap, PrefillWs ws, int32_t *status, hipStream_t stream) {
  plan_extend_kernel<<<dim3(batch), dim3(kExtendThreads), 0, stream>>>(batch, nexus_cu, keep_len, body_len, cache_len,
                                                                        row_cap, max_rows, total_new, ws, status);
  return hipGetLastError();
}

static unsigned extend_chunks(long rows, int row_pieces) {
  long chunks = (rows * row_pieces + kExtendThreads * 4 - 1) / (kExtendThreads * 4);
  if (chunks < 1) chunks = 1;
  if (chunks > 64) chunks = 64;
  return static_cast<unsigned>(chunks);
}

hipError_t launch_extend_stage(int batch, int max_rows, int Hkv, int D, const int32_t *keep_len,
                               const int32_t *body_len, const uint16_t *kc, const uint16_t *vc, const int64_t *row_off,
                               PrefillWs ws, uint16_t *k_stage, uint16_t *v_stage, const int32_t *status,
                               hipStream_t stream) {
  const int row_pieces = Hkv * D / 8;
  extend_stage_kernel<<<dim3(extend_chunks(max_rows, row_pieces), batch), dim3(kExtendThreads), 0, stream>>>(
      keep_len, body_len, kc, vc, row_off, ws, k_stage, v_stage, max_rows, row_pieces, status);
  return hipGetLastError();
}

hipError_t launch_extend_append(int batch, int max_new, int max_rows, int Hkv, int D, const int32_t *nexus_cu,
                                const int32_t *keep_len, uint16_t *kc, uint16_t *vc, const int64_t *row_off,
                                int32_t *cache_len, const uint16_t *k_new, const uint16_t *v_new, PrefillWs ws,
                                const uint16_t *k_stage, const uint16_t *v_stage, const int32_t *status,
                                hipStream_t stream) {
  const int row_pieces = Hkv * D / 8;
  const long rows = static_cast<long>(max_new) + (k_stage != nullptr ? max_rows : 0);
  extend_append_kernel<<<dim3(extend_chunks(rows, row_pieces), batch), dim3(kExtendThreads), 0, stream>>>(
      nexus_cu, keep_len, kc, vc, row_off, cache_len, k_new, v_new, ws, k_stage, v_stage, max_rows, row_pieces,
      status);
  return hipGetLastError();
}

}  // namespace sonic
