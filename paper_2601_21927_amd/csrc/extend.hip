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

namespace sonic {

constexpr int kExtendThreads = 256;

// One workgroup per request: check the lengths, then one descriptor per block of
// up to 32 new Nexus rows.  ReqInfo.nruns carries the number of tail rows after
// the body to the cache update.
__global__ __launch_bounds__(kExtendThreads) void plan_extend_kernel(
    const int32_t *__restrict__ nexus_cu, const int32_t *__restrict__ keep_len, const int32_t *__restrict__ body_len,
    const int32_t *__restrict__ cache_len, const int32_t *__restrict__ row_cap, int max_rows, int total_new,
    PrefillWs ws, int32_t *status) {
  const int b = blockIdx.x;
  const int s = nexus_cu[b];
  const int e = nexus_cu[b + 1];
  const int len = cache_len[b];
  const int keep = keep_len[b];
  const int cap = row_cap[b];
  const int body = body_len != nullptr ? body_len[b] : len - keep;
  bool bad = s < 0 || e < s || e > total_new || keep < 0 || keep > len || len > cap || len > max_rows;
  bad = bad || body < 0 || body > len - keep;
  const int kn = bad ? 0 : e - s;
  const int rest = bad ? 0 : len - keep - body;
  if (bad || keep + kn + rest > cap) {
    if (threadIdx.x == 0) {
      raise_status(status, bad ? SONIC_ERR_BAD_LAYOUT : SONIC_ERR_CAPACITY);
      ws.req[b] = ReqInfo{0, 0, 0, 0, 0, 0};
    }
    return;
  }
  const int nt = (kn + kTileRows - 1) / kTileRows;
  for (int j = threadIdx.x; j < nt; j += kExtendThreads) {
    TileDesc d;
    d.req = b;
    d.p0 = j * kTileRows;
    d.nrows = min(kTileRows, kn - d.p0);
    d.npre = keep + body;  // the kept cache rows and the segment's body
    d.seg_start = 0;       // then every new Nexus row, no causal part
    d.seg_len = kn;
    d.ndiag = 0;
    d.pad = 0;
    ws.tiles[s + j] = d;
  }
  // every block of the request costs the same: all keep + body + kn keys
  const int64_t cost = static_cast<int64_t>(nt) * ((keep + body + kn + kKeyChunk - 1) / kKeyChunk);
  if (threadIdx.x == 0) ws.req[b] = ReqInfo{nt, 0, kn, rest, cost, 0};
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

hipError_t launch_plan_order(int batch, const int32_t *cu, PrefillWs ws, int32_t *status, hipStream_t stream);

hipError_t launch_plan_extend(int batch, int total_new, int max_rows, const int32_t *nexus_cu,
                              const int32_t *keep_len, const int32_t *body_len, const int32_t *cache_len,
                              const int32_t *row_cap, PrefillWs ws, int32_t *status, hipStream_t stream) {
  plan_extend_kernel<<<dim3(batch), dim3(kExtendThreads), 0, stream>>>(nexus_cu, keep_len, body_len, cache_len,
                                                                        row_cap, max_rows, total_new, ws, status);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_plan_order(batch, nexus_cu, ws, status, stream);
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
