// KV compaction: keep system, Nexus and current-query rows (Sec. 3, Fig. 2
// caption; Sec. 3.2 after Eq.(4)), dropping every history body row.
//
// Grid: (chunk of 1024 input tokens, request, slice); the slice count is chosen
// so that the launch has about 2048 workgroups.  Each workgroup
//   1. requests the status word, the request's bounds, first cache row and
//      capacity together;
//   2. requests every role byte it needs at once: the request's tokens before its
//      chunk (16-byte loads, counted four bytes at a time) and its own chunk's
//      (four per thread, in rank order);
//   3. sums the first and ranks the second in one two-value workgroup scan, and
//      lists the chunk's kept positions in LDS;
//   4. copies its slice of those rows (K and V, bitwise), every load of a
//      thread's batch in flight before its stores; dropped rows are never read.
// So a workgroup waits for three memory round trips (bounds, roles, rows), and
// the role bytes a request shares between its chunks are served from L2.
// Destination row = cache_row_off[b] + (kept before) + rank.  Rows past the
// request's capacity are not written; SONIC_ERR_CAPACITY is raised instead.
// role is read only inside its total_tokens bytes.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kCompactThreads = 256;
constexpr int kCompactChunk = 1024;   // input tokens per workgroup
constexpr int kCompactMaxSlices = 32; // workgroups sharing one chunk's copy (grid z)
constexpr int kCountUnroll = 8;       // 16-byte role loads in flight per thread
constexpr int kCopyUnroll = 4;        // 16-byte K and V units in flight per thread

// Kept (not HISTORY_TEXT) bytes of a 32-bit word among its byte lanes [lo, hi).
// Bytes outside the lanes are replaced by the text code; then a byte is dropped
// exactly when it equals the text code, i.e. when y = w ^ 0x01010101 has a zero
// byte, counted with the exact zero-byte test ((y & 7f..) + 7f..) | y.
__device__ __forceinline__ int kept_in_dword(uint32_t w, int lo, int hi) {
  const uint32_t m = static_cast<uint32_t>(((1ull << (8 * hi)) - 1) & ~((1ull << (8 * lo)) - 1));
  const uint32_t x = (w & m) | (0x01010101u & ~m);
  const uint32_t y = x ^ 0x01010101u;
  const uint32_t zero_hi = ~(((y & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | y) & 0x80808080u;
  return 4 - __popc(zero_hi);
}

template <int D>
__global__ __launch_bounds__(kCompactThreads) void compact_kernel(
    const int32_t *__restrict__ cu, const uint8_t *__restrict__ role, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, uint16_t *__restrict__ kc, uint16_t *__restrict__ vc,
    const int64_t *__restrict__ row_off, const int32_t *__restrict__ row_cap, int32_t *__restrict__ cache_len,
    int32_t *__restrict__ keep_idx, int32_t *status, int total_tokens, int Hkv) {
  __shared__ int lds[2 * (kCompactThreads / kWave)];
  __shared__ int16_t kept_pos[kCompactChunk];
  __shared__ int s_ok;
  const int chunk = blockIdx.x;
  const int b = blockIdx.y;
  const int slice = blockIdx.z;
  // one round trip: status, bounds, first cache row and capacity
  const int s = cu[b];
  const int e = cu[b + 1];
  const int cap = row_cap[b];
  const int64_t off0 = row_off[b];
  if (threadIdx.x == 0) s_ok = __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0;
  __syncthreads();
  if (!s_ok) return;
  if (s < 0 || e < s || e > total_tokens) {   // cu_seqlens itself is malformed
    if (threadIdx.x == 0) raise_status(status, SONIC_ERR_BAD_LAYOUT);
    return;
  }
  const int L = e - s;
  const int nchunks = max((L + kCompactChunk - 1) / kCompactChunk, 1);
  if (nchunks > static_cast<int>(gridDim.x)) {
    // max_seqlen understated this request's length: none of its chunks copies anything
    if (chunk == 0 && slice == 0 && threadIdx.x == 0) raise_status(status, SONIC_ERR_INVALID_ARG);
    return;
  }
  if (chunk >= nchunks) return;
  const int c0 = chunk * kCompactChunk;

  // ---- kept tokens before the chunk: role bytes [s, s + c0) in 16-byte words ----
  int before_part = 0;
  {
    const long a = s, z = static_cast<long>(s) + c0;
    const long w_lo = a & ~15L;
    const long w_hi = (z + 15) & ~15L;
    for (long base = w_lo + 16L * threadIdx.x; base < w_hi; base += 16L * kCompactThreads * kCountUnroll) {
      u32x4 x[kCountUnroll];
#pragma unroll
      for (int i = 0; i < kCountUnroll; ++i) {
        const long wb = base + 16L * kCompactThreads * i;
        x[i] = u32x4{0x01010101u, 0x01010101u, 0x01010101u, 0x01010101u};
        if (wb + 16 <= total_tokens) {
          if (wb < w_hi) x[i] = *reinterpret_cast<const u32x4 *>(role + wb);
        } else if (wb < w_hi) {   // the array's last, partial word: byte loads inside the array
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (wb + j < total_tokens)
              x[i][j / 4] = (x[i][j / 4] & ~(0xFFu << (8 * (j % 4)))) |
                            (static_cast<uint32_t>(role[wb + j]) << (8 * (j % 4)));
        }
      }
#pragma unroll
      for (int i = 0; i < kCountUnroll; ++i) {
        const long wb = base + 16L * kCompactThreads * i;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const long db = wb + 4 * j;
          const int lo = static_cast<int>(max(0L, min(4L, a - db)));
          const int hi = static_cast<int>(max(0L, min(4L, z - db)));
          before_part += kept_in_dword(x[i][j], lo, hi);
        }
      }
    }
  }
  // ---- this chunk: thread t looks at tokens c0 + 4t .. 4t+3 ----
  constexpr int PER = kCompactChunk / kCompactThreads;
  bool keep[PER];
  int mine = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int i = c0 + PER * threadIdx.x + j;
    keep[j] = i < L && role[s + i] != kText;
    mine += keep[j];
  }
  int x2[2] = {before_part, mine}, below[2], total[2];
  block_int_scan_n<kCompactThreads, 2>(x2, below, total, lds);
  const int before = total[0];
  const int chunk_kept = total[1];
  int rank = below[1];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    if (keep[j]) kept_pos[rank++] = static_cast<int16_t>(PER * threadIdx.x + j);
  }
  __syncthreads();

  const int64_t dst0 = off0 + before;
  if (chunk == nchunks - 1 && slice == 0 && threadIdx.x == 0) {
    const int n = before + chunk_kept;
    if (n > cap) raise_status(status, SONIC_ERR_CAPACITY);
    else cache_len[b] = n;
  }
  const int slices = gridDim.z;
  const int per_slice = (chunk_kept + slices - 1) / slices;
  const int j0 = slice * per_slice;
  const int j1 = min(chunk_kept, j0 + per_slice);
  const int room = cap - before;   // ranks >= room would overflow the request's rows
  const int jend = min(j1, room);
  if (j1 > room && j0 < j1 && threadIdx.x == 0) raise_status(status, SONIC_ERR_CAPACITY);
  if (jend <= j0) return;

  constexpr int UNITS = D / 8;                 // 16-byte units per head row
  const int row_units = Hkv * UNITS;           // 16-byte units per token row
  for (int j = j0 + threadIdx.x; j < jend; j += kCompactThreads) keep_idx[dst0 + j] = c0 + kept_pos[j];
  const int nunits = (jend - j0) * row_units;
  const u32x4 *ks = reinterpret_cast<const u32x4 *>(k);
  const u32x4 *vs = reinterpret_cast<const u32x4 *>(v);
  u32x4 *kd = reinterpret_cast<u32x4 *>(kc);
  u32x4 *vd = reinterpret_cast<u32x4 *>(vc);
  for (int u0 = threadIdx.x; u0 < nunits; u0 += kCompactThreads * kCopyUnroll) {
    u32x4 ku[kCopyUnroll], vu[kCopyUnroll];
    size_t dst[kCopyUnroll];
#pragma unroll
    for (int i = 0; i < kCopyUnroll; ++i) {
      const int u = u0 + i * kCompactThreads;
      if (u < nunits) {
        const int j = j0 + u / row_units;
        const int w = u % row_units;
        const size_t src = (static_cast<size_t>(s) + c0 + kept_pos[j]) * row_units + w;
        dst[i] = static_cast<size_t>(dst0 + j) * row_units + w;
        ku[i] = ks[src];
        vu[i] = vs[src];
      }
    }
#pragma unroll
    for (int i = 0; i < kCopyUnroll; ++i) {
      if (u0 + i * kCompactThreads < nunits) {
        kd[dst[i]] = ku[i];
        vd[dst[i]] = vu[i];
      }
    }
  }
}

hipError_t launch_compact(int batch, int total_tokens, int max_seqlen, int Hkv, int D, const int32_t *cu,
                          const uint8_t *role,
                          const uint16_t *k, const uint16_t *v, uint16_t *kc, uint16_t *vc, const int64_t *row_off,
                          const int32_t *row_cap, int32_t *cache_len, int32_t *keep_idx, int32_t *status,
                          hipStream_t stream) {
  const int chunks = max(1, (max_seqlen + kCompactChunk - 1) / kCompactChunk);
  const long cb = static_cast<long>(chunks) * batch;
  const int slices = static_cast<int>(max(1L, min(static_cast<long>(kCompactMaxSlices), (2048 + cb - 1) / cb)));
  dim3 grid(chunks, batch, slices);
  if (D == 64)
    compact_kernel<64><<<grid, dim3(kCompactThreads), 0, stream>>>(cu, role, k, v, kc, vc, row_off, row_cap,
                                                                   cache_len, keep_idx, status, total_tokens, Hkv);
  else if (D == 128)
    compact_kernel<128><<<grid, dim3(kCompactThreads), 0, stream>>>(cu, role, k, v, kc, vc, row_off, row_cap,
                                                                    cache_len, keep_idx, status, total_tokens, Hkv);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sonic
