// KV compaction: keep system, Nexus and current-query rows (Sec. 3, Fig. 2
// caption; Sec. 3.2 after Eq.(4)), dropping every history body row.
//
// Grid: (chunk of 1024 input tokens, request, slice); the slice count is chosen
// so that the launch has about 2048 workgroups.  Each workgroup
//   1. counts the kept tokens of its request before its chunk (16-byte role
//      loads, byte-wise compare, popcount, workgroup sum);
//   2. ranks the kept tokens of its chunk with wave ballots and an LDS scan
//      and lists their positions in LDS;
//   3. copies its slice of those rows (K and V, bitwise) with 16-byte vector
//      loads and stores; dropped rows are never read.
// Destination row = cache_row_off[b] + (kept before) + rank.  Rows past the
// request's capacity are not written; SONIC_ERR_CAPACITY is raised instead.
#include "common.h"
#include "scan.h"

namespace sonic {

constexpr int kCompactThreads = 256;
constexpr int kCompactChunk = 1024;   // input tokens per workgroup
constexpr int kCompactMaxSlices = 32; // workgroups sharing one chunk's copy (grid z)

// Kept (non-history-text) bytes of one 32-bit word, restricted to byte lanes [lo, hi).
__device__ __forceinline__ int kept_bytes(uint32_t w, int lo, int hi) {
  int c = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int byte = (w >> (8 * j)) & 0xFF;
    c += (j >= lo && j < hi && byte != kText) ? 1 : 0;
  }
  return c;
}

// Kept tokens among role[a, e) (absolute byte positions), summed over the workgroup.
__device__ int count_kept(const uint8_t *__restrict__ role, long a, long e, int *lds) {
  int c = 0;
  if (e > a) {
    const long w0 = a & ~15L;                       // first 16-byte word touching [a, e)
    const long nwords = ((e + 15) & ~15L) - w0;     // bytes spanned by whole words
    for (long off = static_cast<long>(threadIdx.x) * 16; off < nwords; off += kCompactThreads * 16) {
      const long wb = w0 + off;
      // The aligned 16-byte word holds at least one byte of [a, e), so it lies on a mapped page.
      const u32x4 x = *reinterpret_cast<const u32x4 *>(role + wb);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const long db = wb + 4 * i;
        const int lo = static_cast<int>(max(0L, min(4L, a - db)));
        const int hi = static_cast<int>(max(0L, min(4L, e - db)));
        c += kept_bytes(x[i], lo, hi);
      }
    }
  }
  int total;
  block_int_scan<kCompactThreads>(c, &total, lds);
  return total;
}

template <int D>
__global__ __launch_bounds__(kCompactThreads) void compact_kernel(
    const int32_t *__restrict__ cu, const uint8_t *__restrict__ role, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, uint16_t *__restrict__ kc, uint16_t *__restrict__ vc,
    const int64_t *__restrict__ row_off, const int32_t *__restrict__ row_cap, int32_t *__restrict__ cache_len,
    int32_t *__restrict__ keep_idx, int32_t *status, int total_tokens, int Hkv) {
  __shared__ int lds[kCompactThreads / kWave + 1];
  __shared__ int16_t kept_pos[kCompactChunk];
  __shared__ int s_ok;
  if (!block_status_clear(status, &s_ok)) return;
  const int chunk = blockIdx.x;
  const int b = blockIdx.y;
  const int slice = blockIdx.z;
  const int s = cu[b];
  const int e = cu[b + 1];
  if (s < 0 || e < s || e > total_tokens) {   // cu_seqlens itself is malformed
    if (threadIdx.x == 0) raise_status(status, SONIC_ERR_BAD_LAYOUT);
    return;
  }
  const int L = e - s;
  const int nchunks = (L + kCompactChunk - 1) / kCompactChunk;
  if (chunk >= max(nchunks, 1)) return;
  const int c0 = chunk * kCompactChunk;

  const int before = count_kept(role, s, s + min(c0, L), lds);

  // rank the kept tokens of this chunk: thread t looks at tokens c0 + 4t .. 4t+3
  constexpr int PER = kCompactChunk / kCompactThreads;
  bool keep[PER];
  int mine = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int i = c0 + PER * threadIdx.x + j;
    keep[j] = i < L && role[s + i] != kText;
    mine += keep[j];
  }
  int chunk_kept;
  int rank = block_int_scan<kCompactThreads>(mine, &chunk_kept, lds);
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    if (keep[j]) kept_pos[rank++] = static_cast<int16_t>(PER * threadIdx.x + j);
  }
  __syncthreads();

  const int cap = row_cap[b];
  const int64_t dst0 = row_off[b] + before;
  if (chunk == max(nchunks, 1) - 1 && slice == 0 && threadIdx.x == 0) {
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
  const int total = (jend - j0) * row_units;
  for (int u = threadIdx.x; u < total; u += kCompactThreads) {
    const int j = j0 + u / row_units;
    const int w = u % row_units;
    const size_t src = (static_cast<size_t>(s) + c0 + kept_pos[j]) * row_units + w;
    const size_t dst = static_cast<size_t>(dst0 + j) * row_units + w;
    const u32x4 ku = reinterpret_cast<const u32x4 *>(k)[src];
    const u32x4 vu = reinterpret_cast<const u32x4 *>(v)[src];
    reinterpret_cast<u32x4 *>(kc)[dst] = ku;
    reinterpret_cast<u32x4 *>(vc)[dst] = vu;
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
