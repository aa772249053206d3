// Masked prefill attention (Sec. 3.2) on gfx950 matrix cores.
//
// Work item = (descriptor, kv-head).  A workgroup holds G waves, one per q-head
// of the kv-head's group, so every K/V block staged in LDS serves G heads.
// Each wave owns the 32 query rows of its descriptor for one q-head and walks
// the descriptor's visible keys in steps of 64:
//
//   S^T (64 keys x 32 rows)   = K . Q^T   v_mfma_f32_32x32x16_bf16, fp32 accumulate
//   online softmax over keys  (fp32, exp2 with log2(e) folded into the scale)
//   O^T (d x 32 rows)        += V^T . P^T  v_mfma_f32_32x32x16_bf16, P rounded to bf16
//
// Computing the transposed products leaves each lane with one query row
// (lane % 32) in every accumulator, so row maxima and sums need a single
// cross-lane exchange (lane ^ 32) and rescaling needs no exchange at all.
//
// Only the last one or two 64-key steps of a descriptor can hold masked
// entries (the ragged end of the key list and the causal diagonal); all
// earlier steps are fully visible and skip the predicate.
//
// The grid is persistent: workgroup w serves the queue of XCD (w mod 8); item i
// belongs to queue i mod 8, and items are ordered so that one queue sees one
// kv-head (Hkv = 8) or a fixed subset of kv-heads, which keeps the K/V a queue
// streams inside one XCD's L2.  Queues are filled most-expensive-first.
#include "common.h"

namespace sonic {

// MFMA row m of a 32-key block holds key perm32(m) (bits 2 and 3 swapped), so
// that accumulator element v of lane half g maps to key 8g+v (v < 8) and
// 16+8g+(v-8) (v >= 8): eight consecutive keys per half, which is exactly the
// K-operand layout the P.V product needs.  The permutation is an involution.
__device__ __forceinline__ int perm32(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

__device__ __forceinline__ int acc_key(int v, int g) { return v < 8 ? 8 * g + v : 16 + 8 * g + (v - 8); }

__device__ __forceinline__ int virtual_to_pos(const TileDesc &t, const int32_t *__restrict__ npos, int vk) {
  if (vk < t.r0_end) return vk;
  vk -= t.r0_end;
  if (vk < t.nx) return npos[vk];
  vk -= t.nx;
  if (vk < t.r1_len) return t.r1_start + vk;
  return t.p0 + (vk - t.r1_len);
}

template <int D, int G>
__global__ __launch_bounds__(G * kWave, 2) void prefill_kernel(const int32_t *__restrict__ cu,
                                                            const uint16_t *__restrict__ q,
                                                            const uint16_t *__restrict__ k,
                                                            const uint16_t *__restrict__ v, float *__restrict__ out,
                                                            PrefillWs ws, int Hkv, float scale_log2) {
  constexpr int NT = G * kWave;
  constexpr int DC = D / 8;    // 16-byte chunks per K row
  constexpr int DS = D / 16;   // d steps of the S product
  constexpr int DB = D / 32;   // 32-wide d blocks of the output
  __shared__ __align__(16) uint16_t k_lds[kKeyChunk * D];   // [64 keys][D], chunk-swizzled
  __shared__ __align__(16) uint16_t vt_lds[D * kKeyChunk];  // [D][64 keys], chunk-swizzled
  __shared__ int s_item;

  const int Hq = Hkv * G;
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int n = lane & 31;
  const int g = lane >> 5;
  const int xcd = blockIdx.x % kNumXcd;
  const int nitems = ws.ctrl[0] * Hkv;

  for (;;) {
    if (threadIdx.x == 0) s_item = atomicAdd(&ws.ctrl[8 + xcd], 1) * kNumXcd + xcd;
    __syncthreads();
    const int item = s_item;
    __syncthreads();
    if (item >= nitems) break;
    const int slot = ws.order[item / Hkv];
    const int kvh = item % Hkv;
    const TileDesc t = ws.tiles[slot];
    const int base = cu[t.req];
    const int32_t *npos = ws.nexus_pos + base;
    const int h = kvh * G + wave;
    const int nv = tile_key_count(t);
    const int nF = nv - t.ndiag;

    // Q^T fragments (B operand): lane (row n, half g) holds d = 16*ds + 8*g .. +7.
    bf16x8 qf[DS];
    {
      const bool ok = n < t.nrows;
      const uint16_t *qrow = q + (static_cast<size_t>(base + t.p0 + n) * Hq + h) * D;
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) {
        u32x4 w = {0u, 0u, 0u, 0u};
        if (ok) w = *reinterpret_cast<const u32x4 *>(qrow + 16 * ds + 8 * g);
        qf[ds] = __builtin_bit_cast(bf16x8, w);
      }
    }

    f32x16 oacc[DB];
#pragma unroll
    for (int i = 0; i < DB; ++i) oacc[i] = f32x16{};
    float m_run = -INFINITY;
    float l_run = 0.f;

    const int nchunks = (nv + kKeyChunk - 1) / kKeyChunk;
    for (int c = 0; c < nchunks; ++c) {
      const int vk0 = c * kKeyChunk;
      // ---- stage K (row-major, MFMA row order) and V^T into LDS ----
      for (int task = threadIdx.x; task < kKeyChunk * DC; task += NT) {
        const int r = task / DC;
        const int cc = task % DC;
        const int vk = vk0 + r;
        u32x4 w = {0u, 0u, 0u, 0u};
        if (vk < nv) {
          const int p = virtual_to_pos(t, npos, vk);
          w = *reinterpret_cast<const u32x4 *>(k + (static_cast<size_t>(base + p) * Hkv + kvh) * D + cc * 8);
        }
        const int m = (r & 32) | perm32(r & 31);
        *reinterpret_cast<u32x4 *>(k_lds + (m * DC + (cc ^ (m & 7))) * 8) = w;
      }
      for (int task = threadIdx.x; task < 8 * DC; task += NT) {
        const int dg = task % DC;   // 8 consecutive d
        const int kg = task / DC;   // 8 consecutive keys
        u32x4 rows[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int vk = vk0 + kg * 8 + i;
          rows[i] = u32x4{0u, 0u, 0u, 0u};
          if (vk < nv) {
            const int p = virtual_to_pos(t, npos, vk);
            rows[i] = *reinterpret_cast<const u32x4 *>(v + (static_cast<size_t>(base + p) * Hkv + kvh) * D + dg * 8);
          }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {   // d = 8*dg + j: gather element j of the 8 keys
          u32x4 o;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const uint32_t a = rows[2 * u][j >> 1];
            const uint32_t bb = rows[2 * u + 1][j >> 1];
            o[u] = (j & 1) ? ((a >> 16) | (bb & 0xFFFF0000u)) : ((a & 0xFFFFu) | (bb << 16));
          }
          const int dr = dg * 8 + j;
          *reinterpret_cast<u32x4 *>(vt_lds + (dr * 8 + (kg ^ (dr & 7))) * 8) = o;
        }
      }
      __syncthreads();

      // ---- S^T = K . Q^T for two 32-key blocks ----
      f32x16 sacc[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        sacc[kb] = f32x16{};
        const int m = kb * 32 + n;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
          const bf16x8 a = *reinterpret_cast<const bf16x8 *>(k_lds + (m * DC + ((2 * ds + g) ^ (m & 7))) * 8);
          sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ds], sacc[kb], 0, 0, 0);
        }
      }

      // ---- mask (ragged end / causal diagonal only), online softmax ----
      const bool need_mask = vk0 + kKeyChunk > nF;
      float mloc = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          float x = sacc[kb][e] * scale_log2;
          if (need_mask) {
            const int vk = vk0 + kb * 32 + acc_key(e, g);
            const bool vis = vk < nF || (vk < nv && vk - nF <= n);
            x = vis ? x : -INFINITY;
          }
          sacc[kb][e] = x;
          mloc = fmaxf(mloc, x);
        }
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
      const float m_new = fmaxf(m_run, mloc);
      const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      float lsum = 0.f;
      bf16x8 pb[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x8 lo, hi;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          lo[e] = __builtin_amdgcn_exp2f(sacc[kb][e] - m_new);
          hi[e] = __builtin_amdgcn_exp2f(sacc[kb][8 + e] - m_new);
          lsum += lo[e] + hi[e];
        }
        pb[2 * kb] = __builtin_convertvector(lo, bf16x8);
        pb[2 * kb + 1] = __builtin_convertvector(hi, bf16x8);
      }
      l_run = l_run * corr + lsum;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] *= corr;

      // ---- O^T += V^T . P^T ----
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int dr = db * 32 + n;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const bf16x8 a = *reinterpret_cast<const bf16x8 *>(vt_lds + (dr * 8 + ((2 * ks + g) ^ (dr & 7))) * 8);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[db], 0, 0, 0);
        }
      }
      __syncthreads();
    }

    // ---- normalise and store: lane (n, g) holds d = 32*db + 8*i + 4*g + (0..3) ----
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    const float inv = 1.f / l_tot;
    if (n < t.nrows) {
      float *orow = out + (static_cast<size_t>(base + t.p0 + n) * Hq + h) * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f32x4 o = {oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv, oacc[db][4 * i + 2] * inv,
                     oacc[db][4 * i + 3] * inv};
          *reinterpret_cast<f32x4 *>(orow + db * 32 + 8 * i + 4 * g) = o;
        }
      }
    }
  }
}

template <int D, int G>
static hipError_t launch_prefill_dg(int grid, const int32_t *cu, const uint16_t *q, const uint16_t *k,
                                    const uint16_t *v, float *out, PrefillWs ws, int Hkv, float scale_log2,
                                    hipStream_t stream) {
  prefill_kernel<D, G><<<dim3(grid), dim3(G * kWave), 0, stream>>>(cu, q, k, v, out, ws, Hkv, scale_log2);
  return hipGetLastError();
}

template <int D, int G>
static hipError_t occupancy_dg(int *blocks) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, prefill_kernel<D, G>, G * kWave, 0);
}

#define SONIC_FOR_G(D, X) \
  switch (G) {            \
    case 1: X(D, 1); break; \
    case 2: X(D, 2); break; \
    case 3: X(D, 3); break; \
    case 4: X(D, 4); break; \
    case 5: X(D, 5); break; \
    case 6: X(D, 6); break; \
    case 7: X(D, 7); break; \
    case 8: X(D, 8); break; \
    default: return hipErrorInvalidValue; \
  }

hipError_t prefill_occupancy(int D, int G, int *blocks) {
#define OCC(DD, GG) return occupancy_dg<DD, GG>(blocks)
  if (D == 64) {
    SONIC_FOR_G(64, OCC)
  } else if (D == 128) {
    SONIC_FOR_G(128, OCC)
  }
#undef OCC
  return hipErrorInvalidValue;
}

hipError_t launch_prefill(int D, int G, int grid, const int32_t *cu, const uint16_t *q, const uint16_t *k,
                          const uint16_t *v, float *out, PrefillWs ws, int Hkv, float scale_log2,
                          hipStream_t stream) {
#define LAUNCH(DD, GG) return launch_prefill_dg<DD, GG>(grid, cu, q, k, v, out, ws, Hkv, scale_log2, stream)
  if (D == 64) {
    SONIC_FOR_G(64, LAUNCH)
  } else if (D == 128) {
    SONIC_FOR_G(128, LAUNCH)
  }
#undef LAUNCH
  return hipErrorInvalidValue;
}

}  // namespace sonic
