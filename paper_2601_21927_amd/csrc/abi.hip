// C ABI entry points: argument checks, workspace carving and kernel launches.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <vector>

#include "common.h"

namespace sonic {
hipError_t launch_plan(int batch, int total_tokens, int Hkv, int D, int nexus_scope, const int32_t *cu,
                       const uint8_t *role, const int32_t *turn, const uint16_t *k, const uint16_t *v, PrefillWs ws,
                       int32_t *status, hipStream_t stream);
hipError_t prefill_occupancy(int D, int G, bool stats, int ks, int *blocks);
hipError_t launch_recon(int batch, int total_tokens, int Dm, int max_rows, int num_cus, const int32_t *cu,
                        const uint8_t *role, const int32_t *turn, const uint16_t *h, PrefillWs ws,
                        int4 *items, float *target, float *cos_out, float *ratio_out,
                        int32_t *status, hipStream_t stream);
hipError_t launch_routed_gemm(int T, int K, int N, const uint8_t *role, const uint16_t *x, const uint16_t *w_text,
                              const uint16_t *w_nexus, float *y, int32_t *blk_nexus, int32_t *counts, int32_t *perm,
                              int32_t *status, hipStream_t stream);
hipError_t launch_key_weight(int batch, int T, int Hq, int Hkv, int D, int num_cus, const int32_t *cu,
                             const uint8_t *role, const uint16_t *q, const uint16_t *k, PrefillWs ws,
                             float scale_log2, float *w, int32_t *status, hipStream_t stream);
hipError_t launch_plan_extend(int batch, int total_new, int max_rows, const int32_t *nexus_cu,
                              const int32_t *keep_len, const int32_t *body_len, const int32_t *cache_len,
                              const int32_t *row_cap, PrefillWs ws, int32_t *status, hipStream_t stream);
hipError_t launch_extend_stage(int batch, int max_rows, int Hkv, int D, const int32_t *keep_len,
                               const int32_t *body_len, const uint16_t *kc, const uint16_t *vc, const int64_t *row_off,
                               PrefillWs ws, uint16_t *k_stage, uint16_t *v_stage, const int32_t *status,
                               hipStream_t stream);
hipError_t launch_extend_append(int batch, int max_new, int max_rows, int Hkv, int D, const int32_t *nexus_cu,
                                const int32_t *keep_len, uint16_t *kc, uint16_t *vc, const int64_t *row_off,
                                int32_t *cache_len, const uint16_t *k_new, const uint16_t *v_new, PrefillWs ws,
                                const uint16_t *k_stage, const uint16_t *v_stage, const int32_t *status,
                                hipStream_t stream);
hipError_t launch_prefill(int D, int G, int grid, bool stats, int ks, AttnRows rows, PrefillWs ws, int Hkv, float scale_log2,
                          hipStream_t stream);
hipError_t launch_compact(int batch, int total_tokens, int max_seqlen, int Hkv, int D, const int32_t *cu,
                          const uint8_t *role,
                          const uint16_t *k, const uint16_t *v, uint16_t *kc, uint16_t *vc, const int64_t *row_off,
                          const int32_t *row_cap, int32_t *cache_len, int32_t *keep_idx, int32_t *status,
                          hipStream_t stream);
int decode_splits(int batch, int Hkv, int max_ctx);
size_t decode_ws_layout(int batch, int Hkv, int G, int D, int nsplit, DecodeWs *ws, char *base);
size_t decode_scratch_layout(int batch, int Hkv, int G, int D, int nsplit, DecodeWs *ws, char *base);
hipError_t decode_scratch(hipStream_t stream, char **base);
hipError_t launch_decode(int batch, int Hq, int Hkv, int D, int max_ctx, int nsplit, uint16_t *kc,
                         uint16_t *vc, const int64_t *row_off, const int32_t *row_cap, int32_t *cache_len,
                         const uint8_t *row_role, const uint16_t *q, const uint16_t *k_new, const uint16_t *v_new,
                         float scale_log2, float *out, const DecodeWs &ws, int32_t *status, hipStream_t stream);

namespace {

constexpr int kAbiVersion = 10;
constexpr double kLog2e = 1.4426950408889634;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// softmax_scale == 0 selects the standard scaled dot-product attention scale 1/sqrt(d)
float default_scale(float scale, int d) { return scale == 0.f ? static_cast<float>(1.0 / std::sqrt(double(d))) : scale; }

bool debug_sync() {
  static const bool on = [] {
    const char *e = std::getenv("SONIC_DEBUG_SYNC");
    return e != nullptr && e[0] == '1';
  }();
  return on;
}

// Device facts needed for launch shapes, cached per device.
struct DeviceInfo {
  bool valid = false;
  int num_cus = 0;
  int prefill_blocks[2][2][9] = {};   // [statistics variant][D == 128][G]: resident workgroups per CU
  int prefill_ks2_blocks[2][9] = {};  // the same for the key-split variant, [D == 128][G <= 4]
};

std::mutex g_dev_mutex;
std::vector<DeviceInfo> g_dev;

hipError_t device_info(DeviceInfo **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_dev_mutex);
  if (static_cast<int>(g_dev.size()) <= dev) g_dev.resize(dev + 1);
  DeviceInfo &d = g_dev[dev];
  if (!d.valid) {
    e = hipDeviceGetAttribute(&d.num_cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    for (int st = 0; st < 2; ++st)
      for (int di = 0; di < 2; ++di)
        for (int G = 1; G <= 8; ++G) {
          int blocks = 0;
          e = prefill_occupancy(di ? 128 : 64, G, st != 0, 1, &blocks);
          if (e != hipSuccess) return e;
          d.prefill_blocks[st][di][G] = blocks > 0 ? blocks : 1;
          if (st == 0 && G <= 4) {
            e = prefill_occupancy(di ? 128 : 64, G, false, 2, &blocks);
            if (e != hipSuccess) return e;
            d.prefill_ks2_blocks[di][G] = blocks > 0 ? blocks : 1;
          }
        }
    d.valid = true;
  }
  *out = &d;
  return hipSuccess;
}

int32_t finish(hipError_t e, int32_t *dev_status, hipStream_t stream) {
  if (e != hipSuccess) return SONIC_ERR_HIP;
  if (debug_sync()) {
    if (hipStreamSynchronize(stream) != hipSuccess) return SONIC_ERR_HIP;
    int32_t st = 0;
    if (hipMemcpy(&st, dev_status, sizeof(st), hipMemcpyDeviceToHost) != hipSuccess) return SONIC_ERR_HIP;
    return st;
  }
  return SONIC_OK;
}

// ---------------------------------------------------------------- host grammar
struct HostSeg {
  int body_start, body_len, nexus_len;
};
struct HostParsed {
  int length = 0, system = 0, current = 0;
  std::vector<HostSeg> segs;
};

// Split one request per Eq.(1): SYSTEM* (TEXT+ NEXUS*)* CURRENT*, segment ids
// constant within a segment and strictly increasing across segments.
bool host_parse(const uint8_t *role, const int32_t *turn, int L, HostParsed *out) {
  out->length = L;
  out->segs.clear();
  int p = 0;
  while (p < L && role[p] == kSystem) ++p;
  out->system = p;
  bool have_prev = false;
  int prev_turn = 0;
  while (p < L && role[p] == kText) {
    const int t = turn[p];
    if (have_prev && t <= prev_turn) return false;
    const int b0 = p;
    while (p < L && role[p] == kText && turn[p] == t) ++p;
    const int n0 = p;
    while (p < L && role[p] == kNexus) {
      if (turn[p] != t) return false;
      ++p;
    }
    out->segs.push_back(HostSeg{b0, n0 - b0, p - n0});
    have_prev = true;
    prev_turn = t;
  }
  const int c0 = p;
  while (p < L && role[p] == kCurrent) ++p;
  if (p != L) return false;
  out->current = L - c0;
  return true;
}

}  // namespace
}  // namespace sonic

using namespace sonic;

extern "C" {

int32_t sonic_abi_version(void) { return kAbiVersion; }

const char *sonic_status_string(int32_t s) {
  switch (s) {
    case SONIC_OK: return "ok";
    case SONIC_ERR_INVALID_ARG: return "invalid argument";
    case SONIC_ERR_BAD_LAYOUT: return "role/turn_id layout breaks the augmented-sequence order";
    case SONIC_ERR_CAPACITY: return "cache capacity exceeded";
    case SONIC_ERR_WORKSPACE: return "workspace too small";
    case SONIC_ERR_UNSUPPORTED: return "unsupported shape";
    case SONIC_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t sonic_validate_layout_host(int32_t batch, const int32_t *cu, const uint8_t *role, const int32_t *turn_id,
                                   int32_t *bad_request) {
  if (batch < 0 || cu == nullptr || (batch > 0 && cu[batch] > 0 && (role == nullptr || turn_id == nullptr)))
    return SONIC_ERR_INVALID_ARG;
  if (cu[0] != 0) return SONIC_ERR_INVALID_ARG;
  HostParsed hp;
  for (int b = 0; b < batch; ++b) {
    if (cu[b + 1] < cu[b]) return SONIC_ERR_INVALID_ARG;
    if (!host_parse(role + cu[b], turn_id + cu[b], cu[b + 1] - cu[b], &hp)) {
      if (bad_request) *bad_request = b;
      return SONIC_ERR_BAD_LAYOUT;
    }
  }
  return SONIC_OK;
}

int32_t sonic_layout_stats_host(int32_t batch, const int32_t *cu, const uint8_t *role, const int32_t *turn_id,
                                int32_t nexus_scope, int64_t *visible_pairs, int32_t *kept_rows) {
  if (nexus_scope != SONIC_NEXUS_ALL && nexus_scope != SONIC_NEXUS_UP_TO_OWN) return SONIC_ERR_INVALID_ARG;
  int32_t bad = -1;
  const int32_t st = sonic_validate_layout_host(batch, cu, role, turn_id, &bad);
  if (st != SONIC_OK) return st;
  HostParsed hp;
  for (int b = 0; b < batch; ++b) {
    host_parse(role + cu[b], turn_id + cu[b], cu[b + 1] - cu[b], &hp);
    const int64_t S = hp.system, C = hp.current;
    int64_t k_tot = 0;
    for (const HostSeg &s : hp.segs) k_tot += s.nexus_len;
    // system rows: causal; body row r of segment i: S + (Nexus before i) + r + 1;
    // Nexus row of segment i: S + b_i + K_tot (own and earlier segments only:
    // S + b_i + (Nexus before i) + k_i); current row r: S + K_tot + r + 1.
    int64_t pairs = S * (S + 1) / 2 + C * (S + k_tot) + C * (C + 1) / 2;
    int64_t before = 0;
    for (const HostSeg &s : hp.segs) {
      const int64_t bl = s.body_len, kl = s.nexus_len;
      const int64_t nexus_keys = nexus_scope == SONIC_NEXUS_ALL ? k_tot : before + kl;
      pairs += bl * (S + before) + bl * (bl + 1) / 2 + kl * (S + bl + nexus_keys);
      before += kl;
    }
    if (visible_pairs) visible_pairs[b] = pairs;
    if (kept_rows) kept_rows[b] = static_cast<int32_t>(S + k_tot + C);
  }
  return SONIC_OK;
}

// ---------------------------------------------------------------- prefill
static size_t prefill_ws_layout(int32_t batch, int32_t T, int32_t Hq, int32_t Hkv, int32_t d, PrefillWs *ws,
                                char *base) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return base ? base + o : nullptr;
  };
  const size_t B1 = static_cast<size_t>(batch > 0 ? batch : 1);
  const size_t T1 = static_cast<size_t>(T > 0 ? T : 1);
  char *req = take(sizeof(ReqInfo) * B1);
  char *ppos = take(sizeof(int32_t) * T1);
  char *runs = take(sizeof(int2) * T1);
  char *tiles = take(sizeof(TileDesc) * T1);
  char *order = take(sizeof(int32_t) * T1);
  char *ctrl = take(sizeof(int32_t) * 16);
  const size_t rows_bytes = T1 * static_cast<size_t>(Hkv > 0 ? Hkv : 1) * static_cast<size_t>(d > 0 ? d : 1) * 2;
  char *kpre = take(rows_bytes);
  char *vpre = take(rows_bytes);
  // attention statistics
  char *lse = take(sizeof(float) * T1 * static_cast<size_t>(Hq > 0 ? Hq : 1));
  char *wpart = take(sizeof(float) * T1 * static_cast<size_t>(Hkv > 0 ? Hkv : 1));
  char *kblocks = take(sizeof(int2) * (T1 / 64 + B1 + 1));
  char *ncur = take(sizeof(int32_t) * B1);
  if (ws) {
    ws->req = reinterpret_cast<ReqInfo *>(req);
    ws->prefix_pos = reinterpret_cast<int32_t *>(ppos);
    ws->runs = reinterpret_cast<int2 *>(runs);
    ws->tiles = reinterpret_cast<TileDesc *>(tiles);
    ws->order = reinterpret_cast<int32_t *>(order);
    ws->ctrl = reinterpret_cast<int32_t *>(ctrl);
    ws->k_pre = reinterpret_cast<uint16_t *>(kpre);
    ws->v_pre = reinterpret_cast<uint16_t *>(vpre);
    ws->lse = reinterpret_cast<float *>(lse);
    ws->wpart = reinterpret_cast<float *>(wpart);
    ws->kblocks = reinterpret_cast<int2 *>(kblocks);
    ws->ncur = reinterpret_cast<int32_t *>(ncur);
  }
  return off;
}

size_t sonic_prefill_workspace_bytes(int32_t batch, int32_t total_tokens, int32_t num_q_heads, int32_t num_kv_heads,
                                     int32_t head_dim) {
  if (batch < 0 || total_tokens < 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0) return 0;
  return prefill_ws_layout(batch, total_tokens, num_q_heads, num_kv_heads, head_dim, nullptr, nullptr);
}

int32_t sonic_segment_attn_prefill(int32_t batch, int32_t total_tokens, int32_t Hq, int32_t Hkv, int32_t d,
                                   const int32_t *cu_seqlens, const uint8_t *role, const int32_t *turn_id,
                                   const void *q, const void *k, const void *v, float softmax_scale,
                                   int32_t nexus_scope, float *out, float *nexus_mass, float *key_weight,
                                   void *workspace, size_t workspace_bytes, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (batch < 0 || total_tokens < 0 || Hq <= 0 || Hkv <= 0 || dev_status == nullptr) return SONIC_ERR_INVALID_ARG;
  if (nexus_scope != SONIC_NEXUS_ALL && nexus_scope != SONIC_NEXUS_UP_TO_OWN) return SONIC_ERR_INVALID_ARG;
  if (d != 64 && d != 128) return SONIC_ERR_UNSUPPORTED;
  if (Hq % Hkv != 0) return SONIC_ERR_INVALID_ARG;
  const int G = Hq / Hkv;
  if (G > 8) return SONIC_ERR_UNSUPPORTED;
  if (!std::isfinite(softmax_scale) || softmax_scale < 0.f) return SONIC_ERR_INVALID_ARG;
  softmax_scale = default_scale(softmax_scale, d);
  if (batch == 0 || total_tokens == 0) return SONIC_OK;
  if (!cu_seqlens || !role || !turn_id || !q || !k || !v || !out || !workspace) return SONIC_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) || !aligned(workspace, 256) ||
      !aligned(nexus_mass, 4) || !aligned(key_weight, 4))
    return SONIC_ERR_INVALID_ARG;
  if (static_cast<size_t>(total_tokens) * Hq * d >= (size_t(1) << 40)) return SONIC_ERR_UNSUPPORTED;
  // K/V rows are addressed with 32-bit byte offsets inside one request
  if (static_cast<size_t>(total_tokens) * Hkv * d * 2 >= (size_t(1) << 32)) return SONIC_ERR_UNSUPPORTED;
  PrefillWs ws;
  const size_t need = prefill_ws_layout(batch, total_tokens, Hq, Hkv, d, &ws, static_cast<char *>(workspace));
  if (workspace_bytes < need) return SONIC_ERR_WORKSPACE;
  DeviceInfo *di = nullptr;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return SONIC_ERR_HIP;
  e = launch_plan(batch, total_tokens, Hkv, d, nexus_scope, cu_seqlens, role, turn_id,
                  static_cast<const uint16_t *>(k), static_cast<const uint16_t *>(v), ws, dev_status, stream);
  if (e != hipSuccess) return SONIC_ERR_HIP;
  const bool stats = nexus_mass != nullptr || key_weight != nullptr;
  int grid = di->num_cus * di->prefill_blocks[stats][d == 128][G];
  grid = (grid + kNumXcd - 1) / kNumXcd * kNumXcd;
  AttnRows rows{cu_seqlens, nullptr, static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k),
                static_cast<const uint16_t *>(v), ws.k_pre, ws.v_pre, out, nexus_mass, ws.lse};
  const float scale_log2 = static_cast<float>(softmax_scale * kLog2e);
  e = launch_prefill(d, G, grid, stats, 1, rows, ws, Hkv, scale_log2, stream);
  if (e == hipSuccess && key_weight != nullptr)
    e = launch_key_weight(batch, total_tokens, Hq, Hkv, d, di->num_cus, cu_seqlens, role,
                          static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k), ws, scale_log2,
                          key_weight, dev_status, stream);
  return finish(e, dev_status, stream);
}

// ---------------------------------------------------------------- next-turn Nexus step
// Workspace: the plan (per request, per new row), then the staging rows for the tail
// rows after a segment body (max_rows per request, K and V).
static size_t extend_ws_layout(int32_t batch, int32_t total_new, int32_t max_rows, size_t row_bytes, PrefillWs *ws,
                               uint16_t **k_stage, uint16_t **v_stage, char *base) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return base ? base + o : nullptr;
  };
  const size_t B1 = static_cast<size_t>(batch > 0 ? batch : 1);
  const size_t N1 = static_cast<size_t>(total_new > 0 ? total_new : 1);
  char *req = take(sizeof(ReqInfo) * B1);
  char *tiles = take(sizeof(TileDesc) * N1);
  char *order = take(sizeof(int32_t) * N1);
  char *ctrl = take(sizeof(int32_t) * 16);
  const size_t stage_bytes = B1 * static_cast<size_t>(max_rows > 0 ? max_rows : 1) * row_bytes;
  char *ks = take(stage_bytes);
  char *vs = take(stage_bytes);
  if (ws) {
    *ws = PrefillWs{};
    ws->req = reinterpret_cast<ReqInfo *>(req);
    ws->tiles = reinterpret_cast<TileDesc *>(tiles);
    ws->order = reinterpret_cast<int32_t *>(order);
    ws->ctrl = reinterpret_cast<int32_t *>(ctrl);
    *k_stage = reinterpret_cast<uint16_t *>(ks);
    *v_stage = reinterpret_cast<uint16_t *>(vs);
  }
  return off;
}

size_t sonic_nexus_extend_workspace_bytes(int32_t batch, int32_t total_new, int32_t max_rows, int32_t num_kv_heads,
                                          int32_t head_dim) {
  if (batch < 0 || total_new < 0 || max_rows < 0 || num_kv_heads <= 0 || head_dim <= 0) return 0;
  return extend_ws_layout(batch, total_new, max_rows, static_cast<size_t>(num_kv_heads) * head_dim * 2, nullptr,
                          nullptr, nullptr, nullptr);
}

int32_t sonic_nexus_extend(int32_t batch, int32_t total_new, int32_t Hq, int32_t Hkv, int32_t d, int32_t max_rows,
                           const int32_t *nexus_cu, const int32_t *keep_len, const int32_t *body_len, void *k_cache,
                           void *v_cache, const int64_t *cache_row_off, const int32_t *cache_row_cap,
                           int32_t *cache_len, const void *q, const void *k, const void *v, float softmax_scale,
                           float *out, void *workspace, size_t workspace_bytes, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (batch < 0 || total_new < 0 || Hq <= 0 || Hkv <= 0 || max_rows < 0 || dev_status == nullptr)
    return SONIC_ERR_INVALID_ARG;
  if (d != 64 && d != 128) return SONIC_ERR_UNSUPPORTED;
  if (Hq % Hkv != 0) return SONIC_ERR_INVALID_ARG;
  const int G = Hq / Hkv;
  if (G > 8) return SONIC_ERR_UNSUPPORTED;
  if (batch > 65535) return SONIC_ERR_UNSUPPORTED;
  if (!std::isfinite(softmax_scale) || softmax_scale < 0.f) return SONIC_ERR_INVALID_ARG;
  softmax_scale = default_scale(softmax_scale, d);
  if (batch == 0) return SONIC_OK;
  if (!nexus_cu || !keep_len || !k_cache || !v_cache || !cache_row_off || !cache_row_cap || !cache_len ||
      !workspace || (total_new > 0 && (!q || !k || !v || !out)))
    return SONIC_ERR_INVALID_ARG;
  if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) ||
      !aligned(out, 16) || !aligned(workspace, 256))
    return SONIC_ERR_INVALID_ARG;
  // cache and new rows are addressed with 32-bit byte offsets inside one request
  const size_t row_bytes = static_cast<size_t>(Hkv) * d * 2;
  if (static_cast<size_t>(max_rows) * row_bytes >= (size_t(1) << 32) ||
      static_cast<size_t>(total_new) * row_bytes >= (size_t(1) << 32))
    return SONIC_ERR_UNSUPPORTED;
  PrefillWs ws;
  uint16_t *k_stage = nullptr, *v_stage = nullptr;
  const size_t need = extend_ws_layout(batch, total_new, max_rows, row_bytes, &ws, &k_stage, &v_stage,
                                       static_cast<char *>(workspace));
  if (workspace_bytes < need) return SONIC_ERR_WORKSPACE;
  DeviceInfo *di = nullptr;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return SONIC_ERR_HIP;
  e = launch_plan_extend(batch, total_new, max_rows, nexus_cu, keep_len, body_len, cache_len, cache_row_cap, ws,
                         dev_status, stream);
  if (e != hipSuccess) return SONIC_ERR_HIP;
  if (body_len != nullptr) {
    // the tail rows after the body, staged before the cache update moves them
    e = launch_extend_stage(batch, max_rows, Hkv, d, keep_len, body_len, static_cast<const uint16_t *>(k_cache),
                            static_cast<const uint16_t *>(v_cache), cache_row_off, ws, k_stage, v_stage, dev_status,
                            stream);
    if (e != hipSuccess) return SONIC_ERR_HIP;
  }
  if (total_new > 0) {
    // Fewer work items than twice the CUs (the usual next turn: a few blocks of new
    // rows per request) would leave CUs idle: split each item's keys over two wave
    // groups of one workgroup instead.
    const int64_t item_bound = (static_cast<int64_t>(total_new + kTileRows - 1) / kTileRows + batch) * Hkv;
    const int ks = (G <= 4 && item_bound <= 2 * static_cast<int64_t>(di->num_cus)) ? 2 : 1;
    int grid = di->num_cus * (ks == 2 ? di->prefill_ks2_blocks[d == 128][G] : di->prefill_blocks[0][d == 128][G]);
    grid = (grid + kNumXcd - 1) / kNumXcd * kNumXcd;
    AttnRows rows{nexus_cu, cache_row_off, static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k),
                  static_cast<const uint16_t *>(v), static_cast<const uint16_t *>(k_cache),
                  static_cast<const uint16_t *>(v_cache), out};
    e = launch_prefill(d, G, grid, false, ks, rows, ws, Hkv, static_cast<float>(softmax_scale * kLog2e), stream);
    if (e != hipSuccess) return SONIC_ERR_HIP;
  }
  e = launch_extend_append(batch, total_new, max_rows, Hkv, d, nexus_cu, keep_len, static_cast<uint16_t *>(k_cache),
                           static_cast<uint16_t *>(v_cache), cache_row_off, cache_len,
                           static_cast<const uint16_t *>(k), static_cast<const uint16_t *>(v), ws,
                           body_len != nullptr ? k_stage : nullptr, body_len != nullptr ? v_stage : nullptr,
                           dev_status, stream);
  return finish(e, dev_status, stream);
}

// ---------------------------------------------------------------- role-routed projection
static size_t projection_ws_layout(int32_t T, char *base, int32_t **blk, int32_t **counts, int32_t **perm) {
  const size_t T1 = static_cast<size_t>(T > 0 ? T : 1);
  const size_t nblk = (T1 + 1023) / 1024;
  const size_t b_bytes = align_up(nblk * sizeof(int32_t), 256);
  const size_t c_bytes = 256;
  const size_t p_bytes = align_up(T1 * sizeof(int32_t), 256);
  if (base) {
    *blk = reinterpret_cast<int32_t *>(base);
    *counts = reinterpret_cast<int32_t *>(base + b_bytes);
    *perm = reinterpret_cast<int32_t *>(base + b_bytes + c_bytes);
  }
  return b_bytes + c_bytes + p_bytes;
}

size_t sonic_role_projection_workspace_bytes(int32_t total_tokens) {
  if (total_tokens < 0) return 0;
  return projection_ws_layout(total_tokens, nullptr, nullptr, nullptr, nullptr);
}

int32_t sonic_role_projection(int32_t T, int32_t K, int32_t N, const uint8_t *role, const void *x,
                              const void *w_text, const void *w_nexus, float *y, void *workspace,
                              size_t workspace_bytes, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (T < 0 || K <= 0 || N <= 0 || dev_status == nullptr) return SONIC_ERR_INVALID_ARG;
  if (K % 64 != 0) return SONIC_ERR_UNSUPPORTED;
  // operand rows are addressed by 32-bit byte offsets
  if (static_cast<uint64_t>(T) * K * 2 > 0xFFFFFFFFull || static_cast<uint64_t>(N) * K * 2 > 0xFFFFFFFFull)
    return SONIC_ERR_UNSUPPORTED;
  if (T == 0) return SONIC_OK;
  if (!role || !x || !w_text || !w_nexus || !y || !workspace) return SONIC_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(w_text, 16) || !aligned(w_nexus, 16) || !aligned(y, 4) ||
      !aligned(workspace, 256))
    return SONIC_ERR_INVALID_ARG;
  int32_t *blk = nullptr, *counts = nullptr, *perm = nullptr;
  if (workspace_bytes < projection_ws_layout(T, static_cast<char *>(workspace), &blk, &counts, &perm))
    return SONIC_ERR_WORKSPACE;
  const hipError_t e = launch_routed_gemm(T, K, N, role, static_cast<const uint16_t *>(x),
                                          static_cast<const uint16_t *>(w_text),
                                          static_cast<const uint16_t *>(w_nexus), y, blk, counts, perm, dev_status,
                                          stream);
  return finish(e, dev_status, stream);
}

// ---------------------------------------------------------------- reconstruction targets
static size_t recon_ws_layout(int32_t batch, int32_t T, PrefillWs *ws, int4 **items, char *base) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return base ? base + o : nullptr;
  };
  const size_t B1 = static_cast<size_t>(batch > 0 ? batch : 1);
  const size_t T1 = static_cast<size_t>(T > 0 ? T : 1);
  char *req = take(sizeof(ReqInfo) * B1);
  char *ppos = take(sizeof(int32_t) * T1);
  char *runs = take(sizeof(int2) * T1);
  char *tiles = take(sizeof(TileDesc) * T1);
  char *ctrl = take(sizeof(int32_t) * 16);
  char *it = take(sizeof(int4) * T1);
  if (ws) {
    *ws = PrefillWs{};
    ws->req = reinterpret_cast<ReqInfo *>(req);
    ws->prefix_pos = reinterpret_cast<int32_t *>(ppos);
    ws->runs = reinterpret_cast<int2 *>(runs);
    ws->tiles = reinterpret_cast<TileDesc *>(tiles);
    ws->ctrl = reinterpret_cast<int32_t *>(ctrl);
    *items = reinterpret_cast<int4 *>(it);
  }
  return off;
}

size_t sonic_nexus_recon_workspace_bytes(int32_t batch, int32_t total_tokens) {
  if (batch < 0 || total_tokens < 0) return 0;
  return recon_ws_layout(batch, total_tokens, nullptr, nullptr, nullptr);
}

int32_t sonic_nexus_recon_targets(int32_t batch, int32_t T, int32_t Dm, const int32_t *cu_seqlens,
                                  const uint8_t *role, const int32_t *turn_id, const void *h, int32_t max_rows,
                                  float *target, float *cos_target, float *entropy_ratio, void *workspace,
                                  size_t workspace_bytes, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (batch < 0 || T < 0 || Dm <= 0 || max_rows < 0 || dev_status == nullptr) return SONIC_ERR_INVALID_ARG;
  if (Dm % 8 != 0 || Dm > 16384) return SONIC_ERR_UNSUPPORTED;
  if (batch > 65535) return SONIC_ERR_UNSUPPORTED;
  if (batch == 0 || T == 0) return SONIC_OK;
  if (!cu_seqlens || !role || !turn_id || !h || !workspace || (max_rows > 0 && (!target || !cos_target ||
                                                                                  !entropy_ratio)))
    return SONIC_ERR_INVALID_ARG;
  if (!aligned(h, 16) || !aligned(target, 16) || !aligned(workspace, 256)) return SONIC_ERR_INVALID_ARG;
  PrefillWs ws;
  int4 *items = nullptr;
  if (workspace_bytes < recon_ws_layout(batch, T, &ws, &items, static_cast<char *>(workspace)))
    return SONIC_ERR_WORKSPACE;
  DeviceInfo *di = nullptr;
  hipError_t e = device_info(&di);
  if (e != hipSuccess) return SONIC_ERR_HIP;
  e = launch_recon(batch, T, Dm, max_rows, di->num_cus, cu_seqlens, role, turn_id, static_cast<const uint16_t *>(h),
                   ws, items, target, cos_target, entropy_ratio, dev_status, stream);
  return finish(e, dev_status, stream);
}

// ---------------------------------------------------------------- compaction
int32_t sonic_kv_compact(int32_t batch, int32_t total_tokens, int32_t max_seqlen, int32_t Hkv, int32_t d,
                         const int32_t *cu_seqlens, const uint8_t *role, const void *k, const void *v, void *k_cache,
                         void *v_cache, const int64_t *cache_row_off, const int32_t *cache_row_cap,
                         int32_t *cache_len, int32_t *keep_idx, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (batch < 0 || total_tokens < 0 || max_seqlen < 0 || Hkv <= 0 || dev_status == nullptr)
    return SONIC_ERR_INVALID_ARG;
  if (batch > 65535) return SONIC_ERR_UNSUPPORTED;
  if (d != 64 && d != 128) return SONIC_ERR_UNSUPPORTED;
  if (batch == 0) return SONIC_OK;
  if (!cu_seqlens || !cache_row_off || !cache_row_cap || !cache_len) return SONIC_ERR_INVALID_ARG;
  if (total_tokens > 0 && (!role || !k || !v || !k_cache || !v_cache || !keep_idx)) return SONIC_ERR_INVALID_ARG;
  if (total_tokens > 0 && (!aligned(role, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(k_cache, 16) ||
                           !aligned(v_cache, 16)))
    return SONIC_ERR_INVALID_ARG;
  hipError_t e = launch_compact(batch, total_tokens, max_seqlen, Hkv, d, cu_seqlens, role, static_cast<const uint16_t *>(k),
                                static_cast<const uint16_t *>(v), static_cast<uint16_t *>(k_cache),
                                static_cast<uint16_t *>(v_cache), cache_row_off, cache_row_cap, cache_len, keep_idx,
                                dev_status, stream);
  return finish(e, dev_status, stream);
}

// ---------------------------------------------------------------- decode
static size_t decode_ws_bytes(int32_t batch, int32_t Hq, int32_t d, int32_t nsplit) {
  // counters: per request, then per (request, kv-head) with Hkv <= Hq
  const size_t counters = align_up(static_cast<size_t>(batch) * sizeof(int32_t), 256) +
                          align_up(static_cast<size_t>(batch) * Hq * sizeof(int32_t), 256);
  const size_t records = nsplit > 1 ? static_cast<size_t>(batch) * Hq * nsplit * (d + 2) * sizeof(float) : 0;
  return counters + records;
}

size_t sonic_decode_workspace_bytes(int32_t batch, int32_t Hq, int32_t d, int32_t max_ctx) {
  if (batch <= 0 || Hq <= 0 || max_ctx <= 0) return 256;
  // enough for any kv-head count the call may use (Hkv dividing Hq, Hq / Hkv <= 8)
  int nsplit = 1;
  for (int hkv = 1; hkv <= Hq; ++hkv)
    if (Hq % hkv == 0 && Hq / hkv <= 8) nsplit = std::max(nsplit, decode_splits(batch, hkv, max_ctx));
  return align_up(decode_ws_bytes(batch, Hq, d, nsplit), 256);
}

// Argument checks shared by the two decode entry points.  Returns SONIC_OK with *empty set
// when there is nothing to do, or the status to return.
static int32_t check_decode(int32_t batch, int32_t Hq, int32_t Hkv, int32_t d, int32_t max_ctx, const void *k_cache,
                            const void *v_cache, const int64_t *cache_row_off, const int32_t *cache_row_cap,
                            const int32_t *cache_len, const void *q, const void *k_new, const void *v_new,
                            float *softmax_scale, const float *out, const int32_t *dev_status, bool *empty) {
  *empty = false;
  if (batch < 0 || Hq <= 0 || Hkv <= 0 || max_ctx <= 0 || dev_status == nullptr) return SONIC_ERR_INVALID_ARG;
  if (d != 64 && d != 128) return SONIC_ERR_UNSUPPORTED;
  if (Hq % Hkv != 0) return SONIC_ERR_INVALID_ARG;
  if (Hq / Hkv > 8) return SONIC_ERR_UNSUPPORTED;
  if (batch > 65535 || Hkv > 65535) return SONIC_ERR_UNSUPPORTED;
  if (!std::isfinite(*softmax_scale) || *softmax_scale < 0.f) return SONIC_ERR_INVALID_ARG;
  *softmax_scale = default_scale(*softmax_scale, d);
  if (batch == 0) {
    *empty = true;
    return SONIC_OK;
  }
  if (!k_cache || !v_cache || !cache_row_off || !cache_row_cap || !cache_len || !q || !k_new || !v_new || !out)
    return SONIC_ERR_INVALID_ARG;
  if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(q, 16) || !aligned(k_new, 16) ||
      !aligned(v_new, 16) || !aligned(out, 16))
    return SONIC_ERR_INVALID_ARG;
  return SONIC_OK;
}

int32_t sonic_compressed_decode(int32_t batch, int32_t Hq, int32_t Hkv, int32_t d, int32_t max_ctx, void *k_cache,
                                void *v_cache, const int64_t *cache_row_off, const int32_t *cache_row_cap,
                                int32_t *cache_len, const uint8_t *row_role, const void *q, const void *k_new,
                                const void *v_new, float softmax_scale, float *out, void *workspace,
                                size_t workspace_bytes, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  bool empty = false;
  const int32_t st = check_decode(batch, Hq, Hkv, d, max_ctx, k_cache, v_cache, cache_row_off, cache_row_cap,
                                  cache_len, q, k_new, v_new, &softmax_scale, out, dev_status, &empty);
  if (st != SONIC_OK || empty) return st;
  if (!workspace || !aligned(workspace, 256)) return SONIC_ERR_INVALID_ARG;
  const int nsplit = decode_splits(batch, Hkv, max_ctx);
  if (workspace_bytes < decode_ws_bytes(batch, Hq, d, nsplit)) return SONIC_ERR_WORKSPACE;
  DecodeWs ws;
  decode_ws_layout(batch, Hkv, Hq / Hkv, d, nsplit, &ws, static_cast<char *>(workspace));
  hipError_t e = launch_decode(batch, Hq, Hkv, d, max_ctx, nsplit, static_cast<uint16_t *>(k_cache),
                               static_cast<uint16_t *>(v_cache), cache_row_off, cache_row_cap, cache_len, row_role,
                               static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k_new),
                               static_cast<const uint16_t *>(v_new), static_cast<float>(softmax_scale * kLog2e), out,
                               ws, dev_status, stream);
  return finish(e, dev_status, stream);
}

int32_t sonic_compressed_decode_noalloc(int32_t batch, int32_t Hq, int32_t Hkv, int32_t d, int32_t max_ctx,
                                        void *k_cache, void *v_cache, const int64_t *cache_row_off,
                                        const int32_t *cache_row_cap, int32_t *cache_len, const uint8_t *row_role,
                                        const void *q, const void *k_new, const void *v_new, float softmax_scale,
                                        float *out, int32_t *dev_status, void *stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  bool empty = false;
  const int32_t st = check_decode(batch, Hq, Hkv, d, max_ctx, k_cache, v_cache, cache_row_off, cache_row_cap,
                                  cache_len, q, k_new, v_new, &softmax_scale, out, dev_status, &empty);
  if (st != SONIC_OK || empty) return st;
  const int nsplit = decode_splits(batch, Hkv, max_ctx);
  const size_t need = decode_scratch_layout(batch, Hkv, Hq / Hkv, d, nsplit, nullptr, nullptr);
  if (need == 0 || need > kScratchBytes) return SONIC_ERR_WORKSPACE;
  char *base = nullptr;
  hipError_t e = decode_scratch(stream, &base);
  if (e != hipSuccess) return SONIC_ERR_HIP;
  DecodeWs ws;
  decode_scratch_layout(batch, Hkv, Hq / Hkv, d, nsplit, &ws, base);
  e = launch_decode(batch, Hq, Hkv, d, max_ctx, nsplit, static_cast<uint16_t *>(k_cache),
                    static_cast<uint16_t *>(v_cache), cache_row_off, cache_row_cap, cache_len, row_role,
                    static_cast<const uint16_t *>(q), static_cast<const uint16_t *>(k_new),
                    static_cast<const uint16_t *>(v_new), static_cast<float>(softmax_scale * kLog2e), out, ws,
                    dev_status, stream);
  return finish(e, dev_status, stream);
}

}  // extern "C"
