// hwkv_api.hip -- host side of the C ABI declared in include/hwkv.h:
// policy validation and accounting, grouped-cache layout and allocation, the
// host mirror of sequence lengths, argument validation (always before any
// device work, no state change on error), and the per-call work tables the
// kernels consume.
#include "hwkv.h"

#include <algorithm>
#include <cerrno>
#include <cinttypes>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "hwkv_internal.h"

struct hwkv_policy {
  int32_t n_layers = 0, n_kv_heads = 0, n_q_heads = 0, head_dim = 0;
  int32_t n_sinks = 0, n_levels = 0;
  std::vector<int64_t> level_window;  // 0 = full
  std::vector<int32_t> level_of_unit; // [n_layers * n_kv_heads]
};

struct hwkv_cache {
  hwkv_policy pol;
  int32_t batch = 0;
  int64_t max_ctx = 0;
  // per unit u = layer * n_kv_heads + h
  std::vector<int64_t> window;   // canonical: 0 = full (incl. S + w >= max_ctx)
  std::vector<int64_t> cap;      // rows holding data
  std::vector<int64_t> cap_pad;  // rows allocated (multiple of 64)
  std::vector<int64_t> k_off;    // element offset of (u, seq 0); seq stride
  std::vector<int64_t> v_off;    //   is cap_pad * head_dim
  std::vector<int64_t> n;        // [layer * batch + b] sequence lengths
  int32_t fmt = HWKV_KV_BF16;    // cache format (HWKV_KV_*)
  int32_t elem = 2;              // bytes per stored element
  std::vector<float> k_scale;    // per unit (fp8 scales; 1 otherwise)
  std::vector<float> v_scale;
  // paged caches: full units take pages of kPageTokens rows from a pool
  bool paged = false;
  int64_t n_pages = 0;           // pool size
  int64_t max_pages = 0;         // pages per (full unit, sequence) at max_ctx
  int64_t pool_off = 0;          // element offset of page 0
  size_t table_off = 0;          // byte offset of the device page table
  std::vector<int32_t> full_index;  // per unit: rank among full units, or -1
  std::vector<int32_t> pt_host;  // host copy of the page table
  std::vector<int32_t> held;     // pages held per (full unit, sequence)
  std::vector<int32_t> free_list;  // free pages (taken from the back)
  uint8_t *base = nullptr;
  size_t bytes = 0;
  bool owned = false;
  size_t ws_bytes = 0;
  // kernel timing (profiling): events recorded by decode calls
  bool timing = false;
  std::vector<hipEvent_t> ev_pool;   // created events, reused
  size_t ev_used = 0;                // events recorded since the last read
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string &msg) {
  g_err = msg;
  return code;
}

int ok() {
  g_err.clear();
  return HWKV_OK;
}

bool valid_group(int g) {
  return g == 1 || g == 2 || g == 4 || g == 6 || g == 8;
}

int64_t round_tile(int64_t x) {
  return (x + hwkv::kTile - 1) / hwkv::kTile * hwkv::kTile;
}

// Bytes per stored element of a cache format, or 0 if unknown.
int format_bytes(int32_t fmt) {
  switch (fmt) {
    case HWKV_KV_BF16: return 2;
    case HWKV_KV_F16: return 2;
    case HWKV_KV_FP8_E4M3: return 1;
    default: return 0;
  }
}

// Canonical window and capacity of a finite or full unit at max_ctx.
void unit_shape(const hwkv_policy &p, int32_t u, int64_t max_ctx,
                int64_t *window, int64_t *cap) {
  const int64_t w = p.level_window[p.level_of_unit[u]];
  if (w == 0 || (int64_t)p.n_sinks + w >= max_ctx) {
    *window = 0;
    *cap = max_ctx;
  } else {
    *window = w;
    *cap = p.n_sinks + w;
  }
}

uint64_t round256(uint64_t bytes) { return (bytes + 255) / 256 * 256; }

// Lays out the grouped pools for elements of `elem` bytes; fills per-unit
// vectors when `c` is non-null.  paged: full units get no region; a pool of
// n_pages pages and the page table follow the finite units' regions.
int layout(const hwkv_policy &p, int32_t batch, int64_t max_ctx, int elem,
           bool paged, int64_t n_pages, size_t *bytes, hwkv_cache *c) {
  if (batch < 1) return fail(HWKV_EINVAL, "batch must be >= 1");
  if (paged && (n_pages < 0 || n_pages > (int64_t)INT32_MAX))
    return fail(HWKV_EINVAL, "n_pages must be in [0, 2^31)");
  // the decode kernels address one (unit, sequence) region with 32-bit byte
  // offsets: round_tile(max_ctx) * head_dim * elem must stay below 2^31
  if (max_ctx < 1 ||
      round_tile(max_ctx) * (int64_t)p.head_dim * elem > (int64_t)INT32_MAX)
    return fail(HWKV_EINVAL, "max_ctx must be >= 1 and max_ctx * head_dim * "
                             "element bytes below 2^31 (bytes of one unit's K "
                             "or V)");
  const int32_t U = p.n_layers * p.n_kv_heads;
  const uint64_t D = (uint64_t)p.head_dim;
  std::vector<int64_t> win(U), cap(U), capp(U), koff(U), voff(U);
  for (int32_t u = 0; u < U; ++u) {
    unit_shape(p, u, max_ctx, &win[u], &cap[u]);
    capp[u] = round_tile(cap[u]);
  }
  std::vector<int32_t> fidx(U, -1);
  int32_t n_full = 0;
  if (paged)
    for (int32_t u = 0; u < U; ++u)
      if (win[u] == 0) fidx[u] = n_full++;
  // [level][unit in level][seq] K regions, then the V regions of the level
  uint64_t off = 0;  // elements
  auto mul_ok = [&](uint64_t a, uint64_t b, uint64_t *r) {
    return !__builtin_mul_overflow(a, b, r);
  };
  for (int32_t lv = 0; lv < p.n_levels; ++lv) {
    for (int pass = 0; pass < 2; ++pass) {
      for (int32_t u = 0; u < U; ++u) {
        if (p.level_of_unit[u] != lv) continue;
        if (fidx[u] >= 0) {            // paged full unit: no region
          (pass == 0 ? koff : voff)[u] = -1;
          continue;
        }
        uint64_t region;
        if (!mul_ok((uint64_t)capp[u] * D, (uint64_t)batch, &region) ||
            __builtin_add_overflow(off, region, &off) ||
            off > (uint64_t)INT64_MAX / 4)
          return fail(HWKV_EINVAL, "cache size overflows");
        (pass == 0 ? koff : voff)[u] = (int64_t)(off - region);
      }
    }
  }
  uint64_t total = off * (uint64_t)elem;
  const int64_t max_pages = (max_ctx + hwkv::kPageTokens - 1) / hwkv::kPageTokens;
  uint64_t pool_off = 0, table_off = 0;
  if (paged) {
    // pool: page i at element pool_off + i * 2 * kPageTokens * D
    total = round256(total);
    pool_off = total / (uint64_t)elem;
    uint64_t pool, tab;
    if (!mul_ok((uint64_t)n_pages, 2ull * hwkv::kPageTokens * D * (uint64_t)elem, &pool) ||
        __builtin_add_overflow(total, pool, &total))
      return fail(HWKV_EINVAL, "cache size overflows");
    // table: int32 [full unit][seq][max_pages]; offsets into it are int32
    total = round256(total);
    table_off = total;
    if (!mul_ok((uint64_t)n_full * (uint64_t)batch, (uint64_t)max_pages, &tab) ||
        tab > (uint64_t)INT32_MAX || __builtin_add_overflow(total, tab * 4, &total))
      return fail(HWKV_EINVAL, "page table too large");
    if (total > (uint64_t)INT64_MAX / 4) return fail(HWKV_EINVAL, "cache size overflows");
  }
  *bytes = (size_t)total;
  if (c) {
    c->window = win;
    c->cap = cap;
    c->cap_pad = capp;
    c->k_off = koff;
    c->v_off = voff;
    c->paged = paged;
    if (paged) {
      c->n_pages = n_pages;
      c->max_pages = max_pages;
      c->pool_off = (int64_t)pool_off;
      c->table_off = (size_t)table_off;
      c->full_index = fidx;
      c->pt_host.assign((size_t)n_full * batch * max_pages, -1);
      c->held.assign((size_t)n_full * batch, 0);
      c->free_list.resize((size_t)n_pages);
      for (int64_t i = 0; i < n_pages; ++i)  // page 0 is taken first
        c->free_list[(size_t)i] = (int32_t)(n_pages - 1 - i);
    }
  }
  return HWKV_OK;
}

// Page-table offset of (unit, seq) in a paged cache, or -1 if the unit is
// not paged.
int32_t page_tab_off(const hwkv_cache *c, int32_t u, int32_t seq) {
  if (!c->paged || c->full_index[u] < 0) return -1;
  return (int32_t)(((int64_t)c->full_index[u] * c->batch + seq) * c->max_pages);
}

int32_t *device_page_table(const hwkv_cache *c) {
  return c->paged ? reinterpret_cast<int32_t *>(c->base + c->table_off) : nullptr;
}

// Takes the pages that the full units of `layer` need so that sequence b
// holds rows [0, len[b]) for every (b, len) in `want`, and installs their
// page-table entries on stream s (before the call's kernels, which run
// after them in stream order).  ENOMEM, with nothing changed, if the pool
// has too few free pages.
int take_pages(hwkv_cache *c, int32_t layer,
               const std::vector<std::pair<int32_t, int64_t>> &want, hipStream_t s);

// Shared by hwkv_cache_alloc_format and hwkv_cache_alloc_paged.
int alloc_impl(hwkv_cache **out, const hwkv_policy *p, int32_t batch, int64_t max_ctx,
               int32_t kv_format, const float *k_scale, const float *v_scale, bool paged,
               int64_t n_pages, void *dev_buf, size_t buf_bytes);

int64_t group_size(const hwkv_policy &p) { return p.n_q_heads / p.n_kv_heads; }

// 64-slot tiles of an item with n_valid rows.
int64_t tiles_for(int64_t n_valid) { return (n_valid + hwkv::kTile - 1) / hwkv::kTile; }

// Decode split workgroups of the items of one launch, given their tile
// counts: an item of n tiles gets ceil(n / T) workgroups of at most T tiles,
// with T the least number of tiles per workgroup, from ceil(total / target)
// up, at which the launch has no more than target workgroups (else the
// ceilings of many items together put a third workgroup on some CUs, and
// those CUs' workgroups finish last: on a 16-sequence batch, up to 546
// workgroups for 512 slots took 1,077 us per step against 990 at the
// capped count).  Every item keeps at least one workgroup, so a launch of
// more items than target has one per item.
// The most workgroups plan_workgroups gives a launch of cnt items whose
// tiles add up to at most `tiles`, whatever their lengths.
int64_t max_workgroups(int64_t target, int64_t cnt, int64_t tiles) {
  return std::min(tiles, std::max(target, cnt));
}

void plan_workgroups(const int64_t *tiles, int cnt, int64_t target, int32_t *nwg) {
  int64_t total = 0, longest = 1;
  for (int j = 0; j < cnt; ++j) {
    total += tiles[j];
    longest = std::max(longest, tiles[j]);
  }
  auto count = [&](int64_t t) {
    int64_t n = 0;
    for (int j = 0; j < cnt; ++j) n += (tiles[j] + t - 1) / t;
    return n;
  };
  // count(T) <= total / T + cnt, so the loop ends by T = ceil(total /
  // (target - cnt)) when target > cnt, and at the longest item otherwise
  int64_t T = std::max<int64_t>(1, (total + target - 1) / target);
  while (T < longest && count(T) > target) ++T;
  for (int j = 0; j < cnt; ++j) nwg[j] = (int32_t)((tiles[j] + T - 1) / T);
}

size_t partial_bytes(const hwkv_policy &p) {
  return (size_t)group_size(p) * (size_t)(p.head_dim + 2) * sizeof(float);
}

int64_t &seq_len(hwkv_cache *c, int32_t layer, int32_t b) {
  return c->n[(size_t)layer * c->batch + b];
}

int64_t slot_of(const hwkv_cache *c, int32_t u, int64_t pos) {
  const int64_t w = c->window[u];
  const int64_t S = c->pol.n_sinks;
  if (w == 0 || pos < S) return pos;
  return S + (pos - S) % w;
}

int check_device(hipError_t e, const char *what) {
  if (e == hipSuccess) return HWKV_OK;
  return fail(HWKV_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// The next timing event of the cache (created on first use, then reused);
// the launch it is handed to records it.
int next_event(hwkv_cache *c, hipEvent_t *e) {
  if (c->ev_used == c->ev_pool.size()) {
    hipEvent_t ne;
    const int rc = check_device(hipEventCreate(&ne), "hipEventCreate");
    if (rc != HWKV_OK) return rc;
    c->ev_pool.push_back(ne);
  }
  *e = c->ev_pool[c->ev_used++];
  return HWKV_OK;
}

int take_pages(hwkv_cache *c, int32_t layer,
               const std::vector<std::pair<int32_t, int64_t>> &want, hipStream_t s) {
  if (!c->paged) return HWKV_OK;
  const hwkv_policy &p = c->pol;
  const int32_t H = p.n_kv_heads;
  // count first: nothing changes unless every page is available
  int64_t need_total = 0;
  for (const auto &bw : want)
    for (int32_t h = 0; h < H; ++h) {
      const int32_t pto = page_tab_off(c, layer * H + h, bw.first);
      if (pto < 0) continue;
      const int64_t need = (bw.second + hwkv::kPageTokens - 1) / hwkv::kPageTokens;
      const int64_t have = c->held[(size_t)(pto / c->max_pages)];
      if (need > have) need_total += need - have;
    }
  if (need_total == 0) return HWKV_OK;
  if (need_total > (int64_t)c->free_list.size())
    return fail(HWKV_ENOMEM, "page pool exhausted: " + std::to_string(need_total) +
                                 " pages needed, " + std::to_string(c->free_list.size()) +
                                 " free");
  hwkv::PageUpdateArgs u;
  u.table = device_page_table(c);
  u.n = 0;
  for (const auto &bw : want)
    for (int32_t h = 0; h < H; ++h) {
      const int32_t pto = page_tab_off(c, layer * H + h, bw.first);
      if (pto < 0) continue;
      const int64_t need = (bw.second + hwkv::kPageTokens - 1) / hwkv::kPageTokens;
      int32_t &have = c->held[(size_t)(pto / c->max_pages)];
      for (; have < need; ++have) {
        const int32_t pg = c->free_list.back();
        c->free_list.pop_back();
        c->pt_host[(size_t)pto + have] = pg;
        u.idx[u.n] = pto + have;
        u.page[u.n] = pg;
        if (++u.n == hwkv::kMaxPageUpdates) {
          const int rc = check_device(hwkv::launch_page_update(u, s), "page table launch");
          if (rc != HWKV_OK) return rc;
          u.n = 0;
        }
      }
    }
  if (u.n > 0) return check_device(hwkv::launch_page_update(u, s), "page table launch");
  return HWKV_OK;
}

// Element offsets (2-byte elements) of the prefill-attention staging area:
// for an fp8 cache, per kv head of the layer its K tiles and V rows widened
// to bf16 in the bf16 cache layout (cap_pad rows each); then, for fp8 and
// binary16 caches, the chunk's K and V ([n_tokens][Hkv][D]) as the cache will
// store them.  Returns the bytes (0 for a bf16 cache).
struct StageLayout {
  std::vector<int64_t> k_img, v_img;
  int64_t k_in = 0, v_in = 0;
};
size_t stage_layout(const hwkv_cache *c, int32_t layer, int64_t n_tokens, StageLayout *out) {
  const hwkv_policy &p = c->pol;
  const int64_t D = p.head_dim;
  int64_t off = 0;
  StageLayout L;
  if (c->fmt == HWKV_KV_BF16) {
    if (out) *out = L;
    return 0;
  }
  for (int32_t h = 0; h < p.n_kv_heads && c->fmt == HWKV_KV_FP8_E4M3; ++h) {
    const int32_t u = layer * p.n_kv_heads + h;
    L.k_img.push_back(off);
    off += c->cap_pad[u] * D;
    L.v_img.push_back(off);
    off += c->cap_pad[u] * D;
  }
  off = (off + 127) / 128 * 128;                    // 256-byte aligned
  L.k_in = off;
  off += n_tokens * p.n_kv_heads * D;
  L.v_in = off;
  off += n_tokens * p.n_kv_heads * D;
  if (out) *out = L;
  return (size_t)off * 2;
}

int prefill_attn_impl(hwkv_cache *c, int32_t layer, int32_t seq, int64_t pos0,
                      int64_t n_tokens, const void *q, const void *k, const void *v,
                      float scale, void *out, void *ws, size_t ws_bytes, void *stream) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  // fp8: the units are staged as bf16 code values; fp8 and binary16: the
  // chunk's own keys and values are staged as the cache will store them
  const bool staged = c->fmt == HWKV_KV_FP8_E4M3;
  const bool chunk_staged = c->fmt != HWKV_KV_BF16;
  const hwkv_policy &p = c->pol;
  if (layer < 0 || layer >= p.n_layers || seq < 0 || seq >= c->batch)
    return fail(HWKV_EINVAL, "layer or seq out of range");
  if (n_tokens < 0) return fail(HWKV_EINVAL, "n_tokens must be >= 0");
  if (!std::isfinite(scale) || !(scale > 0.0f))
    return fail(HWKV_EINVAL, "scale must be finite and > 0");
  if (pos0 != seq_len(c, layer, seq))
    return fail(HWKV_ESTATE, "pos0 " + std::to_string(pos0) +
                                 " != sequence length " +
                                 std::to_string(seq_len(c, layer, seq)));
  if (pos0 + n_tokens > c->max_ctx)
    return fail(HWKV_ECAPACITY, "prefill past max_ctx");
  if (n_tokens == 0) return ok();
  if (!q || !k || !v || !out)
    return fail(HWKV_EINVAL, "q, k, v and out must be non-null");
  StageLayout SL;
  if (chunk_staged) {
    const size_t need = stage_layout(c, layer, n_tokens, &SL);
    if (!ws || ws_bytes < need)
      return fail(HWKV_EINVAL, "workspace missing or too small (need " +
                                   std::to_string(need) + " bytes)");
  }
  const int32_t H = p.n_kv_heads;
  const int32_t G = (int32_t)group_size(p);
  const int64_t D = p.head_dim;
  const hipStream_t st = (hipStream_t)stream;
  hwkv::PrefillAttnArgs a;
  std::memset(&a, 0, sizeof a);
  const int64_t p1 = pos0 + n_tokens;
  std::vector<std::pair<int64_t, int32_t>> work;  // (keys of the last token, h)
  for (int32_t h = 0; h < H; ++h) {
    const int32_t u = layer * H + h;
    const int64_t seq_off = (int64_t)seq * c->cap_pad[u] * D;
    if (staged) {         // the bf16 image of the unit
      a.head[h].k_off = SL.k_img[h];
      a.head[h].v_off = SL.v_img[h];
      a.head[h].pto = -1;
      a.head[h].k_scale = c->k_scale[u];
      a.head[h].v_scale = c->v_scale[u];
    } else {
      a.head[h].k_off = c->k_off[u] + seq_off;
      a.head[h].v_off = c->v_off[u] + seq_off;
      a.head[h].pto = page_tab_off(c, u, seq);
      a.head[h].k_scale = 1.0f;
      a.head[h].v_scale = 1.0f;
    }
    a.head[h].window = (int32_t)c->window[u];
    const int64_t w = c->window[u];
    work.push_back({w == 0 ? p1 : std::min(p1, (int64_t)p.n_sinks + w), h});
  }
  std::stable_sort(work.begin(), work.end(),
                   [](const std::pair<int64_t, int32_t> &x,
                      const std::pair<int64_t, int32_t> &y) {
                     return x.first > y.first;
                   });
  for (int32_t r = 0; r < H; ++r) a.head_order[r] = work[r].second;
  const int64_t cols = n_tokens * G;
  const int64_t per = hwkv::prefill_attn_columns_per_block();
  const int64_t nb = (cols + per - 1) / per;
  if (nb * H > (int64_t)INT32_MAX)
    return fail(HWKV_EINVAL, "n_tokens too large for one launch");
  uint16_t *img = static_cast<uint16_t *>(ws);
  if (staged) {
    // the occupied rows of every unit (the keys below pos0), widened
    hwkv::StageArgs sa;
    std::memset(&sa, 0, sizeof sa);
    int64_t max_chunks = 0;
    for (int32_t h = 0; h < H; ++h) {
      const int32_t u = layer * H + h;
      const int64_t seq_off = (int64_t)seq * c->cap_pad[u] * D;
      hwkv::StageUnit &su = sa.unit[h];
      su.src_k_off = c->k_off[u] + seq_off;
      su.src_v_off = c->v_off[u] + seq_off;
      su.dst_k_off = SL.k_img[h];
      su.dst_v_off = SL.v_img[h];
      su.pto = page_tab_off(c, u, seq);
      su.n_rows = (int32_t)std::min(pos0, c->cap[u]);
      max_chunks = std::max(max_chunks, (int64_t)((su.n_rows + 63) / 64) * 64 * (D / 8));
    }
    sa.cache = c->base;
    sa.page_table = device_page_table(c);
    sa.pool_off = c->pool_off;
    sa.image = img;
    sa.n_units = H;
    sa.max_chunks = (int32_t)max_chunks;
    int rc;
    if (max_chunks > 0 &&
        (rc = check_device(hwkv::launch_stage_units((int)D, sa, st), "stage launch")) != HWKV_OK)
      return rc;
    a.cache = img;
  } else {
    a.cache = reinterpret_cast<const uint16_t *>(c->base);
    a.page_table = device_page_table(c);
    a.pool_off = c->pool_off;
  }
  if (chunk_staged) {
    // the chunk's own keys and values as the cache will store them
    hwkv::StageChunkArgs ca;
    std::memset(&ca, 0, sizeof ca);
    ca.fmt = c->fmt;
    ca.k = static_cast<const uint16_t *>(k);
    ca.v = static_cast<const uint16_t *>(v);
    ca.k_out = img + SL.k_in;
    ca.v_out = img + SL.v_in;
    for (int32_t h = 0; h < H; ++h) {
      ca.k_scale[h] = c->k_scale[layer * H + h];
      ca.v_scale[h] = c->v_scale[layer * H + h];
    }
    ca.n_chunks = n_tokens * H * (D / 8);
    ca.n_kv_heads = H;
    const int rc = check_device(hwkv::launch_stage_chunk((int)D, ca, st), "stage launch");
    if (rc != HWKV_OK) return rc;
    a.k = img + SL.k_in;
    a.v = img + SL.v_in;
  } else {
    a.k = static_cast<const uint16_t *>(k);
    a.v = static_cast<const uint16_t *>(v);
  }
  a.q = static_cast<const uint16_t *>(q);
  a.out = static_cast<float *>(out);
  a.p0 = (int32_t)pos0;
  a.n_tokens = (int32_t)n_tokens;
  a.n_kv_heads = H;
  a.group = G;
  a.n_sinks = p.n_sinks;
  a.n_col_blocks = (int32_t)nb;
  a.scale_log2 = scale * 1.4426950408889634f;
  return check_device(hwkv::launch_prefill_attn(p.head_dim, c->fmt == HWKV_KV_F16, a, st),
                      "prefill_attn launch") ==
                 HWKV_OK
             ? ok()
             : HWKV_EDEVICE;
}

// The split partials of hwkv_append_decode_attn_noalloc: a file-scope
// device array (one copy per device, held until the process ends), so that
// the call allocates nothing.  Host code never passes the array's name to a
// kernel or a copy: in host code it stands for the array, not for its device
// address, which scratch_ptr() takes once per device.
constexpr size_t kScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[64] = {};

// The device address of `scratch` on the current device (looked up on the
// first call on each device).
int scratch_ptr(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(HWKV_EDEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(HWKV_EDEVICE, "device index beyond 63");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return fail(HWKV_EDEVICE, std::string("hipGetSymbolAddress(scratch): ") +
                                    hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return HWKV_OK;
}

// Shared validation of a decode call; fills per-item lengths.  static_ws:
// ws is the static scratch (an over-size call is refused with its limit).
int decode_impl(hwkv_cache *c, int32_t layer, const void *k_new,
                const void *v_new, const void *q, float scale, void *out,
                void *ws, size_t ws_bytes, void *stream, bool fused,
                bool static_ws = false) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  const hwkv_policy &p = c->pol;
  if (layer < 0 || layer >= p.n_layers)
    return fail(HWKV_EINVAL, "layer out of range");
  if (!q || !out) return fail(HWKV_EINVAL, "q and out must be non-null");
  if (fused && (!k_new || !v_new))
    return fail(HWKV_EINVAL, "k_new and v_new must be non-null");
  if (!std::isfinite(scale)) return fail(HWKV_EINVAL, "scale must be finite");
  const int32_t H = p.n_kv_heads, B = c->batch;
  const int G = (int)group_size(p);
  // item lengths
  const int n_items_total = B * H;
  std::vector<int32_t> nv(n_items_total), nwg(n_items_total), nslot(n_items_total);
  std::vector<int64_t> tiles(n_items_total);
  for (int32_t b = 0; b < B; ++b) {
    const int64_t n = seq_len(c, layer, b);
    for (int32_t h = 0; h < H; ++h) {
      const int32_t u = layer * H + h;
      int64_t len = n;
      int32_t s_new = -1;
      if (fused) {
        if (c->window[u] == 0 && n >= c->cap[u])
          return fail(HWKV_ECAPACITY, "append past max_ctx on a full unit");
        s_new = (int32_t)slot_of(c, u, n);
        len = n + 1;
      } else if (n == 0) {
        return fail(HWKV_EINVAL, "decode on an empty sequence");
      }
      const int i = b * H + h;
      nv[i] = (int32_t)std::min(len, c->cap[u]);
      tiles[i] = tiles_for(nv[i]);
      nslot[i] = s_new;
    }
  }
  // split workgroups per item, per launch of at most kMaxItems items
  const int64_t target = hwkv::decode_workgroup_target(c->fmt, p.head_dim, G);
  int64_t total_splits = 0;
  for (int i0 = 0; i0 < n_items_total; i0 += hwkv::kMaxItems) {
    const int cnt = std::min(hwkv::kMaxItems, n_items_total - i0);
    plan_workgroups(&tiles[i0], cnt, target, &nwg[i0]);
    for (int j = 0; j < cnt; ++j) total_splits += nwg[i0 + j];
  }
  const size_t need = (size_t)total_splits * partial_bytes(p);
  if (static_ws && need > ws_bytes)
    return fail(HWKV_EINVAL, "the call needs " + std::to_string(need) +
                                 " bytes of split partials, more than the " +
                                 std::to_string(ws_bytes) + "-byte static scratch");
  if (!ws || ws_bytes < need)
    return fail(HWKV_EINVAL, "workspace missing or too small (need " +
                                 std::to_string(need) + " bytes)");
  const hipStream_t s = (hipStream_t)stream;
  if (fused) {  // pages for the appended tokens (the last validation)
    std::vector<std::pair<int32_t, int64_t>> want;
    for (int32_t b = 0; b < B; ++b) want.push_back({b, seq_len(c, layer, b) + 1});
    const int rc = take_pages(c, layer, want, s);
    if (rc != HWKV_OK) return rc;
  }
  // launches of at most kMaxItems items
  int ws_split = 0;
  for (int i0 = 0; i0 < n_items_total; i0 += hwkv::kMaxItems) {
    const int cnt = std::min(hwkv::kMaxItems, n_items_total - i0);
    hwkv::DecodeArgs a;
    std::memset(&a, 0, sizeof a);
    int splits = 0;
    for (int j = 0; j < cnt; ++j) {
      const int i = i0 + j;
      const int32_t b = i / H, h = i % H;
      const int32_t u = layer * H + h;
      const int64_t seq_off = (int64_t)b * c->cap_pad[u] * p.head_dim;
      a.it.k_off[j] = c->k_off[u] + seq_off;
      a.it.v_off[j] = c->v_off[u] + seq_off;
      a.it.n_valid[j] = nv[i];
      a.it.new_slot[j] = nslot[i];
      a.it.q_row[j] = b * p.n_q_heads + h * G;
      a.it.kv_row[j] = b * H + h;
      a.it.k_scale[j] = c->k_scale[u];
      a.it.v_scale[j] = c->v_scale[u];
      a.it.pto[j] = page_tab_off(c, u, b);
      a.it.split_begin[j] = splits;
      splits += nwg[i];
    }
    a.it.split_begin[cnt] = splits;
    // entries past the items: no workgroup begins there (the split kernel
    // counts the items that begin at or before a workgroup)
    for (int j = cnt + 1; j <= hwkv::kMaxItems; ++j) a.it.split_begin[j] = INT32_MAX;
    a.it.n_items = cnt;
    a.it.ws_split0 = ws_split;
    a.cache = c->base;
    a.page_table = device_page_table(c);
    a.pool_off = c->pool_off;
    a.q = static_cast<const uint16_t *>(q);
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.out = static_cast<float *>(out);
    // the call's partials: acc rows of all its launches, then their (m, l)
    a.part_acc = static_cast<float *>(ws);
    a.part_ml = static_cast<float *>(ws) + (size_t)total_splits * G * p.head_dim;
    a.scale_log2 = scale * 1.4426950408889634f;
    const int n_combine =
        cnt * hwkv::decode_combine_blocks_per_item(p.head_dim, G);
    // timing: each kernel's own start and end (four events per launch group)
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    int rc;
    for (int e = 0; c->timing && e < 4; ++e)
      if ((rc = next_event(c, &ev[e])) != HWKV_OK) return rc;
    rc = check_device(
        hwkv::launch_decode_split(c->fmt, p.head_dim, G, a, splits, s, ev[0], ev[1]),
        "decode split launch");
    if (rc != HWKV_OK) return rc;  // earlier launches of this call may run
    rc = check_device(
        hwkv::launch_decode_combine(p.head_dim, G, a, n_combine, s, ev[2], ev[3]),
        "decode merge launch");
    if (rc != HWKV_OK) return rc;
    ws_split += splits;
  }
  if (fused)
    for (int32_t b = 0; b < B; ++b) seq_len(c, layer, b) += 1;
  return ok();
}

}  // namespace

extern "C" {

const char *hwkv_last_error(void) { return g_err.c_str(); }

int hwkv_policy_set(hwkv_policy **out, int32_t n_layers, int32_t n_kv_heads,
                    int32_t n_q_heads, int32_t head_dim, int32_t n_sinks,
                    int32_t n_levels, const int64_t *level_window,
                    const int32_t *level_of_unit) {
  if (!out) return fail(HWKV_EINVAL, "out is null");
  *out = nullptr;
  if (n_layers < 1) return fail(HWKV_EINVAL, "n_layers must be >= 1");
  if (n_kv_heads < 1 || n_kv_heads > hwkv::kMaxItems)
    return fail(HWKV_EINVAL, "n_kv_heads must be in [1, 64]");
  if (n_q_heads < 1 || n_q_heads % n_kv_heads != 0)
    return fail(HWKV_EINVAL, "n_q_heads must be a multiple of n_kv_heads");
  if (!valid_group(n_q_heads / n_kv_heads))
    return fail(HWKV_EINVAL, "GQA group size must be 1, 2, 4, 6 or 8");
  if (head_dim != 64 && head_dim != 128 && head_dim != 256)
    return fail(HWKV_EINVAL, "head_dim must be 64, 128 or 256");
  if (n_sinks < 0) return fail(HWKV_EINVAL, "n_sinks must be >= 0");
  if (n_levels < 1) return fail(HWKV_EINVAL, "n_levels must be >= 1");
  if (!level_window || !level_of_unit)
    return fail(HWKV_EINVAL, "level arrays must be non-null");
  if ((int64_t)n_layers * n_kv_heads > (int64_t(1) << 24))
    return fail(HWKV_EINVAL, "too many units");
  for (int32_t k = 0; k < n_levels; ++k)
    if (level_window[k] < 0)
      return fail(HWKV_EINVAL, "level windows must be > 0 (or 0 for full)");
  const int32_t U = n_layers * n_kv_heads;
  for (int32_t u = 0; u < U; ++u)
    if (level_of_unit[u] < 0 || level_of_unit[u] >= n_levels)
      return fail(HWKV_EINVAL, "level index out of range");
  try {
    hwkv_policy *p = new hwkv_policy;
    p->n_layers = n_layers;
    p->n_kv_heads = n_kv_heads;
    p->n_q_heads = n_q_heads;
    p->head_dim = head_dim;
    p->n_sinks = n_sinks;
    p->n_levels = n_levels;
    p->level_window.assign(level_window, level_window + n_levels);
    p->level_of_unit.assign(level_of_unit, level_of_unit + U);
    *out = p;
  } catch (const std::bad_alloc &) {
    return fail(HWKV_ENOMEM, "host allocation failed");
  }
  return ok();
}

int hwkv_policy_free(hwkv_policy *policy) {
  delete policy;
  return ok();
}

int hwkv_policy_shape(const hwkv_policy *p, int32_t *n_layers, int32_t *n_kv_heads,
                      int32_t *n_q_heads, int32_t *head_dim, int32_t *n_sinks,
                      int32_t *n_levels) {
  if (!p) return fail(HWKV_EINVAL, "policy is null");
  if (n_layers) *n_layers = p->n_layers;
  if (n_kv_heads) *n_kv_heads = p->n_kv_heads;
  if (n_q_heads) *n_q_heads = p->n_q_heads;
  if (head_dim) *head_dim = p->head_dim;
  if (n_sinks) *n_sinks = p->n_sinks;
  if (n_levels) *n_levels = p->n_levels;
  return ok();
}

int hwkv_policy_bytes(const hwkv_policy *p, int64_t ctx, double *bytes) {
  return hwkv_policy_bytes_format(p, ctx, HWKV_KV_BF16, bytes);
}

int hwkv_policy_bytes_format(const hwkv_policy *p, int64_t ctx,
                             int32_t kv_format, double *bytes) {
  if (!p || !bytes) return fail(HWKV_EINVAL, "null argument");
  if (ctx < 1) return fail(HWKV_EINVAL, "ctx must be >= 1");
  const int b = format_bytes(kv_format);
  if (b == 0) return fail(HWKV_EINVAL, "unknown cache format");
  double tot = 0.0;
  const double row = (double)p->head_dim * (double)(b + b);  // d^K b^K + d^V b^V
  for (int32_t lv : p->level_of_unit) {
    const int64_t w = p->level_window[lv];
    const int64_t r = (w == 0) ? ctx : std::min<int64_t>(p->n_sinks + w, ctx);
    tot += (double)r * row;
  }
  *bytes = tot;
  return ok();
}

int hwkv_policy_rate(const hwkv_policy *p, int64_t ctx, double *rate) {
  if (!p || !rate) return fail(HWKV_EINVAL, "null argument");
  double b = 0.0;
  const int rc = hwkv_policy_bytes(p, ctx, &b);
  if (rc != HWKV_OK) return rc;
  const double full = (double)p->level_of_unit.size() * (double)ctx *
                      (double)p->head_dim * 4.0;
  *rate = b / full;
  return ok();
}

int hwkv_cache_bytes(const hwkv_policy *p, int32_t batch, int64_t max_ctx,
                     size_t *bytes) {
  return hwkv_cache_bytes_format(p, batch, max_ctx, HWKV_KV_BF16, bytes);
}

int hwkv_cache_bytes_format(const hwkv_policy *p, int32_t batch,
                            int64_t max_ctx, int32_t kv_format, size_t *bytes) {
  if (!p || !bytes) return fail(HWKV_EINVAL, "null argument");
  const int elem = format_bytes(kv_format);
  if (elem == 0) return fail(HWKV_EINVAL, "unknown cache format");
  const int rc = layout(*p, batch, max_ctx, elem, false, 0, bytes, nullptr);
  return rc == HWKV_OK ? ok() : rc;
}

int hwkv_cache_bytes_paged(const hwkv_policy *p, int32_t batch, int64_t max_ctx,
                           int32_t kv_format, int64_t n_pages, size_t *bytes) {
  if (!p || !bytes) return fail(HWKV_EINVAL, "null argument");
  const int elem = format_bytes(kv_format);
  if (elem == 0) return fail(HWKV_EINVAL, "unknown cache format");
  const int rc = layout(*p, batch, max_ctx, elem, true, n_pages, bytes, nullptr);
  return rc == HWKV_OK ? ok() : rc;
}

int hwkv_cache_alloc(hwkv_cache **out, const hwkv_policy *p, int32_t batch,
                     int64_t max_ctx, void *dev_buf, size_t buf_bytes) {
  return hwkv_cache_alloc_format(out, p, batch, max_ctx, HWKV_KV_BF16, nullptr,
                                 nullptr, dev_buf, buf_bytes);
}

int hwkv_cache_alloc_format(hwkv_cache **out, const hwkv_policy *p,
                            int32_t batch, int64_t max_ctx, int32_t kv_format,
                            const float *k_scale, const float *v_scale,
                            void *dev_buf, size_t buf_bytes) {
  return alloc_impl(out, p, batch, max_ctx, kv_format, k_scale, v_scale, false, 0,
                    dev_buf, buf_bytes);
}

int hwkv_cache_alloc_paged(hwkv_cache **out, const hwkv_policy *p, int32_t batch,
                           int64_t max_ctx, int32_t kv_format, const float *k_scale,
                           const float *v_scale, int64_t n_pages, void *dev_buf,
                           size_t buf_bytes) {
  return alloc_impl(out, p, batch, max_ctx, kv_format, k_scale, v_scale, true, n_pages,
                    dev_buf, buf_bytes);
}

}  // extern "C"

namespace {

int alloc_impl(hwkv_cache **out, const hwkv_policy *p, int32_t batch, int64_t max_ctx,
               int32_t kv_format, const float *k_scale, const float *v_scale, bool paged,
               int64_t n_pages, void *dev_buf, size_t buf_bytes) {
  if (!out || !p) return fail(HWKV_EINVAL, "null argument");
  *out = nullptr;
  const int elem = format_bytes(kv_format);
  if (elem == 0) return fail(HWKV_EINVAL, "unknown cache format");
  const size_t n_units = (size_t)p->n_layers * p->n_kv_heads;
  if (kv_format != HWKV_KV_FP8_E4M3 && (k_scale || v_scale))
    return fail(HWKV_EINVAL, "scales are for fp8 caches only");
  for (const float *sc : {k_scale, v_scale}) {
    if (!sc) continue;
    for (size_t u = 0; u < n_units; ++u)
      if (!(std::isnormal(sc[u]) && sc[u] > 0.f))
        return fail(HWKV_EINVAL, "fp8 scales must be positive, finite and normal");
  }
  hwkv_cache *c = nullptr;
  try {
    c = new hwkv_cache;
    c->pol = *p;
    c->batch = batch;
    c->max_ctx = max_ctx;
    c->fmt = kv_format;
    c->elem = elem;
    c->k_scale.assign(n_units, 1.0f);
    c->v_scale.assign(n_units, 1.0f);
    if (k_scale) c->k_scale.assign(k_scale, k_scale + n_units);
    if (v_scale) c->v_scale.assign(v_scale, v_scale + n_units);
    size_t bytes = 0;
    int rc = layout(*p, batch, max_ctx, elem, paged, n_pages, &bytes, c);
    if (rc != HWKV_OK) {
      delete c;
      return rc;
    }
    c->bytes = bytes;
    c->n.assign((size_t)p->n_layers * batch, 0);
    // workspace: the most partials any call on a layer can take.  A launch
    // of cnt items has at most min(max(target, cnt), its tiles at capacity)
    // workgroups (plan_workgroups), whatever the lengths.
    size_t ws = 0;
    const int64_t target = hwkv::decode_workgroup_target(
        kv_format, p->head_dim, (int)(p->n_q_heads / p->n_kv_heads));
    const int64_t n_items = (int64_t)batch * p->n_kv_heads;
    for (int32_t l = 0; l < p->n_layers; ++l) {
      int64_t parts = 0;
      for (int64_t i0 = 0; i0 < n_items; i0 += hwkv::kMaxItems) {
        const int64_t cnt = std::min<int64_t>(hwkv::kMaxItems, n_items - i0);
        int64_t tiles = 0;
        for (int64_t i = i0; i < i0 + cnt; ++i)
          tiles += tiles_for(c->cap[l * p->n_kv_heads + i % p->n_kv_heads]);
        parts += max_workgroups(target, cnt, tiles);
      }
      ws = std::max(ws, (size_t)parts * partial_bytes(*p));
    }
    c->ws_bytes = ws;
    if (dev_buf) {
      if (buf_bytes < bytes) {
        delete c;
        return fail(HWKV_ENOMEM, "device buffer smaller than cache bytes (" +
                                     std::to_string(bytes) + ")");
      }
      c->base = static_cast<uint8_t *>(dev_buf);
      c->owned = false;
    } else {
      void *ptr = nullptr;
      hipError_t e = hipMalloc(&ptr, bytes ? bytes : 256);
      if (e != hipSuccess) {
        delete c;
        (void)hipGetLastError();
        return fail(e == hipErrorOutOfMemory ? HWKV_ENOMEM : HWKV_EDEVICE,
                    std::string("hipMalloc: ") + hipGetErrorString(e));
      }
      e = hipMemset(ptr, 0, bytes);
      if (e != hipSuccess) {
        (void)hipFree(ptr);
        delete c;
        return fail(HWKV_EDEVICE, std::string("hipMemset: ") + hipGetErrorString(e));
      }
      c->base = static_cast<uint8_t *>(ptr);
      c->owned = true;
    }
  } catch (const std::bad_alloc &) {
    delete c;
    return fail(HWKV_ENOMEM, "host allocation failed");
  }
  *out = c;
  return ok();
}

}  // namespace

extern "C" {

int hwkv_cache_free(hwkv_cache *c) {
  if (!c) return ok();
  int rc = HWKV_OK;
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  if (c->owned && c->base) {
    hipError_t e = hipFree(c->base);
    if (e != hipSuccess) rc = check_device(e, "hipFree");
  }
  delete c;
  return rc == HWKV_OK ? ok() : rc;
}

int hwkv_cache_format(const hwkv_cache *c, int32_t *kv_format, float *k_scale,
                      float *v_scale) {
  if (!c || !kv_format) return fail(HWKV_EINVAL, "null argument");
  *kv_format = c->fmt;
  if (k_scale) std::copy(c->k_scale.begin(), c->k_scale.end(), k_scale);
  if (v_scale) std::copy(c->v_scale.begin(), c->v_scale.end(), v_scale);
  return ok();
}

int hwkv_cache_pages(const hwkv_cache *c, int64_t *total, int64_t *free_pages) {
  if (!c || !total || !free_pages) return fail(HWKV_EINVAL, "null argument");
  *total = c->paged ? c->n_pages : 0;
  *free_pages = c->paged ? (int64_t)c->free_list.size() : 0;
  return ok();
}

int hwkv_cache_reset_seq(hwkv_cache *c, int32_t seq) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  if (seq < 0 || seq >= c->batch) return fail(HWKV_EINVAL, "seq out of range");
  const hwkv_policy &p = c->pol;
  for (int32_t l = 0; l < p.n_layers; ++l) {
    seq_len(c, l, seq) = 0;
    for (int32_t h = 0; h < p.n_kv_heads; ++h) {
      const int32_t pto = page_tab_off(c, l * p.n_kv_heads + h, seq);
      if (pto < 0) continue;
      int32_t &have = c->held[(size_t)(pto / c->max_pages)];
      for (; have > 0; --have) {
        c->free_list.push_back(c->pt_host[(size_t)pto + have - 1]);
        c->pt_host[(size_t)pto + have - 1] = -1;
      }
    }
  }
  return ok();
}

int hwkv_cache_seq_len(const hwkv_cache *c, int32_t layer, int32_t seq,
                       int64_t *n) {
  if (!c || !n) return fail(HWKV_EINVAL, "null argument");
  if (layer < 0 || layer >= c->pol.n_layers || seq < 0 || seq >= c->batch)
    return fail(HWKV_EINVAL, "layer or seq out of range");
  *n = c->n[(size_t)layer * c->batch + seq];
  return ok();
}

int hwkv_cache_unit_info(const hwkv_cache *c, int32_t layer, int32_t kv_head,
                         int64_t *capacity, int64_t *window) {
  if (!c || !capacity || !window) return fail(HWKV_EINVAL, "null argument");
  if (layer < 0 || layer >= c->pol.n_layers || kv_head < 0 ||
      kv_head >= c->pol.n_kv_heads)
    return fail(HWKV_EINVAL, "layer or kv_head out of range");
  const int32_t u = layer * c->pol.n_kv_heads + kv_head;
  *capacity = c->cap[u];
  *window = c->window[u];
  return ok();
}

int hwkv_prefill_write(hwkv_cache *c, int32_t layer, int32_t seq, int64_t pos0,
                       int64_t n_tokens, const void *k, const void *v,
                       void *stream) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  const hwkv_policy &p = c->pol;
  if (layer < 0 || layer >= p.n_layers || seq < 0 || seq >= c->batch)
    return fail(HWKV_EINVAL, "layer or seq out of range");
  if (n_tokens < 0) return fail(HWKV_EINVAL, "n_tokens must be >= 0");
  if (pos0 != seq_len(c, layer, seq))
    return fail(HWKV_ESTATE, "pos0 " + std::to_string(pos0) +
                                 " != sequence length " +
                                 std::to_string(seq_len(c, layer, seq)));
  if (n_tokens == 0) return ok();
  if (!k || !v) return fail(HWKV_EINVAL, "k and v must be non-null");
  const int64_t p0 = pos0, p1 = pos0 + n_tokens;
  const int32_t H = p.n_kv_heads;
  const int64_t S = p.n_sinks;
  for (int32_t h = 0; h < H; ++h) {
    const int32_t u = layer * H + h;
    if (c->window[u] == 0 && p1 > c->cap[u])
      return fail(HWKV_ECAPACITY, "prefill past max_ctx on a full unit");
  }
  {
    const int rc = take_pages(c, layer, {{seq, p1}}, (hipStream_t)stream);
    if (rc != HWKV_OK) return rc;
  }
  hwkv::WriteArgs a;
  std::memset(&a, 0, sizeof a);
  int max_tiles = 0;
  for (int32_t h = 0; h < H; ++h) {
    const int32_t u = layer * H + h;
    const int64_t w = c->window[u];
    const int64_t seq_off = (int64_t)seq * c->cap_pad[u] * p.head_dim;
    hwkv::WriteHead &wh = a.head[h];
    wh.k_off = c->k_off[u] + seq_off;
    wh.v_off = c->v_off[u] + seq_off;
    wh.window = (int32_t)w;
    wh.pto = page_tab_off(c, u, seq);
    wh.k_scale = c->k_scale[u];
    wh.v_scale = c->v_scale[u];
    // slot ranges [lo, hi) written by this chunk
    std::vector<std::pair<int64_t, int64_t>> sr;
    if (w == 0) {
      sr.push_back({p0, p1});
    } else {
      if (p0 < S) sr.push_back({p0, std::min(p1, S)});
      const int64_t start = std::max({p0, p1 - w, S});
      if (start < p1) {
        const int64_t cnt = p1 - start;
        const int64_t f = S + (start - S) % w;
        if (f + cnt <= S + w) {
          sr.push_back({f, f + cnt});
        } else {
          sr.push_back({f, S + w});
          sr.push_back({S, S + (f + cnt - (S + w))});
        }
      }
    }
    // to tile ranges, merged
    std::vector<std::pair<int64_t, int64_t>> tr;
    for (auto &r : sr)
      tr.push_back({r.first / hwkv::kTile, (r.second - 1) / hwkv::kTile + 1});
    std::sort(tr.begin(), tr.end());
    std::vector<std::pair<int64_t, int64_t>> merged;
    for (auto &r : tr) {
      if (!merged.empty() && r.first <= merged.back().second)
        merged.back().second = std::max(merged.back().second, r.second);
      else
        merged.push_back(r);
    }
    int tot = 0;
    for (size_t r = 0; r < merged.size() && r < 3; ++r) {
      wh.tile0[r] = (int32_t)merged[r].first;
      wh.n_tiles[r] = (int32_t)(merged[r].second - merged[r].first);
      tot += wh.n_tiles[r];
    }
    max_tiles = std::max(max_tiles, tot);
  }
  a.cache = c->base;
  a.page_table = device_page_table(c);
  a.pool_off = c->pool_off;
  a.k = static_cast<const uint16_t *>(k);
  a.v = static_cast<const uint16_t *>(v);
  a.p0 = p0;
  a.p1 = p1;
  a.n_kv_heads = H;
  a.n_sinks = p.n_sinks;
  if (max_tiles > 0) {
    const int rc = check_device(
        hwkv::launch_prefill_write(c->fmt, p.head_dim, a, max_tiles,
                                   (hipStream_t)stream),
        "prefill_write launch");
    if (rc != HWKV_OK) return rc;
  }
  seq_len(c, layer, seq) = p1;
  return ok();
}

int hwkv_prefill_attn(hwkv_cache *c, int32_t layer, int32_t seq, int64_t pos0,
                      int64_t n_tokens, const void *q, const void *k,
                      const void *v, float scale, void *out, void *stream) {
  if (c && c->fmt != HWKV_KV_BF16)
    return fail(HWKV_EINVAL, "prefill attention needs a bf16 cache here "
                             "(hwkv_prefill_attn_ws takes fp8 and binary16 caches)");
  return prefill_attn_impl(c, layer, seq, pos0, n_tokens, q, k, v, scale, out,
                           nullptr, 0, stream);
}

int hwkv_prefill_attn_workspace_bytes(const hwkv_cache *c, int64_t n_tokens,
                                      size_t *bytes) {
  if (!c || !bytes) return fail(HWKV_EINVAL, "null argument");
  if (n_tokens < 0) return fail(HWKV_EINVAL, "n_tokens must be >= 0");
  size_t best = 0;
  for (int32_t l = 0; l < c->pol.n_layers; ++l)
    best = std::max(best, stage_layout(c, l, n_tokens, nullptr));
  *bytes = best;
  return ok();
}

int hwkv_prefill_attn_ws(hwkv_cache *c, int32_t layer, int32_t seq, int64_t pos0,
                         int64_t n_tokens, const void *q, const void *k,
                         const void *v, float scale, void *out, void *ws,
                         size_t ws_bytes, void *stream) {
  return prefill_attn_impl(c, layer, seq, pos0, n_tokens, q, k, v, scale, out, ws,
                           ws_bytes, stream);
}

}  // extern "C"

namespace {

size_t replay_rows_bytes(int64_t n_rows) { return (size_t)((n_rows * 4 + 255) / 256 * 256); }

// Upper bound of the replay's splits: a column block visits at most
// ceil(n_hist / 32) key tiles, at most kReplayTilesPerSplit per split.
int64_t replay_max_splits(int64_t n_hist) {
  const int64_t t = (n_hist + 31) / 32;
  return (t + hwkv::kReplayTilesPerSplit - 1) / hwkv::kReplayTilesPerSplit;
}

// Row positions reach the device through a pinned host buffer per device,
// so that their copy is asynchronous on the caller's stream.  A call reuses
// the buffer once the previous call's copy from it (marked by an event) has
// finished, which it has as soon as that call's first kernel ran.
struct RowStage {
  int32_t *host = nullptr;   // pinned, cap entries
  int64_t cap = 0;
  hipEvent_t copied = nullptr;
};
std::mutex g_row_stage_mu;
std::map<int, RowStage> g_row_stage;

// Enqueues the copy of rows[0, n) (as int32) to dst on st.
int stage_rows(const int64_t *rows, int64_t n, void *dst, hipStream_t st) {
  int dev = 0;
  int rc = check_device(hipGetDevice(&dev), "hipGetDevice");
  if (rc != HWKV_OK) return rc;
  std::lock_guard<std::mutex> lock(g_row_stage_mu);
  RowStage &rs = g_row_stage[dev];
  if (!rs.copied) {
    rc = check_device(hipEventCreateWithFlags(&rs.copied, hipEventDisableTiming),
                      "hipEventCreateWithFlags");
    if (rc != HWKV_OK) return rc;
  } else {
    rc = check_device(hipEventSynchronize(rs.copied), "hipEventSynchronize (rows)");
    if (rc != HWKV_OK) return rc;
  }
  if (rs.cap < n) {
    if (rs.host) (void)hipHostFree(rs.host);
    rs.host = nullptr;
    rs.cap = 0;
    const int64_t cap = std::max<int64_t>(n, 1024);
    rc = check_device(hipHostMalloc(reinterpret_cast<void **>(&rs.host), (size_t)cap * 4,
                                    hipHostMallocDefault),
                      "hipHostMalloc (rows)");
    if (rc != HWKV_OK) return rc;
    rs.cap = cap;
  }
  for (int64_t i = 0; i < n; ++i) rs.host[i] = (int32_t)rows[i];
  rc = check_device(hipMemcpyAsync(dst, rs.host, (size_t)n * 4, hipMemcpyHostToDevice, st),
                    "hipMemcpyAsync (rows)");
  if (rc != HWKV_OK) return rc;
  return check_device(hipEventRecord(rs.copied, st), "hipEventRecord (rows)");
}

// Partial sets of the workspace ([n_cols][D + 4] fp32 each): one per split,
// one for the sinks, and two holding the windows' edge (m, l) pairs (at most
// 64 windows x 2 floats <= 2 (D + 4) per column).
int64_t replay_partial_sets(int64_t n_hist) { return replay_max_splits(n_hist) + 3; }

}  // namespace
extern "C" {

int hwkv_calib_workspace_bytes(int32_t n_q_heads, int32_t head_dim, int32_t n_sinks,
                               int64_t n_hist, int64_t n_rows, size_t *bytes) {
  if (!bytes) return fail(HWKV_EINVAL, "bytes is null");
  if (n_rows < 1 || n_rows > (int64_t)(1 << 24) || n_hist < 1 ||
      n_hist > (int64_t)(1 << 24) || n_q_heads < 1 || n_q_heads > 64 * 8 ||
      (head_dim != 64 && head_dim != 128 && head_dim != 256) || n_sinks < 0)
    return fail(HWKV_EINVAL, "bad replay shape");
  const uint64_t part = (uint64_t)replay_partial_sets(n_hist) * (uint64_t)n_rows *
                        (uint64_t)n_q_heads * (uint64_t)(head_dim + 4) * 4u;
  *bytes = replay_rows_bytes(n_rows) + (size_t)part;
  return ok();
}

int hwkv_calib_workspace_bytes_format(int32_t n_kv_heads, int32_t n_q_heads,
                                      int32_t head_dim, int32_t n_sinks, int64_t n_hist,
                                      int64_t n_rows, int32_t kv_format, size_t *bytes) {
  if (!bytes) return fail(HWKV_EINVAL, "bytes is null");
  if (kv_format != HWKV_KV_BF16 && kv_format != HWKV_KV_FP8_E4M3)
    return fail(HWKV_EINVAL, "the replay takes bf16 or fp8 formats");
  if (n_kv_heads < 1 || n_kv_heads > hwkv::kMaxItems)
    return fail(HWKV_EINVAL, "n_kv_heads must be in [1, 64]");
  size_t base = 0;
  const int rc = hwkv_calib_workspace_bytes(n_q_heads, head_dim, n_sinks, n_hist, n_rows, &base);
  if (rc != HWKV_OK) return rc;
  if (kv_format == HWKV_KV_FP8_E4M3)       // the staged trace, 256-byte aligned
    base = (base + 255) / 256 * 256 +
           2 * (size_t)n_hist * (size_t)n_kv_heads * (size_t)head_dim * 2;
  *bytes = base;
  return ok();
}

int hwkv_calib_replay(int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim,
                      int32_t n_sinks, int32_t n_windows,
                      const int64_t *windows, int64_t n_hist, const void *k,
                      const void *v, int64_t n_rows, const int64_t *rows,
                      const void *q, float scale, void *outs, void *scores,
                      void *means, const void *ref_full, void *check, void *ws,
                      size_t ws_bytes, void *stream) {
  return hwkv_calib_replay_format(n_kv_heads, n_q_heads, head_dim, n_sinks, n_windows, windows,
                                  n_hist, k, v, n_rows, rows, q, scale, outs, scores, means,
                                  ref_full, check, HWKV_KV_BF16, nullptr, nullptr, ws, ws_bytes,
                                  stream);
}

int hwkv_calib_replay_format(int32_t n_kv_heads, int32_t n_q_heads, int32_t head_dim,
                             int32_t n_sinks, int32_t n_windows, const int64_t *windows,
                             int64_t n_hist, const void *k, const void *v, int64_t n_rows,
                             const int64_t *rows, const void *q, float scale, void *outs,
                             void *scores, void *means, const void *ref_full, void *check,
                             int32_t kv_format, const float *k_scale, const float *v_scale,
                             void *ws, size_t ws_bytes, void *stream) {
  if (n_kv_heads < 1 || n_kv_heads > hwkv::kMaxItems || n_q_heads < 1 ||
      n_q_heads % n_kv_heads != 0 || !valid_group(n_q_heads / n_kv_heads))
    return fail(HWKV_EINVAL, "n_kv_heads in [1, 64] and n_q_heads = G * n_kv_heads "
                             "with G in {1, 2, 4, 6, 8}");
  if (head_dim != 64 && head_dim != 128 && head_dim != 256)
    return fail(HWKV_EINVAL, "head_dim must be 64, 128 or 256");
  if (n_sinks < 0) return fail(HWKV_EINVAL, "n_sinks must be >= 0");
  if (n_windows < 0 || n_windows > 64 || (n_windows > 0 && !windows))
    return fail(HWKV_EINVAL, "n_windows in [0, 64] with a window array");
  for (int32_t i = 0; i < n_windows; ++i)
    if (windows[i] < 1 || (i > 0 && windows[i] <= windows[i - 1]))
      return fail(HWKV_EINVAL, "windows must be finite (> 0) and strictly increasing");
  if (n_hist < 1 || n_hist > (int64_t)(1 << 24))
    return fail(HWKV_EINVAL, "n_hist must be in [1, 2^24]");
  if (n_rows < 1 || n_rows > (int64_t)(1 << 24) || !rows)
    return fail(HWKV_EINVAL, "n_rows must be in [1, 2^24] with a row array");
  for (int64_t i = 0; i < n_rows; ++i)
    if (rows[i] < 0 || rows[i] >= n_hist || (i > 0 && rows[i] <= rows[i - 1]))
      return fail(HWKV_EINVAL, "rows must be strictly increasing positions in [0, n_hist)");
  if (!std::isfinite(scale) || !(scale > 0.0f))
    return fail(HWKV_EINVAL, "scale must be finite and > 0");
  if (!k || !v || !q || !outs || !ws || (n_windows > 0 && (!scores || !means)))
    return fail(HWKV_EINVAL, "k, v, q, outs, ws (and scores, means) must be non-null");
  if ((ref_full == nullptr) != (check == nullptr))
    return fail(HWKV_EINVAL, "check is required exactly when ref_full is given");
  if (kv_format != HWKV_KV_BF16 && kv_format != HWKV_KV_FP8_E4M3)
    return fail(HWKV_EINVAL, "the replay takes bf16 or fp8 formats (binary16 values are "
                             "not bf16 values)");
  const bool staged = kv_format == HWKV_KV_FP8_E4M3;
  if (!staged && (k_scale || v_scale))
    return fail(HWKV_EINVAL, "scales are for fp8 only");
  for (const float *sc : {k_scale, v_scale}) {
    if (!sc) continue;
    for (int32_t h = 0; h < n_kv_heads; ++h)
      if (!(std::isnormal(sc[h]) && sc[h] > 0.f))
        return fail(HWKV_EINVAL, "fp8 scales must be positive, finite and normal");
  }
  size_t need = 0;
  if (hwkv_calib_workspace_bytes_format(n_kv_heads, n_q_heads, head_dim, n_sinks, n_hist,
                                        n_rows, kv_format, &need) != HWKV_OK)
    return HWKV_EINVAL;
  if (ws_bytes < need) return fail(HWKV_EINVAL, "workspace too small");
  float ks[hwkv::kMaxItems], vs[hwkv::kMaxItems];
  for (int32_t h = 0; h < n_kv_heads; ++h) {
    ks[h] = k_scale ? k_scale[h] : 1.0f;
    vs[h] = v_scale ? v_scale[h] : 1.0f;
  }
  const int32_t G = n_q_heads / n_kv_heads;
  const int64_t per = hwkv::prefill_attn_columns_per_block();
  const int64_t nb = (n_rows * G + per - 1) / per;
  if (nb * n_kv_heads > (int64_t)INT32_MAX ||
      (int64_t)(n_windows + 1) * n_rows * n_q_heads > (int64_t)INT32_MAX)
    return fail(HWKV_EINVAL, "n_rows too large for one launch");
  hipStream_t st = (hipStream_t)stream;

  // row positions to the device, asynchronously
  int rc = stage_rows(rows, n_rows, ws, st);
  if (rc != HWKV_OK) return rc;

  int dev = 0, n_cus = 256;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n_cus < 1)
    n_cus = 256;  // only the split sizes depend on it
  (void)hipGetLastError();
  const size_t vec = (size_t)n_rows * n_q_heads * head_dim;
  float *part = reinterpret_cast<float *>(static_cast<uint8_t *>(ws) +
                                          replay_rows_bytes(n_rows));
  // fp8: the trace's keys and values as a cache of that format stores them,
  // staged after the partials as bf16 code values
  const void *k_src = k, *v_src = v;
  if (staged) {
    size_t base = 0;
    hwkv_calib_workspace_bytes(n_q_heads, head_dim, n_sinks, n_hist, n_rows, &base);
    base = (base + 255) / 256 * 256;
    uint16_t *kst = reinterpret_cast<uint16_t *>(static_cast<uint8_t *>(ws) + base);
    uint16_t *vst = kst + (size_t)n_hist * n_kv_heads * head_dim;
    hwkv::StageChunkArgs ca;
    std::memset(&ca, 0, sizeof ca);
    ca.fmt = HWKV_KV_FP8_E4M3;
    ca.k = static_cast<const uint16_t *>(k);
    ca.v = static_cast<const uint16_t *>(v);
    ca.k_out = kst;
    ca.v_out = vst;
    for (int32_t h = 0; h < n_kv_heads; ++h) {
      ca.k_scale[h] = ks[h];
      ca.v_scale[h] = vs[h];
    }
    ca.n_chunks = n_hist * n_kv_heads * (head_dim / 8);
    ca.n_kv_heads = n_kv_heads;
    rc = check_device(hwkv::launch_stage_chunk(head_dim, ca, st), "stage launch");
    if (rc != HWKV_OK) return rc;
    k_src = kst;
    v_src = vst;
  }
  // One pass over the trace for every candidate.  Splits: the key tiles of
  // the longest column block (its last row's position) in about two
  // workgroups per CU (one runs per CU at a time; a second round of equal
  // splits evens out the column blocks of unequal length better than one
  // round: 884 against 869 TFLOP/s on the 128K trace), never more than the
  // workspace holds, each of at least the minimum size.
  int64_t max_tiles = 1;
  for (int64_t b = 0; b < nb; ++b) {
    const int64_t c1 = std::min((b + 1) * per, n_rows * G) - 1;
    max_tiles = std::max<int64_t>(max_tiles, rows[c1 / G] / 32 + 1);
  }
  const int64_t ws_splits = replay_max_splits(n_hist);
  const int64_t want = std::min<int64_t>(
      ws_splits, std::max<int64_t>(1, 2 * n_cus / (nb * n_kv_heads)));
  const int64_t tps = std::max<int64_t>(
      hwkv::kReplayMinTilesPerSplit,
      std::max<int64_t>((max_tiles + want - 1) / want, (max_tiles + ws_splits - 1) / ws_splits));
  const int64_t n_splits = (max_tiles + tps - 1) / tps;
  const size_t n_cols = (size_t)n_rows * n_q_heads;
  const size_t set = n_cols * (size_t)(head_dim + 4);
  float *win_ml = part + (size_t)(ws_splits + 1) * set;
  hwkv::ReplayAttnArgs ra;
  std::memset(&ra, 0, sizeof ra);
  ra.q = static_cast<const uint16_t *>(q);
  ra.k = static_cast<const uint16_t *>(k_src);
  ra.v = static_cast<const uint16_t *>(v_src);
  ra.rows = static_cast<const int32_t *>(ws);
  ra.part = part;
  ra.win_acc = static_cast<float *>(outs);       // candidate k's rows hold its edge acc
  ra.win_ml = win_ml;
  // a window reaching back past the history holds every key
  for (int32_t c = 0; c < n_windows; ++c)
    ra.windows[c] = (int32_t)std::min<int64_t>(windows[c], n_hist);
  for (int32_t h = 0; h < n_kv_heads; ++h) ra.k_scale[h] = ks[h];
  ra.n_windows = n_windows;
  ra.n_splits = (int32_t)n_splits;
  ra.tiles_per_split = (int32_t)tps;
  ra.n_rows = (int32_t)n_rows;
  ra.n_kv_heads = n_kv_heads;
  ra.group = G;
  ra.n_sinks = n_sinks;
  ra.n_col_blocks = (int32_t)nb;
  ra.scale_log2 = scale * 1.4426950408889634f;
  rc = check_device(hwkv::launch_replay_attn(head_dim, ra, st), "calib replay launch");
  if (rc != HWKV_OK) return rc;
  hwkv::ReplayMergeArgs ma;
  std::memset(&ma, 0, sizeof ma);
  ma.part = part;
  ma.win_ml = win_ml;
  ma.outs = static_cast<float *>(outs);
  ma.rows = ra.rows;
  std::memcpy(ma.windows, ra.windows, sizeof ma.windows);
  for (int32_t h = 0; h < n_kv_heads; ++h) {
    ma.k_scale[h] = ks[h];
    ma.v_scale[h] = vs[h];
  }
  ma.n_windows = n_windows;
  ma.n_splits = (int32_t)n_splits;
  ma.tiles_per_split = (int32_t)tps;
  ma.n_cols = (int32_t)n_cols;
  ma.n_q_heads = n_q_heads;
  ma.group = G;
  ma.n_sinks = n_sinks;
  ma.scale_log2 = ra.scale_log2;
  rc = check_device(hwkv::launch_replay_merge(head_dim, ma, st), "calib merge launch");
  if (rc != HWKV_OK) return rc;
  hwkv::CalibArgs ca;
  ca.outs = static_cast<const float *>(outs);
  ca.ref = static_cast<const float *>(ref_full);
  ca.scores = static_cast<float *>(scores);
  ca.check = static_cast<float *>(check);
  ca.means = static_cast<float *>(means);
  ca.n_cand = n_windows;
  ca.n_rows = (int32_t)n_rows;
  ca.n_q_heads = n_q_heads;
  ca.group = G;
  if (n_windows > 0 || ref_full) {
    rc = check_device(hwkv::launch_calib_scores(head_dim, ca, st), "calib scores launch");
    if (rc != HWKV_OK) return rc;
  }
  if (n_windows > 0) {
    rc = check_device(hwkv::launch_calib_means(ca, st), "calib means launch");
    if (rc != HWKV_OK) return rc;
  }
  return ok();
}

int hwkv_calib_select(int32_t n_kv_heads, int32_t n_windows,
                      const int64_t *windows, int32_t n_sinks, int64_t ctx,
                      const double *means, double tau, int32_t *choice,
                      double *floor) {
  if (n_kv_heads < 1 || n_windows < 0 || (n_windows > 0 && (!windows || !means)) ||
      !choice || n_sinks < 0 || ctx < 1 || !(tau > 0.0 && tau <= 1.0))
    return fail(HWKV_EINVAL, "bad selection arguments (tau must lie in (0, 1])");
  for (int32_t i = 0; i < n_windows; ++i)
    if (windows[i] < 1) return fail(HWKV_EINVAL, "windows must be finite (> 0)");
  double lowest = 1.0;
  for (int32_t h = 0; h < n_kv_heads; ++h) {
    int32_t best = -1;
    int64_t best_cost = 0;
    double best_score = 1.0;
    // candidates in codebook order; the full one (score 1, cost ctx) last
    for (int32_t c = 0; c <= n_windows; ++c) {
      const double score = c < n_windows ? means[(size_t)c * n_kv_heads + h] : 1.0;
      const int64_t cost = c < n_windows ? std::min((int64_t)n_sinks + windows[c], ctx) : ctx;
      if (score >= tau && (best < 0 || cost < best_cost)) {
        best = c;
        best_cost = cost;
        best_score = score;
      }
    }
    choice[h] = best;
    lowest = std::min(lowest, best_score);
  }
  if (floor) *floor = lowest;
  return ok();
}

int hwkv_budget_select(int32_t n_records, const double *rates,
                       const double *floors, double budget, int32_t *chosen) {
  if (n_records < 1 || !rates || !floors || !chosen)
    return fail(HWKV_EINVAL, "need at least one record and non-null arrays");
  int32_t g_best = -1;
  for (int32_t g = 0; g < n_records; ++g) {
    if (!(rates[g] <= budget)) continue;
    if (g_best < 0 || floors[g] > floors[g_best] ||
        (floors[g] == floors[g_best] && rates[g] < rates[g_best]))
      g_best = g;                                  // earlier g wins full ties
  }
  *chosen = g_best;
  return ok();
}

}  // extern "C"

namespace {

const char kArtifactFormat[] = "hwkv-policy/1";

std::string fmt_double(double x) {
  char b[64];
  std::snprintf(b, sizeof b, "%.17g", x);
  return b;
}

// A strict reader for the artifact's JSON subset: one object whose values
// are strings of printable ASCII without escapes, numbers, arrays of
// integers or arrays of arrays of integers.
struct ArtifactReader {
  const char *p, *end;
  bool ok = true;
  void ws() {
    while (p < end && (*p == ' ' || *p == '\n' || *p == '\t' || *p == '\r')) ++p;
  }
  bool eat(char c) {
    ws();
    if (p < end && *p == c) {
      ++p;
      return true;
    }
    return false;
  }
  bool string(std::string *out) {
    ws();
    if (p >= end || *p != '"') return false;
    const char *q = ++p;
    while (p < end && *p != '"') {
      // printable ASCII without escapes: what the writer emits
      if (*p == '\\' || (unsigned char)*p < 0x20 || (unsigned char)*p > 0x7e) return false;
      ++p;
    }
    if (p >= end) return false;
    out->assign(q, p);
    ++p;
    return true;
  }
  // the characters of a JSON number, then strtod / strtoll over them
  bool number_text(std::string *t) {
    ws();
    const char *q = p;
    while (p < end && (std::strchr("+-0123456789.eE", *p) != nullptr)) ++p;
    if (p == q) return false;
    t->assign(q, p);
    return true;
  }
  bool dbl(double *x) {
    std::string t;
    if (!number_text(&t)) return false;
    char *e = nullptr;
    *x = std::strtod(t.c_str(), &e);
    return e && *e == '\0';
  }
  bool i64(int64_t *x) {
    std::string t;
    if (!number_text(&t)) return false;
    if (t.find_first_of(".eE") != std::string::npos) return false;
    char *e = nullptr;
    errno = 0;
    const long long v = std::strtoll(t.c_str(), &e, 10);
    if (!e || *e != '\0' || errno) return false;
    *x = v;
    return true;
  }
  bool u64(uint64_t *x) {
    std::string t;
    if (!number_text(&t)) return false;
    if (t.find_first_not_of("0123456789") != std::string::npos) return false;
    char *e = nullptr;
    errno = 0;
    const unsigned long long v = std::strtoull(t.c_str(), &e, 10);
    if (!e || *e != '\0' || errno) return false;
    *x = v;
    return true;
  }
  bool int_array(std::vector<int64_t> *v) {
    if (!eat('[')) return false;
    v->clear();
    if (eat(']')) return true;
    do {
      int64_t x;
      if (!i64(&x)) return false;
      v->push_back(x);
    } while (eat(','));
    return eat(']');
  }
};

}  // namespace
extern "C" {

int hwkv_policy_serialize(const hwkv_policy *p, const char *artifact_id, uint64_t seed,
                          int32_t grid_index, double tau, double rate, double floor,
                          char *buf, size_t cap, size_t *len) {
  if (!p || !artifact_id || !len) return fail(HWKV_EINVAL, "policy, artifact_id and len required");
  for (const char *c = artifact_id; *c; ++c)
    if ((unsigned char)*c < 0x20 || (unsigned char)*c > 0x7e || *c == '"' || *c == '\\')
      return fail(HWKV_EINVAL, "artifact_id must be printable ASCII without quote or backslash");
  if (!std::isfinite(tau) || !std::isfinite(rate) || !std::isfinite(floor))
    return fail(HWKV_EINVAL, "tau, rate and floor must be finite");
  std::string t = "{\n";
  t += "  \"format\": \"" + std::string(kArtifactFormat) + "\",\n";
  t += "  \"artifact\": \"" + std::string(artifact_id) + "\",\n";
  t += "  \"seed\": " + std::to_string(seed) + ",\n";
  t += "  \"grid_index\": " + std::to_string(grid_index) + ",\n";
  t += "  \"tau\": " + fmt_double(tau) + ",\n";
  t += "  \"rate\": " + fmt_double(rate) + ",\n";
  t += "  \"floor\": " + fmt_double(floor) + ",\n";
  t += "  \"n_layers\": " + std::to_string(p->n_layers) + ",\n";
  t += "  \"n_kv_heads\": " + std::to_string(p->n_kv_heads) + ",\n";
  t += "  \"n_q_heads\": " + std::to_string(p->n_q_heads) + ",\n";
  t += "  \"head_dim\": " + std::to_string(p->head_dim) + ",\n";
  t += "  \"n_sinks\": " + std::to_string(p->n_sinks) + ",\n";
  t += "  \"level_window\": [";
  for (int32_t k = 0; k < p->n_levels; ++k)
    t += (k ? ", " : "") + std::to_string(p->level_window[k]);
  t += "],\n  \"level_of_unit\": [";
  for (int32_t l = 0; l < p->n_layers; ++l) {
    t += l ? ",\n    [" : "\n    [";
    for (int32_t h = 0; h < p->n_kv_heads; ++h)
      t += (h ? ", " : "") + std::to_string(p->level_of_unit[(size_t)l * p->n_kv_heads + h]);
    t += "]";
  }
  t += "\n  ]\n}\n";
  *len = t.size();
  if (!buf) return ok();
  if (cap < t.size() + 1) return fail(HWKV_ENOMEM, "buffer too small for the artifact");
  std::memcpy(buf, t.c_str(), t.size() + 1);
  return ok();
}

int hwkv_policy_deserialize(const char *buf, size_t len, hwkv_policy **out,
                            char *artifact_id, size_t id_cap, uint64_t *seed,
                            int32_t *grid_index, double *tau, double *rate,
                            double *floor) {
  if (!buf || !out) return fail(HWKV_EINVAL, "buf and out required");
  ArtifactReader r{buf, buf + len};
  std::map<std::string, int> seen;
  std::string fmt, id;
  uint64_t sd = 0;
  int64_t gi = 0, L = 0, H = 0, Q = 0, D = 0, S = 0;
  double ta = 0, ra = 0, fl = 0;
  std::vector<int64_t> lw, lou;
  int64_t rows_read = 0;
  if (!r.eat('{')) return fail(HWKV_EINVAL, "artifact: expected an object");
  do {
    std::string key;
    if (!r.string(&key) || !r.eat(':')) return fail(HWKV_EINVAL, "artifact: expected a key");
    if (seen[key]++) return fail(HWKV_EINVAL, "artifact: repeated key " + key);
    bool good;
    if (key == "format") good = r.string(&fmt);
    else if (key == "artifact") good = r.string(&id);
    else if (key == "seed") good = r.u64(&sd);
    else if (key == "grid_index") good = r.i64(&gi);
    else if (key == "tau") good = r.dbl(&ta);
    else if (key == "rate") good = r.dbl(&ra);
    else if (key == "floor") good = r.dbl(&fl);
    else if (key == "n_layers") good = r.i64(&L);
    else if (key == "n_kv_heads") good = r.i64(&H);
    else if (key == "n_q_heads") good = r.i64(&Q);
    else if (key == "head_dim") good = r.i64(&D);
    else if (key == "n_sinks") good = r.i64(&S);
    else if (key == "level_window") good = r.int_array(&lw);
    else if (key == "level_of_unit") {
      good = r.eat('[');
      lou.clear();
      rows_read = 0;
      if (good && !r.eat(']')) {
        do {
          std::vector<int64_t> row;
          good = r.int_array(&row);
          if (!good) break;
          if (rows_read > 0 && (int64_t)row.size() * rows_read != (int64_t)lou.size()) {
            good = false;
            break;
          }
          lou.insert(lou.end(), row.begin(), row.end());
          ++rows_read;
        } while (r.eat(','));
        good = good && r.eat(']');
      }
    } else {
      return fail(HWKV_EINVAL, "artifact: unknown key " + key);
    }
    if (!good) return fail(HWKV_EINVAL, "artifact: malformed value of " + key);
  } while (r.eat(','));
  if (!r.eat('}')) return fail(HWKV_EINVAL, "artifact: expected '}'");
  r.ws();
  if (r.p != r.end) return fail(HWKV_EINVAL, "artifact: trailing characters");
  if (seen.size() != 14) return fail(HWKV_EINVAL, "artifact: missing keys");
  if (fmt != kArtifactFormat) return fail(HWKV_EINVAL, "artifact: unknown format " + fmt);
  if (L < 1 || L > INT32_MAX || H < 1 || H > INT32_MAX || Q > INT32_MAX || D > INT32_MAX ||
      S < 0 || S > INT32_MAX || gi < INT32_MIN || gi > INT32_MAX || lw.size() > INT32_MAX ||
      rows_read != L || (int64_t)lou.size() != L * H)
    return fail(HWKV_EINVAL, "artifact: inconsistent shape");
  std::vector<int32_t> lev(lou.size());
  for (size_t i = 0; i < lou.size(); ++i) {
    if (lou[i] < INT32_MIN || lou[i] > INT32_MAX) return fail(HWKV_EINVAL, "artifact: level");
    lev[i] = (int32_t)lou[i];
  }
  hwkv_policy *p = nullptr;
  const int rc = hwkv_policy_set(&p, (int32_t)L, (int32_t)H, (int32_t)Q, (int32_t)D, (int32_t)S,
                                 (int32_t)lw.size(), lw.data(), lev.data());
  if (rc != HWKV_OK) return rc;
  *out = p;
  if (artifact_id && id_cap > 0) {
    const size_t n = std::min(id.size(), id_cap - 1);
    std::memcpy(artifact_id, id.data(), n);
    artifact_id[n] = '\0';
  }
  if (seed) *seed = sd;
  if (grid_index) *grid_index = (int32_t)gi;
  if (tau) *tau = ta;
  if (rate) *rate = ra;
  if (floor) *floor = fl;
  return ok();
}

int hwkv_append(hwkv_cache *c, int32_t layer, const void *k_new,
                const void *v_new, void *stream) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  const hwkv_policy &p = c->pol;
  if (layer < 0 || layer >= p.n_layers)
    return fail(HWKV_EINVAL, "layer out of range");
  if (!k_new || !v_new) return fail(HWKV_EINVAL, "k_new and v_new must be non-null");
  const int32_t H = p.n_kv_heads, B = c->batch;
  for (int32_t b = 0; b < B; ++b)
    for (int32_t h = 0; h < H; ++h) {
      const int32_t u = layer * H + h;
      if (c->window[u] == 0 && seq_len(c, layer, b) >= c->cap[u])
        return fail(HWKV_ECAPACITY, "append past max_ctx on a full unit");
    }
  {
    std::vector<std::pair<int32_t, int64_t>> want;
    for (int32_t b = 0; b < B; ++b) want.push_back({b, seq_len(c, layer, b) + 1});
    const int rc = take_pages(c, layer, want, (hipStream_t)stream);
    if (rc != HWKV_OK) return rc;
  }
  const int total = B * H;
  for (int i0 = 0; i0 < total; i0 += hwkv::kMaxItems) {
    const int cnt = std::min(hwkv::kMaxItems, total - i0);
    hwkv::AppendArgs a;
    std::memset(&a, 0, sizeof a);
    for (int j = 0; j < cnt; ++j) {
      const int i = i0 + j;
      const int32_t b = i / H, h = i % H;
      const int32_t u = layer * H + h;
      const int64_t seq_off = (int64_t)b * c->cap_pad[u] * p.head_dim;
      a.k_off[j] = c->k_off[u] + seq_off;
      a.v_off[j] = c->v_off[u] + seq_off;
      a.slot[j] = (int32_t)slot_of(c, u, seq_len(c, layer, b));
      a.kv_row[j] = b * H + h;
      a.k_scale[j] = c->k_scale[u];
      a.v_scale[j] = c->v_scale[u];
      a.pto[j] = page_tab_off(c, u, b);
    }
    a.n_items = cnt;
    a.cache = c->base;
    a.page_table = device_page_table(c);
    a.pool_off = c->pool_off;
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    const int rc = check_device(
        hwkv::launch_append(c->fmt, p.head_dim, a, (hipStream_t)stream),
        "append launch");
    if (rc != HWKV_OK) return rc;
  }
  for (int32_t b = 0; b < B; ++b) seq_len(c, layer, b) += 1;
  return ok();
}

int hwkv_decode_workspace_bytes(const hwkv_cache *c, size_t *bytes) {
  if (!c || !bytes) return fail(HWKV_EINVAL, "null argument");
  *bytes = c->ws_bytes;
  return ok();
}

int hwkv_decode_attn(hwkv_cache *c, int32_t layer, const void *q, float scale,
                     void *out, void *ws, size_t ws_bytes, void *stream) {
  return decode_impl(c, layer, nullptr, nullptr, q, scale, out, ws, ws_bytes,
                     stream, false);
}

int hwkv_append_decode_attn(hwkv_cache *c, int32_t layer, const void *k_new,
                            const void *v_new, const void *q, float scale,
                            void *out, void *ws, size_t ws_bytes,
                            void *stream) {
  return decode_impl(c, layer, k_new, v_new, q, scale, out, ws, ws_bytes,
                     stream, true);
}

int hwkv_append_decode_attn_noalloc(hwkv_cache *c, int32_t layer,
                                    const void *k_new, const void *v_new,
                                    const void *q, float scale, void *out,
                                    void *stream) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  void *ws = nullptr;
  const int rc = scratch_ptr(&ws);
  if (rc != HWKV_OK) return rc;
  return decode_impl(c, layer, k_new, v_new, q, scale, out, ws, kScratchBytes, stream, true,
                     true);
}

int hwkv_decode_timing(hwkv_cache *c, int32_t enable) {
  if (!c) return fail(HWKV_EINVAL, "cache is null");
  c->timing = enable != 0;
  return ok();
}

int hwkv_decode_timing_read(hwkv_cache *c, double *split_ms, double *merge_ms,
                            int64_t *launches) {
  if (!c || !split_ms || !merge_ms || !launches)
    return fail(HWKV_EINVAL, "null argument");
  double sp = 0.0, mg = 0.0;
  const size_t n = c->ev_used / 4;
  if (n > 0) {
    int rc = check_device(hipEventSynchronize(c->ev_pool[c->ev_used - 1]),
                          "hipEventSynchronize");
    if (rc != HWKV_OK) return rc;
    for (size_t i = 0; i < n; ++i) {
      float t0 = 0.f, t1 = 0.f;
      rc = check_device(hipEventElapsedTime(&t0, c->ev_pool[4 * i],
                                            c->ev_pool[4 * i + 1]),
                        "hipEventElapsedTime");
      if (rc != HWKV_OK) return rc;
      rc = check_device(hipEventElapsedTime(&t1, c->ev_pool[4 * i + 2],
                                            c->ev_pool[4 * i + 3]),
                        "hipEventElapsedTime");
      if (rc != HWKV_OK) return rc;
      sp += t0;
      mg += t1;
    }
  }
  *split_ms = sp;
  *merge_ms = mg;
  *launches = (int64_t)n;
  c->ev_used = 0;
  return ok();
}

int hwkv_cache_read_unit(const hwkv_cache *c, int32_t layer, int32_t kv_head,
                         int32_t seq, void *host_k, void *host_v,
                         int64_t *n_valid) {
  if (!c || !host_k || !host_v || !n_valid)
    return fail(HWKV_EINVAL, "null argument");
  const hwkv_policy &p = c->pol;
  if (layer < 0 || layer >= p.n_layers || kv_head < 0 ||
      kv_head >= p.n_kv_heads || seq < 0 || seq >= c->batch)
    return fail(HWKV_EINVAL, "layer, kv_head or seq out of range");
  const int32_t u = layer * p.n_kv_heads + kv_head;
  const int64_t D = p.head_dim, cap = c->cap[u], capp = c->cap_pad[u];
  const int64_t E = c->elem;                 // bytes per element
  const int64_t seq_off = (int64_t)seq * capp * D;
  std::vector<uint8_t> tiles;
  try {
    tiles.resize((size_t)(capp * D * E));
  } catch (const std::bad_alloc &) {
    return fail(HWKV_ENOMEM, "host allocation failed");
  }
  int rc = check_device(hipDeviceSynchronize(), "synchronize");
  if (rc != HWKV_OK) return rc;
  const int32_t pto = page_tab_off(c, u, seq);
  if (pto >= 0) {
    // paged: page j holds tiles 4j .. 4j + 3 (K) and rows 256 j .. (V)
    const int64_t PT = hwkv::kPageTokens;
    const int32_t have = c->held[(size_t)(pto / c->max_pages)];
    for (int32_t j = 0; j < have; ++j) {
      const int64_t pg = c->pt_host[(size_t)pto + j];
      const uint8_t *src = c->base + (c->pool_off + pg * 2 * PT * D) * E;
      const int64_t rows = std::min(PT, cap - j * PT);
      rc = check_device(hipMemcpy(tiles.data() + j * PT * D * E, src,
                                  (size_t)(std::min(PT, capp - j * PT) * D * E),
                                  hipMemcpyDeviceToHost), "copy K page");
      if (rc != HWKV_OK) return rc;
      rc = check_device(hipMemcpy(static_cast<uint8_t *>(host_v) + j * PT * D * E,
                                  src + PT * D * E, (size_t)(rows * D * E),
                                  hipMemcpyDeviceToHost), "copy V page");
      if (rc != HWKV_OK) return rc;
    }
  } else {
    rc = check_device(hipMemcpy(tiles.data(), c->base + (c->k_off[u] + seq_off) * E,
                                (size_t)(capp * D * E), hipMemcpyDeviceToHost),
                      "copy K");
    if (rc != HWKV_OK) return rc;
    rc = check_device(hipMemcpy(host_v, c->base + (c->v_off[u] + seq_off) * E,
                                (size_t)(cap * D * E), hipMemcpyDeviceToHost),
                      "copy V");
    if (rc != HWKV_OK) return rc;
  }
  // untile K: [tile][D/8][64][8 elements] -> [slot][D]
  uint8_t *hk = static_cast<uint8_t *>(host_k);
  const int64_t NC = D / 8, LB = 8 * E;
  for (int64_t j = 0; j < cap; ++j) {
    const int64_t t = j / hwkv::kTile, sl = j % hwkv::kTile;
    for (int64_t g = 0; g < NC; ++g)
      std::memcpy(hk + (j * D + g * 8) * E,
                  tiles.data() + ((t * NC + g) * hwkv::kTile + sl) * LB, (size_t)LB);
  }
  *n_valid = std::min(c->n[(size_t)layer * c->batch + seq], cap);
  return ok();
}

}  // extern "C"
