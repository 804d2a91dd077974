// hwkv_internal.h -- types shared by the host API and the gfx950 kernels.
//
// Device layout of one (unit, sequence) region; elements are those of the
// cache format (kv_format.h: 2 bytes for bf16 and f16, 1 byte for fp8), and
// a chunk is 8 elements (16 or 8 bytes):
//   K: cap_pad / 64 tiles; tile t holds slots 64t .. 64t+63 as
//      [head_dim / 8][64 slots][8 channels]   (chunks, slot-minor)
//      so that a wavefront with one lane per slot reads 64 chunks contiguous
//      per channel chunk (lane-per-token q.k without LDS staging or
//      reductions).
//   V: [cap_pad][head_dim] row-major, so that lanes owning channel slices
//      read whole rows contiguously for the p * v accumulation.
// cap_pad = cap rounded up to a multiple of 64.  Regions are grouped by
// window level: for each level, the K regions of its units ([unit][seq]),
// then their V regions.  Offsets below count elements.
//
// Paged caches: full units have no region.  Their rows live in pages of
// kPageTokens rows of one (unit, sequence) -- the K tiles of the page
// ([4 tiles][head_dim / 8][64][8]), then its V rows ([256][head_dim]) -- in
// a pool after the finite units' regions; page j of (unit, sequence) is
// page_table[pto + j], where pto = (full unit index * batch + sequence) *
// pages per max_ctx.  A page holds whole decode and prefill key tiles.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace hwkv {

constexpr int kTile = 64;        // token slots per K tile (= wavefront width)
constexpr int kMaxItems = 64;    // (sequence, kv-head) items per launch
constexpr int kPageTokens = 256; // rows per page of a paged full unit
constexpr int kDecodeWaves = 4;  // waves of a decode split workgroup
#ifndef HWKV_DECODE_WG_PER_CU_X4
#define HWKV_DECODE_WG_PER_CU_X4 8
#endif
// Decode split workgroups a launch aims at, in quarters per CU: the host
// picks the tiles per workgroup so that the launch has about this many
// workgroups (at most as many as the kernel's register budget holds at once):
// two per CU.
constexpr int kDecodeWgPerCuX4 = HWKV_DECODE_WG_PER_CU_X4;

// Decode work of one launch: items are (sequence b, kv head h) pairs of one
// layer; item i owns rows [0, n_valid[i]) of its unit and the launch's split
// workgroups [split_begin[i], split_begin[i + 1]); workgroup j of the item's
// nwg walks the item's 64-slot tiles j, j + nwg, ...
struct DecodeItems {
  int64_t k_off[kMaxItems];      // element offset of the item's K tiles
  int64_t v_off[kMaxItems];      // element offset of the item's V rows
  int32_t n_valid[kMaxItems];    // occupied slots attended (>= 1)
  int32_t new_slot[kMaxItems];   // slot taking the appended token, or -1
  int32_t q_row[kMaxItems];      // b * n_q_heads + h * G (first q head)
  int32_t kv_row[kMaxItems];     // b * n_kv_heads + h (row of k_new/v_new)
  float k_scale[kMaxItems];      // fp8 scales of the item's unit (else 1)
  float v_scale[kMaxItems];
  int32_t pto[kMaxItems];        // page-table offset of a paged unit, or -1
  int32_t split_begin[kMaxItems + 1];
  int32_t n_items;
  int32_t ws_split0;             // first partial of this launch in the call's
                                 // partial arrays
};

struct DecodeArgs {
  DecodeItems it;
  void *cache;                   // cache base
  const uint16_t *q;             // [B][Hq][D]
  const uint16_t *k_new;         // [B][Hkv][D] or null
  const uint16_t *v_new;
  float *out;                    // [B][Hq][D]
  float *part_acc;               // partials: acc [partial][G][D]
  float *part_ml;                //   and (m, l) [partial][G][2]
  const int32_t *page_table;     // paged caches (else null)
  int64_t pool_off;              // element offset of page 0
  float scale_log2;              // scale * log2(e)
};

// Materialisation of one chunk: for kv head h, the tiles listed in up to
// three disjoint ranges [tile0[r], tile0[r] + n_tiles[r]).
struct WriteHead {
  int64_t k_off;                 // element offset of the (unit, seq) K tiles
  int64_t v_off;                 // element offset of its V rows
  int32_t window;                // 0 = full
  int32_t pto;                   // page-table offset of a paged unit, or -1
  int32_t tile0[3];
  int32_t n_tiles[3];
  float k_scale, v_scale;        // fp8 scales of the unit (else 1)
};

struct WriteArgs {
  WriteHead head[kMaxItems];     // one per kv head of the layer
  void *cache;
  const int32_t *page_table;     // paged caches (else null)
  int64_t pool_off;              // element offset of page 0
  const uint16_t *k;             // [n_tokens][Hkv][D]
  const uint16_t *v;
  int64_t p0, p1;                // chunk [p0, p1)
  int32_t n_kv_heads;
  int32_t n_sinks;
};

struct AppendArgs {
  int64_t k_off[kMaxItems];
  int64_t v_off[kMaxItems];
  int32_t slot[kMaxItems];
  int32_t kv_row[kMaxItems];
  float k_scale[kMaxItems];
  float v_scale[kMaxItems];
  int32_t pto[kMaxItems];        // page-table offset of a paged unit, or -1
  int32_t n_items;
  void *cache;
  const int32_t *page_table;     // paged caches (else null)
  int64_t pool_off;              // element offset of page 0
  const uint16_t *k_new;
  const uint16_t *v_new;
};

// Page-table entries to install (table[idx[i]] = page[i]) before the
// kernels of a call that took new pages read them.
constexpr int kMaxPageUpdates = 496;
struct PageUpdateArgs {
  int32_t *table;
  int32_t n;
  int32_t idx[kMaxPageUpdates];
  int32_t page[kMaxPageUpdates];
};

// Prefill attention of one chunk [p0, p0 + n_tokens) of one sequence: per
// kv head the (unit, sequence) region offsets and canonical window; the
// kernel's workgroups visit heads in head_order (most keys first) and each
// head's column blocks from the last token down.
struct PrefillAttnHead {
  int64_t k_off;                 // element offset of the (unit, seq) K tiles
  int64_t v_off;                 // element offset of its V rows
  int32_t window;                // 0 = full
  int32_t pto;                   // page-table offset of a paged unit, or -1
  float k_scale;                 // logit multiplier of the stored keys (fp8: s_K)
  float v_scale;                 // output multiplier (fp8: s_V)
};

struct PrefillAttnArgs {
  PrefillAttnHead head[kMaxItems];
  int32_t head_order[kMaxItems];
  const uint16_t *cache;         // 2-byte elements: bf16 or binary16
  const int32_t *page_table;     // paged caches (else null)
  int64_t pool_off;              // element offset of page 0
  const uint16_t *q;             // [n_tokens][Hq][D]
  const uint16_t *k;             // [n_tokens][Hkv][D]
  const uint16_t *v;
  float *out;                    // [n_tokens][Hq][D]
  int32_t p0;
  int32_t n_tokens;
  int32_t n_kv_heads;
  int32_t group;                 // G = Hq / Hkv
  int32_t n_sinks;
  int32_t n_col_blocks;          // per head: ceil(n_tokens * G / columns)
  float scale_log2;              // scale * log2(e)
};

#ifndef HWKV_PREFILL_WAVES
#define HWKV_PREFILL_WAVES 8
#endif
constexpr int kPrefillWaves = HWKV_PREFILL_WAVES;

// Launchers (return the launch status).  D in {64, 128, 256}; G in
// {1, 2, 4, 6, 8}; fmt one of the HWKV_KV_* formats.  Non-null events e0, e1
// take the kernel's own start and end times (hipExtLaunchKernel), so their
// elapsed time excludes the dispatch of the launch.
hipError_t launch_decode_split(int fmt, int D, int G, const DecodeArgs &a,
                               int n_splits, hipStream_t s, hipEvent_t e0 = nullptr,
                               hipEvent_t e1 = nullptr);
template <int F>
hipError_t launch_decode_split_fmt(int D, int G, const DecodeArgs &a,
                                   int n_splits, hipStream_t s, hipEvent_t e0,
                                   hipEvent_t e1);
hipError_t launch_decode_combine(int D, int G, const DecodeArgs &a,
                                 int n_combine_blocks, hipStream_t s,
                                 hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// split workgroups a launch aims at on the current device
int decode_workgroup_target(int fmt, int D, int G);
int decode_combine_blocks_per_item(int D, int G);  // merge workgroups
hipError_t launch_prefill_write(int fmt, int D, const WriteArgs &a,
                                int max_tiles, hipStream_t s);
hipError_t launch_append(int fmt, int D, const AppendArgs &a, hipStream_t s);
hipError_t launch_page_update(const PageUpdateArgs &a, hipStream_t s);

// Staging of an fp8 cache for prefill attention: rows [0, n_rows) of one
// (unit, sequence) widened to bf16 code values in the bf16 cache layout, and
// a chunk's K or V quantised as the cache stores it and widened.
struct StageUnit {
  int64_t src_k_off, src_v_off;  // fp8 element offsets (unpaged units)
  int64_t dst_k_off, dst_v_off;  // bf16 element offsets in the image
  int32_t pto;                   // page-table offset of a paged unit, or -1
  int32_t n_rows;                // occupied slots to stage
};
struct StageArgs {
  StageUnit unit[kMaxItems];     // one per kv head of the layer
  const uint8_t *cache;          // fp8 cache base
  const int32_t *page_table;
  int64_t pool_off;
  uint16_t *image;               // bf16 image base
  int32_t n_units;
  int32_t max_chunks;            // max over units of n_rows * D / 8 (per K or V)
};
hipError_t launch_stage_units(int D, const StageArgs &a, hipStream_t s);
struct StageChunkArgs {
  int32_t fmt;                   // HWKV_KV_FP8_E4M3 or HWKV_KV_F16
  const uint16_t *k, *v;         // [n_tokens][Hkv][D] bf16 inputs
  uint16_t *k_out, *v_out;       // the same layout: the stored values, as bf16
                                 // code values (fp8) or binary16 (f16)
  float k_scale[kMaxItems];      // per kv head of the layer
  float v_scale[kMaxItems];
  int64_t n_chunks;              // n_tokens * Hkv * D / 8
  int32_t n_kv_heads;
};
hipError_t launch_stage_chunk(int D, const StageChunkArgs &a, hipStream_t s);
int prefill_attn_columns_per_block();   // (token, q head) columns
// f16: the cache, k and v hold binary16 values (else bf16); q is bf16.
hipError_t launch_prefill_attn(int D, bool f16, const PrefillAttnArgs &a, hipStream_t s);

// Calibration scores: for every (row, q head), the stabilised cosine of each
// candidate output against the full one (and of the full one against a
// reference); then per (candidate, kv head) the mean score.
struct CalibArgs {
  const float *outs;             // [n_cand + 1][n_rows][Hq][D], full last
  const float *ref;              // [n_rows][Hq][D] or null
  float *scores;                 // [n_cand][n_rows][Hq]
  float *check;                  // [n_rows][Hq] (if ref)
  float *means;                  // [n_cand][Hkv]
  int32_t n_cand, n_rows, n_q_heads, group;
};
hipError_t launch_calib_scores(int D, const CalibArgs &a, hipStream_t s);

// Calibration replay in one pass: for every sampled row, the keys of the
// traced history are visited once, from the row's position down, and every
// candidate window's partial is taken at the window's edge (the windows are
// nested suffixes of the history, plus the common sink prefix).
constexpr int kMaxWindows = 64;
struct ReplayAttnArgs {
  const uint16_t *q;             // [n_rows][Hq][D] queries of the sampled rows
  const uint16_t *k, *v;         // [n_hist][Hkv][D] traced keys and values
  const int32_t *rows;           // [n_rows] positions, strictly increasing
  float *part;                   // [n_splits + 1][n_cols][D + 4]: the splits'
                                 // partials [m, l, -, -, acc], then the sinks'
  float *win_acc;                // [n_windows][n_cols][D]: a window's acc at its edge
  float *win_ml;                 // [n_windows][n_cols][2]: its (m, l)
  int32_t windows[kMaxWindows];  // finite candidate windows, strictly increasing
  float k_scale[kMaxItems];      // per kv head: the keys' logit scale (fp8; else 1)
  int32_t n_windows, n_splits, tiles_per_split;
  int32_t n_rows, n_kv_heads, group, n_sinks, n_col_blocks;
  float scale_log2;              // scale * log2(e)
};
hipError_t launch_replay_attn(int D, const ReplayAttnArgs &a, hipStream_t s);

// Merge of the one-pass replay: candidate k of column c from the sinks'
// partial, the partials of the splits that lie inside the window and the
// edge partial of the split that holds the window's edge.
struct ReplayMergeArgs {
  const float *part;             // as in ReplayAttnArgs
  const float *win_ml;
  float *outs;                   // [n_windows + 1][n_cols][D], full last; on entry
                                 // a window's rows hold its edge partial's acc
  const int32_t *rows;
  int32_t windows[kMaxWindows];
  float k_scale[kMaxItems];      // per kv head: the keys' logit scale
  float v_scale[kMaxItems];      //   and the values' scale (fp8; else 1)
  int32_t n_windows, n_splits, tiles_per_split;
  int32_t n_cols, n_q_heads, group, n_sinks;
  float scale_log2;
};
hipError_t launch_replay_merge(int D, const ReplayMergeArgs &a, hipStream_t s);
constexpr int kReplayTilesPerSplit = 128;   // 32-key tiles per split, at most
#ifndef HWKV_REPLAY_MIN_TILES
#define HWKV_REPLAY_MIN_TILES 8
#endif
// A short trace takes smaller splits (as many as the workspace holds, of at
// least this many tiles), so that the launch still has workgroups for every
// CU.
constexpr int kReplayMinTilesPerSplit = HWKV_REPLAY_MIN_TILES;
hipError_t launch_calib_means(const CalibArgs &a, hipStream_t s);

}  // namespace hwkv

// Kernel arguments travel by value; the kernarg segment is limited to 4 KiB.
static_assert(sizeof(hwkv::DecodeArgs) <= 4096, "decode kernarg too large");
static_assert(sizeof(hwkv::WriteArgs) <= 4096, "write kernarg too large");
static_assert(sizeof(hwkv::AppendArgs) <= 4096, "append kernarg too large");
static_assert(sizeof(hwkv::PageUpdateArgs) <= 4096, "page update kernarg too large");
static_assert(sizeof(hwkv::StageArgs) <= 4096, "stage kernarg too large");
static_assert(sizeof(hwkv::StageChunkArgs) <= 4096, "stage chunk kernarg too large");
static_assert(sizeof(hwkv::PrefillAttnArgs) <= 4096, "prefill kernarg too large");
static_assert(sizeof(hwkv::ReplayAttnArgs) <= 4096, "replay kernarg too large");
static_assert(sizeof(hwkv::ReplayMergeArgs) <= 4096, "replay merge kernarg too large");
