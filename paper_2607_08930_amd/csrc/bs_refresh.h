// Internal declarations of the dual-cache refresh (full-row attention with
// rotary embedding at explicit position ids) shared by its host entry point
// and its gfx950 kernels.
#pragma once

#include "bs_internal.h"

namespace bs {

constexpr int kRefQ = 128;     // query positions per workgroup (4 waves x 32)
constexpr int kRefKT = 32;     // keys per LDS stage
constexpr int kRefNS = 5;      // LDS stages (5 x 16 KiB of K and V: two workgroups per CU)

// One workgroup: query positions [q0, q0 + kRefQ) of one request row and one
// query head. row < 0 marks an empty slot of the XCD-ordered grid.
struct RefItem {
  int32_t row, off, len, h, q0, pad0, pad1, pad2;
};

struct RefArgs {
  const RefItem* items;
  int Hq, Hkv, G, W;
  float scale_log2e;      // softmax scale * log2(e)
  float nl2b;             // -2 log2(base) / D: inverse frequency of feature pair f is exp2(f * nl2b)
  int rope;               // 0: no rotation
  const uint16_t* q;      // [R][W][Hq][D] projections (not rotated)
  uint16_t* out;          // [R][W][Hq][D]
  const uint16_t* k_cache;  // [R][Hkv][W][D] rotated keys (written by the first launch)
  const uint16_t* v_cache;
};

struct RefKvArgs {
  const bs_req_desc* reqs;
  int Hkv, W;
  float nl2b;
  int rope;
  const uint16_t* k;  // [R][W][Hkv][D]
  const uint16_t* v;
  uint16_t* k_cache;  // [R][Hkv][W][D]
  uint16_t* v_cache;
};

// Rotated keys and the values of every listed request's logical cells into the
// cache (grid: one y-slice per request).
hipError_t launch_refresh_kv(const RefKvArgs& a, int n, int max_len, hipStream_t s);
// Full-row attention over the refreshed cache, one workgroup per item.
hipError_t launch_refresh_attn(const RefArgs& a, int n_items, hipStream_t s);

}  // namespace bs
