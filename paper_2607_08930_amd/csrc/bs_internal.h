// Internal declarations shared by the host entry points and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "blockserve.h"

namespace bs {

// Block geometry of one request (Section "Problem formulation"): block k of
// K = ceil(g / L) covers logical positions [s, s + B), s = p + k L.
struct Geo {
  int s, B, len;
};

__host__ __device__ inline Geo geo_of(const bs_req_desc& r, int L) {
  Geo q;
  q.s = r.p + r.k * L;
  int rem = r.g - r.k * L;
  q.B = rem < L ? rem : L;
  q.len = r.p + r.g;
  return q;
}

// 16 bytes held in registers. A native clang vector (not HIP's uint4 struct):
// loads and copies of it stay plain vector operations, so arrays of them are
// kept in VGPRs instead of being lowered to memcpy into scratch.
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ inline v4u ld16(const void* p) { return *reinterpret_cast<const v4u*>(p); }
__device__ inline void st16(void* p, v4u v) { *reinterpret_cast<v4u*>(p) = v; }

// ---------------------------------------------------------------- attention
// One work item = (request, KV head, key range [t0, t1) of the logical row).
// Items with nsplit > 1 write unnormalised partials that a merge pass combines.
struct AttnItem {
  int32_t req;
  int32_t kvh;
  int32_t t0;
  int32_t t1;
  int32_t split;   // index of this range among the request's ranges
  int32_t nsplit;  // number of ranges of this request (1: write out directly)
  int32_t ws_slot; // first partial slot of this request (nsplit > 1)
  int32_t pad;
};

// Key range length of one split of the bf16 path. Fixed, so the split count of
// a request depends on its own length only (bitwise batch invariance).
constexpr int kAttnSplitKeys = 1024;

struct AttnArgs {
  const bs_req_desc* reqs;
  const AttnItem* items;
  int n_items;
  int L, Hq, Hkv, D, G, RB;  // RB: 32-row blocks per head = ceil(L / 32)
  int R, W;
  float scale_log2e;         // softmax scale * log2(e)
  float scale;               // softmax scale
  const void* q;
  const void* k_new;
  const void* v_new;
  void* k_cache;
  void* v_cache;
  void* out;
  int write_back;
  // split partials: per slot [L][Hq-group rows][D] fp32 O plus m and l
  float* ws_o;
  float* ws_ml;
};

hipError_t launch_attn_f32(const AttnArgs& a, int n_req, hipStream_t s);
hipError_t launch_attn_bf16(const AttnArgs& a, int n_req, int n_slots, hipStream_t s);

// ---------------------------------------------------------------- decode
struct DecPartial {
  float m;    // chunk max
  float s;    // sum exp(x - m) over the chunk
  int32_t a;  // smallest index attaining m
  int32_t pad;
};

constexpr int kDecChunkBytes = 65536;  // logits bytes per row chunk (one workgroup)

struct DecArgs {
  const bs_req_desc* reqs;
  int n, L, V, nchunk;
  const void* logits;
  int64_t row_stride;  // elements
  int32_t* tokens;
  uint8_t* masked;
  float tau;
  int q_min, eos_id;
  int32_t* n_unmasked;
  uint8_t* done;
  uint8_t* eos_seen;
  float* conf_out;
  DecPartial* part;
};

hipError_t launch_decode(const DecArgs& a, bs_dtype dt, hipStream_t s);

// ---------------------------------------------------------------- gather / scatter
hipError_t launch_gather(const bs_req_desc* reqs, int n, int L, const void* src, int64_t stride,
                         int eb, void* dst, int32_t* pos, hipStream_t s);
hipError_t launch_scatter(const bs_req_desc* reqs, int n, int L, const void* src, int eb,
                          void* dst, int64_t stride, hipStream_t s);

// ---------------------------------------------------------------- compaction
struct CopyUnit {
  int32_t seg;    // segment index
  int32_t chunk;  // chunk index within one (layer, tensor, head) run of the segment
};

constexpr int kCopyChunkBytes = 16384;

struct CopyArgs {
  const bs_copy_seg* segs;
  const CopyUnit* units;
  int n_units;
  int n_layers, Hkv;
  int64_t row_bytes;  // D * elem
  const char* src_k;
  const char* src_v;
  int64_t src_ls;
  int W_src;
  const char* stg_k;
  const char* stg_v;
  int64_t stg_ls;
  int W_stg;
  char* dst_k;
  char* dst_v;
  int64_t dst_ls;
  int W_dst;
};

hipError_t launch_compact(const CopyArgs& a, hipStream_t s);

}  // namespace bs
