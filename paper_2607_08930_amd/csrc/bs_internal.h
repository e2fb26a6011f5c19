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
// One work item = (request, KV head) with the request's geometry resolved on
// the host, so a workgroup needs a single scalar load before its first DMA.
// An item may be one piece of a row: keys [64 t0, min(64 t1, len)), with its
// un-normalised output, running max and row sum going to partial slot `part`
// for a merge launch (split-KV); part < 0 marks a whole row (t0 = 0,
// t1 = ceil(len / 64)) written out directly.
struct AttnItem {
  int32_t req;   // request index (row of q / k_new / v_new / out)
  int32_t kvh;   // KV head
  int32_t len;   // logical row length p + g (keys [0, len))
  int32_t s;     // first block position
  int32_t B;     // block length
  int32_t row;   // dense row of the cache
  int32_t off;   // column of logical position 0
  int32_t rb;    // first 32-row block of the block served by this workgroup
  int32_t t0;    // first 64-key tile of this piece
  int32_t t1;    // one past its last tile
  int32_t part;  // partial slot of a split row, or -1
  int32_t pad;
};

// One split row: its pieces wrote partial slots [part0, part0 + nparts).
struct AttnMerge {
  int32_t req, kvh, rb, B;
  int32_t part0, nparts, pad0, pad1;
};

constexpr int kAttnTile = 64;                   // keys per tile of the shared-tile kernel
// floats of one wave's partial at head dimension D: O^T in accumulator order
// (D / 8 groups of 4 per lane, 64 lanes), then the running max (log2 units)
// and the row sum per lane
__host__ __device__ constexpr int part_wave_floats(int D) { return D / 8 * 64 * 4 + 2 * 64; }

struct AttnArgs {
  const bs_req_desc* reqs;
  const AttnItem* items;
  int n_items;
  int L, Hq, Hkv, D, G, RB;  // RB: 32-row blocks per head = ceil(L / 32)
  int RBW;                   // row blocks per workgroup: RB, or 1 when G * RB > 8 waves
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
  // NULL, or where one item per request (KV head 0, first row block) stores
  // the request's block mask word, read from `masked` (dense [R][W] box with
  // row stride msk_rs) for the row reductions that follow
  uint64_t* mask_words;
  const uint8_t* masked;
  int64_t msk_rs;
  // split-KV: partial slots (part_wave_floats(D) per wave of a workgroup) and the
  // rows the merge launch combines from them
  float* parts;
  const AttnMerge* merges;
  int n_merge;
};

constexpr int kMhaWaves = 4;  // waves (independent items) per workgroup of the single-wave bf16 kernel

hipError_t launch_attn_f32(const AttnArgs& a, int n_req, hipStream_t s);
hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------- decode
struct DecPartial {
  float m;    // max over the part
  float s;    // sum exp(x - m) over the part
  int32_t a;  // smallest index attaining m
  int32_t pad;
};

constexpr int kDecChunkBytes = 32768;  // logits bytes streamed per chunk of a row
constexpr int kDecPartChunks = 2;      // chunks per part: one workgroup streams one part of a row

// Parts a row of V elements of `eb` bytes is split into.
inline int dec_parts(int V, int eb) {
  const int64_t chunks = ((int64_t)V * eb + kDecChunkBytes - 1) / kDecChunkBytes;
  return (int)((chunks + kDecPartChunks - 1) / kDecPartChunks);
}

// Decode workspace: [n * L * parts] DecPartial part results, then [n] block
// mask words (bit j of word i: block position j of request i is masked; set
// by the fused step's attention, read by its row reductions).
inline size_t dec_parts_bytes(int n, int L, int parts) { return (size_t)n * L * parts * sizeof(DecPartial); }
inline size_t dec_workspace_bytes(int n, int L, int parts) { return dec_parts_bytes(n, L, parts) + (size_t)n * 8; }

struct DecArgs {
  const bs_req_desc* reqs;
  int n, L, V;
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
  int parts;       // parts per row
  DecPartial* part;
  // tokens/masked layout: compact [n][L] (dense == 0), or the dense [R][W]
  // boxes with these row strides in elements, block cell j of request i at
  // (row_i, off_i + s_i + j)
  int dense;
  int64_t tok_rs, msk_rs;
  int32_t* pos_out;  // [n][L] or NULL: s_i + j for j < B_i, else -1
  // NULL, or the block mask words of the requests (see dec_workspace_bytes):
  // the row reductions then walk a grid ordered by the k-th masked position
  // of each request and skip the descriptor and mask reads
  const uint64_t* words;
};

hipError_t launch_decode(const DecArgs& a, bs_dtype dt, hipStream_t s);

// launch_decode with mark(2) after the row reductions and mark(3) after the
// selection (the step's phase-timing event indices); mark returns a hipError_t.
template <class Mark>
hipError_t launch_decode_marked(const DecArgs& a, bs_dtype dt, hipStream_t s, Mark mark);
hipError_t launch_decode_rows(const DecArgs& a, bs_dtype dt, hipStream_t s);
hipError_t launch_decode_select(const DecArgs& a, hipStream_t s);

template <class Mark>
hipError_t launch_decode_marked(const DecArgs& a, bs_dtype dt, hipStream_t s, Mark mark) {
  hipError_t e = launch_decode_rows(a, dt, s);
  if (e == hipSuccess) e = mark(2);
  if (e == hipSuccess) e = launch_decode_select(a, s);
  if (e == hipSuccess) e = mark(3);
  return e;
}

// ---------------------------------------------------------------- output head
// Logits of the masked block rows from their hidden states, reduced on the fly
// into one DecPartial per (row, 128-entry vocabulary slice), then merged into
// the per-row part the selection reads.
constexpr int kLmNT = 256;  // vocabulary entries per workgroup tile
constexpr int kLmMT = 256;  // hidden rows per workgroup tile
constexpr int kLmKT = 32;   // reduction depth per LDS stage
constexpr int kLmNS = 4;    // LDS stages

inline int lm_parts(int V) { return 2 * ((V + kLmNT - 1) / kLmNT); }

// Workspace: count (16 B) | row list [n L] int32 | per-row parts [n L]
// DecPartial | slice parts [n L][lm_parts(V)] DecPartial.
inline size_t lm_rows_bytes(int n, int L) { return ((size_t)n * L * 4 + 15) / 16 * 16; }
inline size_t lm_workspace_bytes(int n, int L, int V) {
  return 16 + lm_rows_bytes(n, L) + (size_t)n * L * sizeof(DecPartial) +
         (size_t)n * L * lm_parts(V) * sizeof(DecPartial);
}

// Packed output-head matrix: one 16 KiB slab per (256-row vocabulary tile
// vt, 32-wide K slice kt), slab (vt, kt) at element (vt * (d / 32) + kt) *
// 8192, holding rows vt * 256 .. + 256 (rows past V zero) as 64-byte rows
// whose 16-byte chunk c sits in slot c ^ ((row >> 2) & 3) -- the LDS order,
// so a stage of the ring is one contiguous copy.
inline size_t lm_packed_bytes(int V, int d) { return (size_t)((V + kLmNT - 1) / kLmNT) * kLmNT * d * 2; }

struct LmArgs {
  const bs_req_desc* reqs;
  int n, L, d, V;
  const uint16_t* hidden;   // [n][L][d] bf16
  const uint16_t* w;        // packed (see lm_packed_bytes)
  const uint8_t* masked;    // compact [n][L]
  int32_t* count;           // masked rows
  int32_t* rows;            // their compact indices i * L + j, increasing
  DecPartial* slices;       // [n L][parts]
  int parts;
  DecPartial* row_part;     // [n L]: merged, read by the selection
};

hipError_t launch_lm_rows(const LmArgs& a, hipStream_t s);
hipError_t launch_lm_gemm(const LmArgs& a, hipStream_t s);
hipError_t launch_lm_merge(const LmArgs& a, hipStream_t s);
hipError_t launch_lm_pack(const uint16_t* w, int64_t ldw, int V, int d, uint16_t* packed, hipStream_t s);

// ---------------------------------------------------------------- gather / scatter
constexpr int kMaxGather = 4;  // tensors moved by one gather/scatter launch

struct GatherSet {
  int count;
  const void* dense[kMaxGather];   // [R][W] tensors (written by scatter)
  void* compact[kMaxGather];       // [n][L] tensors (written by gather)
  int64_t stride[kMaxGather];      // dense row stride in bytes
  int eb[kMaxGather];              // element bytes: 1, 2, 4, 8 or 16
};

hipError_t launch_gather(const bs_req_desc* reqs, int n, int L, const GatherSet& g, int32_t* pos, hipStream_t s);
hipError_t launch_scatter(const bs_req_desc* reqs, int n, int L, const GatherSet& g, hipStream_t s);

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
