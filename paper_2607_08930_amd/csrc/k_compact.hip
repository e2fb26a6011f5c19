// K4: KV scatter/compaction at a block boundary (Algorithm 1's evict/admit;
// Eq. 1 discussion of the shrinking box). A segment moves `len` positions of
// every (layer, K|V, KV head) run: in the [R][Hkv][W][D] box one such run is a
// contiguous len * D * elem bytes, so the copy is a batched set of contiguous
// byte ranges. Work unit = one 16 KiB chunk of one run; a grid-stride loop
// walks units with the chunk index fastest, so neighbouring workgroups stream
// neighbouring memory. Each thread issues its four 16-byte loads before any
// store. Loads and stores keep the default cache policy: the rows written here
// are read by the step's attention right after, and a non-temporal variant
// made the 32-layer churn step about 5% slower (two paired runs on one
// MI355X), through the attention that follows as much as through the copy.
#include "bs_internal.h"

namespace bs {
namespace {

constexpr int kThreads = 256;
constexpr int kPer = kCopyChunkBytes / (kThreads * 16);  // 4

__global__ __launch_bounds__(kThreads) void k_compact(CopyArgs a) {
  const int64_t total = (int64_t)a.n_units * a.Hkv * 2 * a.n_layers;
  for (int64_t u = blockIdx.x; u < total; u += gridDim.x) {
    const int cu = (int)(u % a.n_units);
    int64_t rest = u / a.n_units;
    const int h = (int)(rest % a.Hkv);
    rest /= a.Hkv;
    const int kv = (int)(rest % 2);
    const int l = (int)(rest / 2);
    const CopyUnit un = a.units[cu];
    const bs_copy_seg sg = a.segs[un.seg];
    const char* sbase;
    int64_t sls;
    int sW;
    if (sg.src_kind == 0) {
      sbase = kv ? a.src_v : a.src_k;
      sls = a.src_ls;
      sW = a.W_src;
    } else {
      sbase = kv ? a.stg_v : a.stg_k;
      sls = a.stg_ls;
      sW = a.W_stg;
    }
    const char* sp = sbase + l * sls + (((int64_t)sg.src_row * a.Hkv + h) * sW + sg.src_col) * a.row_bytes;
    char* dp = (kv ? a.dst_v : a.dst_k) + l * a.dst_ls +
               (((int64_t)sg.dst_row * a.Hkv + h) * a.W_dst + sg.dst_col) * a.row_bytes;
    const int64_t nbytes = (int64_t)sg.len * a.row_bytes;
    const int64_t start = (int64_t)un.chunk * kCopyChunkBytes;
    v4u v[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int64_t o = start + ((int64_t)k * kThreads + threadIdx.x) * 16;
      if (o < nbytes) v[k] = ld16(sp + o);
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int64_t o = start + ((int64_t)k * kThreads + threadIdx.x) * 16;
      if (o < nbytes) st16(dp + o, v[k]);
    }
  }
}

}  // namespace

hipError_t launch_compact(const CopyArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)a.n_units * a.Hkv * 2 * a.n_layers;
  if (total == 0) return hipSuccess;
  const int64_t cap = 256 * 32;  // 32 resident workgroups per CU at most
  const unsigned grid = (unsigned)(total < cap ? total : cap);
  hipLaunchKernelGGL(k_compact, dim3(grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace bs
