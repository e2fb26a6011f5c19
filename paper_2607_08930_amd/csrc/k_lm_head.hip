// Output head fused with confidence-aware parallel decoding (paragraph
// "Vectorized mixed-schedule execution"; the greedy parallel decoding of
// Fast-dLLM, "Implementation details"). The logit of vocabulary entry v at a
// masked block position is the inner product of the position's final hidden
// state with row v of the output-head matrix. The logits are reduced to
// (max, smallest index attaining it, sum of exp(x - max)) as they leave the
// matrix cores and are never stored; the selection then runs unchanged.
//
// k_lm_pack   once per model: lays the output-head matrix out as the
//             contiguous 16 KiB slabs the ring stages copy (the [V][d] layout
//             would read 64 bytes from each of 256 rows 2 d bytes apart).
// k_lm_rows   one workgroup lists the masked rows (j < B_i, masked) of the
//             compact [n][L] block state in increasing order and counts them.
// k_lm_head   C^T = W H^T on v_mfma_f32_32x32x16_bf16 over 256 (vocabulary)
//             x 256 (listed rows) tiles; K moves HBM -> LDS in 32-wide slices
//             through a 4-deep ring by direct DMA. Vocabulary is the MFMA M
//             axis, so a lane holds one row's column of 16 logits per 32x32
//             block: the epilogue reduces 64 logits per lane and exchanges
//             once with the other half-wave. One DecPartial per (row,
//             128-entry vocabulary slice).
// k_lm_merge  one wave per listed row merges its slices into the DecPartial
//             the selection reads.
#include <float.h>
#include <limits.h>

#include "bs_internal.h"
#include "bs_lds.h"

namespace bs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
constexpr float kLog2e = 1.4426950408889634f;

__device__ inline bool listed(const LmArgs& a, int x) {
  const int i = x / a.L, j = x - i * a.L;
  const Geo q = geo_of(a.reqs[i], a.L);
  return j < q.B && a.masked[x] != 0;
}

__global__ __launch_bounds__(1024) void k_lm_rows(LmArgs a) {
  __shared__ int sc[1024];
  const int total = a.n * a.L, t = threadIdx.x;
  const int per = (total + 1023) / 1024;
  const int x0 = min(t * per, total), x1 = min(x0 + per, total);
  int c = 0;
  for (int x = x0; x < x1; ++x) c += listed(a, x) ? 1 : 0;
  sc[t] = c;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {      // inclusive scan of the per-thread counts
    const int v = t >= o ? sc[t - o] : 0;
    __syncthreads();
    sc[t] += v;
    __syncthreads();
  }
  int pos = sc[t] - c;
  for (int x = x0; x < x1; ++x)
    if (listed(a, x)) a.rows[pos++] = x;
  if (t == 1023) *a.count = sc[1023];
}

// LDS rows hold 32 bf16 of K (64 bytes, four 16-byte chunks). Chunk c of tile
// row r sits in slot c ^ ((r >> 2) & 3): the 32 rows one MFMA operand read
// touches then spread two per bank group.
constexpr int kTile = kLmNT * kLmKT;        // elements of one operand tile (W or H): 16 KiB
constexpr int kStage = 2 * kTile;           // W tile, then H tile

__global__ __launch_bounds__(512, 1) void k_lm_head(LmArgs a) {
  static_assert(kLmNT == 256 && kLmMT == 256 && kLmKT == 32 && kLmNS == 4, "tiling below assumes these");
  __shared__ __align__(1024) uint16_t ring[kLmNS * kStage];   // 128 KiB
  const int count = *a.count;
  const int nvt = (a.V + kLmNT - 1) / kLmNT;
  const int nrt = (a.n * a.L + kLmMT - 1) / kLmMT;
  // Workgroups b = x + 8 q run on XCD x. With one or two row tiles in use,
  // XCD x serves row tile x % nact only: that tile's hidden rows stay in its
  // L2 while W streams past, and the XCDs serving a row tile split the
  // vocabulary tiles round-robin (W is read once per row tile). With more
  // row tiles, consecutive q on one XCD take all row tiles of one vocabulary
  // tile, which then share that XCD's L2 copy of the W slab (W is read about
  // once; the hidden rows come from L2 or the Infinity Cache). Measured on
  // the LLaDA-8B and Dream-7B head shapes, each order is the faster one in
  // its range.
  if (count == 0) return;
  const int x = (int)(blockIdx.x & 7), q = (int)(blockIdx.x >> 3);
  const int nact = (count + kLmMT - 1) / kLmMT;
  int vt, rt;
  if (nact <= 2) {
    rt = x % nact;
    const int gsize = (8 - rt + nact - 1) / nact;
    vt = q * gsize + x / nact;
    if (vt >= nvt) return;
  } else {
    const int total = nvt * nrt, per_xcd = (total + 7) / 8;
    const int lin = x * per_xcd + q;
    if (q >= per_xcd || lin >= total) return;
    vt = lin / nrt;
    rt = lin - vt * nrt;
  }
  const int v0 = vt * kLmNT, r0 = rt * kLmMT;
  if (r0 >= count) return;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;

  // DMA: a stage is 32 blocks of 1 KiB (16 tile rows each); wave w issues
  // blocks 4w .. 4w + 3: W rows for w < 4, H rows for w >= 4. Lane l fills
  // slot l & 3 of tile row 16 b + (l >> 2) with global chunk
  // (l & 3) ^ ((l >> 4) & 3).
  const int gch = (lane & 3) ^ ((lane >> 4) & 3);
  const bool wside = w < 4;
  const int b0 = (w & 3) * 4;
  // W comes from the packed slabs (already in LDS order: block b of slab
  // (vt, t) is one contiguous KiB); H rows are gathered through the row list.
  const uint16_t* hp[4];                       // H: listed row's K start + chunk
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int row = 16 * (b0 + q) + (lane >> 2);
    hp[q] = wside ? nullptr : a.hidden + (int64_t)a.rows[min(r0 + row, count - 1)] * a.d + gch * 8;
  }
  const uint32_t ring_lds = lds_addr(ring) + (uint32_t)((wside ? 0 : kTile * 2) + b0 * 1024);
  const uint16_t* wslab = a.w + (int64_t)vt * (a.d / kLmKT) * kTile + b0 * 512;
  // block q of this wave's share of stage t
  auto issue1 = [&](int t, int q) {
    const uint32_t sb = __builtin_amdgcn_readfirstlane(ring_lds + (uint32_t)((t % kLmNS) * kStage * 2));
    if (wside)
      dma16_sv(sb + q * 1024, uniform64(wslab + (int64_t)t * kTile + q * 512), (uint32_t)(lane * 16));
    else
      dma16(sb + q * 1024, hp[q] + t * kLmKT);
  };
  auto issue = [&](int t) {
#pragma unroll
    for (int q = 0; q < 4; ++q) issue1(t, q);
  };

  // MFMA operands: wave (wv, wr) = (w & 1, w >> 1) computes vocabulary rows
  // 128 wv .. + 128 (four 32-row blocks) x hidden rows 64 wr .. + 64 (two).
  // Lane (g, n) reads row n of a block, chunk 2 s + g of the 32-wide slice.
  const int g = lane >> 5, n = lane & 31;
  const int wv = w & 1, wr = w >> 1;
  int off[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) off[s] = n * kLmKT + (((2 * s + g) ^ ((n >> 2) & 3)) * 8);
  f32x16_t acc[4][2];
#pragma unroll
  for (int vb = 0; vb < 4; ++vb)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[vb][rb][r] = 0.0f;

  const int nk = a.d / kLmKT;
#pragma unroll
  for (int t = 0; t < kLmNS - 1; ++t)
    if (t < nk) issue(t);
  for (int t = 0; t < nk; ++t) {
    // stage t landed once only the (at most two) later stages' four blocks each remain
    const int ahead = min(nk - 1 - t, kLmNS - 2);
    if (ahead >= 2)
      wait_vm_c<8>();
    else if (ahead == 1)
      wait_vm_c<4>();
    else
      wait_vm_c<0>();
    // after the barrier every wave is done with stage t - 1, whose slot is
    // refilled: one DMA block after every four MFMAs
    __syncthreads();
    const bool refill = t + kLmNS - 1 < nk;
    const uint16_t* st = ring + (t % kLmNS) * kStage;
    const uint16_t* at = st + (128 * wv) * kLmKT;
    const uint16_t* bt = st + kTile + (64 * wr) * kLmKT;
    bf16x8_t A[2][4], B[2][2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) A[s][vb] = *reinterpret_cast<const bf16x8_t*>(at + 32 * vb * kLmKT + off[s]);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) B[s][rb] = *reinterpret_cast<const bf16x8_t*>(bt + 32 * rb * kLmKT + off[s]);
    }
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
          acc[vb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[s][vb], B[s][rb], acc[vb][rb], 0, 0, 0);
        if (vb & 1) {
          __builtin_amdgcn_sched_barrier(0);
          if (refill) issue1(t + kLmNS - 1, 2 * s + (vb >> 1));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
  }

  // Epilogue: lane (g, n) holds C^T[vocab v][row n] for
  // v = v0 + 128 wv + 32 vb + 8 (r / 4) + 4 g + r % 4.
  const int vbase = v0 + 128 * wv + 4 * g;
  if (v0 + kLmNT > a.V) {                      // ragged last vocabulary tile only
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (vbase + 32 * vb + 8 * (r >> 2) + (r & 3) >= a.V) {
          acc[vb][0][r] = -__builtin_inff();
          acc[vb][1][r] = -__builtin_inff();
        }
  }
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    float mx = -__builtin_inff();
    int am = INT_MAX;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float x = acc[vb][rb][r];
        const int id = vbase + 32 * vb + 8 * (r >> 2) + (r & 3);
        if (x > mx || (x == mx && id < am)) {
          mx = x;
          am = id;
        }
      }
    const float mo = __shfl_xor(mx, 32, 64);
    const int ao = __shfl_xor(am, 32, 64);
    const float M = fmaxf(mx, mo);
    int A = mx == M ? am : INT_MAX;
    if (mo == M) A = min(A, ao);
    const float nm = M == -__builtin_inff() ? 0.0f : -M * kLog2e;   // a slice past V sums to 0
    float sum = 0.0f;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sum += __builtin_amdgcn_exp2f(fmaf(acc[vb][rb][r], kLog2e, nm));
    sum += __shfl_xor(sum, 32, 64);
    const int slot = r0 + 64 * wr + 32 * rb + n;
    if (g == 0 && slot < count) {
      DecPartial p;
      p.m = M;
      p.s = sum;
      p.a = A;
      p.pad = 0;
      a.slices[(int64_t)slot * a.parts + 2 * vt + wv] = p;
    }
  }
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline int wave_min_i(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}

__global__ __launch_bounds__(64) void k_lm_merge(LmArgs a) {
  const int x = blockIdx.x, lane = threadIdx.x;
  if (x >= *a.count) return;
  const DecPartial* p = a.slices + (int64_t)x * a.parts;
  float M = -__builtin_inff();
  for (int k = lane; k < a.parts; k += 64) M = fmaxf(M, p[k].m);
  M = wave_max(M);
  float S = 0.0f;
  int A = INT_MAX;
  for (int k = lane; k < a.parts; k += 64) {
    const DecPartial q = p[k];
    if (q.m != -__builtin_inff()) S += q.s * __builtin_amdgcn_exp2f((q.m - M) * kLog2e);
    if (q.m == M) A = min(A, q.a);
  }
  S = wave_sum(S);
  A = wave_min_i(A);
  if (lane == 0) {
    DecPartial r;
    r.m = M;
    r.s = S;
    r.a = A;
    r.pad = 0;
    a.row_part[a.rows[x]] = r;
  }
}

// One thread per 16-byte chunk of the packed matrix: slab (vt, kt), row r,
// slot s holds W[vt * 256 + r][32 kt + 8 (s ^ ((r >> 2) & 3)) .. + 8], or
// zeros for rows past V.
__global__ __launch_bounds__(256) void k_lm_pack(const uint16_t* w, int64_t ldw, int V, int d, uint16_t* packed) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;      // chunk index
  const int nkt = d / kLmKT;
  const int64_t total = (int64_t)((V + kLmNT - 1) / kLmNT) * nkt * kLmNT * 4;
  if (x >= total) return;
  const int slot = (int)(x & 3), r = (int)((x >> 2) & (kLmNT - 1));
  const int64_t slab = x >> 10;                                     // 1024 chunks per slab
  const int kt = (int)(slab % nkt), vt = (int)(slab / nkt);
  const int v = vt * kLmNT + r;
  v4u val = v4u{0u, 0u, 0u, 0u};
  if (v < V) val = ld16(w + (int64_t)v * ldw + kt * kLmKT + (slot ^ ((r >> 2) & 3)) * 8);
  st16(packed + x * 8, val);
}

}  // namespace

hipError_t launch_lm_pack(const uint16_t* w, int64_t ldw, int V, int d, uint16_t* packed, hipStream_t s) {
  const int64_t chunks = (int64_t)((V + kLmNT - 1) / kLmNT) * (d / kLmKT) * kLmNT * 4;
  hipLaunchKernelGGL(k_lm_pack, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s, w, ldw, V, d, packed);
  return hipGetLastError();
}

hipError_t launch_lm_rows(const LmArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_rows, dim3(1), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_gemm(const LmArgs& a, hipStream_t s) {
  const int nvt = (a.V + kLmNT - 1) / kLmNT;
  const int nrt = (a.n * a.L + kLmMT - 1) / kLmMT;
  // enough workgroups per XCD for either order: nvt covers the one-row-tile
  // order (an XCD serves at most nvt vocabulary tiles), the other needs
  // ceil(nvt * nrt / 8)
  const int per_xcd = max((nvt * nrt + 7) / 8, nvt);
  hipLaunchKernelGGL(k_lm_head, dim3((unsigned)(8 * per_xcd)), dim3(512), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_lm_merge(const LmArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_lm_merge, dim3((unsigned)(a.n * a.L)), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace bs
