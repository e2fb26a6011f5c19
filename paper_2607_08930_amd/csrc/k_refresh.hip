// Dual-cache refresh at a block start (the dual cache of Fast-dLLM that the
// paper integrates, Sections "Experimental setup" and "Diffusion LLM Inference
// Optimization"; position ids of paragraph "Logical positional alignment").
//
// The refresh forward recomputes the KV of every cell of a request's logical
// row and attends every position to the whole row (bidirectional). Per layer
// this file runs the two parts that do not need model weights:
//
// k_refresh_kv   rotary embedding of the keys at their position ids (the
//                count of real tokens before the cell, i.e. the cell's logical
//                position) and the scatter of rotated keys and plain values
//                from the token-major projections into the head-major cache.
//                HBM-bound: every byte is read once and written once.
// k_refresh_attn full-row attention over the refreshed cache, the queries
//                rotated as they are loaded. A workgroup of four waves owns
//                128 query positions of one head, 32 queries per wave
//                (32x32x16 MFMAs), and two workgroups share a CU (two waves
//                per SIMD), so one workgroup's prologue (first tiles, queries
//                and their rotation) runs beside the other's loop. K/V tiles
//                of 32 keys stream HBM/L2 -> LDS by direct DMA through a
//                5-stage ring, two tiles in flight. Inside a wave the loop is
//                software-pipelined by
//                32-key sub-tiles: while the exponentials of sub-tile u run on
//                the VALU, the matrix core computes the scores of u + 1 and
//                accumulates P V of u - 1.
#include "bs_lds.h"
#include "bs_refresh.h"

namespace bs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4;

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ inline uint32_t pack_bf16(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) | ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
}

// Rotate the feature pairs (x1[e], x2[e]) of 8 consecutive features f0 .. f0+7
// of the first half (partners f + D/2 in x2) by the angle pos * exp2(f * nl2b).
// The angle is formed in turns, pos * exp2(f * nl2b - log2(2 pi)); its
// fractional part (exact) feeds the hardware sine and cosine, which take
// turns. The fp32 roundings of the inverse frequency and of the product leave
// an angle error of a few 2^-23 relative, under 4e-4 rad for positions below
// 2048.
__device__ inline void rope8(v4u& x1, v4u& x2, int f0, float pos, float nl2b) {
  constexpr float kNegLog2TwoPi = -2.6514961294723187f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float a[2], b[2];
    a[0] = bf16_lo(x1[w]); a[1] = bf16_hi(x1[w]);
    b[0] = bf16_lo(x2[w]); b[1] = bf16_hi(x2[w]);
    float ya[2], yb[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const float turns = pos * __builtin_amdgcn_exp2f(fmaf((float)(f0 + 2 * w + e), nl2b, kNegLog2TwoPi));
      const float fr = __builtin_amdgcn_fractf(turns);
      const float sn = __builtin_amdgcn_sinf(fr), cs = __builtin_amdgcn_cosf(fr);
      ya[e] = a[e] * cs - b[e] * sn;
      yb[e] = b[e] * cs + a[e] * sn;
    }
    x1[w] = pack_bf16(ya[0], ya[1]);
    x2[w] = pack_bf16(yb[0], yb[1]);
  }
}

// ------------------------------------------------------------------ keys/values
// Thread u of request blockIdx.y: cell t = u / (Hkv * HC), KV head c, and the
// 16-byte chunk pair (ch, ch + HC) of that head's row (features 8 ch .. + 7 and
// their rotation partners D/2 + 8 ch .. + 7).
template <int D>
__global__ __launch_bounds__(256) void k_refresh_kv(RefKvArgs a) {
  constexpr int HC = D / 16;
  const bs_req_desc r = a.reqs[blockIdx.y];
  const int len = r.p + r.g;
  const int u = blockIdx.x * 256 + threadIdx.x;
  if (u >= len * a.Hkv * HC) return;
  const int ch = u % HC, c = (u / HC) % a.Hkv, t = u / (HC * a.Hkv);
  const int64_t src = (((int64_t)r.row * a.W + r.off + t) * a.Hkv + c) * D + ch * 8;
  const int64_t dst = (((int64_t)r.row * a.Hkv + c) * a.W + r.off + t) * D + ch * 8;
  v4u k1 = ld16(a.k + src), k2 = ld16(a.k + src + D / 2);
  const v4u v1 = ld16(a.v + src), v2 = ld16(a.v + src + D / 2);
  if (a.rope) rope8(k1, k2, ch * 8, (float)t, a.nl2b);
  st16(a.k_cache + dst, k1);
  st16(a.k_cache + dst + D / 2, k2);
  st16(a.v_cache + dst, v1);
  st16(a.v_cache + dst + D / 2, v2);
}

// ------------------------------------------------------------------ attention
// XOR swizzle of a cache row's 16-byte slots in LDS (D = 128: 16 slots) for
// an LDS that serves 256 bytes (64 banks of 4 bytes) per cycle. The 32 lanes
// of one transposed V read cover rows r0 .. r0 + 3 (r0 % 4 == 0) at chunks
// 4 t .. 4 t + 3: row bits 0..1 move to slot bits 2..3, so those reads land
// in 16 distinct slots; row bits 2..3 move to slot bits 0..1, so any 16
// consecutive rows still get distinct slots for one chunk (the K reads).
__device__ inline int swz16(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

__device__ inline float vmax(float x, float y) { return __builtin_elementwise_maximum(x, y); }

// lsum + the eight bf16 weights in p (the values the P V MFMA consumes)
__device__ inline float add_weights(float lsum, const bf16x8_t& p) {
  const bf16x2_t one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int k = 0; k < 4; ++k) lsum = __builtin_amdgcn_fdot2_f32_bf16(bf16x2_t{p[2 * k], p[2 * k + 1]}, one, lsum, false);
  return lsum;
}

// NW waves of QW 32-query blocks each (NW * QW * 32 = 256 queries per
// workgroup) share the K/V ring. QW = 2 feeds every LDS fragment to two
// MFMAs but needs about 400 registers (one wave per SIMD, so nothing hides
// the softmax arithmetic and the LDS latency: 20% slower on the Dream-7B
// shape); QW = 1 reads twice the LDS bytes per MFMA and fits two waves per
// SIMD (222 VGPRs), which is what the launch uses.
template <int D, int QW, int NW>
__global__ __launch_bounds__(64 * NW, 2) void k_refresh_attn(RefArgs a) {
  static_assert(D == 128, "the refresh attention is laid out for D = 128");
  static_assert(NW * QW * 32 == kRefQ, "a workgroup covers kRefQ queries");
  constexpr int KT = kRefKT, NS = kRefNS;
  constexpr int NKK = D / 16;        // K-steps of a score MFMA
  constexpr int NDT = D / 32;        // 32-feature output tiles
  constexpr int TILE = KT * D;       // elements of one K (or V) tile
  constexpr int STAGE = 2 * TILE;    // K tile, then V tile
  constexpr int SPT = KT / 32;       // 32-key sub-tiles per tile
  constexpr int PB = STAGE * 2 / 1024 / NW;   // 1 KiB DMA blocks per stage and wave
  constexpr int WPT = NW / 2;        // waves per tensor (K, then V)
  __shared__ __align__(1024) uint16_t ring[NS * STAGE];

  const RefItem it = a.items[blockIdx.x];
  if (it.row < 0) return;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, g = lane >> 5, n = lane & 31;
  const int len = it.len, h = it.h, c = h / a.G;
  const int ntiles = (len + KT - 1) / KT, nsub = (len + 31) / 32;
  const int qbase = it.q0 + 32 * QW * w;             // first query of this wave
  const bool active = qbase < len;                   // wave-uniform

  const int64_t cache_off = (((int64_t)it.row * a.Hkv + c) * a.W + it.off) * D;
  const uint16_t* kcb = a.k_cache + cache_off;
  const uint16_t* vcb = a.v_cache + cache_off;

  // DMA: wave w moves PB blocks of a stage; the first NW/2 waves the K tile,
  // the others the V tile. Block rb of a tile covers its rows 4 rb .. + 3;
  // lane l fills row 4 rb + l / 16, slot l % 16, from global chunk
  // slot ^ swz(row).
  const int tensor = w / WPT;
  const uint16_t* tb_src = tensor ? vcb : kcb;
  const uint32_t ring_lds = lds_addr(ring);
  auto issue = [&](int tile) {
    const uint32_t sbase = __builtin_amdgcn_readfirstlane(ring_lds + (uint32_t)((tile % NS) * STAGE * 2));
    const int t0 = tile * KT;
    if (t0 + KT <= len) {
      const uint64_t base = uniform64(tb_src + (int64_t)t0 * D);
#pragma unroll
      for (int k = 0; k < PB; ++k) {
        const int rb = (w % WPT) * PB + k;
        const int row = rb * 4 + (lane >> 4);
        const int chunk = (lane & 15) ^ swz16(row);
        dma16_sv(sbase + (uint32_t)((tensor * TILE + rb * 4 * D) * 2), base, (uint32_t)(row * D + chunk * 8) * 2u);
      }
    } else {
      // ragged last tile: rows past the row end repeat its last key (masked)
#pragma unroll
      for (int k = 0; k < PB; ++k) {
        const int rb = (w % WPT) * PB + k;
        const int row = rb * 4 + (lane >> 4);
        const int chunk = (lane & 15) ^ swz16(row);
        const int t = min(t0 + row, len - 1);
        dma16(sbase + (uint32_t)((tensor * TILE + rb * 4 * D) * 2), tb_src + (int64_t)t * D + chunk * 8);
      }
    }
  };

  // prologue: tiles 0 .. 2 in flight before the queries load
  issue(0);
  if (ntiles > 1) issue(1);
  if (ntiles > 2) issue(2);

  // queries of this lane's column n of each query block, rotated, as MFMA B
  // operands: feature 16 kk + 8 g + e; the rotation partner of kk < NKK/2 is
  // chunk kk + NKK/2 of the same lane
  bf16x8_t qb[QW][NKK];
#pragma unroll
  for (int b = 0; b < QW; ++b) {
    const int j = min(qbase + 32 * b + n, len - 1);
    const uint16_t* qp = a.q + (((int64_t)it.row * a.W + it.off + j) * a.Hq + h) * D;
    v4u x[NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) x[kk] = ld16(qp + 16 * kk + 8 * g);
    if (a.rope) {
#pragma unroll
      for (int kk = 0; kk < NKK / 2; ++kk) rope8(x[kk], x[kk + NKK / 2], 16 * kk + 8 * g, (float)j, a.nl2b);
    }
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) qb[b][kk] = __builtin_bit_cast(bf16x8_t, x[kk]);
  }

  // loop-invariant LDS element offsets of this lane's K and V fragments
  int koff[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) koff[kk] = n * D + (((2 * kk + g) ^ swz16(n)) * 8);
  const int q16 = lane >> 4, j16 = lane & 15;
  const int vrow = 4 * (q16 >> 1) + (j16 >> 2);
  int voff[NDT][2][2];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int row = 16 * ks + 8 * h2 + vrow;
        const int col = 32 * dt + 16 * (q16 & 1) + 4 * (j16 & 3);
        voff[dt][ks][h2] = row * D + (((col >> 3) ^ swz16(row)) * 8) + (col & 7);
      }

  f32x16_t o[QW][NDT];
#pragma unroll
  for (int b = 0; b < QW; ++b)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) o[b][dt][rr] = 0.0f;
  float mrun[QW], lsum[QW], alpha_pend[QW];
#pragma unroll
  for (int b = 0; b < QW; ++b) {
    mrun[b] = -__builtin_inff();
    lsum[b] = 0.0f;
    alpha_pend[b] = 1.0f;
  }
  bool resc_pend = false;

  // K rows of sub-tile u (32 keys) start at element sub_k(u); its V rows at + TILE
  auto sub_k = [&](int u) { return ((u / SPT) % NS) * STAGE + (u % SPT) * 32 * D; };
  auto vfrag = [&](const uint16_t* vs, int dt, int ks) {
    const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vs + voff[dt][ks][0]));
    const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vs + voff[dt][ks][1]));
    return (bf16x8_t)__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  };
  auto rescale = [&]() {
#pragma unroll
    for (int b = 0; b < QW; ++b)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) o[b][dt][rr] *= alpha_pend[b];
  };

  // tile 0 landed (tiles 1, 2 may still be in flight), visible to all waves
  if (ntiles > 2)
    wait_vm_c<2 * PB>();
  else if (ntiles > 1)
    wait_vm_c<PB>();
  else
    wait_vm_c<0>();
  __syncthreads();

  // two sets of score and probability registers, used in turn by the two
  // halves of each loop trip (no register copies between sub-tiles)
  f32x16_t sA[QW], sB[QW];
  bf16x8_t pA[QW][2], pB[QW][2];
#pragma unroll
  for (int b = 0; b < QW; ++b)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) pA[b][ks][e] = (__bf16)0.0f;
  if (active) {
#pragma unroll
    for (int b = 0; b < QW; ++b)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) sA[b][rr] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(ring + koff[kk]);
#pragma unroll
      for (int b = 0; b < QW; ++b) sA[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qb[b][kk], sA[b], 0, 0, 0);
    }
  }

  // one sub-tile u: sc holds its scores, pprev the probabilities of u - 1;
  // writes the scores of u + 1 to sn and the probabilities of u to pcur
  auto sub_tile = [&](int u, f32x16_t (&sc)[QW], f32x16_t (&sn)[QW], const bf16x8_t (&pprev)[QW][2],
                      bf16x8_t (&pcur)[QW][2]) {
    const int un = u + 1;
    if (un < nsub && un % SPT == 0) {
      // sub-tile un opens tile T: it has landed once only tile T + 1 (if
      // issued) is in flight. Tile T + 2 refills the slot of tile T + 2 - NS;
      // P V runs one sub-tile behind the scores, so this step still reads V
      // of sub-tile T SPT - 2, in tile T - ceil(2 / SPT): the refilled tile
      // must be older than that.
      static_assert(NS >= 3 + (SPT + 1) / SPT, "ring too short for the lagging P V");
      const int T = un / SPT;
      if (T + 1 < ntiles)
        wait_vm_c<PB>();
      else
        wait_vm_c<0>();
      __syncthreads();
      if (T + 2 < ntiles) issue(T + 2);
    }
    if (!active) return;
    // a reference max raised in the previous sub-tile rescales the
    // accumulators now, after P V of its predecessor and before its own (at
    // the top, so the tail stays one basic block in which the exponentials
    // and the MFMAs can interleave)
    if (resc_pend) {
      rescale();
      resc_pend = false;
    }
    // K fragments of sub-tile u + 1 (on the last sub-tile a resident one
    // again, its scores discarded), issued first so their latency hides under
    // the softmax arithmetic; V of u - 1 (of sub-tile 0 at u = 0, with zero
    // weights)
    const uint16_t* kt = ring + sub_k(un < nsub ? un : u);
    const uint16_t* vs = ring + sub_k(u > 0 ? u - 1 : 0) + TILE;
    bf16x8_t kf[NKK];
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) kf[kk] = *reinterpret_cast<const bf16x8_t*>(kt + koff[kk]);
    const int k0 = u * 32;
    if (k0 + 32 > len) {                               // ragged last sub-tile
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int key = k0 + 8 * (rr >> 2) + 4 * g + (rr & 3);
        if (key >= len) {
#pragma unroll
          for (int b = 0; b < QW; ++b) sc[b][rr] = -__builtin_inff();
        }
      }
    }
    // running max per query (log2 units), lazily raised: the reference max
    // moves only when a score exceeds it by 2^8, so the accumulators are
    // rescaled a handful of times per row (alpha = 1 when it stays)
#pragma unroll
    for (int b = 0; b < QW; ++b) {
      float mx = vmax(sc[b][0], sc[b][1]);
#pragma unroll
      for (int rr = 2; rr < 16; ++rr) mx = vmax(mx, sc[b][rr]);
      // the other half-wave holds the other 16 keys of this query
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = vmax(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * a.scale_log2e;
      const bool resc = __builtin_amdgcn_ballot_w64(mx > mrun[b] + 8.0f) != 0;
      const float mnew = resc ? fmaxf(mrun[b], mx) : mrun[b];
      alpha_pend[b] = __builtin_amdgcn_exp2f(mrun[b] - mnew);
      lsum[b] *= alpha_pend[b];
      mrun[b] = mnew;
      resc_pend |= resc;
    }
    // probabilities of sub-tile u on the VALU, interleaved with the matrix
    // core's scores of u + 1 and P V of u - 1
#pragma unroll
    for (int b = 0; b < QW; ++b) {
      const float nm = -mrun[b];
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const float pr = __builtin_amdgcn_exp2f(fmaf(sc[b][rr], a.scale_log2e, nm));
        pcur[b][rr >> 3][rr & 7] = (__bf16)pr;
      }
      lsum[b] = add_weights(add_weights(lsum[b], pcur[b][0]), pcur[b][1]);
    }
#pragma unroll
    for (int b = 0; b < QW; ++b)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) sn[b][rr] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk)
#pragma unroll
      for (int b = 0; b < QW; ++b) sn[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qb[b][kk], sn[b], 0, 0, 0);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t va = vfrag(vs, dt, ks);
#pragma unroll
        for (int b = 0; b < QW; ++b)
          o[b][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pprev[b][ks], o[b][dt], 0, 0, 0);
      }
    // schedule: the max/rescale arithmetic, then one MFMA per few VALU ops
    __builtin_amdgcn_sched_group_barrier(0x002, 20 * QW, 0);
#pragma unroll
    for (int i = 0; i < 16 * QW; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    }
  };

  int u = 0;
  for (; u + 1 < nsub; u += 2) {
    sub_tile(u, sA, sB, pA, pB);
    sub_tile(u + 1, sB, sA, pB, pA);
  }
  if (u < nsub) {                                   // odd count: the last sub-tile's probabilities end in pB
    sub_tile(u, sA, sB, pA, pB);
#pragma unroll
    for (int b = 0; b < QW; ++b) {
      pA[b][0] = pB[b][0];
      pA[b][1] = pB[b][1];
    }
  }
  if (!active) return;
  if (resc_pend) rescale();
  {
    const uint16_t* vs = ring + sub_k(nsub - 1) + TILE;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8_t va = vfrag(vs, dt, ks);
#pragma unroll
        for (int b = 0; b < QW; ++b)
          o[b][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pA[b][ks], o[b][dt], 0, 0, 0);
      }
  }

  // lane (g, n): O^T[feature 32 dt + 8 (rr / 4) + 4 g + rr % 4][query n of block b]
  typedef uint32_t v2u __attribute__((ext_vector_type(2)));
#pragma unroll
  for (int b = 0; b < QW; ++b) {
    const int j = qbase + 32 * b + n;
    const float lt = lsum[b] + __shfl_xor(lsum[b], 32, 64);
    if (j < len) {
      const float inv = 1.0f / lt;
      uint16_t* op = a.out + (((int64_t)it.row * a.W + it.off + j) * a.Hq + h) * D;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const uint32_t w0 = pack_bf16(o[b][dt][4 * rq + 0] * inv, o[b][dt][4 * rq + 1] * inv);
          const uint32_t w1 = pack_bf16(o[b][dt][4 * rq + 2] * inv, o[b][dt][4 * rq + 3] * inv);
          *reinterpret_cast<v2u*>(op + dt * 32 + 8 * rq + 4 * g) = v2u{w0, w1};
        }
    }
  }
}

}  // namespace

hipError_t launch_refresh_kv(const RefKvArgs& a, int n, int max_len, hipStream_t s) {
  constexpr int D = 128;
  const int64_t units = (int64_t)max_len * a.Hkv * (D / 16);
  const dim3 grid((unsigned)((units + 255) / 256), (unsigned)n);
  hipLaunchKernelGGL(k_refresh_kv<D>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_refresh_attn(const RefArgs& a, int n_items, hipStream_t s) {
  constexpr int QW = 1, NW = kRefQ / (32 * QW);
  hipLaunchKernelGGL((k_refresh_attn<128, QW, NW>), dim3((unsigned)n_items), dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

}  // namespace bs
