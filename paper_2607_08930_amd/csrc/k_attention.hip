// K2: dual-cache block attention (paragraph "Vectorized mixed-schedule
// execution"; dual cache of Fast-dLLM as integrated by the paper).
//
// The keys of request i are its logical row [0, p + g): cached prefix
// [0, s), the fresh block [s, s + B) read from k_new/v_new, and the cached
// masked suffix [s + B, p + g). Key t of the row is therefore fetched either
// from cache cell off + t of the request's dense row or from fresh row t - s;
// the stale block slot and the padding are never read. With write_back the
// fresh rows are also stored into the cache slot from the LDS tile that holds
// them (in-place KV update at the physical offsets of the active block), so
// they are read from memory once.
//
// bf16 path (gfx950 MFMA): one workgroup per (request, KV head) and one wave
// per (query head of the group, 32-row block of the active block), so the K/V
// tiles staged in LDS are shared by the whole query group (GQA). Per 32-key
// sub-tile a wave computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (keys on
// the M axis, queries on N), which leaves every lane holding one query's
// column: the online-softmax max/sum need one cross-half exchange only. The
// probabilities are then fed straight from the accumulator registers as the B
// operand of O^T += V^T P^T; V is staged transposed in LDS (transposed in
// registers, 8x8 bf16 blocks) so each lane reads its 8 keys of one feature
// with two 8-byte LDS reads. Softmax statistics and accumulators are fp32.
//
// fp32 path: one wave per (request, query head, block row); lane t scores key
// t of each 64-key chunk, the weights are broadcast by lane shuffles for P V.
#include <float.h>

#include "bs_internal.h"
#include "bs_lds.h"

namespace bs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

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

// ------------------------------------------------------------------ fp32
__global__ __launch_bounds__(256) void k_attn_f32(AttnArgs a, int jblocks) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int jb = blockIdx.x % jblocks;
  const int rest = blockIdx.x / jblocks;
  const int h = rest % a.Hq;
  const int i = rest / a.Hq;
  const int j = jb * 4 + w;
  if (j >= a.L) return;
  const bs_req_desc r = a.reqs[i];
  const Geo q = geo_of(r, a.L);
  const int c = h / a.G;
  const int D = a.D;
  float* op = static_cast<float*>(a.out) + (((int64_t)i * a.L + j) * a.Hq + h) * D;
  if (j >= q.B) {
    for (int d = lane; d < D; d += 64) op[d] = 0.0f;
    return;
  }
  const float* qp = static_cast<const float*>(a.q) + (((int64_t)i * a.L + j) * a.Hq + h) * D;
  const int64_t fresh_stride = (int64_t)a.Hkv * D;
  const float* knb = static_cast<const float*>(a.k_new) + ((int64_t)i * a.L * a.Hkv + c) * D;
  const float* vnb = static_cast<const float*>(a.v_new) + ((int64_t)i * a.L * a.Hkv + c) * D;
  float* kcb = static_cast<float*>(a.k_cache) + (((int64_t)r.row * a.Hkv + c) * a.W + r.off) * D;
  float* vcb = static_cast<float*>(a.v_cache) + (((int64_t)r.row * a.Hkv + c) * a.W + r.off) * D;
  const int bs = q.s, be = q.s + q.B;

  float o[4] = {0.f, 0.f, 0.f, 0.f};
  float mrun = -__builtin_inff(), l = 0.0f;
  for (int t0 = 0; t0 < q.len; t0 += 64) {
    const int t = t0 + lane;
    float sc = -__builtin_inff();
    if (t < q.len) {
      const float* kp = (t >= bs && t < be) ? knb + (int64_t)(t - bs) * fresh_stride : kcb + (int64_t)t * D;
      float acc = 0.0f;
      for (int d = 0; d < D; d += 4) {
        const float4 kv = *reinterpret_cast<const float4*>(kp + d);
        const float4 qv = *reinterpret_cast<const float4*>(qp + d);
        acc = fmaf(qv.x, kv.x, acc);
        acc = fmaf(qv.y, kv.y, acc);
        acc = fmaf(qv.z, kv.z, acc);
        acc = fmaf(qv.w, kv.w, acc);
      }
      sc = acc * a.scale;
    }
    const float mnew = fmaxf(mrun, wave_max(sc));
    const float alpha = expf(mrun - mnew);
    const float p = (t < q.len) ? expf(sc - mnew) : 0.0f;
    l = l * alpha + wave_sum(p);
#pragma unroll
    for (int u = 0; u < 4; ++u) o[u] *= alpha;
    mrun = mnew;
    const int nk = min(64, q.len - t0);
    for (int tt = 0; tt < nk; ++tt) {
      const float pt = __shfl(p, tt, 64);
      const int tk = t0 + tt;
      const float* vp = (tk >= bs && tk < be) ? vnb + (int64_t)(tk - bs) * fresh_stride : vcb + (int64_t)tk * D;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int d = lane + 64 * u;
        if (d < D) o[u] = fmaf(pt, vp[d], o[u]);
      }
    }
  }
  const float inv = 1.0f / l;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int d = lane + 64 * u;
    if (d < D) op[d] = o[u] * inv;
  }
  if (a.write_back && (h % a.G) == 0) {
    for (int d = lane; d < D; d += 64) {
      kcb[(int64_t)(bs + j) * D + d] = knb[(int64_t)j * fresh_stride + d];
      vcb[(int64_t)(bs + j) * D + d] = vnb[(int64_t)j * fresh_stride + d];
    }
  }
}

// ------------------------------------------------------------------ bf16 MFMA
// Tiles move HBM -> LDS by direct DMA (global_load_lds_dwordx4: lane l of a
// wave instruction fills bytes [16 l, 16 l + 16) of a 1 KiB LDS block), through
// a ring of NS stages per group, so loads occupy no registers and NS - 1 tiles
// stay in flight while one is consumed. Rows are stored with their 16-byte
// chunks XOR-swizzled (slot = chunk ^ swz(row)); the permutation is applied on
// the global side, since each lane picks which chunk it fetches. K is read as
// the MFMA A operand with one 16-byte LDS read; V is read with the LDS
// transpose load (ds_read_b64_tr_b16), which hands each lane 4 consecutive keys
// of one feature: two of them form the 8-key A operand of O^T += V^T P^T.
// The DMA is issued through inline assembly and waited for with explicit
// vmcnt counts: the compiler's waitcnt pass cannot see it, and would otherwise
// drain every stage in flight before reading the current one. The K/V tiles
// are read once, with the non-temporal hint (measured: LLaDA-8B layer
// attention 60.4 -> 57.3 us).
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// max without the canonicalisation fmaxf needs in IEEE mode (scores are finite
// or -inf, so NaN propagation never applies)
__device__ inline float vmax(float x, float y) { return __builtin_elementwise_maximum(x, y); }

// Combine lane l with lane l ^ 32 (the two key halves of a query column):
// v_permlane32_swap exchanges the 32-lane halves of two registers in the
// VALU, with no LDS round trip; both halves combine (low, high) in that order.
__device__ inline void xhalf(float v, float& lo, float& hi) {
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  lo = __uint_as_float(sw[0]);
  hi = __uint_as_float(sw[1]);
}
__device__ inline float xhalf_max(float v) {
  float lo, hi;
  xhalf(v, lo, hi);
  return vmax(lo, hi);
}
__device__ inline float xhalf_sum(float v) {
  float lo, hi;
  xhalf(v, lo, hi);
  return lo + hi;
}

// lsum += sum of the eight bf16 weights in p (the values the P V MFMA uses)
__device__ inline float add_weights(float lsum, const bf16x8_t& p) {
  const bf16x2_t one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int k = 0; k < 4; ++k) lsum = __builtin_amdgcn_fdot2_f32_bf16(bf16x2_t{p[2 * k], p[2 * k + 1]}, one, lsum, false);
  return lsum;
}
// XOR swizzle of a row's 16-byte slots. D = 128 (16 slots), for an LDS that
// serves 256 bytes (64 banks of 4 bytes) per cycle: the 32 lanes of one
// transposed V read cover rows r0 .. r0 + 3 (r0 % 4 == 0) at chunks
// 4 t .. 4 t + 3, and row bits 0..1 moved to slot bits 2..3 put them in 16
// distinct slots; row bits 2..3 moved to slot bits 0..1 keep any 16
// consecutive rows on distinct slots for one chunk (the K reads). D = 64
// (8 slots): rows r0..r0+3 differ in bits 1..2 and any 8 consecutive rows get
// distinct slots for one chunk.
template <int NCH>
__device__ inline int swz(int row) {
  if constexpr (NCH == 16) return ((row & 3) << 2) | ((row >> 2) & 3);
  return ((row & 3) << 1) | ((row >> 2) & 1);
}

// compile-time flag passed to a generic lambda
template <bool B>
struct Flag {
  static constexpr bool value = B;
};

// One (request, KV head) item processed by GW waves that share its K/V tiles:
// wave wg of the group serves query head c * G + wg / RBW and rows
// 32 * (rb + wg % RBW) .. + 32 of the block (RBW row blocks per workgroup,
// starting at the item's rb). SHARED = false is the single-wave case
// (GW = 1): the wave owns its ring, so no barrier is needed anywhere.
//
// The DMA of a stage (2 * BPT blocks of 1 KiB) is issued by the NI waves
// I0 .. I0 + NI - 1 only, PB = 2 * BPT / NI blocks each, so every count and
// offset of the issue sequence is a compile-time constant plus one per-wave
// base: no per-block branch, and the waits are compile-time vmcnt values.
// The other waves see a stage through the barrier that follows the issuers'
// waits.
//
// The work item is taken by value: the DMA's inline assembly clobbers memory,
// so fields read through a reference would be loaded again after every issue,
// as vector loads whose waits also drain the DMA in flight (measured: 2.6 us
// of the skewed Dream-7B batch's attention).
template <int D, int KT, int NS, bool SHARED, int NI, int I0>
__device__ inline void attn_item(const AttnArgs& a, const AttnItem it, uint16_t* ring, int GW, int wg,
                                 int lane) {
  constexpr int NKK = D / 16;
  constexpr int NDT = D / 32;
  constexpr int NCH = D / 8;                      // 16-byte chunks per row
  constexpr int RPB = 64 / NCH;                   // rows per 1 KiB DMA block
  constexpr int BPT = KT / RPB;                   // blocks per K (or V) tile
  constexpr int TILE = KT * D;                    // elements of one K (or V) tile
  constexpr int STAGE = 2 * TILE;                 // K tile then V tile
  constexpr int RPI = BPT / NI;                   // blocks per tile and issuing wave
  constexpr int PB = 2 * RPI;                     // blocks per stage and issuing wave
  static_assert(BPT % NI == 0, "issuing waves must split a tile evenly");
  const int g = lane >> 5, n = lane & 31;
  const int c = it.kvh;
  const int h = c * a.G + wg / a.RBW;
  const int j = (it.rb + wg % a.RBW) * 32 + n;
  const int bs = it.s, be = it.s + it.B, len = it.len;

  const int64_t cache_off = (((int64_t)it.row * a.Hkv + c) * a.W + it.off) * D;
  const uint16_t* kcb = static_cast<const uint16_t*>(a.k_cache) + cache_off;
  const uint16_t* vcb = static_cast<const uint16_t*>(a.v_cache) + cache_off;
  const int64_t fstride = (int64_t)a.Hkv * D;
  const uint16_t* knb = static_cast<const uint16_t*>(a.k_new) + ((int64_t)it.req * a.L * a.Hkv + c) * D;
  const uint16_t* vnb = static_cast<const uint16_t*>(a.v_new) + ((int64_t)it.req * a.L * a.Hkv + c) * D;

  // Block k of issuing wave u = wg - I0 is block (k % RPI) * NI + u of tensor
  // k / RPI (K, then V): it covers tile rows [rb * RPB, rb * RPB + RPB), and
  // lane l fills slot l % NCH of row rb * RPB + l / NCH with global chunk
  // slot ^ swz(row).
  const bool issuer = (unsigned)(wg - I0) < (unsigned)NI;
  const int u = issuer ? wg - I0 : 0;
  const int urow = u * RPB + lane / NCH, dslot = lane % NCH;
  const uint32_t ring_lds = lds_addr(ring) + (uint32_t)(u * RPB * D * 2);
  auto row_of = [&](int r) { return r * NI * RPB + urow; };
  auto chunk_of = [&](int row) { return dslot ^ swz<NCH>(row); };
  auto issue = [&](int stage, int tb) {
    const uint32_t sbase = __builtin_amdgcn_readfirstlane(ring_lds + (uint32_t)(stage * STAGE * 2));
    if (tb + KT <= len && (tb + KT <= bs || tb >= be)) {
      // whole tile inside the cached part of the row: uniform base + lane offset
      const uint64_t kb = uniform64(kcb + (int64_t)tb * D), vb = uniform64(vcb + (int64_t)tb * D);
#pragma unroll
      for (int k = 0; k < PB; ++k) {
        const int tensor = k / RPI, r = k % RPI;
        const int row = row_of(r);
        dma16_sv_once(sbase + (uint32_t)((tensor * TILE + r * NI * RPB * D) * 2), tensor ? vb : kb,
                 (uint32_t)(row * D + chunk_of(row) * 8) * 2u);
      }
    } else {
      // tile holds fresh block rows or runs past the row end: per-lane sources
#pragma unroll
      for (int k = 0; k < PB; ++k) {
        const int tensor = k / RPI, r = k % RPI;
        const int row = row_of(r);
        const int t = min(tb + row, len - 1);        // rows past the end repeat a valid key (masked later)
        const bool fresh = (t >= bs) & (t < be);
        const uint16_t* src = tensor ? (fresh ? vnb + (int64_t)(t - bs) * fstride : vcb + (int64_t)t * D)
                                     : (fresh ? knb + (int64_t)(t - bs) * fstride : kcb + (int64_t)t * D);
        dma16_once(sbase + (uint32_t)((tensor * TILE + r * NI * RPB * D) * 2), src + chunk_of(row) * 8);
      }
    }
  };
  // issuing waves: wait until at most x (< NS) stages of this wave's DMA are
  // in flight (a count above the 6-bit vmcnt field waits for everything)
  auto wait_stages = [&](int x) {
    static_assert(NS <= 4, "wait counts are encoded up to three stages");
    if (x <= 0)
      wait_vm_c<0>();
    else if (x == 1)
      wait_vm_c<PB>();
    else if (x == 2)
      wait_vm_c<2 * PB>();
    else
      wait_vm_c<3 * PB>();
  };

  // In-place KV update. Group loop: the fresh block rows that a tile holds
  // (keys [tb, tb + KT) within [bs, be), staged from k_new / v_new) go into
  // the cache slot [off + s, off + s + B) straight from LDS, so they are read
  // from memory once. A store counts in vmcnt like the DMA, so a store issued
  // in the loop would make the next stage wait drain it too: the stores come
  // from the waves that issue no DMA (when the group has any); they are
  // non-temporal whole rows, like the output below. The single-wave loop
  // issues them itself, as plain stores, and counts them in its waits: a wait
  // two tiles later covers them, and non-temporal stores were measured to
  // hold that wait up (LLaDA-8B layer attention 57.0 -> 60.7 us). Only the
  // row-block-0 workgroup of an item stores them.
  const bool do_wb = a.write_back && it.rb == 0;
  uint16_t* kcw = static_cast<uint16_t*>(a.k_cache) + cache_off;
  uint16_t* vcw = static_cast<uint16_t*>(a.v_cache) + cache_off;
  // chunk cid of the tile's fresh rows (K then V) by lane
  // (wg - w0) * 64 + lane of the storing waves [w0, GW)
  auto write_back_tile = [&](const uint16_t* st, int tb) {
    const int r0 = max(bs, tb) - tb, r1 = min(be, tb + KT) - tb;
    const int w0 = GW > NI ? NI : 0;
    if (!do_wb || r0 >= r1 || wg < w0) return;
    const int nc = (r1 - r0) * NCH;               // chunks per tensor
    const int gt = (wg - w0) * 64 + lane, gth = (GW - w0) * 64;
#pragma unroll
    for (int tensor = 0; tensor < 2; ++tensor) {
      const uint16_t* src = st + tensor * TILE;
      uint16_t* dst = tensor ? vcw : kcw;
      for (int cid = gt; cid < nc; cid += gth) {
        const int row = r0 + cid / NCH, c = cid % NCH;
        const v4u v = *reinterpret_cast<const v4u*>(src + row * D + ((c ^ swz<NCH>(row)) * 8));
        __builtin_nontemporal_store(v, reinterpret_cast<v4u*>(dst + (int64_t)(tb + row) * D + c * 8));
      }
    }
  };
  // tiles of this item: keys [64 t0, min(64 t1, len)) of the row (the whole
  // row, or one piece of it), in KT-key tiles from tb0
  constexpr int TPU = kAttnTile / KT;             // KT-key tiles per 64-key unit
  const int tb0 = it.t0 * kAttnTile;
  const int ntiles = min((len + KT - 1) / KT, it.t1 * TPU) - it.t0 * TPU;
  // The request's block mask word, in the fused step (one item per request:
  // KV head 0, first row block, its first wave): lane j reads mask cell j of
  // the block, by inline assembly so the compiler adds no wait of its own;
  // issued before the DMA, so every later wait of this wave covers it, and
  // consumed after the last one.
  const bool word_owner = a.mask_words != nullptr && it.kvh == 0 && it.rb == 0 && it.t0 == 0 && wg == 0;
  uint32_t mcell = 0;
  if (word_owner) {
    const uint8_t* mp = a.masked + it.row * a.msk_rs + it.off + it.s + (lane < it.B ? lane : 0);
    asm volatile("global_load_ubyte %0, %1, off" : "=v"(mcell) : "v"(mp) : "memory");
  }
  // prologue: stages 0 .. NS-2 (issued before anything else so the first
  // tiles are in flight while the queries load)
  if (issuer) {
#pragma unroll
    for (int st = 0; st < NS - 1; ++st)
      if (st < ntiles) issue(st, tb0 + st * KT);
  }

  // queries of this lane's column as MFMA B operands: feature d = 16 kk + 8 g + e
  bf16x8_t qb[NKK];
  {
    const bool qv = j < it.B;
    const uint16_t* qp = static_cast<const uint16_t*>(a.q) + (((int64_t)it.req * a.L + min(j, it.B - 1)) * a.Hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      v4u t = ld16(qp + 16 * kk + 8 * g);
      if (!qv) t = v4u{0u, 0u, 0u, 0u};
      qb[kk] = __builtin_bit_cast(bf16x8_t, t);
    }
  }
  // loop-invariant parts of this lane's LDS read addresses (elements)
  int koff[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) koff[kk] = n * D + (((2 * kk + g) ^ swz<NCH>(n)) * 8);
  const int q16 = lane >> 4, j16 = lane & 15;
  const int vrow = 4 * (q16 >> 1) + (j16 >> 2);              // + sub*32 + 16 ks + 8 h2
  int voff[NDT][2][2];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int row = 16 * ks + 8 * h2 + vrow;                // row within a 32-key sub-tile
        const int col = 32 * dt + 16 * (q16 & 1) + 4 * (j16 & 3);
        voff[dt][ks][h2] = row * D + (((col >> 3) ^ swz<NCH>(row)) * 8) + (col & 7);
      }

  f32x16_t o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) o[dt][rr] = 0.0f;
  float mrun = -__builtin_inff(), lsum = 0.0f;
  if constexpr (SHARED) {
    static_assert(KT == 64 && NS == 4, "the group loop refills the slot of tile t - 1 while tiles t .. t + 2 are held");
    // Software pipeline over 64-key tiles, two MFMA blocks per tile, each
    // interleaved with the VALU work of the same wave (a wave's MFMAs overlap
    // only its own VALU work), in an order fixed by scheduling fences:
    //   block 1: P V of tile t - 1 (16 MFMAs) beside the max of tile t's
    //            scores, the rescale decision, the scaled scores and half of
    //            the exponentials;
    //   barrier: tile t + 1 resident, every wave done with tile t - 1, whose
    //            slot is refilled with tile t + 3;
    //   block 2: scores of tile t + 1 (16 MFMAs) beside the other
    //            exponentials, their bf16 conversion and the row sums.
    // (16 MFMAs per block at D = 128; 8 at D = 64.)

    // pin(x): x is computed here; keeps the compiler from sinking the
    // arithmetic past the scheduling fences into the block that uses it
    auto pin = [](float& x) { asm volatile("" : "+v"(x)); };
    const float sl2e = a.scale_log2e;
    f32x16_t sa, sb;           // scores of tile t (keys 0..31 and 32..63 of the tile)
    float ex[32];              // tile t: scaled scores, then their exponentials
    bf16x8_t pp[2][2];         // probabilities of the last converted tile: [half][ks]
    constexpr int NSC = 2 * NKK, NPV = 4 * NDT;   // score and P V MFMAs per tile
    auto kread = [&](const uint16_t* kt, int j) -> bf16x8_t {   // A operand of score MFMA j
      return *reinterpret_cast<const bf16x8_t*>(kt + (j & 1) * 32 * D + koff[j >> 1]);
    };
    auto vread = [&](const uint16_t* vt, int i) -> bf16x8_t {   // A operand of P V MFMA i
      const int dt = i % NDT, ks = (i / NDT) & 1, hh = i / (2 * NDT);
      const uint16_t* vs = vt + hh * 32 * D;
      const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vs + voff[dt][ks][0]));
      const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vs + voff[dt][ks][1]));
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    auto sfrag = [&](int j) -> f32x16_t& { return (j & 1) ? sb : sa; };
    // P V of one tile, no interleaving (the last tile, after the loop)
    auto pv_plain = [&](const uint16_t* vt) {
#pragma unroll
      for (int i = 0; i < NPV; ++i)
        o[i % NDT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vread(vt, i), pp[i / (2 * NDT)][(i / NDT) & 1],
                                                            o[i % NDT], 0, 0, 0);
    };
    auto mask_ragged = [&](int tb) {
      if (tb + KT > len) {                         // ragged last tile only
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int key = tb + 8 * (rr >> 2) + 4 * g + (rr & 3);
          if (key >= len) sa[rr] = -__builtin_inff();
          if (key + 32 >= len) sb[rr] = -__builtin_inff();
        }
      }
    };

    // tile 0 resident (the later prologue stages may still be in flight)
    if (issuer) wait_stages(min(ntiles - 1, NS - 2));
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      sa[rr] = 0.0f;
      sb[rr] = 0.0f;
    }
#pragma unroll
    for (int j = 0; j < NSC; ++j)
      sfrag(j) = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kread(ring, j), qb[j >> 1], sfrag(j), 0, 0, 0);

    auto body = [&](auto first_tag, int tile) {
      constexpr bool FIRST = decltype(first_tag)::value;
      const int tb = tb0 + tile * KT;
      const uint16_t* vprev = ring + ((tile + NS - 1) % NS) * STAGE + TILE;
      mask_ragged(tb);
      // ---- block 1
      bf16x8_t vf[3];
      if constexpr (!FIRST) {
        vf[0] = vread(vprev, 0);
        vf[1] = vread(vprev, 1);
      }
      float m8[8];
      float mx = 0.0f, alpha = 1.0f;
      bool resc = false;
      __builtin_amdgcn_sched_barrier(0);
      // sixteen slots of VALU work; the NPV MFMAs are spread evenly over them
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if constexpr (!FIRST) {
          if ((i * NPV) % 16 == 0) {
            const int m = i * NPV / 16;
            if (m + 2 < NPV) vf[(m + 2) % 3] = vread(vprev, m + 2);
            o[m % NDT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[m % 3], pp[m / (2 * NDT)][(m / NDT) & 1],
                                                                o[m % NDT], 0, 0, 0);
          }
        }
        if (i < 2) {
#pragma unroll
          for (int k = 4 * i; k < 4 * i + 4; ++k)
            m8[k] = vmax(vmax(sa[2 * k], sa[2 * k + 1]), vmax(sb[2 * k], sb[2 * k + 1]));
        } else if (i == 2) {
          mx = vmax(vmax(vmax(m8[0], m8[1]), vmax(m8[2], m8[3])), vmax(vmax(m8[4], m8[5]), vmax(m8[6], m8[7])));
          mx = xhalf_max(mx) * sl2e;              // log2 units
          pin(mx);
        } else if (i == 3) {
          // lazy rescale: keep the reference max until a score exceeds it by
          // 2^8, so the O accumulators are rescaled a handful of times per row
          resc = __builtin_amdgcn_ballot_w64(mx > mrun + 8.0f) != 0;
          const float mnew = resc ? fmaxf(mrun, mx) : mrun;
          alpha = __builtin_amdgcn_exp2f(mrun - mnew);
          lsum *= alpha;
          mrun = mnew;
        } else if (i < 8) {
#pragma unroll
          for (int r = 8 * (i - 4); r < 8 * (i - 4) + 8; ++r) {
            ex[r] = fmaf(r < 16 ? sa[r] : sb[r - 16], sl2e, -mrun);
            pin(ex[r]);
          }
        } else {
          ex[2 * (i - 8)] = __builtin_amdgcn_exp2f(ex[2 * (i - 8)]);
          ex[2 * (i - 8) + 1] = __builtin_amdgcn_exp2f(ex[2 * (i - 8) + 1]);
          pin(ex[2 * (i - 8)]);
          pin(ex[2 * (i - 8) + 1]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (!FIRST) {
        if (resc) {                                // rare: after the P V of tile t - 1
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int rr = 0; rr < 16; ++rr) o[dt][rr] *= alpha;
        }
      }
      // ---- barrier: tile + 1 landed (stages up to tile + NS - 2 were
      // issued); every wave is done with tile - 1, whose slot is refilled
      if (tile + 1 < ntiles) {
        if (issuer) wait_stages(min(ntiles - 1, tile + NS - 2) - tile - 1);
        __syncthreads();
        const int nxt = tile + NS - 1;
        if (issuer && nxt < ntiles) issue(nxt % NS, tb0 + nxt * KT);
      }
      // ---- block 2 (on the last tile the scores read a resident slot and
      // are discarded)
      const uint16_t* knext = ring + ((tile + 1) % NS) * STAGE;
      bf16x8_t kf[3];
      kf[0] = kread(knext, 0);
      kf[1] = kread(knext, 1);
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        sa[rr] = 0.0f;
        sb[rr] = 0.0f;
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        if ((j * NSC) % 16 == 0) {
          const int m = j * NSC / 16;
          if (m + 2 < NSC) kf[(m + 2) % 3] = kread(knext, m + 2);
          sfrag(m) = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[m % 3], qb[m >> 1], sfrag(m), 0, 0, 0);
        }
        if (j < 8) {
          ex[16 + 2 * j] = __builtin_amdgcn_exp2f(ex[16 + 2 * j]);
          ex[17 + 2 * j] = __builtin_amdgcn_exp2f(ex[17 + 2 * j]);
          pin(ex[16 + 2 * j]);
          pin(ex[17 + 2 * j]);
        } else {
          // values 4 (j - 8) .. + 3 -> bf16 pairs, and their sum
          const int v0 = 4 * (j - 8);
          bf16x8_t& dst = pp[v0 >> 4][(v0 >> 3) & 1];
#pragma unroll
          for (int e = 0; e < 4; ++e) dst[(v0 & 7) + e] = (__bf16)ex[v0 + e];
          if ((v0 & 7) == 4) {
            lsum = add_weights(lsum, dst);
            pin(lsum);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      write_back_tile(ring + (tile % NS) * STAGE, tb);
    };
    if (ntiles > 0) body(Flag<true>{}, 0);
    for (int tile = 1; tile < ntiles; ++tile) body(Flag<false>{}, tile);
    pv_plain(ring + ((ntiles + NS - 1) % NS) * STAGE + TILE);
  } else {
    // The fresh block rows a tile holds are stored from the LDS tile after
    // the tile is consumed, always as SPT full store instructions per tensor
    // (a lane whose row lies outside the block stores a block row's chunk
    // again, the same bytes to the same address), so the next tile's wait
    // knows how many vmcnt entries the stores add behind its stage: with two
    // stages, stage t + 1 is issued before tile t's stores and stage t + 2
    // after them.
    static_assert(NS == 2, "the store count in the waits assumes one stage ahead");
    constexpr int SPT = KT * NCH / 64;
    bool stored = false;                          // the previous tile issued 2 SPT stores
    for (int tile = 0; tile < ntiles; ++tile) {
      const int nxt = tile + NS - 1;
      const bool ahead = nxt < ntiles;
      if (ahead) issue(nxt % NS, tb0 + nxt * KT);
      // this tile's stage has landed once only the next stage's DMA (if
      // issued) and the previous tile's stores (if any) remain
      if (ahead) {
        if (stored)
          wait_vm_c<PB + 2 * SPT>();
        else
          wait_vm_c<PB>();
      } else {
        if (stored)
          wait_vm_c<2 * SPT>();
        else
          wait_vm_c<0>();
      }
      const uint16_t* kt = ring + (tile % NS) * STAGE;
      const uint16_t* vtl = kt + TILE;
      const int tb = tb0 + tile * KT;
  #pragma unroll
      for (int sub = 0; sub < KT / 32; ++sub) {
        const int sb = tb + sub * 32;
        if (sb >= len) break;
        f32x16_t sacc;
  #pragma unroll
        for (int rr = 0; rr < 16; ++rr) sacc[rr] = 0.0f;
  #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
          const bf16x8_t ka = *reinterpret_cast<const bf16x8_t*>(kt + sub * 32 * D + koff[kk]);
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[kk], sacc, 0, 0, 0);
        }
        // lane (g, n) holds S^T[key 8 (rr / 4) + 4 g + rr % 4][query n] (unscaled)
        if (sb + 32 > len) {                       // ragged last sub-tile only
  #pragma unroll
          for (int rr = 0; rr < 16; ++rr)
            if (sb + 8 * (rr >> 2) + 4 * g + (rr & 3) >= len) sacc[rr] = -__builtin_inff();
        }
        float mx = sacc[0];
#pragma unroll
        for (int rr = 1; rr < 16; ++rr) mx = vmax(mx, sacc[rr]);
        mx = xhalf_max(mx) * a.scale_log2e;      // log2 units
        // lazy rescale: keep the reference max until a score exceeds it by 2^8,
        // so the O accumulators are rescaled a handful of times per row
        if (__builtin_amdgcn_ballot_w64(mx > mrun + 8.0f)) {
          const float mnew = fmaxf(mrun, mx);
          const float alpha = __builtin_amdgcn_exp2f(mrun - mnew);
          lsum *= alpha;
  #pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
  #pragma unroll
            for (int rr = 0; rr < 16; ++rr) o[dt][rr] *= alpha;
          mrun = mnew;
        }
        bf16x8_t pb0, pb1;
        const float nm = -mrun;
  #pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sacc[rr], a.scale_log2e, nm));
          if (rr < 8)
            pb0[rr] = (__bf16)p;
          else
            pb1[rr - 8] = (__bf16)p;
        }
        lsum = add_weights(add_weights(lsum, pb0), pb1);
        const uint16_t* vs = vtl + sub * 32 * D;
  #pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
  #pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vs + voff[dt][ks][0]));
            const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vs + voff[dt][ks][1]));
            const bf16x8_t va = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, ks ? pb1 : pb0, o[dt], 0, 0, 0);
          }
      }
      // the wave consumed its LDS reads through the MFMAs above before its
      // next issue overwrites the slot
      stored = do_wb && tb < be && tb + KT > bs;
      if (stored) {
        // every LDS read first, then the stores (one LDS latency, not 2 SPT)
        const int r0 = max(bs, tb) - tb, r1 = min(be, tb + KT) - tb;
        v4u wv[2][SPT];
        int wrow[SPT];
#pragma unroll
        for (int k = 0; k < SPT; ++k) wrow[k] = min(max(k * (64 / NCH) + lane / NCH, r0), r1 - 1);
        const int c = lane % NCH;
#pragma unroll
        for (int tensor = 0; tensor < 2; ++tensor)
#pragma unroll
          for (int k = 0; k < SPT; ++k)
            wv[tensor][k] = *reinterpret_cast<const v4u*>(kt + tensor * TILE + wrow[k] * D + ((c ^ swz<NCH>(wrow[k])) * 8));
#pragma unroll
        for (int tensor = 0; tensor < 2; ++tensor)
#pragma unroll
          for (int k = 0; k < SPT; ++k)
            st16((tensor ? vcw : kcw) + (int64_t)(tb + wrow[k]) * D + c * 8, wv[tensor][k]);
      }
    }
  }
  const float lt = xhalf_sum(lsum);
  if (it.part >= 0) {
    // One piece of a split row: the un-normalised O^T (accumulator order,
    // whole 16-byte groups per lane), the running max in log2 units and the
    // row sum go to the piece's partial slot for the merge launch.
    constexpr int OFL = NDT * 16 * 64;
    float* pw = a.parts + ((int64_t)it.part * GW + wg) * part_wave_floats(D);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq)
        __builtin_nontemporal_store(f32x4_t{o[dt][4 * rq], o[dt][4 * rq + 1], o[dt][4 * rq + 2], o[dt][4 * rq + 3]},
                                    reinterpret_cast<f32x4_t*>(pw + ((dt * 4 + rq) * 64 + lane) * 4));
    __builtin_nontemporal_store(mrun, pw + OFL + lane);
    __builtin_nontemporal_store(lt, pw + OFL + 64 + lane);
  } else {
    // Output: lane (g, n) holds O^T[feature dt*32 + 8 (rr / 4) + 4 g + rr % 4]
    // [query n]. The wave's 32 x D tile is staged row-major in LDS (rows padded
    // by 16 bytes against bank conflicts) and stored as whole rows, 16 bytes per
    // lane, instead of 8-byte pieces scattered over 32 rows. The stores are
    // non-temporal: the output is not read again by the step, and whole lines
    // written around the L2 leave no dirty lines for the kernels that follow
    // to evict (measured: the Dream-7B step's decode rows 61.5 -> 57.7 us).
    if constexpr (SHARED) __syncthreads();          // every wave is done with the ring
    constexpr int SROW = D + 8;                     // staged row stride (elements)
    uint16_t* stg = ring + (SHARED ? wg * 32 * SROW : 0);
    {
      const float inv = (j < it.B) ? 1.0f / lt : 0.0f;
      typedef uint32_t v2u __attribute__((ext_vector_type(2)));
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const __bf16 b0 = (__bf16)(o[dt][4 * rq + 0] * inv);
          const __bf16 b1 = (__bf16)(o[dt][4 * rq + 1] * inv);
          const __bf16 b2 = (__bf16)(o[dt][4 * rq + 2] * inv);
          const __bf16 b3 = (__bf16)(o[dt][4 * rq + 3] * inv);
          const uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, b0) | ((uint32_t)__builtin_bit_cast(uint16_t, b1) << 16);
          const uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, b2) | ((uint32_t)__builtin_bit_cast(uint16_t, b3) << 16);
          *reinterpret_cast<v2u*>(stg + n * SROW + dt * 32 + 8 * rq + 4 * g) = v2u{w0, w1};
        }
    }
    {
      constexpr int RPW = 64 / NCH;                 // rows per wave instruction
      const int jb = (it.rb + wg % a.RBW) * 32;     // first block row of this wave
#pragma unroll
      for (int k = 0; k < 32 / RPW; ++k) {
        const int row = k * RPW + lane / NCH, c = lane % NCH;
        const v4u v = *reinterpret_cast<const v4u*>(stg + row * SROW + c * 8);
        if (jb + row < a.L) {
          uint16_t* op = static_cast<uint16_t*>(a.out) + (((int64_t)it.req * a.L + jb + row) * a.Hq + h) * D;
          __builtin_nontemporal_store(v, reinterpret_cast<v4u*>(op + c * 8));
        }
      }
    }
  }
  if (word_owner) {
    wait_vm_c<0>();
    asm volatile("" : "+v"(mcell));                 // read only after the wait
    const uint64_t bits = __ballot(lane < it.B && mcell != 0);
    if (lane == 0) a.mask_words[it.req] = bits;
  }
}

// One query head per KV head and at most 32 block rows (MHA with L <= 32):
// NW independent waves per workgroup, each owning one item and an NS-stage
// ring of 32-key tiles.
template <int D, int NS, int NW>
__global__ __launch_bounds__(64 * NW, 1) void k_attn_bf16_wave(AttnArgs a) {
  constexpr int STAGE = 2 * 32 * D;
  __shared__ __align__(1024) uint16_t lds[NW * NS * STAGE];
  // the wave index is wave-uniform: through readfirstlane every quantity
  // derived from it (item, DMA block, base pointers) lives in SGPRs
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int idx = blockIdx.x * NW + w;
  if (idx >= a.n_items) return;
  attn_item<D, 32, NS, false, 1, 0>(a, a.items[idx], lds + w * NS * STAGE, 1, 0, threadIdx.x & 63);
}

// GW = G * ceil(L / 32) >= 2 waves share each item's 64-key tiles; the first
// NI <= GW of them issue its DMA.
template <int D, int NS, int NI>
__global__ __launch_bounds__(512, 1) void k_attn_bf16_group(AttnArgs a) {
  constexpr int STAGE = 2 * 64 * D;
  __shared__ __align__(1024) uint16_t lds[NS * STAGE];
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  attn_item<D, 64, NS, true, NI, 0>(a, a.items[blockIdx.x], lds, blockDim.x >> 6, w, threadIdx.x & 63);
}

// Split-KV merge. Wave (r, wg, k) combines group k (4 of the lane's output
// features) of split row r for wave slot wg of its pieces' workgroups, which
// serve query head kvh * G + wg / RBW and 32 block rows (row block
// rb + wg % RBW). Lane (g, n) folds the pieces' partials of its query column
// with a running max m: the sums so far are scaled by 2^(m_old - m) and piece
// p's by 2^(m_p - m) (the log-sum-exp merge of softmax pieces), eight pieces'
// loads in flight at a time; the quotient is written like the attention's own
// output (bf16; rows B .. L - 1 as zeros). Every load of a wave is one
// contiguous 256 B or 1 KiB run.
template <int D>
__global__ __launch_bounds__(256) void k_attn_merge(AttnArgs a) {
  constexpr int NG = D / 8;                       // groups of 4 floats per lane
  constexpr int OFL = NG * 64 * 4;
  constexpr int CH = 8;                           // pieces per batch of loads
  const int GW = a.G * a.RBW;
  const int wv = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (wv >= a.n_merge * GW * NG) return;
  const int k = wv % NG, wg = (wv / NG) % GW;
  const AttnMerge mg = a.merges[wv / (NG * GW)];
  const int g = lane >> 5, n = lane & 31;
  const int h = mg.kvh * a.G + wg / a.RBW;
  const int j = (mg.rb + wg % a.RBW) * 32 + n;
  const int64_t pstride = (int64_t)GW * part_wave_floats(D);
  const float* pw = a.parts + ((int64_t)mg.part0 * GW + wg) * part_wave_floats(D);
  f32x4_t acc = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  float m = -__builtin_inff(), l = 0.0f;
  for (int p0 = 0; p0 < mg.nparts; p0 += CH) {
    float mp[CH], lp[CH];
    f32x4_t op[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      if (p0 + i < mg.nparts) {
        const float* pp = pw + (p0 + i) * pstride;
        mp[i] = pp[OFL + lane];
        lp[i] = pp[OFL + 64 + lane];
        op[i] = *reinterpret_cast<const f32x4_t*>(pp + (k * 64 + lane) * 4);
      } else {
        mp[i] = -__builtin_inff();
        lp[i] = 0.0f;
        op[i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      }
    }
    float mn = m;
#pragma unroll
    for (int i = 0; i < CH; ++i) mn = fmaxf(mn, mp[i]);
    const float sa = __builtin_amdgcn_exp2f(m - mn);
    l *= sa;
    acc *= sa;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const float sb = __builtin_amdgcn_exp2f(mp[i] - mn);     // 0 for the padding entries
      l = fmaf(lp[i], sb, l);
      acc += op[i] * sb;
    }
    m = mn;
  }
  if (j >= a.L) return;
  const float inv = j < mg.B ? 1.0f / l : 0.0f;
  // group k = 4 dt + rq holds features 32 dt + 8 rq + 4 g .. + 3
  uint16_t* op = static_cast<uint16_t*>(a.out) + (((int64_t)mg.req * a.L + j) * a.Hq + h) * D +
                 32 * (k >> 2) + 8 * (k & 3) + 4 * g;
  typedef uint32_t v2u __attribute__((ext_vector_type(2)));
  uint32_t w2[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const __bf16 lo = (__bf16)(acc[2 * e] * inv), hi = (__bf16)(acc[2 * e + 1] * inv);
    w2[e] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
  }
  __builtin_nontemporal_store(v2u{w2[0], w2[1]}, reinterpret_cast<v2u*>(op));
}

template <int D>
hipError_t launch_bf16_d(const AttnArgs& a, int GW, hipStream_t s) {
  if (GW == 1) {
    constexpr int NS = 2, NW = kMhaWaves;
    hipLaunchKernelGGL((k_attn_bf16_wave<D, NS, NW>), dim3((a.n_items + NW - 1) / NW), dim3(64 * NW), 0, s, a);
  } else if (GW < 4) {
    hipLaunchKernelGGL((k_attn_bf16_group<D, 4, 2>), dim3(a.n_items), dim3(64 * GW), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_attn_bf16_group<D, 4, 4>), dim3(a.n_items), dim3(64 * GW), 0, s, a);
  }
  if (a.n_merge > 0)
    hipLaunchKernelGGL((k_attn_merge<D>), dim3((a.n_merge * GW * (D / 8) + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const AttnArgs& a, int n_req, hipStream_t s) {
  const int jblocks = (a.L + 3) / 4;
  const dim3 grid((unsigned)((int64_t)n_req * a.Hq * jblocks)), block(256);
  hipLaunchKernelGGL(k_attn_f32, grid, block, 0, s, a, jblocks);
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t s) {
  const int GW = a.G * a.RBW;
  if (a.D == 128) return launch_bf16_d<128>(a, GW, s);
  if (a.D == 64) return launch_bf16_d<64>(a, GW, s);
  return hipErrorInvalidValue;
}

}  // namespace bs
