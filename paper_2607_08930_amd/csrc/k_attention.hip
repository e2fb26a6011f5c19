// K2: dual-cache block attention (paragraph "Vectorized mixed-schedule
// execution"; dual cache of Fast-dLLM as integrated by the paper).
//
// The keys of request i are its logical row [0, p + g): cached prefix
// [0, s), the fresh block [s, s + B) read from k_new/v_new, and the cached
// masked suffix [s + B, p + g). Key t of the row is therefore fetched either
// from cache cell off + t of the request's dense row or from fresh row t - s;
// the stale block slot and the padding are never read. With write_back the
// fresh rows are also stored into the cache slot as they stream past
// (in-place KV update at the physical offsets of the active block).
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

namespace bs {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

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
// A workgroup serves one (request, KV head). Its waves form S key-split
// groups of GW = G * RB waves: the waves of a group share one K/V tile in LDS
// (one wave per query head of the group and 32-row block), and group s takes
// tiles s, s + S, ... of the request's key range. After the loop the groups'
// (max, sum, O) partials are merged through LDS, so splitting a row never
// costs HBM traffic.
template <int D, int KT, int S, int GTMIN>
struct TileCfg {
  static constexpr int KS = D + 8;                  // K tile row stride (elements), 16-byte rows
  static constexpr int VS = KT + 4;                 // V^T row stride (elements), 8-byte aligned
  static constexpr int KCH = KT * D / 8;            // 16-byte chunks of a K tile
  static constexpr int VBLK = (KT / 8) * (D / 8);   // 8x8 blocks of a V tile
  static constexpr int MAXK = (KCH + GTMIN - 1) / GTMIN;
  static constexpr int MAXV = (VBLK + GTMIN - 1) / GTMIN;
  static constexpr int TILE_ELEMS = KT * KS + D * VS;
};

template <int D, int KT, int S, int GTMIN, int MAXT, int MINW>
__global__ __launch_bounds__(MAXT, MINW) void k_attn_bf16(AttnArgs a) {
  using C = TileCfg<D, KT, S, GTMIN>;
  constexpr int NKK = D / 16;
  constexpr int NDT = D / 32;
  // tiles during the loop; the split groups' partials after it
  constexpr int MERGE_FLOATS = (S - 1) * ((MAXT / 64) / S) * 64 * (2 + NDT * 16);
  constexpr int TILE_BYTES = S * C::TILE_ELEMS * 2;
  constexpr int LDS_BYTES = TILE_BYTES > MERGE_FLOATS * 4 ? TILE_BYTES : MERGE_FLOATS * 4;
  __shared__ __align__(16) uint16_t lds[LDS_BYTES / 2];

  const AttnItem it = a.items[blockIdx.x];
  const bs_req_desc r = a.reqs[it.req];
  const Geo q = geo_of(r, a.L);
  const int GW = a.G * a.RB;                       // waves per split group
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, g = lane >> 5, n = lane & 31;
  const int grp = w / GW, wg = w - grp * GW;
  const int gth = GW * 64, gt = tid - grp * gth;   // threads of this group, index within it
  const int c = it.kvh;
  const int h = c * a.G + wg / a.RB;
  const int j = (wg % a.RB) * 32 + n;
  const int bs = q.s, be = q.s + q.B;
  uint16_t* ks = lds + grp * C::TILE_ELEMS;
  uint16_t* vt = ks + KT * C::KS;

  const int64_t cache_off = (((int64_t)r.row * a.Hkv + c) * a.W + r.off) * D;
  const uint16_t* kcb = static_cast<const uint16_t*>(a.k_cache) + cache_off;
  const uint16_t* vcb = static_cast<const uint16_t*>(a.v_cache) + cache_off;
  uint16_t* kcw = static_cast<uint16_t*>(a.k_cache) + cache_off;
  uint16_t* vcw = static_cast<uint16_t*>(a.v_cache) + cache_off;
  const int64_t fstride = (int64_t)a.Hkv * D;
  const uint16_t* knb = static_cast<const uint16_t*>(a.k_new) + ((int64_t)it.req * a.L * a.Hkv + c) * D;
  const uint16_t* vnb = static_cast<const uint16_t*>(a.v_new) + ((int64_t)it.req * a.L * a.Hkv + c) * D;
  // source of logical key t (clamped into the row; rows past the range are masked later)
  auto krow = [&](int t) -> const uint16_t* {
    t = min(t, it.t1 - 1);
    const bool fresh = (t >= bs) & (t < be);
    return fresh ? knb + (int64_t)(t - bs) * fstride : kcb + (int64_t)t * D;
  };
  auto vrow = [&](int t) -> const uint16_t* {
    t = min(t, it.t1 - 1);
    const bool fresh = (t >= bs) & (t < be);
    return fresh ? vnb + (int64_t)(t - bs) * fstride : vcb + (int64_t)t * D;
  };

  // queries of this lane's column as MFMA B operands: feature d = 16 kk + 8 g + e
  bf16x8_t qb[NKK];
  {
    const bool qv = j < q.B;
    const uint16_t* qp = static_cast<const uint16_t*>(a.q) + (((int64_t)it.req * a.L + min(j, q.B - 1)) * a.Hq + h) * D;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      v4u t = ld16(qp + 16 * kk + 8 * g);
      if (!qv) t = v4u{0u, 0u, 0u, 0u};
      qb[kk] = __builtin_bit_cast(bf16x8_t, t);
    }
  }

  v4u kreg[C::MAXK];
  v4u vreg[C::MAXV * 8];
  auto load_tile = [&](int tb) {
#pragma unroll
    for (int k = 0; k < C::MAXK; ++k) {
      const int cid = min(gt + k * gth, C::KCH - 1);
      kreg[k] = ld16(krow(tb + cid / (D / 8)) + (cid % (D / 8)) * 8);
    }
#pragma unroll
    for (int k = 0; k < C::MAXV; ++k) {
      const int bid = min(gt + k * gth, C::VBLK - 1);
      const int kg = bid / (D / 8), dc = bid % (D / 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) vreg[k * 8 + e] = ld16(vrow(tb + kg * 8 + e) + dc * 8);
    }
  };
  // registers -> LDS (K as is, V transposed in 8x8 blocks)
  auto store_tile = [&](int tb) {
#pragma unroll
    for (int k = 0; k < C::MAXK; ++k) {
      const int cid = gt + k * gth;
      if (cid < C::KCH) {
        const int tt = cid / (D / 8), dc = cid % (D / 8);
        st16(&ks[tt * C::KS + dc * 8], kreg[k]);
      }
    }
#pragma unroll
    for (int k = 0; k < C::MAXV; ++k) {
      const int bid = gt + k * gth;
      if (bid < C::VBLK) {
        const int kg = bid / (D / 8), dc = bid % (D / 8);
#pragma unroll
        for (int dd = 0; dd < 8; ++dd) {
          uint32_t o4[4];
#pragma unroll
          for (int qi = 0; qi < 4; ++qi) {
            const uint32_t lo = vreg[k * 8 + 2 * qi][dd >> 1];
            const uint32_t hi = vreg[k * 8 + 2 * qi + 1][dd >> 1];
            o4[qi] = (dd & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
          }
          uint2* dst = reinterpret_cast<uint2*>(&vt[(dc * 8 + dd) * C::VS + kg * 8]);
          dst[0] = make_uint2(o4[0], o4[1]);
          dst[1] = make_uint2(o4[2], o4[3]);
        }
      }
    }
  };

  f32x16_t o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) o[dt][rr] = 0.0f;
  float mrun = -__builtin_inff(), lsum = 0.0f;
  const int ntiles = (it.t1 - it.t0 + KT - 1) / KT;
  const int rounds = (ntiles + S - 1) / S;   // identical for every group: barriers stay uniform
  if (grp < ntiles) load_tile(it.t0 + grp * KT);
  for (int rd = 0; rd < rounds; ++rd) {
    const int tile = rd * S + grp;
    const bool active = tile < ntiles;
    const int tb = it.t0 + tile * KT;
    __syncthreads();
    if (active) store_tile(tb);
    __syncthreads();
    if (tile + S < ntiles) load_tile(tb + S * KT);
    if (active) {
#pragma unroll
      for (int sub = 0; sub < KT / 32; ++sub) {
        const int sb = tb + sub * 32;
        if (sb >= it.t1) break;
        f32x16_t sacc;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) sacc[rr] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
          const bf16x8_t ka = *reinterpret_cast<const bf16x8_t*>(&ks[(sub * 32 + n) * C::KS + 16 * kk + 8 * g]);
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[kk], sacc, 0, 0, 0);
        }
        // lane (g, n) holds S^T[key 8 (rr / 4) + 4 g + rr % 4][query n]
        float mx = -__builtin_inff();
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int key = sb + 8 * (rr >> 2) + 4 * g + (rr & 3);
          sacc[rr] = key < it.t1 ? sacc[rr] * a.scale_log2e : -__builtin_inff();
          mx = fmaxf(mx, sacc[rr]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float mnew = fmaxf(mrun, mx);
        const float alpha = __builtin_amdgcn_exp2f(mrun - mnew);
        bf16x8_t pb0, pb1;
        float ps = 0.0f;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const float p = __builtin_amdgcn_exp2f(sacc[rr] - mnew);
          ps += p;
          if (rr < 8)
            pb0[rr] = (__bf16)p;
          else
            pb1[rr - 8] = (__bf16)p;
        }
        lsum = lsum * alpha + ps;
        mrun = mnew;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) o[dt][rr] *= alpha;
#pragma unroll
          for (int kst = 0; kst < 2; ++kst) {
            const uint16_t* vp = &vt[(dt * 32 + n) * C::VS + sub * 32 + 16 * kst + 4 * g];
            typedef uint32_t v2u __attribute__((ext_vector_type(2)));
            const v2u lo = *reinterpret_cast<const v2u*>(vp);
            const v2u hi = *reinterpret_cast<const v2u*>(vp + 8);
            const bf16x8_t va = __builtin_bit_cast(bf16x8_t, v4u{lo.x, lo.y, hi.x, hi.y});
            o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, kst ? pb1 : pb0, o[dt], 0, 0, 0);
          }
        }
      }
    }
  }
  float lt = lsum + __shfl_xor(lsum, 32, 64);
  if constexpr (S > 1) {
    // merge the key-split groups: groups 1..S-1 park (m, l, O) in LDS
    float* mb = reinterpret_cast<float*>(lds);                  // [S-1][GW][64][2]
    float* ob = mb + (S - 1) * GW * 64 * 2;                     // [S-1][GW][NDT*16][64]
    __syncthreads();
    if (grp > 0) {
      const int slot = (grp - 1) * GW + wg;
      mb[(slot * 64 + lane) * 2 + 0] = mrun;
      mb[(slot * 64 + lane) * 2 + 1] = lt;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) ob[((int64_t)slot * NDT * 16 + dt * 16 + rr) * 64 + lane] = o[dt][rr];
    }
    __syncthreads();
    if (grp == 0) {
      float M = mrun;
#pragma unroll
      for (int s2 = 1; s2 < S; ++s2) M = fmaxf(M, mb[(((s2 - 1) * GW + wg) * 64 + lane) * 2]);
      const float f0 = __builtin_amdgcn_exp2f(mrun - M);
      lt *= f0;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) o[dt][rr] *= f0;
#pragma unroll
      for (int s2 = 1; s2 < S; ++s2) {
        const int slot = (s2 - 1) * GW + wg;
        const float fs = __builtin_amdgcn_exp2f(mb[(slot * 64 + lane) * 2] - M);
        lt += mb[(slot * 64 + lane) * 2 + 1] * fs;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) o[dt][rr] += ob[((int64_t)slot * NDT * 16 + dt * 16 + rr) * 64 + lane] * fs;
      }
    }
  }
  // in-place KV update: the fresh block rows of this KV head go to the cache
  // slot [off + s, off + s + B) (the item whose key range holds the block)
  if (a.write_back && it.t0 <= bs && bs < it.t1) {
    constexpr int MAXWB = (64 * D / 8 + MAXT / 2 - 1) / (MAXT / 2);
    const int nth = blockDim.x, nch = q.B * (D / 8);
    v4u kw[MAXWB], vw[MAXWB];
#pragma unroll
    for (int u = 0; u < MAXWB; ++u) {
      const int cid = min(tid + u * nth, nch - 1);
      const int64_t src = (int64_t)(cid / (D / 8)) * fstride + (cid % (D / 8)) * 8;
      kw[u] = ld16(knb + src);
      vw[u] = ld16(vnb + src);
    }
#pragma unroll
    for (int u = 0; u < MAXWB; ++u) {
      const int cid = tid + u * nth;
      if (cid < nch) {
        const int64_t dst = (int64_t)(bs + cid / (D / 8)) * D + (cid % (D / 8)) * 8;
        st16(kcw + dst, kw[u]);
        st16(vcw + dst, vw[u]);
      }
    }
  }
  // lane (g, n): O^T[feature dt*32 + 8 (rr / 4) + 4 g + rr % 4][query n]
  if (grp == 0 && j < a.L) {
    const float inv = (j < q.B) ? 1.0f / lt : 0.0f;
    uint16_t* op = static_cast<uint16_t*>(a.out) + (((int64_t)it.req * a.L + j) * a.Hq + h) * D;
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
        *reinterpret_cast<uint2*>(op + dt * 32 + 8 * rq + 4 * g) = make_uint2(w0, w1);
      }
  }
}

// Launch shapes: GW = G * ceil(L / 32) waves share a tile; MHA (GW = 1) splits
// each row four ways inside the workgroup, GW 2..4 two ways, GW 5..8 not at all.
int attn_splits(int GW) { return GW == 1 ? 4 : (GW <= 4 ? 2 : 1); }

template <int D>
hipError_t launch_bf16_d(const AttnArgs& a, int GW, hipStream_t s) {
  const int S = attn_splits(GW);
  const dim3 grid(a.n_items), block(64 * GW * S);
  if (S == 4)
    hipLaunchKernelGGL((k_attn_bf16<D, 32, 4, 64, 256, 1>), grid, block, 0, s, a);
  else if (S == 2)
    hipLaunchKernelGGL((k_attn_bf16<D, 32, 2, 128, 512, 1>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((k_attn_bf16<D, 64, 1, 320, 512, 1>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const AttnArgs& a, int n_req, hipStream_t s) {
  const int jblocks = (a.L + 3) / 4;
  const dim3 grid((unsigned)((int64_t)n_req * a.Hq * jblocks)), block(256);
  hipLaunchKernelGGL(k_attn_f32, grid, block, 0, s, a, jblocks);
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const AttnArgs& a, int n_req, int n_slots, hipStream_t s) {
  (void)n_req;
  (void)n_slots;
  const int GW = a.G * a.RB;
  if (a.D == 128) return launch_bf16_d<128>(a, GW, s);
  if (a.D == 64) return launch_bf16_d<64>(a, GW, s);
  return hipErrorInvalidValue;
}

}  // namespace bs
