// K3: confidence-aware parallel decode (paragraph "Vectorized mixed-schedule
// execution"; greedy decoding, "Implementation details").
//
// Pass 1 (k_decode_rows): one 256-thread workgroup per (masked row, 64 KiB
// chunk of the vocabulary). Every thread issues all 16 of its 16-byte loads
// up front, then reduces in registers: chunk max, then sum exp(x - max), then
// the smallest index attaining the max. Rows that are not masked, and rows past
// the request's block, exit before reading anything.
// Pass 2 (k_decode_select): one wave per request; lane j merges row j's chunk
// partials in chunk order (deterministic), derives the confidence, and the wave
// ranks the masked positions to apply the threshold/quota rule in place.
#include <float.h>
#include <limits.h>

#include "bs_internal.h"

namespace bs {
namespace {

constexpr int kThreads = 256;
constexpr int kVecBytes = 16;
constexpr int kLoads = kDecChunkBytes / (kThreads * kVecBytes);  // 16
constexpr float kLog2e = 1.4426950408889634f;

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

// Elements of one 16-byte vector as fp32.
template <typename T>
struct Lanes;
template <>
struct Lanes<uint16_t> {  // bf16
  static constexpr int N = 8;
  __device__ static inline float get(const v4u& v, int e) {
    const uint32_t w = v[e >> 1];
    return __uint_as_float((e & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
  // element e -> -inf when `drop`
  __device__ static inline void mask(v4u& v, int e, bool drop) {
    const uint32_t w = v[e >> 1];
    const uint32_t m = (e & 1) ? ((w & 0x0000FFFFu) | 0xFF800000u) : ((w & 0xFFFF0000u) | 0x0000FF80u);
    v[e >> 1] = drop ? m : w;
  }
};
template <>
struct Lanes<float> {
  static constexpr int N = 4;
  __device__ static inline float get(const v4u& v, int e) { return __uint_as_float(v[e]); }
  __device__ static inline void mask(v4u& v, int e, bool drop) { v[e] = drop ? 0xFF800000u : v[e]; }
};

template <typename T>
__global__ __launch_bounds__(kThreads) void k_decode_rows(DecArgs a) {
  constexpr int N = Lanes<T>::N;
  constexpr int CH = kDecChunkBytes / sizeof(T);
  const int c = blockIdx.x % a.nchunk;
  const int row = blockIdx.x / a.nchunk;
  const int i = row / a.L, j = row - i * a.L;
  const Geo q = geo_of(a.reqs[i], a.L);
  if (j >= q.B || a.masked[row] == 0) return;
  const T* x = static_cast<const T*>(a.logits) + (int64_t)row * a.row_stride;
  const int v0 = c * CH;
  const int v1 = min(a.V, v0 + CH);
  const int tid = threadIdx.x;

  // Branch-free loads: a vector that starts past the row end re-reads the
  // chunk's first vector; elements at or past V are then set to -inf. A vector
  // that starts before V stays inside the row's padded stride.
  v4u buf[kLoads];
#pragma unroll
  for (int u = 0; u < kLoads; ++u) {
    const int e = v0 + (u * kThreads + tid) * N;
    buf[u] = ld16(x + (e < v1 ? e : v0));
  }
  if (v0 + CH > a.V) {  // last chunk of the row: mask the ragged end
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      const int e = v0 + (u * kThreads + tid) * N;
#pragma unroll
      for (int k = 0; k < N; ++k) Lanes<T>::mask(buf[u], k, e + k >= v1);
    }
  }
  // chunk max
  float m = -__builtin_inff();
#pragma unroll
  for (int u = 0; u < kLoads; ++u)
#pragma unroll
    for (int e = 0; e < N; ++e) m = fmaxf(m, Lanes<T>::get(buf[u], e));
  __shared__ float sm[kThreads / 64];
  __shared__ float ss[kThreads / 64];
  __shared__ int sa[kThreads / 64];
  const int w = tid >> 6, lane = tid & 63;
  float wm = wave_max(m);
  if (lane == 0) sm[w] = wm;
  __syncthreads();
  float M = sm[0];
#pragma unroll
  for (int k = 1; k < kThreads / 64; ++k) M = fmaxf(M, sm[k]);
  // sum of exp(x - M) with independent partial sums per vector lane
  const float mb = M * kLog2e;
  float acc[N];
#pragma unroll
  for (int e = 0; e < N; ++e) acc[e] = 0.0f;
#pragma unroll
  for (int u = 0; u < kLoads; ++u)
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] += __builtin_amdgcn_exp2f(fmaf(Lanes<T>::get(buf[u], e), kLog2e, -mb));
  float s = 0.0f;
#pragma unroll
  for (int e = 0; e < N; ++e) s += acc[e];
  // smallest index holding M (only threads whose own max is M scan)
  int arg = INT_MAX;
  if (m == M) {
#pragma unroll
    for (int u = 0; u < kLoads; ++u)
#pragma unroll
      for (int e = 0; e < N; ++e) {
        const int idx = v0 + (u * kThreads + tid) * N + e;
        if (Lanes<T>::get(buf[u], e) == M && idx < arg) arg = idx;
      }
  }
  float ws_ = wave_sum(s);
  int wa = wave_min_i(arg);
  if (lane == 0) {
    ss[w] = ws_;
    sa[w] = wa;
  }
  __syncthreads();
  if (tid == 0) {
    float S = 0.0f;
    int A = INT_MAX;
    for (int k = 0; k < kThreads / 64; ++k) {
      S += ss[k];
      A = min(A, sa[k]);
    }
    DecPartial pr;
    pr.m = M;
    pr.s = S;
    pr.a = A;
    pr.pad = 0;
    a.part[(int64_t)row * a.nchunk + c] = pr;
  }
}

__global__ __launch_bounds__(256) void k_decode_select(DecArgs a) {
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + wv;
  if (i >= a.n) return;
  const Geo q = geo_of(a.reqs[i], a.L);
  const int j = lane;
  const int64_t cell = (int64_t)i * a.L + j;
  const bool inb = j < q.B;
  const bool m = inb && a.masked[cell] != 0;
  float conf = -1.0f;
  int arg = 0;
  if (m) {
    const DecPartial* pp = a.part + cell * a.nchunk;
    float M = pp[0].m;
    arg = pp[0].a;
    for (int c = 1; c < a.nchunk; ++c)
      if (pp[c].m > M) {
        M = pp[c].m;
        arg = pp[c].a;
      }
    float S = 0.0f;
    for (int c = 0; c < a.nchunk; ++c) S += pp[c].s * __builtin_amdgcn_exp2f((pp[c].m - M) * kLog2e);
    conf = 1.0f / S;
  }
  const unsigned long long bm = __ballot(m);
  const unsigned long long bt = __ballot(m && conf >= a.tau);
  const int nM = __popcll(bm);
  const int nT = __popcll(bt);
  const int nsel = min(nM, max(a.q_min, nT));
  // rank among masked positions: higher confidence first, then smaller j
  int rank = 0;
  for (int jj = 0; jj < 64; ++jj) {
    const float cj = __shfl(conf, jj, 64);
    if (((bm >> jj) & 1ull) && (cj > conf || (cj == conf && jj < j))) ++rank;
  }
  const bool sel = m && rank < nsel;
  int tok = 0;
  bool still = false;
  if (j < a.L) {
    tok = a.tokens[cell];
    still = a.masked[cell] != 0;
    if (sel) {
      tok = arg;
      still = false;
      a.tokens[cell] = arg;
      a.masked[cell] = 0;
    }
    if (a.conf_out) a.conf_out[cell] = m ? conf : -1.0f;
  }
  const bool e = inb && !still && a.eos_id >= 0 && tok == a.eos_id;
  const unsigned long long be = __ballot(e);
  if (lane == 0) {
    a.n_unmasked[i] = nsel;
    a.done[i] = (nsel == nM) ? 1 : 0;
    a.eos_seen[i] = be ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_decode(const DecArgs& a, bs_dtype dt, hipStream_t s) {
  const int64_t rows = (int64_t)a.n * a.L;
  const dim3 g1((unsigned)(rows * a.nchunk)), b1(kThreads);
  if (dt == BS_BF16)
    hipLaunchKernelGGL(k_decode_rows<uint16_t>, g1, b1, 0, s, a);
  else
    hipLaunchKernelGGL(k_decode_rows<float>, g1, b1, 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_decode_select, dim3((a.n + 3) / 4), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bs
