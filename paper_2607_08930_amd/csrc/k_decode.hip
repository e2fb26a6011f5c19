// K3: confidence-aware parallel decode (paragraph "Vectorized mixed-schedule
// execution"; greedy decoding, "Implementation details").
//
// Two launches. k_decode_parts: a masked row is split into parts of
// kDecPartChunks chunks of 32 KiB and one 256-thread workgroup streams one
// part (rows that are not masked exit at once). Within a part the chunks are
// register double buffered: the next chunk's eight 16-byte loads per thread
// are in flight while the current one is reduced. Each thread keeps an online
// (max, sum of exp(x - max)) and the first vector holding its max; the
// workgroup merges the threads' results, and only threads holding the part max
// re-read that one vector to find the smallest index attaining it. The part
// result (max, sum, argmax) goes to the workspace.
// k_decode_select: one wave per request merges every row's parts and runs the
// selection. The launch boundary orders the two, so no workgroup waits on
// another and no cache maintenance is needed inside either kernel.
#include <float.h>
#include <limits.h>

#include "bs_internal.h"

namespace bs {
namespace {

constexpr int kThreads = 256;
constexpr int kLoads = kDecChunkBytes / (kThreads * 16);  // 8
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// max without the canonicalisation fmaxf needs in IEEE mode: every value
// reduced here is a finite logit or -inf (masked tail), never NaN
__device__ inline float vmax(float x, float y) { return __builtin_elementwise_maximum(x, y); }

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = vmax(v, __shfl_xor(v, o, 64));
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

// Loads of one chunk: vector u of thread tid starts at element v0 + (u*256 + tid)*N,
// with the non-temporal hint (a logits row is read once; measured: Dream-7B
// layer decode rows 56.6 -> 54.6 us).
// A vector that starts past the row end re-reads the chunk's first vector (a
// valid address); elements at or past V are masked when the chunk is folded.
// A vector starting before V stays inside the row's padded 16-byte stride.
template <typename T>
__device__ inline void load_chunk(v4u (&buf)[kLoads], const T* x, int v0, int V, int tid) {
  constexpr int N = Lanes<T>::N;
#pragma unroll
  for (int u = 0; u < kLoads; ++u) {
    const int e = v0 + (u * kThreads + tid) * N;
    buf[u] = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(x + (e < V ? e : v0)));
  }
}

template <typename T>
__device__ inline void mask_tail(v4u (&buf)[kLoads], int v0, int V, int tid) {
  constexpr int N = Lanes<T>::N;
  constexpr int CH = kDecChunkBytes / sizeof(T);
  if (v0 + CH > V) {  // last chunk of the row only
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      const int e = v0 + (u * kThreads + tid) * N;
#pragma unroll
      for (int k = 0; k < N; ++k) Lanes<T>::mask(buf[u], k, e + k >= V);
    }
  }
}

// Running reduction of one thread over its elements, in increasing index
// order: exact max `mt` with the start `vbest` of the first 16-byte vector
// holding it, and the sum `s` of exp(x - mb / log2 e). The shift mb (log2
// domain) is raised lazily, only when a vector's max exceeds it by more than
// 8, so every term stays below 2^8 and the sum far from overflow; `thr` is
// that bound in logit units, (mb + 8) ln 2, so the common case costs one
// compare per vector. mb starts at -FLT_MAX rather than -inf so that -inf
// elements contribute exp2(-inf) = 0.
struct RowAcc {
  float mt = -__builtin_inff();
  int vbest = 0;
  float mb = -FLT_MAX;
  float thr = -FLT_MAX;
  float s = 0.0f;
};

template <typename T>
__device__ inline void fold_vector(const v4u& v, int e0, RowAcc& r) {
  constexpr int N = Lanes<T>::N;
  float f[N];
#pragma unroll
  for (int k = 0; k < N; ++k) f[k] = Lanes<T>::get(v, k);
  float vm = f[0];
#pragma unroll
  for (int k = 1; k < N; ++k) vm = vmax(vm, f[k]);
  if (vm > r.mt) {
    r.mt = vm;
    r.vbest = e0;
  }
  if (vm > r.thr) {
    // rare (a handful of times per row): a real branch, not a select, so the
    // common path does not evaluate the rescale
    asm volatile("");
    const float nb = vm * kLog2e;
    r.s *= __builtin_amdgcn_exp2f(r.mb - nb);
    r.mb = nb;
    r.thr = (nb + 8.0f) * kLn2;
  }
  float acc = __builtin_amdgcn_exp2f(fmaf(f[0], kLog2e, -r.mb));
#pragma unroll
  for (int k = 1; k < N; ++k) acc += __builtin_amdgcn_exp2f(fmaf(f[k], kLog2e, -r.mb));
  r.s += acc;
}

template <typename T>
__device__ inline void fold_chunk(v4u (&buf)[kLoads], int v0, int V, int tid, RowAcc& r) {
  constexpr int N = Lanes<T>::N;
  mask_tail<T>(buf, v0, V, tid);
#pragma unroll
  for (int u = 0; u < kLoads; ++u) fold_vector<T>(buf[u], v0 + (u * kThreads + tid) * N, r);
}

// Selection of request i by one wave (lane j = block position j): merge the
// row's part results, apply n = min(|M|, max(q_min, #{c >= tau})) to the
// most confident positions (ties: smallest j), update tokens/mask in place.
// Cell of block position j < B_i of request i in the token / mask state.
__device__ inline int64_t state_cell(const DecArgs& a, const bs_req_desc& r, const Geo& q, int i, int j, int64_t rs) {
  return a.dense ? (int64_t)r.row * rs + r.off + q.s + j : (int64_t)i * a.L + j;
}

__device__ inline void select_request(const DecArgs& a, int i, int lane) {
  const int j = lane;
  const int64_t cell = (int64_t)i * a.L + j;   // compact index: logits rows, part results, conf_out
  // The part results do not depend on the descriptor: their loads are issued
  // first so that they travel together with the descriptor's.
  constexpr int kUnroll = 8;
  const DecPartial* pp = a.part + (j < a.L ? cell : (int64_t)i * a.L) * a.parts;
  DecPartial pr[kUnroll];
#pragma unroll
  for (int p = 0; p < kUnroll; ++p) pr[p] = pp[min(p, a.parts - 1)];
  const bs_req_desc rq = a.reqs[i];
  const Geo q = geo_of(rq, a.L);
  const bool inb = j < q.B;
  const int64_t tc = inb ? state_cell(a, rq, q, i, j, a.tok_rs) : 0;
  const int64_t mc = inb ? state_cell(a, rq, q, i, j, a.msk_rs) : 0;
  const int tok0 = inb ? a.tokens[tc] : 0;
  const bool m = inb && a.masked[mc] != 0;
  float conf = -1.0f;
  int arg = 0;
  if (m) {
    float M = -__builtin_inff();
#pragma unroll
    for (int p = 0; p < kUnroll; ++p) M = fmaxf(M, pr[p].m);   // repeats of the last part change nothing
    for (int p = kUnroll; p < a.parts; ++p) M = fmaxf(M, pp[p].m);
    // parts without a finite logit (m = -inf, s = 0) add nothing; they are
    // skipped so that (-inf) - M never reaches the exponential
    float S = 0.0f;
    int A = INT_MAX;
#pragma unroll
    for (int p = 0; p < kUnroll; ++p)
      if (p < a.parts) {
        if (pr[p].m != -__builtin_inff()) S += pr[p].s * __builtin_amdgcn_exp2f((pr[p].m - M) * kLog2e);
        if (pr[p].m == M) A = min(A, pr[p].a);
      }
    for (int p = kUnroll; p < a.parts; ++p) {
      const DecPartial x = pp[p];
      if (x.m != -__builtin_inff()) S += x.s * __builtin_amdgcn_exp2f((x.m - M) * kLog2e);
      if (x.m == M) A = min(A, x.a);
    }
    conf = 1.0f / S;
    arg = A;
  }
  const unsigned long long bm = __ballot(m);
  const unsigned long long bt = __ballot(m && conf >= a.tau);
  const int nM = __popcll(bm);
  const int nT = __popcll(bt);
  const int nsel = min(nM, max(a.q_min, nT));
  // rank among masked positions: higher confidence first, then smaller j
  // (lane jj's confidence is read through the scalar unit)
  int rank = 0;
  const int cbits = __float_as_int(conf);
  for (unsigned long long rest = bm; rest; rest &= rest - 1) {
    const int jj = __builtin_ctzll(rest);
    const float cj = __int_as_float(__builtin_amdgcn_readlane(cbits, jj));
    if (cj > conf || (cj == conf && jj < j)) ++rank;
  }
  const bool sel = m && rank < nsel;
  int tok = tok0;
  bool still = m;
  if (sel) {
    tok = arg;
    still = false;
    a.tokens[tc] = arg;
    a.masked[mc] = 0;
  }
  if (j < a.L) {
    if (a.conf_out) a.conf_out[cell] = m ? conf : -1.0f;
    if (a.pos_out) a.pos_out[cell] = inb ? q.s + j : -1;
  }
  const bool e = inb && !still && a.eos_id >= 0 && tok == a.eos_id;
  const unsigned long long be = __ballot(e);
  if (lane == 0) {
    a.n_unmasked[i] = nsel;
    a.done[i] = (nsel == nM) ? 1 : 0;
    a.eos_seen[i] = be ? 1 : 0;
  }
}

// Stream NC chunks starting at chunk c0 (two register buffers; every load is
// issued unconditionally, so only the buffer about to be folded is waited for).
template <typename T, int NC>
__device__ inline void stream_part(const T* x, int c0, int V, int tid, RowAcc& r) {
  constexpr int CH = kDecChunkBytes / sizeof(T);
  v4u buf[2][kLoads];
  load_chunk<T>(buf[0], x, c0 * CH, V, tid);
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    if (k + 1 < NC) load_chunk<T>(buf[(k + 1) & 1], x, (c0 + k + 1) * CH, V, tid);
    fold_chunk<T>(buf[k & 1], (c0 + k) * CH, V, tid, r);
  }
}

template <typename T>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_decode_parts(DecArgs a) {
  constexpr int N = Lanes<T>::N;
  constexpr int CH = kDecChunkBytes / sizeof(T);
  static_assert(kDecPartChunks >= 1 && kDecPartChunks <= 4, "stream_part is instantiated for 1..4 chunks");
  int row, part;
  if (a.words) {
    // fused step: workgroup (k, i, part), k outermost, streams part `part` of
    // the k-th masked position of request i; k past the request's count exits
    // (those workgroups come last in the grid)
    const int t = blockIdx.x / a.parts;
    part = blockIdx.x - t * a.parts;
    const int k = t / a.n, i = t - k * a.n;
    uint64_t bits = a.words[i];
    if (k >= __popcll(bits)) return;
    for (int r = 0; r < k; ++r) bits &= bits - 1;
    row = i * a.L + __builtin_ctzll(bits);
  } else {
    row = blockIdx.x / a.parts;
    part = blockIdx.x - row * a.parts;
    const int i = row / a.L, j = row - i * a.L;
    const bs_req_desc rq = a.reqs[i];
    const Geo q = geo_of(rq, a.L);
    if (j >= q.B || a.masked[state_cell(a, rq, q, i, j, a.msk_rs)] == 0) return;
  }
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const T* x = static_cast<const T*>(a.logits) + (int64_t)row * a.row_stride;
  const int nchunk = (a.V + CH - 1) / CH;
  const int c0 = part * kDecPartChunks;
  const int nc = min(kDecPartChunks, nchunk - c0);   // >= 1: parts = ceil(nchunk / kDecPartChunks)

  RowAcc r;
  switch (nc) {
    case 1: stream_part<T, 1>(x, c0, a.V, tid, r); break;
    case 2: stream_part<T, (kDecPartChunks >= 2 ? 2 : 1)>(x, c0, a.V, tid, r); break;
    case 3: stream_part<T, (kDecPartChunks >= 3 ? 3 : 1)>(x, c0, a.V, tid, r); break;
    default: stream_part<T, kDecPartChunks>(x, c0, a.V, tid, r); break;
  }
  // part max and sum across the workgroup
  __shared__ float sm[kThreads / 64];
  __shared__ float ss[kThreads / 64];
  __shared__ int sa[kThreads / 64];
  const float wm = wave_max(r.mt);
  if (lane == 0) sm[w] = wm;
  __syncthreads();
  float M = sm[0];
#pragma unroll
  for (int k = 1; k < kThreads / 64; ++k) M = vmax(M, sm[k]);
  // r.mb <= r.mt * log2 e <= M * log2 e, so the factor is at most 1. A part
  // whose logits are all -inf (M = -inf) sums to 0: its threads hold s = 0
  // and mb = -FLT_MAX, and exp2(mb - M) would be exp2(+inf).
  const float sc = M == -__builtin_inff() ? 0.0f : r.s * __builtin_amdgcn_exp2f(r.mb - M * kLog2e);
  // smallest index holding M: threads whose max is M re-read the one vector
  // where they first saw it
  int arg = INT_MAX;
  if (r.mt == M) {
    const v4u v = ld16(x + r.vbest);
#pragma unroll
    for (int e = N - 1; e >= 0; --e)
      if (Lanes<T>::get(v, e) == M && r.vbest + e < a.V) arg = r.vbest + e;
  }
  const float wsum = wave_sum(sc);
  const int wa = wave_min_i(arg);
  if (lane == 0) {
    ss[w] = wsum;
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
    a.part[(int64_t)row * a.parts + part] = pr;
  }
}

__global__ __launch_bounds__(64) void k_decode_select(DecArgs a) {
  select_request(a, blockIdx.x, threadIdx.x);
}

}  // namespace

hipError_t launch_decode_rows(const DecArgs& a, bs_dtype dt, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)a.n * a.L * a.parts)), block(kThreads);
  if (dt == BS_BF16)
    hipLaunchKernelGGL(k_decode_parts<uint16_t>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(k_decode_parts<float>, grid, block, 0, s, a);
  return hipGetLastError();
}

hipError_t launch_decode_select(const DecArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_decode_select, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_decode(const DecArgs& a, bs_dtype dt, hipStream_t s) {
  return launch_decode_marked(a, dt, s, [](int) { return hipSuccess; });
}

}  // namespace bs
