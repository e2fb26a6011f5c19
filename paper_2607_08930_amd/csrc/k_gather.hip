// K1: gather of the active blocks into compact [n][L] tensors and the inverse
// scatter (paragraph "Vectorized mixed-schedule execution"). One thread per
// compact cell (i, j) moves that cell of every tensor of the call (token ids
// and mask bits travel in one launch); an element is 1..16 bytes, moved as
// one word.
#include "bs_internal.h"

namespace bs {
namespace {

template <int EB>
struct Word;
template <> struct Word<1> { using T = uint8_t; };
template <> struct Word<2> { using T = uint16_t; };
template <> struct Word<4> { using T = uint32_t; };
template <> struct Word<8> { using T = uint2; };
template <> struct Word<16> { using T = v4u; };

template <int EB>
__device__ inline void move(const char* src, char* dst) {
  using T = typename Word<EB>::T;
  *reinterpret_cast<T*>(dst) = *reinterpret_cast<const T*>(src);
}
template <int EB>
__device__ inline void zero(char* dst) {
  using T = typename Word<EB>::T;
  *reinterpret_cast<T*>(dst) = T{};
}

__device__ inline void move_any(int eb, const char* src, char* dst) {
  switch (eb) {
    case 1: move<1>(src, dst); break;
    case 2: move<2>(src, dst); break;
    case 4: move<4>(src, dst); break;
    case 8: move<8>(src, dst); break;
    default: move<16>(src, dst); break;
  }
}
__device__ inline void zero_any(int eb, char* dst) {
  switch (eb) {
    case 1: zero<1>(dst); break;
    case 2: zero<2>(dst); break;
    case 4: zero<4>(dst); break;
    case 8: zero<8>(dst); break;
    default: zero<16>(dst); break;
  }
}

__global__ __launch_bounds__(256) void k_gather(const bs_req_desc* __restrict__ reqs, int n, int L, GatherSet g,
                                                int32_t* __restrict__ pos) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * L) return;
  const int i = t / L, j = t - i * L;
  const bs_req_desc r = reqs[i];
  const Geo q = geo_of(r, L);
  const bool in = j < q.B;
  for (int k = 0; k < g.count; ++k) {
    char* d = static_cast<char*>(g.compact[k]) + (int64_t)t * g.eb[k];
    if (in)
      move_any(g.eb[k], static_cast<const char*>(g.dense[k]) + (int64_t)r.row * g.stride[k] +
                            (int64_t)(r.off + q.s + j) * g.eb[k], d);
    else
      zero_any(g.eb[k], d);
  }
  if (pos) pos[t] = in ? q.s + j : -1;
}

__global__ __launch_bounds__(256) void k_scatter(const bs_req_desc* __restrict__ reqs, int n, int L, GatherSet g) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * L) return;
  const int i = t / L, j = t - i * L;
  const bs_req_desc r = reqs[i];
  const Geo q = geo_of(r, L);
  if (j >= q.B) return;
  for (int k = 0; k < g.count; ++k)
    move_any(g.eb[k], static_cast<const char*>(g.compact[k]) + (int64_t)t * g.eb[k],
             static_cast<char*>(const_cast<void*>(g.dense[k])) + (int64_t)r.row * g.stride[k] + (int64_t)(r.off + q.s + j) * g.eb[k]);
}

}  // namespace

hipError_t launch_gather(const bs_req_desc* reqs, int n, int L, const GatherSet& g, int32_t* pos, hipStream_t s) {
  hipLaunchKernelGGL(k_gather, dim3((n * L + 255) / 256), dim3(256), 0, s, reqs, n, L, g, pos);
  return hipGetLastError();
}

hipError_t launch_scatter(const bs_req_desc* reqs, int n, int L, const GatherSet& g, hipStream_t s) {
  hipLaunchKernelGGL(k_scatter, dim3((n * L + 255) / 256), dim3(256), 0, s, reqs, n, L, g);
  return hipGetLastError();
}

}  // namespace bs
