// K1: gather of the active blocks into compact [n][L] tensors and the inverse
// scatter (paragraph "Vectorized mixed-schedule execution"). One thread per
// compact cell (i, j); an element is 1..16 bytes and is moved as one word.
#include "bs_internal.h"

namespace bs {
namespace {

template <int EB>
struct Word;
template <> struct Word<1> { using T = uint8_t; };
template <> struct Word<2> { using T = uint16_t; };
template <> struct Word<4> { using T = uint32_t; };
template <> struct Word<8> { using T = uint2; };
template <> struct Word<16> { using T = uint4; };

template <int EB>
__global__ __launch_bounds__(256) void k_gather(const bs_req_desc* __restrict__ reqs, int n, int L,
                                                const char* __restrict__ src, int64_t stride,
                                                char* __restrict__ dst, int32_t* __restrict__ pos) {
  using T = typename Word<EB>::T;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * L) return;
  const int i = t / L, j = t - i * L;
  const bs_req_desc r = reqs[i];
  const Geo q = geo_of(r, L);
  T v{};
  int p = -1;
  if (j < q.B) {
    v = *reinterpret_cast<const T*>(src + (int64_t)r.row * stride + (int64_t)(r.off + q.s + j) * EB);
    p = q.s + j;
  }
  reinterpret_cast<T*>(dst)[t] = v;
  if (pos) pos[t] = p;
}

template <int EB>
__global__ __launch_bounds__(256) void k_scatter(const bs_req_desc* __restrict__ reqs, int n, int L,
                                                 const char* __restrict__ src, char* __restrict__ dst,
                                                 int64_t stride) {
  using T = typename Word<EB>::T;
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * L) return;
  const int i = t / L, j = t - i * L;
  const bs_req_desc r = reqs[i];
  const Geo q = geo_of(r, L);
  if (j >= q.B) return;
  *reinterpret_cast<T*>(dst + (int64_t)r.row * stride + (int64_t)(r.off + q.s + j) * EB) =
      reinterpret_cast<const T*>(src)[t];
}

}  // namespace

hipError_t launch_gather(const bs_req_desc* reqs, int n, int L, const void* src, int64_t stride,
                         int eb, void* dst, int32_t* pos, hipStream_t s) {
  const int total = n * L;
  const dim3 grid((total + 255) / 256), block(256);
  const char* sp = static_cast<const char*>(src);
  char* dp = static_cast<char*>(dst);
  switch (eb) {
    case 1: hipLaunchKernelGGL(k_gather<1>, grid, block, 0, s, reqs, n, L, sp, stride, dp, pos); break;
    case 2: hipLaunchKernelGGL(k_gather<2>, grid, block, 0, s, reqs, n, L, sp, stride, dp, pos); break;
    case 4: hipLaunchKernelGGL(k_gather<4>, grid, block, 0, s, reqs, n, L, sp, stride, dp, pos); break;
    case 8: hipLaunchKernelGGL(k_gather<8>, grid, block, 0, s, reqs, n, L, sp, stride, dp, pos); break;
    case 16: hipLaunchKernelGGL(k_gather<16>, grid, block, 0, s, reqs, n, L, sp, stride, dp, pos); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_scatter(const bs_req_desc* reqs, int n, int L, const void* src, int eb,
                          void* dst, int64_t stride, hipStream_t s) {
  const int total = n * L;
  const dim3 grid((total + 255) / 256), block(256);
  const char* sp = static_cast<const char*>(src);
  char* dp = static_cast<char*>(dst);
  switch (eb) {
    case 1: hipLaunchKernelGGL(k_scatter<1>, grid, block, 0, s, reqs, n, L, sp, dp, stride); break;
    case 2: hipLaunchKernelGGL(k_scatter<2>, grid, block, 0, s, reqs, n, L, sp, dp, stride); break;
    case 4: hipLaunchKernelGGL(k_scatter<4>, grid, block, 0, s, reqs, n, L, sp, dp, stride); break;
    case 8: hipLaunchKernelGGL(k_scatter<8>, grid, block, 0, s, reqs, n, L, sp, dp, stride); break;
    case 16: hipLaunchKernelGGL(k_scatter<16>, grid, block, 0, s, reqs, n, L, sp, dp, stride); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace bs
