// Broadcast chain step: in step s the link from rank root+k to rank root+k+1
// carries chunk s-k (paper sections 4 and 5: variables broadcast from one process
// to all).  Block row y is link k; every link whose chunk index is in range copies
// that chunk's bytes with 16-byte vectors, the short last unit byte by byte.
#include "internal.hpp"

namespace hvdx {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnits = 2;  // 16-byte units per lane per pass

template <bool VEC_OK>
__global__ __launch_bounds__(kBlock) void bcast_step_kernel(RankPtrs bufs, BcastArgs a) {
  const int k = blockIdx.y;
  const int64_t j = (int64_t)a.step - k;
  if (j < 0 || j >= a.n) return;
  const int src = (a.root + k) % a.n;
  const int dst = (src + 1) % a.n;
  const int64_t u0 = j * a.q + (j < a.rem ? j : a.rem);
  const int64_t units = a.q + (j < a.rem ? 1 : 0);
  const int64_t lo = u0 * 16 < a.nbytes ? u0 * 16 : a.nbytes;
  const int64_t hi = (u0 + units) * 16 < a.nbytes ? (u0 + units) * 16 : a.nbytes;
  const unsigned char* __restrict__ s = static_cast<const unsigned char*>(bufs.p[src]);
  unsigned char* __restrict__ d = static_cast<unsigned char*>(bufs.p[dst]);
  const int64_t full = VEC_OK ? (hi - lo) / 16 : 0;  // whole units in the chunk
  const int64_t gtid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * kBlock;
  const u32x4* __restrict__ s4 = reinterpret_cast<const u32x4*>(s + lo);
  u32x4* __restrict__ d4 = reinterpret_cast<u32x4*>(d + lo);
  for (int64_t base = (int64_t)blockIdx.x * kBlock * kUnits + threadIdx.x; base < full;
       base += gthreads * kUnits) {
    u32x4 v[kUnits];
#pragma unroll
    for (int u = 0; u < kUnits; ++u)
      if (base + u * kBlock < full) v[u] = __builtin_nontemporal_load(s4 + base + u * kBlock);
#pragma unroll
    for (int u = 0; u < kUnits; ++u)
      if (base + u * kBlock < full) __builtin_nontemporal_store(v[u], d4 + base + u * kBlock);
  }
  for (int64_t e = lo + full * 16 + gtid; e < hi; e += gthreads) d[e] = s[e];
}

}  // namespace

hipError_t launch_bcast_step(const RankPtrs& bufs, const BcastArgs& a, bool vector_ok, hipStream_t stream) {
  const int64_t longest = a.q + (a.rem ? 1 : 0);
  int64_t bx = (longest + (int64_t)kBlock * kUnits - 1) / ((int64_t)kBlock * kUnits);
  if (bx < 1) bx = 1;
  if (bx > (1 << 20)) bx = 1 << 20;
  const dim3 grid((unsigned)bx, (unsigned)(a.n - 1));
  if (vector_ok)
    HVDX_LAUNCH((bcast_step_kernel<true>), grid, dim3(kBlock), 0, stream, bufs, a);
  else
    HVDX_LAUNCH((bcast_step_kernel<false>), grid, dim3(kBlock), 0, stream, bufs, a);
  return hipGetLastError();
}

}  // namespace hvdx
