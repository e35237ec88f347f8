// Tensor Fusion copy-in and copy-out kernels (paper section 7, steps 3 and 5).
//
// The iteration space is the fusion buffer, not the tensor list: block x owns one
// tile of buffer positions and serves it for every rank.  Each lane handles one
// 16-byte vector of the buffer, so load balance does not depend on how ragged the
// tensors are (Inception-V3 mixes 32-element batch-norm vectors with 2M-element
// weights).  A block finds the tensors that overlap its tile once, stages their
// offsets and ends in LDS, and reuses them for all N ranks; per rank it stages the
// N tensor pointers of that rank.  A lane binary-searches the LDS table for its
// vector's tensor.  Vectors entirely inside one tensor with a 16-byte aligned
// source take the vector path; tensor tails, padding and unaligned tensors take a
// per-element path.  Padding is written as zero by the copy-in and skipped by the
// copy-out.

#include "internal.hpp"

namespace hvdx {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

constexpr int kTileVecs = kBlock * 4;  // 16-byte buffer vectors per block tile
constexpr int kLdsTensors = 1024 + 8;  // tensors a tile can stage in LDS

template <typename TB>
struct BufVec {
  static constexpr int n = 16 / sizeof(TB);  // buffer elements per 16 bytes
};

// Convert and move VEC = 16/sizeof(TB) elements between a tensor of type TT and
// the buffer of type TB (TT == TB, or TT = float and TB = _Float16).
template <typename TT, typename TB>
struct Mover;

template <>
struct Mover<float, float> {
  __device__ static void to_buf(const float* src, float* dst) {
    *reinterpret_cast<f32x4*>(dst) = *reinterpret_cast<const f32x4*>(src);
  }
  __device__ static void from_buf(const float* src, float* dst) {
    *reinterpret_cast<f32x4*>(dst) = *reinterpret_cast<const f32x4*>(src);
  }
  __device__ static float cvt_in(float v) { return v; }
  __device__ static float cvt_out(float v) { return v; }
};

template <>
struct Mover<_Float16, _Float16> {
  __device__ static void to_buf(const _Float16* src, _Float16* dst) {
    *reinterpret_cast<f16x8*>(dst) = *reinterpret_cast<const f16x8*>(src);
  }
  __device__ static void from_buf(const _Float16* src, _Float16* dst) {
    *reinterpret_cast<f16x8*>(dst) = *reinterpret_cast<const f16x8*>(src);
  }
  __device__ static _Float16 cvt_in(_Float16 v) { return v; }
  __device__ static _Float16 cvt_out(_Float16 v) { return v; }
};

template <>
struct Mover<float, _Float16> {  // tensor binary32, buffer binary16
  __device__ static void to_buf(const float* src, _Float16* dst) {
    const f32x4 lo = reinterpret_cast<const f32x4*>(src)[0];
    const f32x4 hi = reinterpret_cast<const f32x4*>(src)[1];
    f16x8 h;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      h[k] = (_Float16)lo[k];
      h[k + 4] = (_Float16)hi[k];
    }
    *reinterpret_cast<f16x8*>(dst) = h;
  }
  __device__ static void from_buf(const _Float16* src, float* dst) {
    const f16x8 h = *reinterpret_cast<const f16x8*>(src);
    f32x4 lo, hi;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      lo[k] = (float)h[k];
      hi[k] = (float)h[k + 4];
    }
    reinterpret_cast<f32x4*>(dst)[0] = lo;
    reinterpret_cast<f32x4*>(dst)[1] = hi;
  }
  __device__ static _Float16 cvt_in(float v) { return (_Float16)v; }
  __device__ static float cvt_out(_Float16 v) { return (float)v; }
};

__device__ __forceinline__ void store_zero(float* p) { *reinterpret_cast<f32x4*>(p) = (f32x4)(0.0f); }
__device__ __forceinline__ void store_zero(_Float16* p) {
  *reinterpret_cast<f16x8*>(p) = (f16x8)((_Float16)0.0f);
}

// Last tensor t in [lo, hi) whose offset is <= p, or lo - 1 if none (global memory).
__device__ int64_t find_tensor_global(const int64_t* offset, int64_t lo, int64_t hi, int64_t p) {
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (offset[mid] <= p) lo = mid + 1;
    else hi = mid;
  }
  return lo - 1;
}

struct TileTable {
  int64_t t0;       // first tensor that can own a position of the tile (may be -1)
  int nt;           // tensors t0 .. t0+nt-1 cover the tile
  bool in_lds;      // their offsets/ends are staged in LDS
};

// Thread 0 locates the tile's tensors; everyone stages their offsets and ends.
__device__ TileTable stage_tile(const int64_t* offset, const int64_t* numel, int ntensors, int64_t p0, int64_t p1,
                                int64_t* s_off, int64_t* s_end, int64_t* s_meta) {
  if (threadIdx.x == 0) {
    const int64_t t0 = find_tensor_global(offset, 0, ntensors, p0);
    const int64_t t1 = find_tensor_global(offset, t0 < 0 ? 0 : t0, ntensors, p1 - 1);
    s_meta[0] = t0;
    s_meta[1] = t1 - t0 + 1;
  }
  __syncthreads();
  TileTable tt;
  tt.t0 = s_meta[0];
  tt.nt = (int)s_meta[1];
  tt.in_lds = tt.nt <= kLdsTensors;
  if (tt.in_lds) {
    for (int j = threadIdx.x; j < tt.nt; j += kBlock) {
      const int64_t t = tt.t0 + j;
      if (t >= 0) {
        s_off[j] = offset[t];
        s_end[j] = offset[t] + numel[t];
      } else {  // positions before the first tensor are padding
        s_off[j] = INT64_MIN;
        s_end[j] = INT64_MIN;
      }
    }
  }
  __syncthreads();
  return tt;
}

// Index j (into the tile table) of the tensor owning buffer position p, or -1.
__device__ __forceinline__ int lookup(const TileTable& tt, const int64_t* s_off, const int64_t* offset, int64_t p) {
  if (tt.in_lds) {
    int lo = 0, hi = tt.nt;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s_off[mid] <= p) lo = mid + 1;
      else hi = mid;
    }
    return lo - 1;
  }
  const int64_t lo = tt.t0 < 0 ? 0 : tt.t0;
  return (int)(find_tensor_global(offset, lo, tt.t0 + tt.nt, p) - tt.t0);
}

__device__ __forceinline__ int64_t tensor_begin(const TileTable& tt, const int64_t* s_off, const int64_t* offset,
                                                int j) {
  if (tt.in_lds) return s_off[j];
  const int64_t t = tt.t0 + j;
  return t >= 0 ? offset[t] : INT64_MIN;
}

__device__ __forceinline__ int64_t tensor_end(const TileTable& tt, const int64_t* s_end, const int64_t* offset,
                                              const int64_t* numel, int j) {
  if (tt.in_lds) return s_end[j];
  const int64_t t = tt.t0 + j;
  return t >= 0 ? offset[t] + numel[t] : INT64_MIN;
}

template <typename TT, typename TB>
__global__ __launch_bounds__(kBlock) void pack_kernel(const void* const* __restrict__ srcs,
                                                      const int64_t* __restrict__ numel,
                                                      const int64_t* __restrict__ offset, int ntensors, RankPtrs bufs,
                                                      int64_t count, int nranks) {
  constexpr int V = BufVec<TB>::n;
  __shared__ int64_t s_off[kLdsTensors], s_end[kLdsTensors], s_meta[2];
  __shared__ const TT* s_ptr[kLdsTensors];
  const int64_t p0 = (int64_t)blockIdx.x * kTileVecs * V;
  const int64_t p1 = p0 + (int64_t)kTileVecs * V < count ? p0 + (int64_t)kTileVecs * V : count;
  const TileTable tt = stage_tile(offset, numel, ntensors, p0, p1, s_off, s_end, s_meta);

  for (int r = 0; r < nranks; ++r) {
    if (tt.in_lds) {
      for (int j = threadIdx.x; j < tt.nt; j += kBlock) {
        const int64_t t = tt.t0 + j;
        s_ptr[j] = t >= 0 ? static_cast<const TT*>(srcs[(int64_t)r * ntensors + t]) : nullptr;
      }
      __syncthreads();
    }
    TB* __restrict__ buf = static_cast<TB*>(bufs.p[r]);
    for (int u = 0; u < kTileVecs / kBlock; ++u) {
      const int64_t p = p0 + (int64_t)(u * kBlock + threadIdx.x) * V;
      if (p >= p1) break;
      const int j = lookup(tt, s_off, offset, p);
      const int64_t beg = j >= 0 ? tensor_begin(tt, s_off, offset, j) : INT64_MIN;
      const int64_t end = j >= 0 ? tensor_end(tt, s_end, offset, numel, j) : INT64_MIN;
      const TT* src = nullptr;
      if (j >= 0 && tt.t0 + j >= 0)
        src = tt.in_lds ? s_ptr[j] : static_cast<const TT*>(srcs[(int64_t)r * ntensors + tt.t0 + j]);
      if (j >= 0 && p + V <= end && p + V <= count &&
          (reinterpret_cast<uintptr_t>(src + (p - beg)) & 15) == 0) {
        Mover<TT, TB>::to_buf(src + (p - beg), buf + p);
        continue;
      }
      if (j >= 0 && p >= end && p + V <= count) {
        // the whole vector may be padding: check that no later tensor starts inside it
        const int jn = lookup(tt, s_off, offset, p + V - 1);
        if (jn == j) {
          store_zero(buf + p);
          continue;
        }
      }
      for (int k = 0; k < V; ++k) {  // tails, padding, unaligned tensors
        const int64_t pe = p + k;
        if (pe >= count) break;
        const int jk = lookup(tt, s_off, offset, pe);
        TB v = (TB)0;
        if (jk >= 0 && pe < tensor_end(tt, s_end, offset, numel, jk)) {
          const TT* sk = tt.in_lds ? s_ptr[jk] : static_cast<const TT*>(srcs[(int64_t)r * ntensors + tt.t0 + jk]);
          v = Mover<TT, TB>::cvt_in(sk[pe - tensor_begin(tt, s_off, offset, jk)]);
        }
        buf[pe] = v;
      }
    }
    if (tt.in_lds) __syncthreads();  // s_ptr is rewritten for the next rank
  }
}

template <typename TT, typename TB>
__global__ __launch_bounds__(kBlock) void unpack_kernel(RankPtrs bufs, int64_t count, void* const* __restrict__ dsts,
                                                        const int64_t* __restrict__ numel,
                                                        const int64_t* __restrict__ offset, int ntensors,
                                                        int nranks) {
  constexpr int V = BufVec<TB>::n;
  __shared__ int64_t s_off[kLdsTensors], s_end[kLdsTensors], s_meta[2];
  __shared__ TT* s_ptr[kLdsTensors];
  const int64_t p0 = (int64_t)blockIdx.x * kTileVecs * V;
  const int64_t p1 = p0 + (int64_t)kTileVecs * V < count ? p0 + (int64_t)kTileVecs * V : count;
  const TileTable tt = stage_tile(offset, numel, ntensors, p0, p1, s_off, s_end, s_meta);

  for (int r = 0; r < nranks; ++r) {
    if (tt.in_lds) {
      for (int j = threadIdx.x; j < tt.nt; j += kBlock) {
        const int64_t t = tt.t0 + j;
        s_ptr[j] = t >= 0 ? static_cast<TT*>(dsts[(int64_t)r * ntensors + t]) : nullptr;
      }
      __syncthreads();
    }
    const TB* __restrict__ buf = static_cast<const TB*>(bufs.p[r]);
    for (int u = 0; u < kTileVecs / kBlock; ++u) {
      const int64_t p = p0 + (int64_t)(u * kBlock + threadIdx.x) * V;
      if (p >= p1) break;
      const int j = lookup(tt, s_off, offset, p);
      if (j >= 0 && tt.t0 + j >= 0) {
        const int64_t beg = tensor_begin(tt, s_off, offset, j);
        const int64_t end = tensor_end(tt, s_end, offset, numel, j);
        TT* dst = tt.in_lds ? s_ptr[j] : static_cast<TT*>(dsts[(int64_t)r * ntensors + tt.t0 + j]);
        if (p + V <= end && (reinterpret_cast<uintptr_t>(dst + (p - beg)) & 15) == 0) {
          Mover<TT, TB>::from_buf(buf + p, dst + (p - beg));
          continue;
        }
      }
      for (int k = 0; k < V; ++k) {  // tails, padding, unaligned tensors
        const int64_t pe = p + k;
        if (pe >= count) break;
        const int jk = lookup(tt, s_off, offset, pe);
        if (jk >= 0 && pe < tensor_end(tt, s_end, offset, numel, jk)) {
          TT* dk = tt.in_lds ? s_ptr[jk] : static_cast<TT*>(dsts[(int64_t)r * ntensors + tt.t0 + jk]);
          dk[pe - tensor_begin(tt, s_off, offset, jk)] = Mover<TT, TB>::cvt_out(buf[pe]);
        }
      }
    }
    if (tt.in_lds) __syncthreads();
  }
}

unsigned tiles_for(int64_t count, int buf_dtype) {
  const int64_t v = buf_dtype == HVDX_FLOAT32 ? 4 : 8;
  const int64_t per = (int64_t)kTileVecs * v;
  return (unsigned)((count + per - 1) / per);
}

}  // namespace

hipError_t launch_pack(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                       int src_dtype, const RankPtrs& bufs, int64_t count, int buf_dtype, int nranks,
                       hipStream_t stream) {
  const dim3 grid(tiles_for(count, buf_dtype));
  if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    hipLaunchKernelGGL((pack_kernel<float, float>), grid, dim3(kBlock), 0, stream, srcs, numel, offset, ntensors,
                       bufs, count, nranks);
  else if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT16)
    hipLaunchKernelGGL((pack_kernel<float, _Float16>), grid, dim3(kBlock), 0, stream, srcs, numel, offset,
                       ntensors, bufs, count, nranks);
  else
    hipLaunchKernelGGL((pack_kernel<_Float16, _Float16>), grid, dim3(kBlock), 0, stream, srcs, numel, offset,
                       ntensors, bufs, count, nranks);
  return hipGetLastError();
}

hipError_t launch_unpack(const RankPtrs& bufs, int64_t count, int buf_dtype, void* const* dsts,
                         const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                         hipStream_t stream) {
  const dim3 grid(tiles_for(count, buf_dtype));
  if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    hipLaunchKernelGGL((unpack_kernel<float, float>), grid, dim3(kBlock), 0, stream, bufs, count, dsts, numel,
                       offset, ntensors, nranks);
  else if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT16)
    hipLaunchKernelGGL((unpack_kernel<float, _Float16>), grid, dim3(kBlock), 0, stream, bufs, count, dsts, numel,
                       offset, ntensors, nranks);
  else
    hipLaunchKernelGGL((unpack_kernel<_Float16, _Float16>), grid, dim3(kBlock), 0, stream, bufs, count, dsts,
                       numel, offset, ntensors, nranks);
  return hipGetLastError();
}

}  // namespace hvdx
