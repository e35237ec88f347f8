// Ring-allreduce step kernels (paper section 3: N-1 adding steps, then N-1
// replacing steps).  One launch performs one step for all N simulated ranks:
// block row y is chunk c, whose message in adding step s goes from rank (c+s)
// mod N to (c+s+1) mod N and in replacing step s from (c-1+s) mod N to (c+s) mod N.
//
// The work is a memory stream (one add per 12 bytes in binary32), so the kernels
// are shaped for HBM: 16-byte loads and stores, several independent vectors in
// flight per lane, and a grid-stride loop over each chunk.  A vector never
// straddles two chunks: elements before the chunk's first 16-byte boundary and
// after its last one take a scalar path, so any partition of any count works.
//
// Rounding: every addition is the IEEE sum rounded to nearest even in the
// element type (v_add_f32, v_pk_add_f16, with denormals kept); AVERAGE divides the
// finished sum once, by multiplying with 1/N when N is a power of two (exact
// scaling, same result) and by a correctly rounded division otherwise.

#include "internal.hpp"

namespace hvdx {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

template <typename T>
struct Vec;
template <>
struct Vec<float> {
  using type = f32x4;
  static constexpr int n = 4;
};
template <>
struct Vec<_Float16> {
  using type = f16x8;
  static constexpr int n = 8;
};


template <int DIV>
__device__ __forceinline__ float finish(float v, const RingArgs& a) {
  if constexpr (DIV == DIV_POW2) return v * a.inv;
  if constexpr (DIV == DIV_TRUE) return v / a.nf;
  return v;
}

// receiver's value + sender's value, and the AVERAGE divide when DIV says so
template <int DIV>
__device__ __forceinline__ float combine1(float local, float recv, const RingArgs& a) {
  return finish<DIV>(local + recv, a);
}
template <int DIV>
__device__ __forceinline__ _Float16 combine1(_Float16 local, _Float16 recv, const RingArgs& a) {
  _Float16 s = local + recv;
  if constexpr (DIV == DIV_NONE) return s;
  return (_Float16)finish<DIV>((float)s, a);
}
template <int DIV>
__device__ __forceinline__ f32x4 combine(f32x4 local, f32x4 recv, const RingArgs& a) {
  f32x4 s = local + recv;
  if constexpr (DIV != DIV_NONE) {
#pragma unroll
    for (int k = 0; k < 4; ++k) s[k] = finish<DIV>(s[k], a);
  }
  return s;
}
template <int DIV>
__device__ __forceinline__ f16x8 combine(f16x8 local, f16x8 recv, const RingArgs& a) {
  f16x8 s = local + recv;
  if constexpr (DIV != DIV_NONE) {
#pragma unroll
    for (int k = 0; k < 8; ++k) s[k] = (_Float16)finish<DIV>((float)s[k], a);
  }
  return s;
}

struct Chunk {
  int64_t start, len;
};

__device__ __forceinline__ Chunk chunk_of(int c, const RingArgs& a) {
  const int64_t cc = c;
  return {cc * a.q + (cc < a.rem ? cc : a.rem), a.q + (cc < a.rem ? 1 : 0)};
}

// Sender of chunk c in adding step s and in replacing step s (both mod n); the
// receiver is the next rank on the ring.
__device__ __forceinline__ int rs_sender(int c, int s, int n) { return (c + s) % n; }
__device__ __forceinline__ int ag_sender(int c, int s, int n) { return (c + s + n - 1) % n; }

// Elements [0, head) of a chunk precede its first 16-byte boundary.
template <typename T>
__device__ __forceinline__ int64_t head_elems(const void* p, int64_t len) {
  const uintptr_t mis = reinterpret_cast<uintptr_t>(p) & 15;
  const int64_t h = mis ? (int64_t)((16 - mis) / sizeof(T)) : 0;
  return h < len ? h : len;
}

// ---- launch policies ---------------------------------------------------------------
//
// Two shapes, chosen by the size of one rank buffer.  Measured on MI355X: when a
// step's working set (about 3x a rank buffer) fits the 256 MB Infinity Cache the
// best reduce-scatter keeps loads cached and streams its stores non-temporally
// (the next step re-reads what this one wrote from the cache), and the best
// all-gather is plain with two vectors per lane; when it does not fit, one vector
// per lane with every access non-temporal streams closest to the HBM limit.
template <int U_, int BS_, bool NTL_, bool NTS_>
struct Policy {
  static constexpr int U = U_;      // 16-byte vectors per lane and stream
  static constexpr int BS = BS_;    // threads per block
  static constexpr bool NTL = NTL_; // non-temporal loads
  static constexpr bool NTS = NTS_; // non-temporal stores
};
using RsCached = Policy<4, 256, false, true>;
using RsStream = Policy<1, 256, true, true>;
using AgCached = Policy<2, 512, false, false>;
using AgStream = Policy<1, 256, true, true>;
using C16Cached = Policy<2, 256, false, false>;
using C16Stream = Policy<1, 256, true, true>;
constexpr int64_t kStreamBytes = 128ll << 20;  // rank buffers at least this large stream

template <bool NT, typename V>
__device__ __forceinline__ V vload(const V* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  return *p;
}
template <bool NT, typename V>
__device__ __forceinline__ void vstore(V* p, V v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// ---- plain ring (buffers of type T) ---------------------------------------------------

template <typename T, int DIV, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_step_kernel(RankPtrs bufs, RingArgs a) {
  using VT = typename Vec<T>::type;
  constexpr int V = Vec<T>::n;
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = rs_sender(c, a.step, a.n);
  const int rcv = (snd + 1) % a.n;
  const T* __restrict__ src = static_cast<const T*>(bufs.p[snd]) + ch.start;
  T* __restrict__ dst = static_cast<T*>(bufs.p[rcv]) + ch.start;

  const int64_t head = VEC_OK ? head_elems<T>(dst, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / V;
  const int64_t tail = head + nvec * V;
  const int64_t gtid = (int64_t)blockIdx.x * BS + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * BS;
  for (int64_t e = gtid; e < head; e += gthreads) dst[e] = combine1<DIV>(dst[e], src[e], a);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) dst[e] = combine1<DIV>(dst[e], src[e], a);

  const VT* __restrict__ s4 = reinterpret_cast<const VT*>(src + head);
  VT* __restrict__ d4 = reinterpret_cast<VT*>(dst + head);
  for (int64_t base = (int64_t)blockIdx.x * BS * U + threadIdx.x; base < nvec; base += gthreads * U) {
    VT x[U], y[U];
    if (base + (U - 1) * BS < nvec) {  // whole tile: all loads in flight at once
#pragma unroll
      for (int u = 0; u < U; ++u) {
        x[u] = vload<P::NTL>(s4 + base + u * BS);
        y[u] = vload<P::NTL>(d4 + base + u * BS);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) vstore<P::NTS>(d4 + base + u * BS, combine<DIV>(y[u], x[u], a));
      continue;
    }
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + u * BS;
      if (i < nvec) d4[i] = combine<DIV>(d4[i], s4[i], a);
    }
  }
}

template <typename T, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void ag_step_kernel(RankPtrs bufs, RingArgs a) {
  using VT = typename Vec<T>::type;
  constexpr int V = Vec<T>::n;
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = ag_sender(c, a.step, a.n);
  const int rcv = (snd + 1) % a.n;
  const T* __restrict__ src = static_cast<const T*>(bufs.p[snd]) + ch.start;
  T* __restrict__ dst = static_cast<T*>(bufs.p[rcv]) + ch.start;

  const int64_t head = VEC_OK ? head_elems<T>(dst, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / V;
  const int64_t tail = head + nvec * V;
  const int64_t gtid = (int64_t)blockIdx.x * BS + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * BS;
  for (int64_t e = gtid; e < head; e += gthreads) dst[e] = src[e];
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) dst[e] = src[e];

  const VT* __restrict__ s4 = reinterpret_cast<const VT*>(src + head);
  VT* __restrict__ d4 = reinterpret_cast<VT*>(dst + head);
  for (int64_t base = (int64_t)blockIdx.x * BS * U + threadIdx.x; base < nvec; base += gthreads * U) {
    VT x[U];
    if (base + (U - 1) * BS < nvec) {
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = vload<P::NTL>(s4 + base + u * BS);
#pragma unroll
      for (int u = 0; u < U; ++u) vstore<P::NTS>(d4 + base + u * BS, x[u]);
      continue;
    }
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + u * BS;
      if (i < nvec) d4[i] = s4[i];
    }
  }
}

// ---- compressed ring: binary32 buffers, binary16 on the wire ------------------------
//
// Rank r's binary16 wire copy lives at wire + r * wire_stride.  In adding step s the
// receiver rounds its own binary32 value to binary16 and adds the sender's binary16
// partial (at s = 0 the sender's own value, rounded on first touch); the sum goes to
// the receiver's wire copy.  In replacing step s the receiver takes the sender's wire
// value and stores it widened into its binary32 buffer (and on its wire, unless
// nobody forwards it again); at s = 0 the owner also widens its own result.

__device__ __forceinline__ f16x8 to_f16x8(f32x4 lo, f32x4 hi) {
  f16x8 h;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    h[k] = (_Float16)lo[k];
    h[k + 4] = (_Float16)hi[k];
  }
  return h;
}

__device__ __forceinline__ void from_f16x8(f16x8 h, f32x4& lo, f32x4& hi) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    lo[k] = (float)h[k];
    hi[k] = (float)h[k + 4];
  }
}

template <int DIV, bool FIRST, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_step_c16_kernel(RankPtrs x, _Float16* wire, RingArgs a) {
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = rs_sender(c, a.step, a.n);
  const int rcv = (snd + 1) % a.n;
  const float* __restrict__ xs = static_cast<const float*>(x.p[snd]) + ch.start;
  const float* __restrict__ xr = static_cast<const float*>(x.p[rcv]) + ch.start;
  const _Float16* __restrict__ ws = wire + (int64_t)snd * a.wire_stride + ch.start;
  _Float16* __restrict__ wr = wire + (int64_t)rcv * a.wire_stride + ch.start;

  const int64_t head = VEC_OK ? head_elems<_Float16>(wr, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / 8;
  const int64_t tail = head + nvec * 8;
  const int64_t gtid = (int64_t)blockIdx.x * BS + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * BS;
  auto one = [&](int64_t e) {
    const _Float16 sent = FIRST ? (_Float16)xs[e] : ws[e];
    wr[e] = combine1<DIV>((_Float16)xr[e], sent, a);
  };
  for (int64_t e = gtid; e < head; e += gthreads) one(e);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) one(e);

  const f32x4* __restrict__ xs4 = reinterpret_cast<const f32x4*>(xs + head);
  const f32x4* __restrict__ xr4 = reinterpret_cast<const f32x4*>(xr + head);
  const f16x8* __restrict__ ws8 = reinterpret_cast<const f16x8*>(ws + head);
  f16x8* __restrict__ wr8 = reinterpret_cast<f16x8*>(wr + head);
  for (int64_t base = (int64_t)blockIdx.x * BS * U + threadIdx.x; base < nvec; base += gthreads * U) {
    f16x8 sent[U], mine[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + u * BS;
      if (i < nvec) {
        mine[u] = to_f16x8(vload<P::NTL>(xr4 + 2 * i), vload<P::NTL>(xr4 + 2 * i + 1));
        sent[u] = FIRST ? to_f16x8(vload<P::NTL>(xs4 + 2 * i), vload<P::NTL>(xs4 + 2 * i + 1))
                        : vload<P::NTL>(ws8 + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + u * BS;
      if (i < nvec) vstore<P::NTS>(wr8 + i, combine<DIV>(mine[u], sent[u], a));
    }
  }
}

template <bool FIRST, bool LAST, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void ag_step_c16_kernel(RankPtrs x, _Float16* wire, RingArgs a) {
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = ag_sender(c, a.step, a.n);
  const int rcv = (snd + 1) % a.n;
  float* __restrict__ xs = static_cast<float*>(x.p[snd]) + ch.start;
  float* __restrict__ xr = static_cast<float*>(x.p[rcv]) + ch.start;
  const _Float16* __restrict__ ws = wire + (int64_t)snd * a.wire_stride + ch.start;
  _Float16* __restrict__ wr = wire + (int64_t)rcv * a.wire_stride + ch.start;

  const int64_t head = VEC_OK ? head_elems<_Float16>(wr, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / 8;
  const int64_t tail = head + nvec * 8;
  const int64_t gtid = (int64_t)blockIdx.x * BS + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * BS;
  auto one = [&](int64_t e) {
    const _Float16 h = ws[e];
    const float f = (float)h;
    if (FIRST) xs[e] = f;
    xr[e] = f;
    if (!LAST) wr[e] = h;
  };
  for (int64_t e = gtid; e < head; e += gthreads) one(e);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) one(e);

  f32x4* __restrict__ xs4 = reinterpret_cast<f32x4*>(xs + head);
  f32x4* __restrict__ xr4 = reinterpret_cast<f32x4*>(xr + head);
  const f16x8* __restrict__ ws8 = reinterpret_cast<const f16x8*>(ws + head);
  f16x8* __restrict__ wr8 = reinterpret_cast<f16x8*>(wr + head);
  for (int64_t base = (int64_t)blockIdx.x * BS * U + threadIdx.x; base < nvec; base += gthreads * U) {
    f16x8 h[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + u * BS;
      if (i < nvec) h[u] = vload<P::NTL>(ws8 + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + u * BS;
      if (i < nvec) {
        f32x4 lo, hi;
        from_f16x8(h[u], lo, hi);
        if (FIRST) {
          vstore<P::NTS>(xs4 + 2 * i, lo);
          vstore<P::NTS>(xs4 + 2 * i + 1, hi);
        }
        vstore<P::NTS>(xr4 + 2 * i, lo);
        vstore<P::NTS>(xr4 + 2 * i + 1, hi);
        if (!LAST) vstore<P::NTS>(wr8 + i, h[u]);
      }
    }
  }
}

// One rank, compressed: the result is the value rounded to binary16 and widened.
__global__ __launch_bounds__(kBlock) void roundtrip_c16_kernel(float* x, int64_t count) {
  const int64_t gthreads = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < count; e += gthreads)
    x[e] = (float)(_Float16)x[e];
}

// ---- grid sizing and dispatch --------------------------------------------------------

// Blocks per chunk: enough for one pass over the longest chunk, at least 1.
dim3 step_grid(const RingArgs& a, int elems_per_vec, int unroll, int bs) {
  const int64_t longest = a.q + (a.rem ? 1 : 0);
  const int64_t vecs = longest / elems_per_vec + 2;
  int64_t bx = (vecs + (int64_t)bs * unroll - 1) / ((int64_t)bs * unroll);
  if (bx < 1) bx = 1;
  if (bx > (1 << 20)) bx = 1 << 20;
  return dim3((unsigned)bx, (unsigned)a.n, 1);
}

bool streams(const RingArgs& a, int esize) { return (a.q + 1) * a.n * (int64_t)esize >= kStreamBytes; }

template <typename T, typename P>
void rs_launch(const RankPtrs& bufs, const RingArgs& a, int divmode, bool vec_ok, hipStream_t st) {
  const dim3 grid = step_grid(a, Vec<T>::n, P::U, P::BS);
#define HVDX_RS(DIV, VOK) hipLaunchKernelGGL((rs_step_kernel<T, DIV, VOK, P>), grid, dim3(P::BS), 0, st, bufs, a)
  if (vec_ok) {
    if (divmode == DIV_NONE) HVDX_RS(DIV_NONE, true);
    else if (divmode == DIV_POW2) HVDX_RS(DIV_POW2, true);
    else HVDX_RS(DIV_TRUE, true);
  } else {
    if (divmode == DIV_NONE) HVDX_RS(DIV_NONE, false);
    else if (divmode == DIV_POW2) HVDX_RS(DIV_POW2, false);
    else HVDX_RS(DIV_TRUE, false);
  }
#undef HVDX_RS
}

template <typename T>
hipError_t rs_dispatch(const RankPtrs& bufs, const RingArgs& a, int divmode, bool vec_ok, hipStream_t st) {
  if (streams(a, sizeof(T))) rs_launch<T, RsStream>(bufs, a, divmode, vec_ok, st);
  else rs_launch<T, RsCached>(bufs, a, divmode, vec_ok, st);
  return hipGetLastError();
}

template <typename T, typename P>
void ag_launch(const RankPtrs& bufs, const RingArgs& a, bool vec_ok, hipStream_t st) {
  const dim3 grid = step_grid(a, Vec<T>::n, P::U, P::BS);
  if (vec_ok)
    hipLaunchKernelGGL((ag_step_kernel<T, true, P>), grid, dim3(P::BS), 0, st, bufs, a);
  else
    hipLaunchKernelGGL((ag_step_kernel<T, false, P>), grid, dim3(P::BS), 0, st, bufs, a);
}

template <typename T>
hipError_t ag_dispatch(const RankPtrs& bufs, const RingArgs& a, bool vec_ok, hipStream_t st) {
  if (streams(a, sizeof(T))) ag_launch<T, AgStream>(bufs, a, vec_ok, st);
  else ag_launch<T, AgCached>(bufs, a, vec_ok, st);
  return hipGetLastError();
}

template <typename P>
void rs_c16_launch(const RankPtrs& x, _Float16* w, const RingArgs& a, int divmode, bool vector_ok,
                   hipStream_t stream) {
  const dim3 grid = step_grid(a, 8, P::U, P::BS);
  const bool first = a.step == 0;
#define HVDX_RSC(DIV, F, VOK) \
  hipLaunchKernelGGL((rs_step_c16_kernel<DIV, F, VOK, P>), grid, dim3(P::BS), 0, stream, x, w, a)
#define HVDX_RSC_V(DIV, F) \
  if (vector_ok) HVDX_RSC(DIV, F, true); else HVDX_RSC(DIV, F, false)
#define HVDX_RSC_F(DIV) \
  if (first) { HVDX_RSC_V(DIV, true); } else { HVDX_RSC_V(DIV, false); }
  if (divmode == DIV_NONE) {
    HVDX_RSC_F(DIV_NONE)
  } else if (divmode == DIV_POW2) {
    HVDX_RSC_F(DIV_POW2)
  } else {
    HVDX_RSC_F(DIV_TRUE)
  }
#undef HVDX_RSC_F
#undef HVDX_RSC_V
#undef HVDX_RSC
}

template <typename P>
void ag_c16_launch(const RankPtrs& x, _Float16* w, const RingArgs& a, bool vector_ok, hipStream_t stream) {
  const dim3 grid = step_grid(a, 8, P::U, P::BS);
  const bool first = a.step == 0, last = a.step == a.n - 2;
#define HVDX_AGC(F, L, VOK) \
  hipLaunchKernelGGL((ag_step_c16_kernel<F, L, VOK, P>), grid, dim3(P::BS), 0, stream, x, w, a)
#define HVDX_AGC_V(F, L) \
  if (vector_ok) HVDX_AGC(F, L, true); else HVDX_AGC(F, L, false)
  if (first && last) {
    HVDX_AGC_V(true, true);
  } else if (first) {
    HVDX_AGC_V(true, false);
  } else if (last) {
    HVDX_AGC_V(false, true);
  } else {
    HVDX_AGC_V(false, false);
  }
#undef HVDX_AGC_V
#undef HVDX_AGC
}

}  // namespace

hipError_t launch_rs_step(const RankPtrs& bufs, const RingArgs& a, int dtype, int divmode, bool vector_ok,
                          hipStream_t stream) {
  return dtype == HVDX_FLOAT32 ? rs_dispatch<float>(bufs, a, divmode, vector_ok, stream)
                               : rs_dispatch<_Float16>(bufs, a, divmode, vector_ok, stream);
}

hipError_t launch_ag_step(const RankPtrs& bufs, const RingArgs& a, int dtype, bool vector_ok, hipStream_t stream) {
  return dtype == HVDX_FLOAT32 ? ag_dispatch<float>(bufs, a, vector_ok, stream)
                               : ag_dispatch<_Float16>(bufs, a, vector_ok, stream);
}

hipError_t launch_rs_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, int divmode, bool vector_ok,
                              hipStream_t stream) {
  _Float16* w = static_cast<_Float16*>(wire);
  if (streams(a, 4)) rs_c16_launch<C16Stream>(x, w, a, divmode, vector_ok, stream);
  else rs_c16_launch<C16Cached>(x, w, a, divmode, vector_ok, stream);
  return hipGetLastError();
}

hipError_t launch_ag_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, bool vector_ok, hipStream_t stream) {
  _Float16* w = static_cast<_Float16*>(wire);
  if (streams(a, 4)) ag_c16_launch<C16Stream>(x, w, a, vector_ok, stream);
  else ag_c16_launch<C16Cached>(x, w, a, vector_ok, stream);
  return hipGetLastError();
}

hipError_t launch_roundtrip_c16(void* x, int64_t count, hipStream_t stream) {
  int64_t blocks = (count + kBlock * 4 - 1) / (kBlock * 4);
  if (blocks < 1) blocks = 1;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(roundtrip_c16_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, static_cast<float*>(x),
                     count);
  return hipGetLastError();
}

}  // namespace hvdx
