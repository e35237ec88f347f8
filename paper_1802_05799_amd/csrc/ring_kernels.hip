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

#include "ring_math.hpp"

namespace hvdx {
namespace {

// ---- launch policies ---------------------------------------------------------------
//
// Two shapes, chosen by the size of one rank buffer.  Measured on MI355X: when a
// step's working set (about 3x a rank buffer) fits the 256 MB Infinity Cache the
// best reduce-scatter keeps loads cached and streams its stores non-temporally
// (the next step re-reads what this one wrote from the cache), and the best
// all-gather is plain with two vectors per lane; when it does not fit, one vector
// per lane with every access non-temporal, in 64-thread blocks, streams closest to
// the HBM limit.  The
// fused step N-2/0 (two reads, two writes) does best with one vector per lane in
// both regimes.  Each shape can be replaced at build time (-DHVDX_RS_CACHED=...).
template <int U_, int BS_, bool NTL_, bool NTS_, bool WAVE_ = false>
struct Policy {
  static constexpr int U = U_;      // 16-byte vectors per lane and stream
  static constexpr int BS = BS_;    // threads per block
  static constexpr bool NTL = NTL_; // non-temporal loads
  static constexpr bool NTS = NTS_; // non-temporal stores
  static constexpr bool WAVE = WAVE_;  // a wavefront's U vectors are contiguous (else block-strided)
};
#ifndef HVDX_RS_CACHED
#define HVDX_RS_CACHED Policy<2, 256, false, true>
#endif
#ifndef HVDX_RS_STREAM  // 64-thread blocks: 78% -> 82% of peak on VGG-16's fc6 against 256
#define HVDX_RS_STREAM Policy<1, 64, true, true>
#endif
#ifndef HVDX_AG_CACHED
#define HVDX_AG_CACHED Policy<2, 512, false, false>
#endif
#ifndef HVDX_AG_STREAM  // 64-thread blocks: 76.5% -> 77.7% (binary32), 78% -> 80% (compressed ring)
#define HVDX_AG_STREAM Policy<1, 64, true, true>
#endif
// Replacing step N-3 is the last one launched on its own before the fused copy-out,
// which reads what it writes.  With cached stores its dirty lines were written back
// while the copy-out streamed (77.5% of peak for the copy-out against 79% with this
// step's stores streamed): streaming them took 0.5-0.7% off the ResNet-50 step, the
// other workloads unchanged.  On the earlier replacing steps streamed stores lose
// more than that, since the next step re-reads their output from the caches.
#ifndef HVDX_AG_LAST_CACHED
#define HVDX_AG_LAST_CACHED Policy<2, 512, false, true>
#endif
#ifndef HVDX_RSAG_CACHED  // two reads and two writes per vector: one vector per lane measured best
#define HVDX_RSAG_CACHED Policy<1, 256, false, true>
#endif
#ifndef HVDX_RSAG_STREAM  // cached stores: replacing step 1 reads rank c's copy (VGG-16's fc6: 80% -> 84%)
#define HVDX_RSAG_STREAM Policy<1, 64, true, false>
#endif
#ifndef HVDX_C16_CACHED
#define HVDX_C16_CACHED Policy<2, 256, false, false>
#endif
#ifndef HVDX_RS16_CACHED  // binary16 buffers (more elements per vector, shorter chunks)
#define HVDX_RS16_CACHED HVDX_RS_CACHED
#endif
#ifndef HVDX_AG16_CACHED
#define HVDX_AG16_CACHED HVDX_AG_CACHED
#endif
using RsCached = HVDX_RS_CACHED;
using Rs16Cached = HVDX_RS16_CACHED;
using Ag16Cached = HVDX_AG16_CACHED;
using RsStream = HVDX_RS_STREAM;
using AgCached = HVDX_AG_CACHED;
using AgStream = HVDX_AG_STREAM;
using AgLastCached = HVDX_AG_LAST_CACHED;
using RsAgCached = HVDX_RSAG_CACHED;
using RsAgStream = HVDX_RSAG_STREAM;
using C16Cached = HVDX_C16_CACHED;
#ifndef HVDX_C16_RS_STREAM
#define HVDX_C16_RS_STREAM Policy<1, 64, true, true>
#endif
#ifndef HVDX_C16_AG_STREAM  // replacing step 0 writes 4x what it reads: cached stores measured faster
#define HVDX_C16_AG_STREAM Policy<2, 256, false, false>
#endif
#ifndef HVDX_C16_RSAG_STREAM  // cached stores, as for the binary32 fused step (VGG-16 fp16's fc6: 81.5% -> 84.5%)
#define HVDX_C16_RSAG_STREAM Policy<1, 64, true, false>
#endif
using C16RsStream = HVDX_C16_RS_STREAM;
using C16RsAgStream = HVDX_C16_RSAG_STREAM;
using C16AgStream = HVDX_C16_AG_STREAM;
constexpr int64_t kStreamBytes = 128ll << 20;  // rank buffers at least this large stream

// Vector u of this lane in a block's span of BS*U vectors starting at blk.
template <typename P>
__device__ __forceinline__ int64_t lane_vec(int64_t blk, int u) {
  if constexpr (P::WAVE) return blk + (int64_t)(threadIdx.x >> 6) * 64 * P::U + u * 64 + (threadIdx.x & 63);
  return blk + (int64_t)u * P::BS + threadIdx.x;
}

// The cached (working set fits the Infinity Cache) shapes per buffer type.
template <typename T>
struct CachedShape {
  using rs = RsCached;
  using ag = AgCached;
};
template <>
struct CachedShape<_Float16> {
  using rs = Rs16Cached;
  using ag = Ag16Cached;
};

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
__device__ __forceinline__ void rs_step_body(const RankPtrs& bufs, const RingArgs& a, int64_t bx, int64_t gx) {
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
  const int64_t gtid = bx * BS + threadIdx.x;
  const int64_t gthreads = gx * BS;
  for (int64_t e = gtid; e < head; e += gthreads) dst[e] = combine1<DIV>(dst[e], src[e], a);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) dst[e] = combine1<DIV>(dst[e], src[e], a);

  const VT* __restrict__ s4 = reinterpret_cast<const VT*>(src + head);
  VT* __restrict__ d4 = reinterpret_cast<VT*>(dst + head);
  for (int64_t blk = bx * BS * U; blk < nvec; blk += gthreads * U) {
    VT x[U], y[U];
    if (blk + BS * U <= nvec) {  // whole tile: all loads in flight at once
#pragma unroll
      for (int u = 0; u < U; ++u) {
        x[u] = vload<P::NTL>(s4 + lane_vec<P>(blk, u));
        y[u] = vload<P::NTL>(d4 + lane_vec<P>(blk, u));
      }
#pragma unroll
      for (int u = 0; u < U; ++u) vstore<P::NTS>(d4 + lane_vec<P>(blk, u), combine<DIV>(y[u], x[u], a));
      continue;
    }
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) d4[i] = combine<DIV>(d4[i], s4[i], a);
    }
  }
}

template <typename T, int DIV, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_step_kernel(RankPtrs bufs, RingArgs a) {
  rs_step_body<T, DIV, VEC_OK, P>(bufs, a, blockIdx.x, gridDim.x);
}

// The same step of two rings (two fusion buffers) in one launch: block columns
// [0, x0) serve ring 0 as its own grid would, columns [x0, gridDim.x) ring 1.
template <typename T, int DIV, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_step_pair_kernel(RingPair m, int x0) {
  const int z = (int)blockIdx.x >= x0 ? 1 : 0;
  rs_step_body<T, DIV, VEC_OK, P>(m.bufs[z], m.a[z], z ? (int64_t)blockIdx.x - x0 : (int64_t)blockIdx.x,
      z ? (int64_t)gridDim.x - x0 : (int64_t)x0);
}

template <typename T, bool VEC_OK, typename P>
__device__ __forceinline__ void ag_step_body(const RankPtrs& bufs, const RingArgs& a, int64_t bx, int64_t gx) {
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
  const int64_t gtid = bx * BS + threadIdx.x;
  const int64_t gthreads = gx * BS;
  for (int64_t e = gtid; e < head; e += gthreads) dst[e] = src[e];
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) dst[e] = src[e];

  const VT* __restrict__ s4 = reinterpret_cast<const VT*>(src + head);
  VT* __restrict__ d4 = reinterpret_cast<VT*>(dst + head);
  for (int64_t blk = bx * BS * U; blk < nvec; blk += gthreads * U) {
    VT x[U];
    if (blk + BS * U <= nvec) {
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = vload<P::NTL>(s4 + lane_vec<P>(blk, u));
#pragma unroll
      for (int u = 0; u < U; ++u) vstore<P::NTS>(d4 + lane_vec<P>(blk, u), x[u]);
      continue;
    }
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) d4[i] = s4[i];
    }
  }
}

template <typename T, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void ag_step_kernel(RankPtrs bufs, RingArgs a) {
  ag_step_body<T, VEC_OK, P>(bufs, a, blockIdx.x, gridDim.x);
}

// The same step of two rings (two fusion buffers) in one launch: block columns
// [0, x0) serve ring 0 as its own grid would, columns [x0, gridDim.x) ring 1.
template <typename T, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void ag_step_pair_kernel(RingPair m, int x0) {
  const int z = (int)blockIdx.x >= x0 ? 1 : 0;
  ag_step_body<T, VEC_OK, P>(m.bufs[z], m.a[z], z ? (int64_t)blockIdx.x - x0 : (int64_t)blockIdx.x,
      z ? (int64_t)gridDim.x - x0 : (int64_t)x0);
}

// ---- compressed ring: binary32 buffers, binary16 on the wire ------------------------
//
// Rank r's binary16 wire copy lives at wire + r * wire_stride.  In adding step s the
// receiver rounds its own binary32 value to binary16 and adds the sender's binary16
// partial (at s = 0 the sender's own value, rounded on first touch); the sum goes to
// the receiver's wire copy.  Replacing step 0 widens the owner's binary16 result into
// its own and the receiver's binary32 buffers; every later replacing step forwards a
// binary16 number already held exactly in binary32, so it is the plain binary32 copy.

__device__ __forceinline__ f16x8 to_f16x8(f32x4 lo, f32x4 hi) {
  f16x8 h;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    h[k] = (_Float16)lo[k];
    h[k + 4] = (_Float16)hi[k];
  }
  return h;
}

__device__ __forceinline__ f16x4 narrow4(f32x4 x) {
  f16x4 h;
#pragma unroll
  for (int k = 0; k < 4; ++k) h[k] = (_Float16)x[k];
  return h;
}

__device__ __forceinline__ f32x4 widen4(f16x4 h) {
  f32x4 x;
#pragma unroll
  for (int k = 0; k < 4; ++k) x[k] = (float)h[k];
  return x;
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
  for (int64_t blk = (int64_t)blockIdx.x * BS * U; blk < nvec; blk += gthreads * U) {
    f16x8 sent[U], mine[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) {
        mine[u] = to_f16x8(vload<P::NTL>(xr4 + 2 * i), vload<P::NTL>(xr4 + 2 * i + 1));
        sent[u] = FIRST ? to_f16x8(vload<P::NTL>(xs4 + 2 * i), vload<P::NTL>(xs4 + 2 * i + 1))
                        : vload<P::NTL>(ws8 + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) vstore<P::NTS>(wr8 + i, combine<DIV>(mine[u], sent[u], a));
    }
  }
}

// Replacing step 0: the owner (c-1) of chunk c widens its binary16 result into its
// own binary32 buffer and into rank c's.  The later replacing steps forward values
// that are binary16 numbers held exactly in binary32, so they are plain binary32
// copies (ag_step_kernel<float>): the same bits as narrowing, sending and widening
// again, moved 4 bytes in and 4 out per element.
template <bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void ag_first_c16_kernel(RankPtrs x, const _Float16* wire, RingArgs a) {
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = ag_sender(c, 0, a.n);
  const int rcv = (snd + 1) % a.n;
  float* __restrict__ xs = static_cast<float*>(x.p[snd]) + ch.start;
  float* __restrict__ xr = static_cast<float*>(x.p[rcv]) + ch.start;
  const _Float16* __restrict__ ws = wire + (int64_t)snd * a.wire_stride + ch.start;

  // four elements per lane: 16-byte binary32 stores, 8-byte binary16 loads, each
  // contiguous across the wavefront (the binary32 side fixes the alignment)
  const int64_t head = VEC_OK ? head_elems<float>(xs, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / 4;
  const int64_t tail = head + nvec * 4;
  const int64_t gtid = (int64_t)blockIdx.x * BS + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * BS;
  auto one = [&](int64_t e) {
    const float f = (float)ws[e];
    xs[e] = f;
    xr[e] = f;
  };
  for (int64_t e = gtid; e < head; e += gthreads) one(e);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) one(e);

  f32x4* __restrict__ xs4 = reinterpret_cast<f32x4*>(xs + head);
  f32x4* __restrict__ xr4 = reinterpret_cast<f32x4*>(xr + head);
  const f16x4* __restrict__ ws4 = reinterpret_cast<const f16x4*>(ws + head);
  for (int64_t blk = (int64_t)blockIdx.x * BS * U; blk < nvec; blk += gthreads * U) {
    f16x4 h[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) h[u] = vload<P::NTL>(ws4 + i);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) {
        const f32x4 f = widen4(h[u]);
        vstore<P::NTS>(xs4 + i, f);
        vstore<P::NTS>(xr4 + i, f);
      }
    }
  }
}

// ---- the last adding step fused with the first replacing step -----------------------
//
// In adding step N-2 the owner (c-1) of chunk c completes its sum from the sender
// (c-2); in replacing step 0 the owner sends it on to rank c.  One kernel does both:
// it writes the finished (averaged) chunk to the owner and to rank c, which saves
// reading it back.  The buffers end exactly as after the two steps.

template <typename T, int DIV, bool VEC_OK, typename P>
__device__ __forceinline__ void rs_ag_step_body(const RankPtrs& bufs, const RingArgs& a, int64_t bx, int64_t gx) {
  using VT = typename Vec<T>::type;
  constexpr int V = Vec<T>::n;
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = rs_sender(c, a.n - 2, a.n);
  const int own = (snd + 1) % a.n;
  // with N = 2 the sender is rank c itself, so src and nxt alias (each element is
  // read before the same lane writes it): no __restrict__ on them
  const T* src = static_cast<const T*>(bufs.p[snd]) + ch.start;
  T* __restrict__ dst = static_cast<T*>(bufs.p[own]) + ch.start;
  T* nxt = static_cast<T*>(bufs.p[c]) + ch.start;

  const int64_t head = VEC_OK ? head_elems<T>(dst, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / V;
  const int64_t tail = head + nvec * V;
  const int64_t gtid = bx * BS + threadIdx.x;
  const int64_t gthreads = gx * BS;
  auto one = [&](int64_t e) {
    const T v = combine1<DIV>(dst[e], src[e], a);
    dst[e] = v;
    nxt[e] = v;
  };
  for (int64_t e = gtid; e < head; e += gthreads) one(e);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) one(e);

  const VT* s4 = reinterpret_cast<const VT*>(src + head);
  VT* __restrict__ d4 = reinterpret_cast<VT*>(dst + head);
  VT* n4 = reinterpret_cast<VT*>(nxt + head);
  for (int64_t blk = bx * BS * U; blk < nvec; blk += gthreads * U) {
    VT x[U], y[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) {
        x[u] = vload<P::NTL>(s4 + i);
        y[u] = vload<P::NTL>(d4 + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) {
        const VT v = combine<DIV>(y[u], x[u], a);
        vstore<P::NTS>(d4 + i, v);
        vstore<P::NTS>(n4 + i, v);
      }
    }
  }
}

template <typename T, int DIV, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_ag_step_kernel(RankPtrs bufs, RingArgs a) {
  rs_ag_step_body<T, DIV, VEC_OK, P>(bufs, a, blockIdx.x, gridDim.x);
}

// The same step of two rings (two fusion buffers) in one launch: block columns
// [0, x0) serve ring 0 as its own grid would, columns [x0, gridDim.x) ring 1.
template <typename T, int DIV, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_ag_step_pair_kernel(RingPair m, int x0) {
  const int z = (int)blockIdx.x >= x0 ? 1 : 0;
  rs_ag_step_body<T, DIV, VEC_OK, P>(m.bufs[z], m.a[z], z ? (int64_t)blockIdx.x - x0 : (int64_t)blockIdx.x,
      z ? (int64_t)gridDim.x - x0 : (int64_t)x0);
}

// Compressed: the finished binary16 sum goes, widened, to the owner's and rank c's
// binary32 buffers; no wire copy is written (the replacing steps forward binary32).
template <int DIV, bool FIRST, bool VEC_OK, typename P>
__global__ __launch_bounds__(P::BS) void rs_ag_step_c16_kernel(RankPtrs x, const _Float16* wire, RingArgs a) {
  constexpr int BS = P::BS, U = P::U;
  const int c = blockIdx.y;
  const Chunk ch = chunk_of(c, a);
  const int snd = rs_sender(c, a.n - 2, a.n);
  const int own = (snd + 1) % a.n;
  // with N = 2 the sender is rank c itself: xs/xn and ws/wn alias (read before written)
  const float* xs = static_cast<const float*>(x.p[snd]) + ch.start;
  float* __restrict__ xo = static_cast<float*>(x.p[own]) + ch.start;
  float* xn = static_cast<float*>(x.p[c]) + ch.start;
  const _Float16* ws = wire + (int64_t)snd * a.wire_stride + ch.start;

  // four elements per lane, so that the binary32 loads and both binary32 stores are
  // 16 bytes per lane and contiguous across the wavefront
  const int64_t head = VEC_OK ? head_elems<float>(xo, ch.len) : ch.len;
  const int64_t nvec = (ch.len - head) / 4;
  const int64_t tail = head + nvec * 4;
  const int64_t gtid = (int64_t)blockIdx.x * BS + threadIdx.x;
  const int64_t gthreads = (int64_t)gridDim.x * BS;
  auto one = [&](int64_t e) {
    const _Float16 sent = FIRST ? (_Float16)xs[e] : ws[e];
    const float f = (float)combine1<DIV>((_Float16)xo[e], sent, a);
    xo[e] = f;
    xn[e] = f;
  };
  for (int64_t e = gtid; e < head; e += gthreads) one(e);
  for (int64_t e = tail + gtid; e < ch.len; e += gthreads) one(e);

  const f32x4* xs4 = reinterpret_cast<const f32x4*>(xs + head);
  f32x4* __restrict__ xo4 = reinterpret_cast<f32x4*>(xo + head);
  f32x4* xn4 = reinterpret_cast<f32x4*>(xn + head);
  const f16x4* ws4 = reinterpret_cast<const f16x4*>(ws + head);
  for (int64_t blk = (int64_t)blockIdx.x * BS * U; blk < nvec; blk += gthreads * U) {
    f16x4 sent[U], mine[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) {
        mine[u] = narrow4(vload<P::NTL>(xo4 + i));
        sent[u] = FIRST ? narrow4(vload<P::NTL>(xs4 + i)) : vload<P::NTL>(ws4 + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = lane_vec<P>(blk, u);
      if (i < nvec) {
        const f32x4 f = widen4(combine<DIV>(mine[u], sent[u], a));
        vstore<P::NTS>(xo4 + i, f);
        vstore<P::NTS>(xn4 + i, f);
      }
    }
  }
}

// ---- the ring's fold computed directly -----------------------------------------------
//
// Element e of chunk c ends as FIN(((x_c + x_{c+1}) + ...) + x_{c+N-1}) on every rank,
// the ring's summation order.  One kernel reads the N values of each element once,
// adds them in that order in registers (binary16 after rounding each input when
// compressing) and writes the result to all N ranks: 2N element reads and writes
// instead of the ring's 5(N-1), with identical bits, but without the per-step
// messages of a real ring.


template <typename T, bool COMP>
struct FoldTypes;
template <>
struct FoldTypes<float, false> {
  using acc = float;
  __device__ static float in(float v) { return v; }
  __device__ static float out(float v) { return v; }
};
template <>
struct FoldTypes<_Float16, false> {
  using acc = _Float16;
  __device__ static _Float16 in(_Float16 v) { return v; }
  __device__ static _Float16 out(_Float16 v) { return v; }
};
template <>
struct FoldTypes<float, true> {  // binary32 data, binary16 arithmetic
  using acc = _Float16;
  __device__ static _Float16 in(float v) { return (_Float16)v; }
  __device__ static float out(_Float16 v) { return (float)v; }
};

constexpr int kFoldBatch = 8;  // ranks whose loads are in flight together

// Four elements as one access: 16 bytes of binary32, 8 of binary16.
template <typename T>
struct Four;
template <>
struct Four<float> {
  using type = f32x4;
};
template <>
struct Four<_Float16> {
  using type = f16x4;
};

template <int DIV>
__device__ __forceinline__ float fold_finish(float v, const RingArgs& a) {
  return finish<DIV>(v, a);
}
template <int DIV>
__device__ __forceinline__ _Float16 fold_finish(_Float16 v, const RingArgs& a) {
  return finish16<DIV>(v, a);
}

template <typename T, int DIV, bool COMP, bool VEC_OK>
__global__ __launch_bounds__(kBlock) void fold_kernel(RankPtrs bufs, RingArgs a, int64_t count) {
  using F = FoldTypes<T, COMP>;
  using A = typename F::acc;
  constexpr int V = 4;  // elements per lane (16 bytes of binary32, 8 of binary16)
  const int64_t nv = (count + V - 1) / V;
  const int n = a.n;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nv; i += (int64_t)gridDim.x * kBlock) {
    const int64_t e0 = i * V;
    const int64_t c0 = chunk_index(e0, a);
    const bool whole = VEC_OK && e0 + V <= count && chunk_index(e0 + V - 1, a) == c0;
    if (whole) {  // one aligned 4-element access per rank, contiguous across the wavefront
      using VT = typename Four<T>::type;
      A acc[V];
      VT v[kFoldBatch];
      for (int k0 = 0; k0 < n; k0 += kFoldBatch) {
#pragma unroll
        for (int kk = 0; kk < kFoldBatch; ++kk) {
          const int k = k0 + kk;
          if (k < n)
            v[kk] = *reinterpret_cast<const VT*>(static_cast<const T*>(bufs.p[(c0 + k) % n]) + e0);
        }
#pragma unroll
        for (int kk = 0; kk < kFoldBatch; ++kk) {
          const int k = k0 + kk;
          if (k < n) {
#pragma unroll
            for (int j = 0; j < V; ++j) acc[j] = k == 0 ? F::in(v[kk][j]) : (A)(acc[j] + F::in(v[kk][j]));
          }
        }
      }
      VT out;
#pragma unroll
      for (int j = 0; j < V; ++j) out[j] = F::out(fold_finish<DIV>(acc[j], a));
      for (int r = 0; r < n; ++r)
        *reinterpret_cast<VT*>(static_cast<T*>(bufs.p[r]) + e0) = out;
      continue;
    }
    for (int64_t e = e0; e < e0 + V && e < count; ++e) {  // vectors that cross a chunk edge
      const int64_t c = chunk_index(e, a);
      A acc = F::in(static_cast<const T*>(bufs.p[c])[e]);
      for (int k = 1; k < n; ++k) acc = (A)(acc + F::in(static_cast<const T*>(bufs.p[(c + k) % n])[e]));
      acc = fold_finish<DIV>(acc, a);
      for (int r = 0; r < n; ++r) static_cast<T*>(bufs.p[r])[e] = F::out(acc);
    }
  }
}

// ---- a small ring in one launch ----------------------------------------------------
//
// For buffers so small that each step's launch costs more than its messages: one
// thread runs all 2(N-1) steps for one 16-byte vector (or, where a vector crosses a
// chunk edge or the buffers are not 16-byte aligned, for each of its elements), each
// step still reading the sender's buffer and writing the receiver's in memory.

template <typename T, int DIV, bool VEC_OK>
__global__ __launch_bounds__(kBlock) void chain_kernel(RankPtrs bufs, RingArgs a, int64_t count) {
  using VT = typename Vec<T>::type;
  constexpr int V = Vec<T>::n;
  const int64_t nv = (count + V - 1) / V;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < nv; i += (int64_t)gridDim.x * kBlock) {
    const int64_t e0 = i * V;
    const int64_t c0 = chunk_index(e0, a);
    if (VEC_OK && e0 + V <= count && chunk_index(e0 + V - 1, a) == c0) {
      ring_chain<T, VT, DIV>(bufs, e0, (int)c0, a);
      continue;
    }
    for (int64_t e = e0; e < e0 + V && e < count; ++e) ring_chain<T, T, DIV>(bufs, e, (int)chunk_index(e, a), a);
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
#define HVDX_RS(DIV, VOK) HVDX_LAUNCH((rs_step_kernel<T, DIV, VOK, P>), grid, dim3(P::BS), 0, st, bufs, a)
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
  else rs_launch<T, typename CachedShape<T>::rs>(bufs, a, divmode, vec_ok, st);
  return hipGetLastError();
}

template <typename T, typename P>
void ag_launch(const RankPtrs& bufs, const RingArgs& a, bool vec_ok, hipStream_t st) {
  const dim3 grid = step_grid(a, Vec<T>::n, P::U, P::BS);
  if (vec_ok)
    HVDX_LAUNCH((ag_step_kernel<T, true, P>), grid, dim3(P::BS), 0, st, bufs, a);
  else
    HVDX_LAUNCH((ag_step_kernel<T, false, P>), grid, dim3(P::BS), 0, st, bufs, a);
}

template <typename T>
hipError_t ag_dispatch(const RankPtrs& bufs, const RingArgs& a, bool vec_ok, hipStream_t st) {
  if (streams(a, sizeof(T))) ag_launch<T, AgStream>(bufs, a, vec_ok, st);
  else if (a.step == a.n - 3) ag_launch<T, AgLastCached>(bufs, a, vec_ok, st);
  else ag_launch<T, typename CachedShape<T>::ag>(bufs, a, vec_ok, st);
  return hipGetLastError();
}

template <typename P>
void rs_c16_launch(const RankPtrs& x, _Float16* w, const RingArgs& a, int divmode, bool vector_ok,
                   hipStream_t stream) {
  const dim3 grid = step_grid(a, 8, P::U, P::BS);
  const bool first = a.step == 0;
#define HVDX_RSC(DIV, F, VOK) \
  HVDX_LAUNCH((rs_step_c16_kernel<DIV, F, VOK, P>), grid, dim3(P::BS), 0, stream, x, w, a)
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
void ag_first_c16_launch(const RankPtrs& x, const _Float16* w, const RingArgs& a, bool vector_ok, hipStream_t stream) {
  const dim3 grid = step_grid(a, 4, P::U, P::BS);
  if (vector_ok) HVDX_LAUNCH((ag_first_c16_kernel<true, P>), grid, dim3(P::BS), 0, stream, x, w, a);
  else HVDX_LAUNCH((ag_first_c16_kernel<false, P>), grid, dim3(P::BS), 0, stream, x, w, a);
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

namespace {

// Two rings in one launch: ring 0's columns of blocks (each column one row per chunk),
// then ring 1's, each ring with as many columns as its own step needs, so no block is
// launched without work; *x0 is the first column of ring 1.
dim3 pair_grid(const RingPair& m, int elems_per_vec, int unroll, int bs, int* x0) {
  const dim3 g0 = step_grid(m.a[0], elems_per_vec, unroll, bs), g1 = step_grid(m.a[1], elems_per_vec, unroll, bs);
  *x0 = (int)g0.x;
  return dim3(g0.x + g1.x, (unsigned)m.a[0].n, 1);
}

// Both rings take the launch shape of the longer one.
bool pair_streams(const RingPair& m, int esize) { return streams(m.a[0].q >= m.a[1].q ? m.a[0] : m.a[1], esize); }

template <typename T, typename P>
void rs_pair_launch(const RingPair& m, int divmode, hipStream_t st) {
  int x0;
  const dim3 grid = pair_grid(m, Vec<T>::n, P::U, P::BS, &x0);
  if (divmode == DIV_NONE)
    HVDX_LAUNCH((rs_step_pair_kernel<T, DIV_NONE, true, P>), grid, dim3(P::BS), 0, st, m, x0);
  else if (divmode == DIV_POW2)
    HVDX_LAUNCH((rs_step_pair_kernel<T, DIV_POW2, true, P>), grid, dim3(P::BS), 0, st, m, x0);
  else HVDX_LAUNCH((rs_step_pair_kernel<T, DIV_TRUE, true, P>), grid, dim3(P::BS), 0, st, m, x0);
}

template <typename T, typename P>
void rs_ag_pair_launch(const RingPair& m, int divmode, hipStream_t st) {
  int x0;
  const dim3 grid = pair_grid(m, Vec<T>::n, P::U, P::BS, &x0);
  if (divmode == DIV_NONE)
    HVDX_LAUNCH((rs_ag_step_pair_kernel<T, DIV_NONE, true, P>), grid, dim3(P::BS), 0, st, m, x0);
  else if (divmode == DIV_POW2)
    HVDX_LAUNCH((rs_ag_step_pair_kernel<T, DIV_POW2, true, P>), grid, dim3(P::BS), 0, st, m, x0);
  else HVDX_LAUNCH((rs_ag_step_pair_kernel<T, DIV_TRUE, true, P>), grid, dim3(P::BS), 0, st, m, x0);
}

template <typename T, typename P>
void ag_pair_launch(const RingPair& m, hipStream_t st) {
  int x0;
  const dim3 grid = pair_grid(m, Vec<T>::n, P::U, P::BS, &x0);
  HVDX_LAUNCH((ag_step_pair_kernel<T, true, P>), grid, dim3(P::BS), 0, st, m, x0);
}

template <typename T>
hipError_t rs_pair_dispatch(const RingPair& m, int divmode, hipStream_t st) {
  if (pair_streams(m, sizeof(T))) rs_pair_launch<T, RsStream>(m, divmode, st);
  else rs_pair_launch<T, typename CachedShape<T>::rs>(m, divmode, st);
  return hipGetLastError();
}

template <typename T>
hipError_t rs_ag_pair_dispatch(const RingPair& m, int divmode, hipStream_t st) {
  if (pair_streams(m, sizeof(T))) rs_ag_pair_launch<T, RsAgStream>(m, divmode, st);
  else rs_ag_pair_launch<T, RsAgCached>(m, divmode, st);
  return hipGetLastError();
}

template <typename T>
hipError_t ag_pair_dispatch(const RingPair& m, hipStream_t st) {
  if (pair_streams(m, sizeof(T))) ag_pair_launch<T, AgStream>(m, st);
  else if (m.a[0].step == m.a[0].n - 3) ag_pair_launch<T, AgLastCached>(m, st);
  else ag_pair_launch<T, typename CachedShape<T>::ag>(m, st);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rs_step_pair(const RingPair& m, int dtype, int divmode, hipStream_t stream) {
  return dtype == HVDX_FLOAT32 ? rs_pair_dispatch<float>(m, divmode, stream)
                               : rs_pair_dispatch<_Float16>(m, divmode, stream);
}

hipError_t launch_rs_ag_step_pair(const RingPair& m, int dtype, int divmode, hipStream_t stream) {
  return dtype == HVDX_FLOAT32 ? rs_ag_pair_dispatch<float>(m, divmode, stream)
                               : rs_ag_pair_dispatch<_Float16>(m, divmode, stream);
}

hipError_t launch_ag_step_pair(const RingPair& m, int dtype, hipStream_t stream) {
  return dtype == HVDX_FLOAT32 ? ag_pair_dispatch<float>(m, stream) : ag_pair_dispatch<_Float16>(m, stream);
}

hipError_t launch_rs_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, int divmode, bool vector_ok,
                              hipStream_t stream) {
  _Float16* w = static_cast<_Float16*>(wire);
  if (streams(a, 4)) rs_c16_launch<C16RsStream>(x, w, a, divmode, vector_ok, stream);
  else rs_c16_launch<C16Cached>(x, w, a, divmode, vector_ok, stream);
  return hipGetLastError();
}

hipError_t launch_ag_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, bool vector_ok, hipStream_t stream) {
  if (a.step > 0) return ag_dispatch<float>(x, a, vector_ok, stream);  // binary16 values held in binary32
  const _Float16* w = static_cast<const _Float16*>(wire);
  if (streams(a, 4)) ag_first_c16_launch<C16AgStream>(x, w, a, vector_ok, stream);
  else ag_first_c16_launch<C16Cached>(x, w, a, vector_ok, stream);
  return hipGetLastError();
}

hipError_t launch_roundtrip_c16(void* x, int64_t count, hipStream_t stream) {
  int64_t blocks = (count + kBlock * 4 - 1) / (kBlock * 4);
  if (blocks < 1) blocks = 1;
  if (blocks > 65536) blocks = 65536;
  HVDX_LAUNCH(roundtrip_c16_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, static_cast<float*>(x),
                     count);
  return hipGetLastError();
}

hipError_t launch_rs_ag_step(const RankPtrs& bufs, const RingArgs& a, int dtype, int divmode, bool vector_ok,
                             hipStream_t stream) {
#define HVDX_RSAG(T, P, DIV, VOK) \
  HVDX_LAUNCH((rs_ag_step_kernel<T, DIV, VOK, P>), step_grid(a, Vec<T>::n, P::U, P::BS), dim3(P::BS), 0, \
                     stream, bufs, a)
#define HVDX_RSAG_V(T, P, DIV) \
  if (vector_ok) HVDX_RSAG(T, P, DIV, true); else HVDX_RSAG(T, P, DIV, false)
#define HVDX_RSAG_D(T, P) \
  if (divmode == DIV_NONE) { HVDX_RSAG_V(T, P, DIV_NONE); } \
  else if (divmode == DIV_POW2) { HVDX_RSAG_V(T, P, DIV_POW2); } \
  else { HVDX_RSAG_V(T, P, DIV_TRUE); }
  if (dtype == HVDX_FLOAT32) {
    if (streams(a, 4)) { HVDX_RSAG_D(float, RsAgStream) } else { HVDX_RSAG_D(float, RsAgCached) }
  } else {
    if (streams(a, 2)) { HVDX_RSAG_D(_Float16, RsAgStream) } else { HVDX_RSAG_D(_Float16, RsAgCached) }
  }
#undef HVDX_RSAG_D
#undef HVDX_RSAG_V
#undef HVDX_RSAG
  return hipGetLastError();
}

namespace {
template <typename P>
void rs_ag_c16_launch(const RankPtrs& x, _Float16* w, const RingArgs& a, int divmode, bool vector_ok,
                      hipStream_t stream) {
  const dim3 grid = step_grid(a, 4, P::U, P::BS);
  const bool first = a.n == 2;  // step N-2 is also the first adding step when N = 2
#define HVDX_RAC(DIV, F, VOK) \
  HVDX_LAUNCH((rs_ag_step_c16_kernel<DIV, F, VOK, P>), grid, dim3(P::BS), 0, stream, x, w, a)
#define HVDX_RAC_V(DIV, F) \
  if (vector_ok) HVDX_RAC(DIV, F, true); else HVDX_RAC(DIV, F, false)
#define HVDX_RAC_D(F) \
  if (divmode == DIV_NONE) { HVDX_RAC_V(DIV_NONE, F); } \
  else if (divmode == DIV_POW2) { HVDX_RAC_V(DIV_POW2, F); } \
  else { HVDX_RAC_V(DIV_TRUE, F); }
  if (first) {
    HVDX_RAC_D(true)
  } else {
    HVDX_RAC_D(false)
  }
#undef HVDX_RAC_D
#undef HVDX_RAC_V
#undef HVDX_RAC
}
}  // namespace

hipError_t launch_rs_ag_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, int divmode, bool vector_ok,
                                 hipStream_t stream) {
  _Float16* w = static_cast<_Float16*>(wire);
  if (streams(a, 4)) rs_ag_c16_launch<C16RsAgStream>(x, w, a, divmode, vector_ok, stream);
  else rs_ag_c16_launch<C16Cached>(x, w, a, divmode, vector_ok, stream);
  return hipGetLastError();
}

hipError_t launch_chain(const RankPtrs& bufs, const RingArgs& a, int64_t count, int dtype, int divmode,
                        bool vector_ok, hipStream_t stream) {
  const int64_t v = dtype == HVDX_FLOAT32 ? 4 : 8;
  int64_t blocks = ((count + v - 1) / v + kBlock - 1) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > 65536) blocks = 65536;
  const dim3 grid((unsigned)blocks), block(kBlock);
#define HVDX_CHAIN(T, DIV) \
  if (vector_ok) HVDX_LAUNCH((chain_kernel<T, DIV, true>), grid, block, 0, stream, bufs, a, count); \
  else HVDX_LAUNCH((chain_kernel<T, DIV, false>), grid, block, 0, stream, bufs, a, count)
#define HVDX_CHAIN_D(T) \
  if (divmode == DIV_NONE) { HVDX_CHAIN(T, DIV_NONE); } \
  else if (divmode == DIV_POW2) { HVDX_CHAIN(T, DIV_POW2); } \
  else { HVDX_CHAIN(T, DIV_TRUE); }
  if (dtype == HVDX_FLOAT32) {
    HVDX_CHAIN_D(float)
  } else {
    HVDX_CHAIN_D(_Float16)
  }
#undef HVDX_CHAIN_D
#undef HVDX_CHAIN
  return hipGetLastError();
}

hipError_t launch_fold(const RankPtrs& bufs, const RingArgs& a, int64_t count, int dtype, int compress, int divmode,
                       bool vector_ok, hipStream_t stream) {
  int64_t blocks = (count / 4 + kBlock) / kBlock;
  if (blocks < 1) blocks = 1;
  if (blocks > (1 << 20)) blocks = 1 << 20;
  const dim3 grid((unsigned)blocks), block(kBlock);
#define HVDX_FOLD(T, C, DIV) \
  if (vector_ok) HVDX_LAUNCH((fold_kernel<T, DIV, C, true>), grid, block, 0, stream, bufs, a, count); \
  else HVDX_LAUNCH((fold_kernel<T, DIV, C, false>), grid, block, 0, stream, bufs, a, count)
#define HVDX_FOLD_D(T, C) \
  if (divmode == DIV_NONE) { HVDX_FOLD(T, C, DIV_NONE); } \
  else if (divmode == DIV_POW2) { HVDX_FOLD(T, C, DIV_POW2); } \
  else { HVDX_FOLD(T, C, DIV_TRUE); }
  if (compress == HVDX_COMPRESS_FP16) {
    HVDX_FOLD_D(float, true)
  } else if (dtype == HVDX_FLOAT32) {
    HVDX_FOLD_D(float, false)
  } else {
    HVDX_FOLD_D(_Float16, false)
  }
#undef HVDX_FOLD_D
#undef HVDX_FOLD
  return hipGetLastError();
}

}  // namespace hvdx
