// Device helpers shared by the ring and the copy kernels: vector types, the ring's
// partition and schedule (paper section 3), and its arithmetic (the adding step's
// sum, the AVERAGE divide).  Internal to the library.
#pragma once

#include "internal.hpp"

namespace hvdx {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

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

// binary16 finish: scaling by 1/N = 2^-k is done in binary16 itself (one rounding of
// the exact product, the same bits as through binary32); going through binary32
// lets the compiler select v_fma_mix with a +0 addend, which turns -0 into +0.
template <int DIV>
__device__ __forceinline__ _Float16 finish16(_Float16 v, const RingArgs& a) {
  if constexpr (DIV == DIV_POW2) return v * (_Float16)a.inv;
  if constexpr (DIV == DIV_TRUE) return (_Float16)((float)v / a.nf);
  return v;
}

// receiver's value + sender's value, and the AVERAGE divide when DIV says so
template <int DIV>
__device__ __forceinline__ float combine1(float local, float recv, const RingArgs& a) {
  return finish<DIV>(local + recv, a);
}
template <int DIV>
__device__ __forceinline__ _Float16 combine1(_Float16 local, _Float16 recv, const RingArgs& a) {
  return finish16<DIV>(local + recv, a);
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
  if constexpr (DIV == DIV_POW2) s = s * (f16x8)((_Float16)a.inv);
  if constexpr (DIV == DIV_TRUE) {
#pragma unroll
    for (int k = 0; k < 8; ++k) s[k] = finish16<DIV>(s[k], a);
  }
  return s;
}

template <int DIV>
__device__ __forceinline__ f16x4 combine(f16x4 local, f16x4 recv, const RingArgs& a) {
  f16x4 s = local + recv;
  if constexpr (DIV == DIV_POW2) s = s * (f16x4)((_Float16)a.inv);
  if constexpr (DIV == DIV_TRUE) {
#pragma unroll
    for (int k = 0; k < 4; ++k) s[k] = finish16<DIV>(s[k], a);
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

// Index of the chunk holding element e.
__device__ __forceinline__ int64_t chunk_index(int64_t e, const RingArgs& a) {
  const int64_t big = a.rem * (a.q + 1);  // elements in the first rem (longer) chunks
  return e < big ? e / (a.q + 1) : a.rem + (e - big) / a.q;
}

// The adding step's result for a scalar or a 16-byte vector (receiver's value first).
template <int DIV>
__device__ __forceinline__ float add_step(float local, float recv, const RingArgs& a) {
  return combine1<DIV>(local, recv, a);
}
template <int DIV>
__device__ __forceinline__ _Float16 add_step(_Float16 local, _Float16 recv, const RingArgs& a) {
  return combine1<DIV>(local, recv, a);
}
template <int DIV>
__device__ __forceinline__ f32x4 add_step(f32x4 local, f32x4 recv, const RingArgs& a) {
  return combine<DIV>(local, recv, a);
}
template <int DIV>
__device__ __forceinline__ f16x8 add_step(f16x8 local, f16x8 recv, const RingArgs& a) {
  return combine<DIV>(local, recv, a);
}
template <int DIV>
__device__ __forceinline__ f16x4 add_step(f16x4 local, f16x4 recv, const RingArgs& a) {
  return combine<DIV>(local, recv, a);
}

// The whole ring for the elements at e (one T, or one 16-byte vector A of them, all in
// chunk c), in the ring's order: adding steps 0..N-2, then replacing steps 0..N-2, each
// reading the sender's buffer and writing the receiver's.  Elements never meet other
// elements on the ring, so one thread can run an element's steps back to back.
template <typename T, typename A, int DIV>
__device__ __forceinline__ void ring_chain(const RankPtrs& bufs, int64_t e, int c, const RingArgs& a) {
  auto at = [&](int r) { return reinterpret_cast<A*>(static_cast<T*>(bufs.p[r]) + e); };
  const int n = a.n;
  int snd = c;  // adding step s: chunk c goes from rank c+s to c+s+1
  for (int s = 0; s < n - 1; ++s) {
    const int rcv = snd + 1 == n ? 0 : snd + 1;
    const A x = *at(snd);
    A* pr = at(rcv);
    *pr = s == n - 2 ? add_step<DIV>(*pr, x, a) : add_step<DIV_NONE>(*pr, x, a);
    snd = rcv;
  }
  for (int s = 0; s < n - 1; ++s) {  // snd is the owner, c-1; replacing step s: c-1+s to c+s
    const int rcv = snd + 1 == n ? 0 : snd + 1;
    *at(rcv) = *at(snd);
    snd = rcv;
  }
}

}  // namespace
}  // namespace hvdx
