// Tensor Fusion copy-in and copy-out kernels (paper section 7, steps 3 and 5), and the
// ring steps of a fusion buffer run on the ranks' tensors (further below).
//
// The iteration space is the fusion buffer, not the tensor list: block x owns one
// tile of buffer positions and serves it for every rank.  Each lane handles one
// 16-byte vector of the buffer, so load balance does not depend on how ragged the
// tensors are (Inception-V3 mixes 32-element batch-norm vectors with 2M-element
// weights).  A block finds the tensors that overlap its tile once, stages their
// offsets and ends in LDS, together with the tensor pointers of the ranks it
// serves, and reuses them for all of those ranks.  A lane binary-searches the LDS table for its
// vector's tensor.  Vectors entirely inside one tensor with a 16-byte aligned
// source take the vector path; tensor tails, padding and unaligned tensors take a
// per-element path.  Padding is written as zero by the copy-in and skipped by the
// copy-out.

#include "ring_math.hpp"

namespace hvdx {
namespace {


// Shape of a copy kernel: POS buffer vectors per lane in a row (a row is BS*POS
// vectors for BS threads per block), SUB rows per block (one tensor lookup serves them all), RB ranks whose
// loads are in flight together, RPB ranks per block (0 = all), non-temporal
// loads/stores, and the lane layout.  Measured on MI355X with the workloads' buckets:
// a block's prologue (two rounds of dependent loads to find its tensors) has to be
// amortized over enough data, yet a plain copy streams fastest with only one or two
// 16-byte loads in flight per lane (83% of peak against 78% with four).  The
// copy-out serves two ranks per block one after the other, two block-strided
// vectors per lane, in 256-thread blocks, and loads the first rank's vectors before
// the tensor lookup: against both ranks' four loads at once in 512-thread blocks it
// went from 75% to 78% of peak on ResNet-50's buffers (71% to 75% on Inception-V3's,
// 68% to 74% on VGG-16's; each step 1% faster); without the early loads this shape
// was no better.  The copy-in's loads need the lookup first; it is best with both
// ranks' two vectors per lane in flight at once (one vector per lane lost 8 points;
// four ranks per block in two batches lost 0.8% of the ResNet-50 step once tiles
// inside one tensor skip the per-vector classification).  One rank per block with
// one vector per lane (the best pattern for a plain copy between many buffers) lost
// to the prologue even with 8 rows; more rows or wavefront-contiguous lanes did not
// help either.
#ifndef HVDX_LDS_TENSORS
#define HVDX_LDS_TENSORS 64
#endif
template <int POS_, int RB_, int RPB_, bool NTL_, bool NTS_, bool WAVE_ = false, int SUB_ = 1, int BS_ = kBlock>
struct CopyCfg {
  static_assert(BS_ >= 128 && BS_ % 64 == 0, "the tile lookup takes two wavefronts");
  static constexpr int BS = BS_;  // threads per block
  static constexpr int POS = POS_, RB = RB_, RPB = RPB_;
  static constexpr bool NTL = NTL_, NTS = NTS_;
  static constexpr bool WAVE = WAVE_;  // a wavefront's POS vectors are contiguous (else block-strided)
  static constexpr int SUB = SUB_;     // rows of BS*POS vectors a block moves one after another
  static constexpr int kRowVecs = BS_ * POS_;
  static constexpr int kTileVecs = kRowVecs * SUB_;  // a block's tile: one tensor lookup serves all its rows
  // A tile's tensors staged in LDS; a tile that spans more looks its tensors up in
  // global memory instead.
  static constexpr int kLdsTensors = kTileVecs + 8 < HVDX_LDS_TENSORS ? kTileVecs + 8 : HVDX_LDS_TENSORS;
};
#ifndef HVDX_PACK_CFG
#define HVDX_PACK_CFG CopyCfg<2, 2, 2, true, true>
#endif
#ifndef HVDX_UNPACK_CFG
#define HVDX_UNPACK_CFG CopyCfg<2, 1, 2, true, true>
#endif
#ifndef HVDX_PACK16_CFG
#define HVDX_PACK16_CFG CopyCfg<2, 2, 2, true, true>
#endif
#ifndef HVDX_UNPACK16_CFG
#define HVDX_UNPACK16_CFG CopyCfg<2, 1, 2, true, true>
#endif
using PackCfg = HVDX_PACK_CFG;      // binary32 buffers
using UnpackCfg = HVDX_UNPACK_CFG;
using Pack16Cfg = HVDX_PACK16_CFG;  // binary16 buffers
using Unpack16Cfg = HVDX_UNPACK16_CFG;
#ifndef HVDX_UNPACK_EARLY  // copy-out: buffer loads issued before the tensor lookup
#define HVDX_UNPACK_EARLY 1
#endif
#ifndef HVDX_COPY_ATTR
#define HVDX_COPY_ATTR
#endif
#ifndef HVDX_LDS_PTRS
#define HVDX_LDS_PTRS 256
#endif
constexpr int kLdsPtrs = HVDX_LDS_PTRS;  // (rank, tensor) pointers a tile can stage in LDS

// Vector u of this lane within its block's tile.
template <typename Cfg>
__device__ __forceinline__ int tile_vec(int u) {
  if constexpr (Cfg::WAVE) return (threadIdx.x >> 6) * 64 * Cfg::POS + u * 64 + (threadIdx.x & 63);
  return u * Cfg::BS + threadIdx.x;
}

// Elements a lane moves as one vector: 16 bytes on the wider side, so that every load
// and store instruction of a wavefront covers one contiguous run of memory (binary32
// tensors with a binary16 buffer: 16-byte tensor vectors, 8-byte buffer vectors).
template <typename TT, typename TB>
struct BufVec {
  static constexpr int n = 16 / (sizeof(TT) > sizeof(TB) ? sizeof(TT) : sizeof(TB));
};

// Host side: the same count from the data types.
inline int64_t vec_elems(int tensor_dtype, int buf_dtype) {
  return tensor_dtype == HVDX_FLOAT32 || buf_dtype == HVDX_FLOAT32 ? 4 : 8;
}

// Convert and move BufVec<TT, TB>::n elements between a tensor of type TT and the
// buffer of type TB (TT == TB, or TT = float and TB = _Float16).
template <typename TT, typename TB>
struct Mover;

__device__ __forceinline__ bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// 16-byte loads and stores of the copy kernels, with optional non-temporal hints
template <bool NT, typename V>
__device__ __forceinline__ V ld16(const V* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  return *p;
}
template <bool NT, typename V>
__device__ __forceinline__ void st16(V* p, V v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

template <>
struct Mover<float, float> {
  using buf_vec = f32x4;
  // 4 tensor elements -> one buffer vector (tensor side may be unaligned, unless the
  // caller has checked it: ALIGNED)
  template <bool NT, bool ALIGNED = false>
  __device__ static f32x4 load(const float* src) {
    if (ALIGNED || aligned16(src)) return ld16<NT>(reinterpret_cast<const f32x4*>(src));
    return f32x4{src[0], src[1], src[2], src[3]};
  }
  template <bool NT, bool ALIGNED = false>
  __device__ static void store(float* dst, f32x4 v) {
    if (ALIGNED || aligned16(dst)) {
      st16<NT>(reinterpret_cast<f32x4*>(dst), v);
      return;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) dst[k] = v[k];
  }
  __device__ static float cvt_in(float v) { return v; }
  __device__ static float cvt_out(float v) { return v; }
};

template <>
struct Mover<_Float16, _Float16> {
  using buf_vec = f16x8;
  template <bool NT, bool ALIGNED = false>
  __device__ static f16x8 load(const _Float16* src) {
    if (ALIGNED || aligned16(src)) return ld16<NT>(reinterpret_cast<const f16x8*>(src));
    f16x8 h;
#pragma unroll
    for (int k = 0; k < 8; ++k) h[k] = src[k];
    return h;
  }
  template <bool NT, bool ALIGNED = false>
  __device__ static void store(_Float16* dst, f16x8 v) {
    if (ALIGNED || aligned16(dst)) {
      st16<NT>(reinterpret_cast<f16x8*>(dst), v);
      return;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) dst[k] = v[k];
  }
  __device__ static _Float16 cvt_in(_Float16 v) { return v; }
  __device__ static _Float16 cvt_out(_Float16 v) { return v; }
};

template <>
struct Mover<float, _Float16> {  // tensor binary32 (16-byte vectors), buffer binary16 (8-byte vectors)
  using buf_vec = f16x4;
  template <bool NT, bool ALIGNED = false>
  __device__ static f16x4 load(const float* src) {
    const f32x4 x = ALIGNED || aligned16(src) ? ld16<NT>(reinterpret_cast<const f32x4*>(src))
                                   : f32x4{src[0], src[1], src[2], src[3]};
    f16x4 h;
#pragma unroll
    for (int k = 0; k < 4; ++k) h[k] = (_Float16)x[k];
    return h;
  }
  template <bool NT, bool ALIGNED = false>
  __device__ static void store(float* dst, f16x4 h) {
    f32x4 x;
#pragma unroll
    for (int k = 0; k < 4; ++k) x[k] = (float)h[k];
    if (ALIGNED || aligned16(dst)) {
      st16<NT>(reinterpret_cast<f32x4*>(dst), x);
      return;
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) dst[k] = x[k];
  }
  __device__ static _Float16 cvt_in(float v) { return (_Float16)v; }
  __device__ static float cvt_out(_Float16 v) { return (float)v; }
};

// Zero one buffer vector (padding).
template <typename VB, typename TB>
__device__ __forceinline__ void store_zero(TB* p) {
  *reinterpret_cast<VB*>(p) = (VB)((TB)0);
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

// Last tensor t in [lo, hi) with offset[t] <= p, or lo - 1 if none, found by one
// 64-lane wavefront: each round the lanes probe 64 evenly spaced offsets and a ballot
// narrows the range 64-fold (two rounds cover 4096 tensors).  Every lane of the
// calling wavefront must take part; all get the answer.
__device__ int64_t find_tensor_wave(const int64_t* offset, int64_t lo, int64_t hi, int64_t p) {
  const int lane = threadIdx.x & 63;
  while (lo < hi) {
    const int64_t n = hi - lo;
    const int64_t idx = lo + ((lane + 1) * n + 63) / 64 - 1;  // non-decreasing in lane, last = hi - 1
    const unsigned long long mask = __ballot(offset[idx] <= p);
    const int cnt = __popcll(mask);  // offsets are ascending: the true lanes come first
    if (cnt == 64) {
      lo = hi;
    } else {
      const int64_t stop = lo + ((int64_t)(cnt + 1) * n + 63) / 64 - 1;  // probe of lane cnt: > p
      if (cnt > 0) lo = lo + ((int64_t)cnt * n + 63) / 64;              // one past the probe of lane cnt-1
      hi = stop;
    }
  }
  return lo - 1;
}

// Waves 0 and 1 locate the tile's first and last tensor at the same time; then the
// whole block stages their offsets and ends, and the tile's (rank, tensor) pointers
// of slots [r0, r1) (slot v is rank (v + rot) mod n), in one pass: two rounds of
// global loads per block in all.
template <int LDS_TENSORS>
__device__ TileTable stage_tile(const int64_t* offset, const int64_t* numel, int ntensors, int64_t p0, int64_t p1,
                                const void* const* ptrs, int r0, int r1, int rot, int n, int64_t* s_off,
                                int64_t* s_end, int64_t* s_meta, const void** s_ptr, bool* ptrs_in_lds) {
  const int wave = threadIdx.x >> 6;
  if (wave < 2) {
    const int64_t t = find_tensor_wave(offset, 0, ntensors, wave == 0 ? p0 : p1 - 1);
    if ((threadIdx.x & 63) == 0) s_meta[wave] = t;
  }
  __syncthreads();
  TileTable tt;
  tt.t0 = s_meta[0];
  tt.nt = (int)(s_meta[1] - s_meta[0] + 1);
  tt.in_lds = tt.nt <= LDS_TENSORS;
  const int nr = r1 - r0;
  const bool pin = tt.in_lds && (int64_t)tt.nt * nr <= kLdsPtrs;
  const int work = pin ? tt.nt * nr : (tt.in_lds ? tt.nt : 0);
  for (int idx = threadIdx.x; idx < work; idx += blockDim.x) {
    if (idx < tt.nt) {
      const int64_t t = tt.t0 + idx;
      s_off[idx] = t >= 0 ? offset[t] : INT64_MIN;  // positions before the first tensor are padding
      s_end[idx] = t >= 0 ? offset[t] + numel[t] : INT64_MIN;
    }
    if (pin) {
      const int rr = idx / tt.nt;
      const int64_t t = tt.t0 + (idx - rr * tt.nt);
      const int rank = (r0 + rr + rot) % n;
      s_ptr[idx] = t >= 0 ? ptrs[(int64_t)rank * ntensors + t] : nullptr;
    }
  }
  *ptrs_in_lds = pin;
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

// What one lane does with one 16-byte buffer vector, the same for every rank.
enum PosClass { POS_NONE = 0, POS_VEC = 1, POS_ZERO = 2, POS_EDGE = 3 };

struct Pos {
  int64_t p;    // buffer position of the vector's first element
  int t;        // tensor owning it (POS_VEC); tensor counts are int
  int64_t li;   // index of that element inside the tensor (POS_VEC)
  int cls;
};

// Classify buffer vector [p, p+V): inside one tensor, all padding, or an edge that
// needs the element-by-element path (tensor tails, unaligned tensor offsets).  Only
// positions in [cs, ce) belong to the block: the kernels fused with a ring step work
// on one ring chunk per block, and a vector that reaches outside it takes the
// element path, which skips the positions of the neighbouring chunk.
template <int V>
__device__ __forceinline__ Pos classify(const TileTable& tt, const int64_t* s_off, const int64_t* s_end,
                                        const int64_t* offset, const int64_t* numel, int64_t p, int64_t p1,
                                        int64_t cs, int64_t ce) {
  Pos q{p, -1, 0, POS_NONE};
  if (p >= p1 || p + V <= cs) return q;  // past the tile, or wholly before the block's chunk
  const int j = lookup(tt, s_off, offset, p);
  const int64_t t = tt.t0 + j;
  const int64_t beg = t >= 0 ? tensor_begin(tt, s_off, offset, j) : INT64_MIN;
  const int64_t end = t >= 0 ? tensor_end(tt, s_end, offset, numel, j) : INT64_MIN;
  q.cls = POS_EDGE;
  if (p >= cs && p + V <= ce) {
    if (t >= 0 && p + V <= end) {
      q.cls = POS_VEC;
      q.t = (int)t;
      q.li = p - beg;
    } else if (p >= end && lookup(tt, s_off, offset, p + V - 1) == j) {
      q.cls = POS_ZERO;  // no tensor element anywhere in the vector
    }
  }
  return q;
}

// The ring's chunk partition: chunk c starts at c*q + min(c, rem) and holds q
// elements, one more for the first rem chunks.
__device__ __forceinline__ int64_t chunk_start(int c, int64_t q, int64_t rem) { return c * q + (c < rem ? c : rem); }

// Which buffer positions and ranks a block serves.  Plain copies: grid (tiles, rank
// groups), tile x covers [x*T, x*T + T) of the buffer.  Fused with a ring step: grid
// (tiles per chunk, chunks, rank groups); chunk c's tiles are the buffer's own tiles
// from the one holding its first position on (so every access keeps the alignment
// of the plain copy), and the block serves only [cs, ce) of its tile.
struct BlockSpan {
  int64_t p0, p1, cs, ce;
  int c;  // ring chunk (fused kernels), else 0
  int rbeg, rend;
};

template <bool RING>
__device__ __forceinline__ BlockSpan block_span(int64_t tile_elems, int64_t count, int nranks, int rpb, int64_t q,
                                                int64_t rem, int group, int64_t bx) {
  BlockSpan b;
  if constexpr (RING) {
    b.c = blockIdx.y;
    b.cs = chunk_start(b.c, q, rem);
    b.ce = b.cs + q + (b.c < rem ? 1 : 0);
    b.p0 = (b.cs & ~(tile_elems - 1)) + bx * tile_elems;  // tile_elems is a power of two
    b.p1 = b.p0 + tile_elems < b.ce ? b.p0 + tile_elems : b.ce;
  } else {
    b.c = 0;
    b.cs = 0;
    b.ce = count;
    b.p0 = bx * tile_elems;
    b.p1 = b.p0 + tile_elems < count ? b.p0 + tile_elems : count;
  }
  b.rbeg = group * rpb;
  b.rend = b.rbeg + rpb < nranks ? b.rbeg + rpb : nranks;
  return b;
}

// A tile wholly inside one tensor and, fused with a ring step, one chunk: every
// lane's vectors are whole vectors of that tensor (the common case for large
// tensors), so the copy needs no per-vector classification.  Block-uniform.
template <typename Cfg, int V>
__device__ __forceinline__ bool whole_tile(const TileTable& tt, const BlockSpan& bs, const int64_t* s_off,
                                           const int64_t* s_end, const int64_t* offset, const int64_t* numel) {
  const int64_t end = bs.p0 + (int64_t)Cfg::kTileVecs * V;
  if (Cfg::SUB != 1 || tt.nt != 1 || tt.t0 < 0 || bs.p0 < bs.cs || end > bs.ce) return false;
  return tensor_begin(tt, s_off, offset, 0) <= bs.p0 && end <= tensor_end(tt, s_end, offset, numel, 0);
}

// The tile's (rank, tensor) pointers, staged in LDS when they fit so that the data
// loads do not wait behind dependent pointer loads.  A block serves "slots" [r0, r0+nr);
// slot v is rank (v + rot) mod n (rot = 0 except in the copy-in fused with a ring step).
struct PtrTable {
  const void* const* g;  // rank-major device table
  const void* const* s;  // LDS copy, s[(v - r0) * nt + j], or null
  int64_t t0, ntensors;
  int nt, r0, rot, n;
  __device__ __forceinline__ int rank(int v) const { return v + rot < n ? v + rot : v + rot - n; }
  __device__ __forceinline__ const void* get(int v, int64_t t) const {
    return s ? s[(v - r0) * nt + (int)(t - t0)] : g[(int64_t)rank(v) * ntensors + t];
  }
};

// Copy-in.  With RING it is fused with the ring's first adding step (paper section 3,
// the first round of the ring's adding half): in chunk c the receiving rank c+1
// stores its own value plus rank c's, so the buffers end in the state the copy-in and
// that step leave, without reading the sender's buffer back.
// A block's slots start at its chunk's sender, so slot 0 (sender) and slot 1
// (receiver) are one load batch of the first rank group.
//
// Each row of the tile is moved in two passes: whole vectors (and all-padding ones)
// first, for every rank, then the rare edge vectors element by element.  Keeping the
// element path out of the vector pass keeps the vector pass's registers low enough
// for full occupancy.
template <typename TT, typename TB, typename Cfg, bool RING>
__device__ __forceinline__ void pack_body(const void* const* __restrict__ srcs, const int64_t* __restrict__ numel,
                                          const int64_t* __restrict__ offset, int ntensors, const RankPtrs& bufs,
                                          int64_t count, int nranks, int rpb, int64_t q, int64_t rem, int skip_sender,
                                          int group, int64_t bx) {
  static_assert(!RING || (Cfg::RB >= 2 && (Cfg::RPB == 0 || Cfg::RPB >= 2)),
                "the fused copy-in needs the sender and receiver in one load batch");
  constexpr int V = BufVec<TT, TB>::n;
  using VB = typename Mover<TT, TB>::buf_vec;
  constexpr int kPosPerLane = Cfg::POS, kRankBatch = Cfg::RB, kTileVecs = Cfg::kTileVecs;
  __shared__ int64_t s_off[Cfg::kLdsTensors], s_end[Cfg::kLdsTensors], s_meta[2];
  __shared__ const void* s_ptr[kLdsPtrs];
  static_assert((kTileVecs & (kTileVecs - 1)) == 0, "tiles are a power of two vectors");
  const BlockSpan bs = block_span<RING>((int64_t)kTileVecs * V, count, nranks, rpb, q, rem, group, bx);
  if (bs.p0 >= bs.p1) return;  // past the end of a shorter chunk: the whole block leaves
  const int rot = bs.c;
  bool pin;
  const TileTable tt = stage_tile<Cfg::kLdsTensors>(offset, numel, ntensors, bs.p0, bs.p1, srcs, bs.rbeg, bs.rend,
                                                    rot, nranks, s_off, s_end, s_meta, s_ptr, &pin);
  const PtrTable pt{srcs, pin ? s_ptr : nullptr, tt.t0, ntensors, tt.nt, bs.rbeg, rot, nranks};
  const int receiver = bs.c + 1 == nranks ? 0 : bs.c + 1;  // of chunk c in adding step 0

  if (whole_tile<Cfg, V>(tt, bs, s_off, s_end, offset, numel)) {  // no per-vector classification needed
    const int64_t li0 = bs.p0 - tensor_begin(tt, s_off, offset, 0);
    for (int v0 = bs.rbeg; v0 < bs.rend; v0 += kRankBatch) {
      VB v[kRankBatch][kPosPerLane];
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int slot = v0 + rr;
        if (slot >= bs.rend) continue;
        const TT* src = static_cast<const TT*>(pt.get(slot, tt.t0)) + li0;
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u)
          v[rr][u] = Mover<TT, TB>::template load<Cfg::NTL>(src + tile_vec<Cfg>(u) * V);
      }
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int slot = v0 + rr;
        if (slot >= bs.rend) break;
        if (RING && skip_sender && slot == 0) continue;  // the sender's copy of its own chunk is never read
        TB* __restrict__ buf = static_cast<TB*>(bufs.p[pt.rank(slot)]) + bs.p0;
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u) {
          VB x = v[rr][u];
          if (RING && rr > 0 && slot == 1) x = x + v[rr > 0 ? rr - 1 : 0][u];  // receiver: own + sender's
          st16<Cfg::NTS>(reinterpret_cast<VB*>(buf + tile_vec<Cfg>(u) * V), x);
        }
      }
    }
    return;
  }

  for (int row = 0; row < Cfg::SUB; ++row) {
    const int64_t r0 = bs.p0 + (int64_t)row * Cfg::kRowVecs * V;
    if (r0 >= bs.p1) break;
    Pos pos[kPosPerLane];
    bool edges = false;
#pragma unroll
    for (int u = 0; u < kPosPerLane; ++u) {
      pos[u] = classify<V>(tt, s_off, s_end, offset, numel, r0 + (int64_t)tile_vec<Cfg>(u) * V, bs.p1, bs.cs, bs.ce);
      edges |= pos[u].cls == POS_EDGE;
    }

    for (int v0 = bs.rbeg; v0 < bs.rend; v0 += kRankBatch) {
      VB v[kRankBatch][kPosPerLane];
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int slot = v0 + rr;
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u)
          if (slot < bs.rend && pos[u].cls == POS_VEC)
            v[rr][u] = Mover<TT, TB>::template load<Cfg::NTL>(static_cast<const TT*>(pt.get(slot, pos[u].t)) +
                                                              pos[u].li);
      }
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int slot = v0 + rr;
        if (slot >= bs.rend) break;
        if (RING && skip_sender && slot == 0) continue;  // the sender's copy of its own chunk is never read
        TB* __restrict__ buf = static_cast<TB*>(bufs.p[pt.rank(slot)]);
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u) {
          if (pos[u].cls == POS_VEC) {
            VB x = v[rr][u];
            if (RING && rr > 0 && slot == 1) x = x + v[rr > 0 ? rr - 1 : 0][u];  // receiver: own + sender's
            st16<Cfg::NTS>(reinterpret_cast<VB*>(buf + pos[u].p), x);
          } else if (pos[u].cls == POS_ZERO) {
            store_zero<VB>(buf + pos[u].p);  // padding: zero, and zero + zero for a receiver
          }
        }
      }
    }

    if (!edges) continue;
    for (int slot = bs.rbeg; slot < bs.rend; ++slot) {
      if (RING && skip_sender && slot == 0) continue;
      const int r = pt.rank(slot);
      TB* __restrict__ buf = static_cast<TB*>(bufs.p[r]);
      for (int u = 0; u < kPosPerLane; ++u) {
        if (pos[u].cls != POS_EDGE) continue;
        for (int k = 0; k < V; ++k) {
          const int64_t pe = pos[u].p + k;
          if (pe >= bs.ce) break;
          if (pe < bs.cs) continue;
          const int jk = lookup(tt, s_off, offset, pe);
          const int64_t tk = tt.t0 + jk;
          const bool in_tensor = tk >= 0 && pe < tensor_end(tt, s_end, offset, numel, jk);
          const int64_t li = in_tensor ? pe - tensor_begin(tt, s_off, offset, jk) : 0;
          TB val = (TB)0;
          if (in_tensor) {
            val = Mover<TT, TB>::cvt_in(static_cast<const TT*>(pt.get(slot, tk))[li]);
            if (RING && r == receiver)
              val = val + Mover<TT, TB>::cvt_in(static_cast<const TT*>(srcs[(int64_t)bs.c * ntensors + tk])[li]);
          }
          buf[pe] = val;
        }
      }
    }
  }
}

template <typename TT, typename TB, typename Cfg, bool RING>
__global__ __launch_bounds__(Cfg::BS) HVDX_COPY_ATTR void pack_kernel(const void* const* __restrict__ srcs,
                                                                    const int64_t* __restrict__ numel,
                                                                    const int64_t* __restrict__ offset, int ntensors,
                                                                    RankPtrs bufs, int64_t count, int nranks, int rpb,
                                                                    int64_t q, int64_t rem, int skip_sender) {
  pack_body<TT, TB, Cfg, RING>(srcs, numel, offset, ntensors, bufs, count, nranks, rpb, q, rem, skip_sender,
                               RING ? (int)blockIdx.z : (int)blockIdx.y, blockIdx.x);
}

// The fused copy-in of two fusion buffers in one launch: block columns [0, x0) serve
// buffer 0's chunk tiles, [x0, gridDim.x) buffer 1's, so neither has idle blocks.
template <typename TT, typename TB, typename Cfg>
__global__ __launch_bounds__(Cfg::BS) HVDX_COPY_ATTR void pack_pair_kernel(CopyPair m, int nranks, int rpb,
                                                                         int x0) {
  const int b = (int)blockIdx.x >= x0 ? 1 : 0;
  pack_body<TT, TB, Cfg, true>(static_cast<const void* const*>(m.t[b]), m.numel[b], m.offset[b], m.ntensors[b],
                               m.bufs[b], m.count[b], nranks, rpb, m.q[b], m.rem[b], 1, blockIdx.z,
                               (int64_t)blockIdx.x - b * x0);
}

// Copy-out.  With RING it is fused with the ring's last replacing step: in chunk c
// that step hands rank c-3's final values to rank c-2, so rank c-2 copies them out
// from rank c-3's buffer (mod N) and its own buffer keeps the chunk's older values.
// Two passes per row, as in the copy-in.
template <typename TT, typename TB, typename Cfg, bool RING>
__device__ __forceinline__ void unpack_body(const RankPtrs& bufs, int64_t count, void* const* __restrict__ dsts,
                                            const int64_t* __restrict__ numel, const int64_t* __restrict__ offset,
                                            int ntensors, int nranks, int rpb, int64_t q, int64_t rem, int group,
                                            int64_t bx) {
  constexpr int V = BufVec<TT, TB>::n;
  using VB = typename Mover<TT, TB>::buf_vec;
  constexpr int kPosPerLane = Cfg::POS, kRankBatch = Cfg::RB, kTileVecs = Cfg::kTileVecs;
  __shared__ int64_t s_off[Cfg::kLdsTensors], s_end[Cfg::kLdsTensors], s_meta[2];
  __shared__ const void* s_ptr[kLdsPtrs];
  static_assert((kTileVecs & (kTileVecs - 1)) == 0, "tiles are a power of two vectors");
  const BlockSpan bs = block_span<RING>((int64_t)kTileVecs * V, count, nranks, rpb, q, rem, group, bx);
  if (bs.p0 >= bs.p1) return;  // past the end of a shorter chunk: the whole block leaves
  // the rank that receives chunk c in the last replacing step, which reads its sender's buffer
  const int receiver = RING ? (bs.c + nranks - 2) % nranks : -1;
  // Rank batch rb's buffer vectors at the tile's whole-row positions (the positions
  // every lane serves in row 0).
  auto load_batch = [&](VB (&v)[kRankBatch][kPosPerLane], int rb) {
#pragma unroll
    for (int rr = 0; rr < kRankBatch; ++rr) {
      const int r = rb + rr;
      const int from = r == receiver ? (r == 0 ? nranks - 1 : r - 1) : r;
      const TB* __restrict__ buf = static_cast<const TB*>(bufs.p[r < bs.rend ? from : bs.rbeg]) + bs.p0;
#pragma unroll
      for (int u = 0; u < kPosPerLane; ++u)
        if (r < bs.rend) v[rr][u] = ld16<Cfg::NTL>(reinterpret_cast<const VB*>(buf + tile_vec<Cfg>(u) * V));
    }
  };
  // Where the buffer is read does not depend on the tensors: when the whole tile lies
  // inside the buffer, the first rank batch is loaded before the tensor lookup, whose
  // dependent loads and barriers then overlap those loads' latency.
  const bool early = HVDX_UNPACK_EARLY && Cfg::SUB == 1 && bs.p0 + (int64_t)kTileVecs * V <= count;
  VB pre[kRankBatch][kPosPerLane];
  if (early) load_batch(pre, bs.rbeg);
  bool pin;
  const TileTable tt = stage_tile<Cfg::kLdsTensors>(offset, numel, ntensors, bs.p0, bs.p1, dsts, bs.rbeg, bs.rend, 0,
                                                    nranks, s_off, s_end, s_meta, s_ptr, &pin);
  const PtrTable pt{dsts, pin ? s_ptr : nullptr, tt.t0, ntensors, tt.nt, bs.rbeg, 0, nranks};

  if (whole_tile<Cfg, V>(tt, bs, s_off, s_end, offset, numel)) {  // no per-vector classification needed
    const int64_t li0 = bs.p0 - tensor_begin(tt, s_off, offset, 0);
    for (int rb = bs.rbeg; rb < bs.rend; rb += kRankBatch) {
      VB v[kRankBatch][kPosPerLane];
      if (early && rb == bs.rbeg) {
#pragma unroll
        for (int rr = 0; rr < kRankBatch; ++rr)
#pragma unroll
          for (int u = 0; u < kPosPerLane; ++u) v[rr][u] = pre[rr][u];
      } else {
        load_batch(v, rb);
      }
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int r = rb + rr;
        if (r >= bs.rend) break;
        TT* dst = static_cast<TT*>(const_cast<void*>(pt.get(r, tt.t0))) + li0;
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u)
          Mover<TT, TB>::template store<Cfg::NTS>(dst + tile_vec<Cfg>(u) * V, v[rr][u]);
      }
    }
    return;
  }

  for (int row = 0; row < Cfg::SUB; ++row) {
    const int64_t r0 = bs.p0 + (int64_t)row * Cfg::kRowVecs * V;
    if (r0 >= bs.p1) break;
    Pos pos[kPosPerLane];
    bool edges = false;
#pragma unroll
    for (int u = 0; u < kPosPerLane; ++u) {
      pos[u] = classify<V>(tt, s_off, s_end, offset, numel, r0 + (int64_t)tile_vec<Cfg>(u) * V, bs.p1, bs.cs, bs.ce);
      edges |= pos[u].cls == POS_EDGE;
    }

    for (int rb = bs.rbeg; rb < bs.rend; rb += kRankBatch) {
      VB v[kRankBatch][kPosPerLane];
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int r = rb + rr;
        const int from = r == receiver ? (r == 0 ? nranks - 1 : r - 1) : r;
        const TB* __restrict__ buf = static_cast<const TB*>(bufs.p[r < bs.rend ? from : bs.rbeg]);
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u) {
          if (r >= bs.rend || pos[u].cls != POS_VEC) continue;
          // row 0's positions are the ones loaded early
          v[rr][u] = early && row == 0 && rb == bs.rbeg ? pre[rr][u]
                                                        : ld16<Cfg::NTL>(reinterpret_cast<const VB*>(buf + pos[u].p));
        }
      }
#pragma unroll
      for (int rr = 0; rr < kRankBatch; ++rr) {
        const int r = rb + rr;
        if (r >= bs.rend) break;
#pragma unroll
        for (int u = 0; u < kPosPerLane; ++u)
          if (pos[u].cls == POS_VEC)
            Mover<TT, TB>::template store<Cfg::NTS>(static_cast<TT*>(const_cast<void*>(pt.get(r, pos[u].t))) +
                                                        pos[u].li,
                                                    v[rr][u]);
      }
    }

    if (!edges) continue;
    for (int r = bs.rbeg; r < bs.rend; ++r) {
      const int from = r == receiver ? (r == 0 ? nranks - 1 : r - 1) : r;
      const TB* __restrict__ buf = static_cast<const TB*>(bufs.p[from]);
      for (int u = 0; u < kPosPerLane; ++u) {
        if (pos[u].cls != POS_EDGE) continue;
        for (int k = 0; k < V; ++k) {
          const int64_t pe = pos[u].p + k;
          if (pe >= bs.ce) break;
          if (pe < bs.cs) continue;
          const int jk = lookup(tt, s_off, offset, pe);
          const int64_t tk = tt.t0 + jk;
          if (tk >= 0 && pe < tensor_end(tt, s_end, offset, numel, jk)) {
            TT* dk = static_cast<TT*>(const_cast<void*>(pt.get(r, tk)));
            dk[pe - tensor_begin(tt, s_off, offset, jk)] = Mover<TT, TB>::cvt_out(buf[pe]);
          }
        }
      }
    }
  }
}

template <typename TT, typename TB, typename Cfg, bool RING>
__global__ __launch_bounds__(Cfg::BS) HVDX_COPY_ATTR void unpack_kernel(RankPtrs bufs, int64_t count,
                                                                      void* const* __restrict__ dsts,
                                                                      const int64_t* __restrict__ numel,
                                                                      const int64_t* __restrict__ offset, int ntensors,
                                                                      int nranks, int rpb, int64_t q, int64_t rem) {
  unpack_body<TT, TB, Cfg, RING>(bufs, count, dsts, numel, offset, ntensors, nranks, rpb, q, rem,
                                 RING ? (int)blockIdx.z : (int)blockIdx.y, blockIdx.x);
}

// The fused copy-out of two fusion buffers in one launch (columns as pack_pair_kernel).
template <typename TT, typename TB, typename Cfg>
__global__ __launch_bounds__(Cfg::BS) HVDX_COPY_ATTR void unpack_pair_kernel(CopyPair m, int nranks, int rpb,
                                                                           int x0) {
  const int b = (int)blockIdx.x >= x0 ? 1 : 0;
  unpack_body<TT, TB, Cfg, true>(m.bufs[b], m.count[b], m.t[b], m.numel[b], m.offset[b], m.ntensors[b], nranks, rpb,
                                 m.q[b], m.rem[b], blockIdx.z, (int64_t)blockIdx.x - b * x0);
}

// ---- a small fusion buffer's whole cycle in one launch ------------------------------
//
// For buffers so small that launches cost more than their data: each thread takes one
// 16-byte buffer vector through the copy-in for every rank, all 2(N-1) ring steps
// (ring_chain: each step reads the sender's buffer and writes the receiver's) and the
// copy-out for every rank.  Vectors of padding only are skipped (their values never
// reach a tensor and the buffers are scratch afterwards); edge vectors go element by
// element.  A block serves one tile of 256 vectors for all ranks.
using SmallCfg = CopyCfg<1, 1, 0, false, false>;

template <typename TT, typename TB, int DIV>
__global__ __launch_bounds__(kBlock) void small_cycle_kernel(const void* const* __restrict__ tensors,
                                                             const int64_t* __restrict__ numel,
                                                             const int64_t* __restrict__ offset, int ntensors,
                                                             RankPtrs bufs, RingArgs a, int64_t count) {
  using Cfg = SmallCfg;
  using M = Mover<TT, TB>;
  using VB = typename M::buf_vec;
  constexpr int V = BufVec<TT, TB>::n;
  __shared__ int64_t s_off[Cfg::kLdsTensors], s_end[Cfg::kLdsTensors], s_meta[2];
  __shared__ const void* s_ptr[kLdsPtrs];
  const int n = a.n;
  const int64_t p0 = (int64_t)blockIdx.x * Cfg::kTileVecs * V;
  const int64_t p1 = p0 + (int64_t)Cfg::kTileVecs * V < count ? p0 + (int64_t)Cfg::kTileVecs * V : count;
  if (p0 >= p1) return;
  bool pin;
  const TileTable tt = stage_tile<Cfg::kLdsTensors>(offset, numel, ntensors, p0, p1, tensors, 0, n, 0, n, s_off,
                                                    s_end, s_meta, s_ptr, &pin);
  const PtrTable pt{tensors, pin ? s_ptr : nullptr, tt.t0, ntensors, tt.nt, 0, 0, n};
  const Pos ps = classify<V>(tt, s_off, s_end, offset, numel, p0 + (int64_t)threadIdx.x * V, p1, 0, count);
  auto buf = [&](int r) { return static_cast<TB*>(bufs.p[r]); };
  auto ten = [&](int r, int64_t t) { return static_cast<TT*>(const_cast<void*>(pt.get(r, t))); };
  if (ps.cls == POS_VEC) {
    for (int r = 0; r < n; ++r)
      st16<false>(reinterpret_cast<VB*>(buf(r) + ps.p), M::template load<false>(ten(r, ps.t) + ps.li));
    const int64_t c0 = chunk_index(ps.p, a);
    if (chunk_index(ps.p + V - 1, a) == c0) {
      ring_chain<TB, VB, DIV>(bufs, ps.p, (int)c0, a);
    } else {
      for (int k = 0; k < V; ++k) ring_chain<TB, TB, DIV>(bufs, ps.p + k, (int)chunk_index(ps.p + k, a), a);
    }
    for (int r = 0; r < n; ++r)
      M::template store<false>(ten(r, ps.t) + ps.li, *reinterpret_cast<const VB*>(buf(r) + ps.p));
  } else if (ps.cls == POS_EDGE) {
    for (int k = 0; k < V; ++k) {
      const int64_t pe = ps.p + k;
      if (pe >= count) break;
      const int jk = lookup(tt, s_off, offset, pe);
      const int64_t tk = tt.t0 + jk;
      if (tk < 0 || pe >= tensor_end(tt, s_end, offset, numel, jk)) continue;  // padding
      const int64_t li = pe - tensor_begin(tt, s_off, offset, jk);
      for (int r = 0; r < n; ++r) buf(r)[pe] = M::cvt_in(ten(r, tk)[li]);
      ring_chain<TB, TB, DIV>(bufs, pe, (int)chunk_index(pe, a), a);
      for (int r = 0; r < n; ++r) ten(r, tk)[li] = M::cvt_out(buf(r)[pe]);
    }
  }
}

// ---- the fused copies driven by tile tables -------------------------------------------
//
// The same two copies as pack_kernel<..., true> and unpack_kernel<..., true> inside the
// fused cycle, but each block reads its tile (a stretch of one tensor, or of padding,
// inside one ring chunk, cut once on the host by hvdx_fuse_copy_tiles) and moves it for
// one rank, one 16-byte vector (on the wider side) per lane.  No tensor search, no LDS,
// no barrier: the block's only dependent loads are its tile and a tensor pointer, and the
// copy-out issues its buffer loads before the pointer arrives.  Measured on MI355X, a copy
// between many buffers streams fastest in exactly this shape (one rank, one vector per
// lane per block), and the copy-out's tiles start on the tensors' own tile bounds, so each
// wavefront's stores cover whole cache lines of the tensor it writes.

// Copy-in with the ring's adding step 0 (paper section 3), in the fused cycle: block row y
// is rank c+1+y of the tile's chunk c, so row 0 is the chunk's receiver, which stores its
// own value plus the sender's; the sender (rank c) stores nothing, as in the cycle's
// lookup kernel (replacing step 0 overwrites its copy before anything reads it).
template <typename TT, typename TB, int U>
__global__ __launch_bounds__(kTileLanes) void pack_tiles_kernel(TiledCopy k, int nranks) {
  using M = Mover<TT, TB>;
  using VB = typename M::buf_vec;
  constexpr int V = BufVec<TT, TB>::n;
  const int b = (int64_t)blockIdx.x >= k.x0 ? 1 : 0;
  const hvdx_copy_tile tl = k.tiles[b][b ? (int64_t)blockIdx.x - k.x0 : (int64_t)blockIdx.x];
  const bool receiver = blockIdx.y == 0;
  int r = tl.chunk + 1 + (int)blockIdx.y;
  if (r >= nranks) r -= nranks;
  TB* __restrict__ buf = static_cast<TB*>(k.m.bufs[b].p[r]) + tl.pos;
  if (tl.tensor < 0) {  // padding: zero, and zero + zero for the receiver
    for (int e = threadIdx.x; e < tl.len; e += kTileLanes) buf[e] = (TB)0;
    return;
  }
  const int64_t nt = k.m.ntensors[b];
  const TT* __restrict__ src = static_cast<const TT*>(k.m.t[b][(int64_t)r * nt + tl.tensor]) + tl.li;
  const TT* __restrict__ snd =
      receiver ? static_cast<const TT*>(k.m.t[b][(int64_t)tl.chunk * nt + tl.tensor]) + tl.li : src;
  auto one = [&](int e) {
    TB v = M::cvt_in(src[e]);
    if (receiver) v = v + M::cvt_in(snd[e]);
    buf[e] = v;
  };
  if (aligned16(src) && aligned16(snd) && reinterpret_cast<uintptr_t>(buf) % sizeof(VB) == 0) {
    VB x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {  // lane vectors u*256 apart: each instruction one contiguous run
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (i + V <= tl.len) {
        x[u] = M::template load<true>(src + i);
        if (receiver) x[u] = x[u] + M::template load<true>(snd + i);  // own value plus the sender's
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (i + V <= tl.len) st16<true>(reinterpret_cast<VB*>(buf + i), x[u]);
      else
        for (int e = i; e < tl.len && e < i + V; ++e) one(e);  // the tile's last, partial vector
    }
  } else {
    for (int e = threadIdx.x; e < tl.len; e += kTileLanes) one(e);  // copies not vector-aligned here
  }
}

// Copy-out with the ring's last replacing step: in chunk c that step hands rank c-3's
// final values to rank c-2, which copies them out of rank c-3's buffer (mod N).
template <typename TT, typename TB, int U>
__global__ __launch_bounds__(kTileLanes) void unpack_tiles_kernel(TiledCopy k, int nranks) {
  using M = Mover<TT, TB>;
  using VB = typename M::buf_vec;
  constexpr int V = BufVec<TT, TB>::n;
  const int b = (int64_t)blockIdx.x >= k.x0 ? 1 : 0;
  const hvdx_copy_tile tl = k.tiles[b][b ? (int64_t)blockIdx.x - k.x0 : (int64_t)blockIdx.x];
  const int r = blockIdx.y;
  int rc = tl.chunk - 2;  // the rank receiving chunk c in replacing step N-2
  if (rc < 0) rc += nranks;
  const int from = r == rc ? (r == 0 ? nranks - 1 : r - 1) : r;
  const TB* __restrict__ buf = static_cast<const TB*>(k.m.bufs[b].p[from]) + tl.pos;
  const bool bvec = reinterpret_cast<uintptr_t>(buf) % sizeof(VB) == 0;
  VB x[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {  // the buffer loads go out before the tensor pointer arrives
    const int i = (u * kTileLanes + threadIdx.x) * V;
    if (bvec && i + V <= tl.len) x[u] = ld16<true>(reinterpret_cast<const VB*>(buf + i));
  }
  TT* __restrict__ dst = static_cast<TT*>(const_cast<void*>(k.m.t[b][(int64_t)r * k.m.ntensors[b] + tl.tensor])) +
                         tl.li;
  if (bvec && aligned16(dst)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (i + V <= tl.len) M::template store<true>(dst + i, x[u]);
      else
        for (int e = i; e < tl.len && e < i + V; ++e) dst[e] = M::cvt_out(buf[e]);
    }
  } else {
    for (int e = threadIdx.x; e < tl.len; e += kTileLanes) dst[e] = M::cvt_out(buf[e]);
  }
}

// The block index a tile kernel works on.  The blocks the hardware hands to one of the 8
// XCDs (block b goes to XCD b mod 8) take one contiguous run of tiles, so two neighbouring
// tiles that share a cache line (a tile's reads on the side it does not write start off
// the lines) mostly share that XCD's L2; a bijection on [0, gridDim.x) for any grid size.
// Measured on MI355X against block b taking tile run b: ResNet-50 and Inception-V3 -2%
// per step (their ring steps +1 to +3 points of peak), VGG-16 -0.3%, VGG-16 fp16 unchanged.
#ifndef HVDX_XCD_BLOCKS
#define HVDX_XCD_BLOCKS 1
#endif
__device__ __forceinline__ int64_t tile_block() {
  const int64_t b = blockIdx.x;
  if constexpr (HVDX_XCD_BLOCKS) {
    const int64_t g = gridDim.x, q = g / 8, r = g % 8, x = b % 8;
    return x * q + (x < r ? x : r) + b / 8;
  }
  return b;
}

// The bucket that tile g of a TiledRing launch belongs to, and g's index in its table.
__device__ __forceinline__ int ring_bucket(const TiledRing& k, int64_t g, int64_t* local) {
  int b = 0;
#pragma unroll
  for (int i = 1; i < kRingBuckets; ++i)
    if (i < k.nbuckets && g >= k.end[i - 1]) b = i;
  *local = b ? g - k.end[b - 1] : g;
  return b;
}

// ---- the ring on the tensors ------------------------------------------------------------
//
// With every rank in one memory, a replacing step can write the chunk it delivers
// straight into the receiver's output tensors instead of its fusion buffer, and the
// next step forwards it from there: each rank's tensors then end holding the result
// with no copy-out.  Likewise an adding step can read the receiver's own elements of
// its chunk from its tensors, where the copy-in would have taken them (in adding step s
// rank c+s+1 touches chunk c for the first time): no copy-in, and the fusion buffers
// hold only the partial sums received.  The messages and their order are the ring's;
// only where a rank's own input is read and where a received chunk is stored change.
// The kernels run over the plan's tile tables (each tile inside one tensor and one ring
// chunk): the adding steps over the copy-in's (on the buffer's tile grid), the others
// over the copy-out's (on the tensor's).  With binary32 tensors and binary16 buffers
// this is the compressed ring: elements rounded where first read, binary16 partial
// sums, binary32 values (binary16 results held exactly) in the replacing steps.
// Padding tiles have no tensor and are skipped.

// Adding step N-2 and replacing step 0 of chunk c: the owner (rank c-1) completes its
// sum from the sender's (c-2) buffer, and the finished value goes to the owner's and
// rank c's tensors.  The owner's copy is not read again and streams; rank c's is the
// sender's input in replacing step 1 and stays in the caches.  OWN_T: the owner's own
// value is read from its tensors (the adding steps never copied it into its buffer);
// each lane reads an element there before it writes the result over it.
#ifndef HVDX_RSAGT_NTL  // non-temporal buffer loads: the buffers are not read again
#define HVDX_RSAGT_NTL true
#endif
#ifndef HVDX_RSAGT_NXT_NTS  // rank c's copy: replacing step 1 reads it
#define HVDX_RSAGT_NXT_NTS false
#endif
template <typename TT, typename TB, int DIV, bool OWN_T, int U>
__global__ __launch_bounds__(kTileLanes) void rs_ag_tiles_kernel(TiledRing k, RingArgs a) {
  using M = Mover<TT, TB>;
  using VB = typename M::buf_vec;
  constexpr int V = BufVec<TT, TB>::n;
  constexpr size_t VBB = sizeof(VB);
  int64_t li;
  const int b = ring_bucket(k, tile_block(), &li);
  const hvdx_copy_tile tl = k.tiles[b][li];
  if (tl.tensor < 0) return;
  const int n = a.n;
  const int c = tl.chunk;
  const int own = c == 0 ? n - 1 : c - 1;
  const int snd = own == 0 ? n - 1 : own - 1;
  const int64_t nt = k.ntensors[b];
  const TB* bs = static_cast<const TB*>(k.bufs[b * n + snd]) + tl.pos;
  const TB* bo = static_cast<const TB*>(k.bufs[b * n + own]) + tl.pos;  // not read with OWN_T
  TT* d_own;
  TT* d_nxt;
  VB mine[U], sent[U];
  bool vec;
  auto aligned_b = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % VBB == 0; };
  if constexpr (OWN_T) {  // the owner's own value from its tensors: the pointers first
    d_own = static_cast<TT*>(const_cast<void*>(k.t[b][(int64_t)own * nt + tl.tensor])) + tl.li;
    d_nxt = static_cast<TT*>(const_cast<void*>(k.t[b][(int64_t)c * nt + tl.tensor])) + tl.li;
    vec = aligned16(d_own) && aligned_b(bs) && aligned16(d_nxt);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (vec && i + V <= tl.len) {
        mine[u] = M::template load<HVDX_RSAGT_NTL, true>(d_own + i);
        sent[u] = ld16<HVDX_RSAGT_NTL>(reinterpret_cast<const VB*>(bs + i));
      }
    }
  } else {
    const bool bvec = aligned_b(bo) && aligned_b(bs);
#pragma unroll
    for (int u = 0; u < U; ++u) {  // the buffer loads go out before the tensor pointers arrive
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (bvec && i + V <= tl.len) {
        mine[u] = ld16<HVDX_RSAGT_NTL>(reinterpret_cast<const VB*>(bo + i));
        sent[u] = ld16<HVDX_RSAGT_NTL>(reinterpret_cast<const VB*>(bs + i));
      }
    }
    d_own = static_cast<TT*>(const_cast<void*>(k.t[b][(int64_t)own * nt + tl.tensor])) + tl.li;
    d_nxt = static_cast<TT*>(const_cast<void*>(k.t[b][(int64_t)c * nt + tl.tensor])) + tl.li;
    vec = bvec && aligned16(d_own) && aligned16(d_nxt);
  }
  auto one = [&](int e) {  // with OWN_T each lane reads its element before it writes over it
    const TB m = OWN_T ? M::cvt_in(d_own[e]) : bo[e];
    const TT v = M::cvt_out(combine1<DIV>(m, bs[e], a));
    d_own[e] = v;
    d_nxt[e] = v;
  };
  if (vec) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (i + V <= tl.len) {
        const VB v = combine<DIV>(mine[u], sent[u], a);
        M::template store<true, true>(d_own + i, v);
        M::template store<HVDX_RSAGT_NXT_NTS, true>(d_nxt + i, v);
      } else {
        for (int e = i; e < tl.len && e < i + V; ++e) one(e);  // the tile's last, partial vector
      }
    }
  } else {
    for (int e = threadIdx.x; e < tl.len; e += kTileLanes) one(e);
  }
}

// Adding step s <= N-3 with every rank's own values read from its tensors (the copy-in
// fused with the step that first reads each chunk): rank c+s+1 adds its own elements of
// chunk c to what rank c+s sent (its partial sum in its buffer, or at s = 0 its own
// elements, also from its tensors) and keeps the sum in its buffer.  Over the copy-in's
// tiles (on the buffer's tile grid); padding is skipped (nothing reads it).  Tensor
// loads are non-temporal (each element is read once in the adding steps), the sender's
// partial sum too (read once), the stores cached (the next step reads them).
#ifndef HVDX_ADDT_TPB
#define HVDX_ADDT_TPB 2
#endif
#ifndef HVDX_ADDT_NTL
#define HVDX_ADDT_NTL true
#endif
#ifndef HVDX_ADDT_NTS
#define HVDX_ADDT_NTS false
#endif
template <typename TT, typename TB, bool FIRST, int TPB, int U>
__global__ __launch_bounds__(kTileLanes) void add_tiles_kernel(TiledRing k, int step, int64_t ntiles) {
  using M = Mover<TT, TB>;
  using VB = typename M::buf_vec;
  constexpr int V = BufVec<TT, TB>::n;
  constexpr size_t VBB = sizeof(VB);
  const TT* mine[TPB];
  const TT* sent_t[TPB];  // the sender's tensor (step 0)
  const TB* sent_b[TPB];  // the sender's buffer (later steps)
  TB* out[TPB];
  int len[TPB];
  bool vec[TPB];
  auto aligned_b = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % VBB == 0; };
#pragma unroll
  for (int j = 0; j < TPB; ++j) {
    const int64_t g = tile_block() * TPB + j;
    len[j] = 0;
    mine[j] = nullptr;
    sent_t[j] = nullptr;
    sent_b[j] = nullptr;
    out[j] = nullptr;
    vec[j] = false;
    if (g >= ntiles) continue;
    int64_t loc;
    const int b = ring_bucket(k, g, &loc);
    const hvdx_copy_tile tl = k.tiles[b][loc];
    if (tl.tensor < 0) continue;
    const int n = k.nranks;
    int snd = tl.chunk + step;  // chunk < N and step <= N-3: below 2N
    if (snd >= n) snd -= n;
    const int rcv = snd + 1 == n ? 0 : snd + 1;
    const int64_t nt = k.ntensors[b];
    mine[j] = static_cast<const TT*>(k.t[b][(int64_t)rcv * nt + tl.tensor]) + tl.li;
    if (FIRST) sent_t[j] = static_cast<const TT*>(k.t[b][(int64_t)snd * nt + tl.tensor]) + tl.li;
    else sent_b[j] = static_cast<const TB*>(k.bufs[b * n + snd]) + tl.pos;
    out[j] = static_cast<TB*>(k.bufs[b * n + rcv]) + tl.pos;
    len[j] = tl.len;
    vec[j] = aligned16(mine[j]) && (FIRST ? aligned16(sent_t[j]) : aligned_b(sent_b[j])) && aligned_b(out[j]);
  }
  VB x[TPB][U], y[TPB][U];
#pragma unroll
  for (int j = 0; j < TPB; ++j)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (vec[j] && i + V <= len[j]) {
        x[j][u] = M::template load<HVDX_ADDT_NTL, true>(mine[j] + i);
        y[j][u] = FIRST ? M::template load<HVDX_ADDT_NTL, true>(sent_t[j] + i)
                        : ld16<HVDX_ADDT_NTL>(reinterpret_cast<const VB*>(sent_b[j] + i));
      }
    }
  auto one = [&](int j, int e) {
    out[j][e] = M::cvt_in(mine[j][e]) + (FIRST ? M::cvt_in(sent_t[j][e]) : sent_b[j][e]);
  };
#pragma unroll
  for (int j = 0; j < TPB; ++j) {
    if (vec[j]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = (u * kTileLanes + threadIdx.x) * V;
        if (i + V <= len[j]) st16<HVDX_ADDT_NTS>(reinterpret_cast<VB*>(out[j] + i), x[j][u] + y[j][u]);
        else
          for (int e = i; e < len[j] && e < i + V; ++e) one(j, e);
      }
    } else {
      for (int e = threadIdx.x; e < len[j]; e += kTileLanes) one(j, e);
    }
  }
}

// Replacing step s >= 1 of chunk c: rank c-1+s's tensors to rank c+s's (mod N).  The
// receiver's copy is the next step's input (cached stores) except in the last step.  A
// block moves TPB consecutive tiles, all of their loads in flight before any store.
// Measured on MI355X (ResNet-50, Inception-V3, VGG-16): one tile per block 72-79% of
// peak, two 79-81%, four 78-81%; non-temporal loads +6 points against cached ones (the
// sender's copy is not read again); streamed stores in every step lose 5-10 points
// (the next step reads them).
#ifndef HVDX_AGT_TPB
#define HVDX_AGT_TPB 2
#endif
#ifndef HVDX_AGT_NTL
#define HVDX_AGT_NTL true
#endif
#ifndef HVDX_AGT_NTS
#define HVDX_AGT_NTS false
#endif
template <typename T, bool LAST, int TPB, int U>
__global__ __launch_bounds__(kTileLanes) void ag_tiles_kernel(TiledRing k, int step, int64_t ntiles) {
  using VT = typename Vec<T>::type;
  constexpr int V = Vec<T>::n;
  const T* src[TPB];
  T* dst[TPB];
  int len[TPB];
  bool vec[TPB];
#pragma unroll
  for (int j = 0; j < TPB; ++j) {
    const int64_t g = tile_block() * TPB + j;
    len[j] = 0;
    src[j] = nullptr;
    dst[j] = nullptr;
    vec[j] = false;
    if (g >= ntiles) continue;
    int64_t loc;
    const int b = ring_bucket(k, g, &loc);
    const hvdx_copy_tile tl = k.tiles[b][loc];
    if (tl.tensor < 0) continue;
    const int n = k.nranks;
    int snd = tl.chunk + step - 1;  // chunk < N and step <= N-2: below 2N
    if (snd >= n) snd -= n;
    const int rcv = snd + 1 == n ? 0 : snd + 1;
    const int64_t nt = k.ntensors[b];
    src[j] = static_cast<const T*>(k.t[b][(int64_t)snd * nt + tl.tensor]) + tl.li;
    dst[j] = static_cast<T*>(const_cast<void*>(k.t[b][(int64_t)rcv * nt + tl.tensor])) + tl.li;
    len[j] = tl.len;
    vec[j] = aligned16(src[j]) && aligned16(dst[j]);
  }
  VT x[TPB][U];
#pragma unroll
  for (int j = 0; j < TPB; ++j)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = (u * kTileLanes + threadIdx.x) * V;
      if (vec[j] && i + V <= len[j]) x[j][u] = ld16<HVDX_AGT_NTL>(reinterpret_cast<const VT*>(src[j] + i));
    }
#pragma unroll
  for (int j = 0; j < TPB; ++j) {
    if (vec[j]) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = (u * kTileLanes + threadIdx.x) * V;
        if (i + V <= len[j]) st16<LAST || HVDX_AGT_NTS>(reinterpret_cast<VT*>(dst[j] + i), x[j][u]);
        else
          for (int e = i; e < len[j] && e < i + V; ++e) dst[j][e] = src[j][e];
      }
    } else {
      for (int e = threadIdx.x; e < len[j]; e += kTileLanes) dst[j][e] = src[j][e];
    }
  }
}

// ---- the broadcast chain over many tensors ------------------------------------------
//
// One chain step (paper sections 4 and 5; reading B2): block row y is link k, from rank
// root+k to rank root+k+1, carrying chunk step-k of the virtual byte space in which the
// call's tensors lie end to end, each starting on a 16-byte boundary.  A block copies
// one tile of its chunk.  It finds the tile's tensors as the copy kernels do (positions
// are bytes here, and the two ranks of the link are the tile's two pointer slots); a
// tile inside one tensor whose two copies are 16-byte aligned there is moved as whole
// vectors, otherwise each lane takes its 16-byte units one by one: a unit inside one
// tensor with both copies aligned as a vector, a tensor's short last unit or an
// unaligned copy byte by byte.  Bytes between tensors belong to none and are skipped.
using BcastCfg = CopyCfg<2, 1, 2, true, true>;
typedef unsigned int b32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(BcastCfg::BS) void bcast_tensors_step_kernel(BcastTensorsArgs a) {
  using Cfg = BcastCfg;
  constexpr int V = 16;  // bytes per unit
  constexpr int64_t kTileBytes = (int64_t)Cfg::kTileVecs * V;
  __shared__ int64_t s_off[Cfg::kLdsTensors], s_end[Cfg::kLdsTensors], s_meta[2];
  __shared__ const void* s_ptr[kLdsPtrs];
  const int k = blockIdx.y;
  const int64_t j = (int64_t)a.step - k;
  if (j < 0 || j >= a.n) return;  // this link carries nothing in this step
  const int src = (a.root + k) % a.n;
  const int64_t u0 = j * a.q + (j < a.rem ? j : a.rem);
  const int64_t units = a.q + (j < a.rem ? 1 : 0);
  const int64_t lo = u0 * V < a.total ? u0 * V : a.total;
  const int64_t hi = (u0 + units) * V < a.total ? (u0 + units) * V : a.total;
  const int64_t p0 = lo + (int64_t)blockIdx.x * kTileBytes;
  if (p0 >= hi) return;  // past the end of a shorter chunk: the whole block leaves
  const int64_t p1 = p0 + kTileBytes < hi ? p0 + kTileBytes : hi;
  bool pin;
  // slot 0 is the sending rank, slot 1 the receiving one
  const TileTable tt = stage_tile<Cfg::kLdsTensors>(a.voff, a.nbytes, a.ntensors, p0, p1, a.ptrs, 0, 2, src, a.n,
                                                    s_off, s_end, s_meta, s_ptr, &pin);
  const PtrTable pt{a.ptrs, pin ? s_ptr : nullptr, tt.t0, a.ntensors, tt.nt, 0, src, a.n};

  if (tt.nt == 1 && tt.t0 >= 0 && p1 - p0 == kTileBytes) {  // block-uniform
    const int64_t beg = tensor_begin(tt, s_off, a.voff, 0);
    const int64_t end = tensor_end(tt, s_end, a.voff, a.nbytes, 0);
    const unsigned char* s = static_cast<const unsigned char*>(pt.get(0, tt.t0)) + (p0 - beg);
    unsigned char* d = static_cast<unsigned char*>(const_cast<void*>(pt.get(1, tt.t0))) + (p0 - beg);
    if (beg <= p0 && p1 <= end && aligned16(s) && aligned16(d)) {
      b32x4 v[Cfg::POS];
#pragma unroll
      for (int u = 0; u < Cfg::POS; ++u) v[u] = ld16<Cfg::NTL>(reinterpret_cast<const b32x4*>(s + tile_vec<Cfg>(u) * V));
#pragma unroll
      for (int u = 0; u < Cfg::POS; ++u) st16<Cfg::NTS>(reinterpret_cast<b32x4*>(d + tile_vec<Cfg>(u) * V), v[u]);
      return;
    }
  }

  for (int u = 0; u < Cfg::POS; ++u) {
    const int64_t p = p0 + (int64_t)tile_vec<Cfg>(u) * V;
    if (p >= p1) continue;
    const int jt = lookup(tt, s_off, a.voff, p);
    const int64_t t = tt.t0 + jt;
    if (t < 0) continue;  // before the first tensor
    const int64_t beg = tensor_begin(tt, s_off, a.voff, jt);
    const int64_t end = tensor_end(tt, s_end, a.voff, a.nbytes, jt);
    if (p >= end) continue;  // between two tensors
    // tensor t starts at or before p (lookup), so bytes [p, stop) are its own
    const int64_t stop = p + V < end ? (p + V < p1 ? p + V : p1) : (end < p1 ? end : p1);
    const unsigned char* s = static_cast<const unsigned char*>(pt.get(0, t)) + (p - beg);
    unsigned char* d = static_cast<unsigned char*>(const_cast<void*>(pt.get(1, t))) + (p - beg);
    if (stop - p == V && aligned16(s) && aligned16(d)) {
      st16<Cfg::NTS>(reinterpret_cast<b32x4*>(d), ld16<Cfg::NTL>(reinterpret_cast<const b32x4*>(s)));
    } else {
      for (int64_t e = 0; e < stop - p; ++e) d[e] = s[e];
    }
  }
}

template <typename Cfg>
unsigned tiles_for(int64_t count, int64_t vec) {
  const int64_t per = (int64_t)Cfg::kTileVecs * vec;
  return (unsigned)((count + per - 1) / per);
}

template <typename Cfg>
int ranks_per_block(int nranks) { return Cfg::RPB > 0 && Cfg::RPB < nranks ? Cfg::RPB : nranks; }

// Plain: (tiles, rank groups).  Fused with a ring step: (tiles a chunk can meet --
// its length plus up to a tile of slack before its start -- chunks, rank groups).
template <typename Cfg, bool RING>
dim3 copy_grid(int64_t count, int64_t vec, int nranks) {
  const int rpb = ranks_per_block<Cfg>(nranks);
  const unsigned groups = (unsigned)((nranks + rpb - 1) / rpb);
  if (!RING) return dim3(tiles_for<Cfg>(count, vec), groups);
  const int64_t tile = (int64_t)Cfg::kTileVecs * vec;
  const int64_t longest = count / nranks + (count % nranks ? 1 : 0);
  return dim3(tiles_for<Cfg>(longest + tile - 1, vec), (unsigned)nranks, groups);
}

template <typename Cfg, bool RING>
void pack_with(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors, int src_dtype,
               const RankPtrs& bufs, int64_t count, int buf_dtype, int nranks, int skip_sender, hipStream_t stream) {
  const int rpb = ranks_per_block<Cfg>(nranks);
  const dim3 grid = copy_grid<Cfg, RING>(count, vec_elems(src_dtype, buf_dtype), nranks);
  const int64_t q = count / nranks, rem = count % nranks;
  if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((pack_kernel<float, float, Cfg, RING>), grid, dim3(Cfg::BS), 0, stream, srcs, numel, offset,
                       ntensors, bufs, count, nranks, rpb, q, rem, skip_sender);
  else if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT16)
    HVDX_LAUNCH((pack_kernel<float, _Float16, Cfg, RING>), grid, dim3(Cfg::BS), 0, stream, srcs, numel,
                       offset, ntensors, bufs, count, nranks, rpb, q, rem, skip_sender);
  else
    HVDX_LAUNCH((pack_kernel<_Float16, _Float16, Cfg, RING>), grid, dim3(Cfg::BS), 0, stream, srcs, numel,
                       offset, ntensors, bufs, count, nranks, rpb, q, rem, skip_sender);
}

template <typename Cfg, bool RING>
void unpack_with(const RankPtrs& bufs, int64_t count, int buf_dtype, void* const* dsts, const int64_t* numel,
                 const int64_t* offset, int ntensors, int dst_dtype, int nranks, hipStream_t stream) {
  const int rpb = ranks_per_block<Cfg>(nranks);
  const dim3 grid = copy_grid<Cfg, RING>(count, vec_elems(dst_dtype, buf_dtype), nranks);
  const int64_t q = count / nranks, rem = count % nranks;
  if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((unpack_kernel<float, float, Cfg, RING>), grid, dim3(Cfg::BS), 0, stream, bufs, count, dsts,
                       numel, offset, ntensors, nranks, rpb, q, rem);
  else if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT16)
    HVDX_LAUNCH((unpack_kernel<float, _Float16, Cfg, RING>), grid, dim3(Cfg::BS), 0, stream, bufs, count,
                       dsts, numel, offset, ntensors, nranks, rpb, q, rem);
  else
    HVDX_LAUNCH((unpack_kernel<_Float16, _Float16, Cfg, RING>), grid, dim3(Cfg::BS), 0, stream, bufs, count,
                       dsts, numel, offset, ntensors, nranks, rpb, q, rem);
}

// Two buffers in one launch: buffer 0's chunk-tile columns (x0 of them), then buffer 1's.
template <typename Cfg>
dim3 pair_grid(const CopyPair& m, int64_t vec, int nranks, unsigned* x0) {
  const dim3 g0 = copy_grid<Cfg, true>(m.count[0], vec, nranks), g1 = copy_grid<Cfg, true>(m.count[1], vec, nranks);
  *x0 = g0.x;
  return dim3(g0.x + g1.x, (unsigned)nranks, g0.z);
}

template <typename Cfg>
void pack_pair_with(const CopyPair& m, int src_dtype, int buf_dtype, int nranks, hipStream_t stream) {
  const int rpb = ranks_per_block<Cfg>(nranks);
  unsigned x0;
  const dim3 grid = pair_grid<Cfg>(m, vec_elems(src_dtype, buf_dtype), nranks, &x0);
  if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((pack_pair_kernel<float, float, Cfg>), grid, dim3(Cfg::BS), 0, stream, m, nranks, rpb, (int)x0);
  else if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT16)
    HVDX_LAUNCH((pack_pair_kernel<float, _Float16, Cfg>), grid, dim3(Cfg::BS), 0, stream, m, nranks, rpb,
                (int)x0);
  else
    HVDX_LAUNCH((pack_pair_kernel<_Float16, _Float16, Cfg>), grid, dim3(Cfg::BS), 0, stream, m, nranks, rpb,
                (int)x0);
}

template <typename Cfg>
void unpack_pair_with(const CopyPair& m, int buf_dtype, int dst_dtype, int nranks, hipStream_t stream) {
  const int rpb = ranks_per_block<Cfg>(nranks);
  unsigned x0;
  const dim3 grid = pair_grid<Cfg>(m, vec_elems(dst_dtype, buf_dtype), nranks, &x0);
  if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((unpack_pair_kernel<float, float, Cfg>), grid, dim3(Cfg::BS), 0, stream, m, nranks, rpb,
                (int)x0);
  else if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT16)
    HVDX_LAUNCH((unpack_pair_kernel<float, _Float16, Cfg>), grid, dim3(Cfg::BS), 0, stream, m, nranks, rpb,
                (int)x0);
  else
    HVDX_LAUNCH((unpack_pair_kernel<_Float16, _Float16, Cfg>), grid, dim3(Cfg::BS), 0, stream, m, nranks, rpb,
                (int)x0);
}

}  // namespace

hipError_t launch_pack(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                       int src_dtype, const RankPtrs& bufs, int64_t count, int buf_dtype, int nranks, bool ring,
                       bool skip_sender, hipStream_t stream) {
  const int skip = ring && skip_sender ? 1 : 0;
  if (buf_dtype == HVDX_FLOAT32) {
    if (ring)
      pack_with<PackCfg, true>(srcs, numel, offset, ntensors, src_dtype, bufs, count, buf_dtype, nranks, skip, stream);
    else
      pack_with<PackCfg, false>(srcs, numel, offset, ntensors, src_dtype, bufs, count, buf_dtype, nranks, 0, stream);
  } else {
    if (ring)
      pack_with<Pack16Cfg, true>(srcs, numel, offset, ntensors, src_dtype, bufs, count, buf_dtype, nranks, skip,
                                 stream);
    else
      pack_with<Pack16Cfg, false>(srcs, numel, offset, ntensors, src_dtype, bufs, count, buf_dtype, nranks, 0, stream);
  }
  return hipGetLastError();
}

hipError_t launch_pack_pair(const CopyPair& m, int src_dtype, int buf_dtype, int nranks, hipStream_t stream) {
  if (buf_dtype == HVDX_FLOAT32) pack_pair_with<PackCfg>(m, src_dtype, buf_dtype, nranks, stream);
  else pack_pair_with<Pack16Cfg>(m, src_dtype, buf_dtype, nranks, stream);
  return hipGetLastError();
}

hipError_t launch_unpack_pair(const CopyPair& m, int buf_dtype, int dst_dtype, int nranks, hipStream_t stream) {
  if (buf_dtype == HVDX_FLOAT32) unpack_pair_with<UnpackCfg>(m, buf_dtype, dst_dtype, nranks, stream);
  else unpack_pair_with<Unpack16Cfg>(m, buf_dtype, dst_dtype, nranks, stream);
  return hipGetLastError();
}

hipError_t launch_small_cycle(const void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                              int tensor_dtype, const RankPtrs& bufs, const RingArgs& a, int64_t count, int buf_dtype,
                              int divmode, hipStream_t stream) {
  const dim3 grid(tiles_for<SmallCfg>(count, vec_elems(tensor_dtype, buf_dtype))), block(kBlock);
#define HVDX_SMALL(TT, TB, DIV) \
  HVDX_LAUNCH((small_cycle_kernel<TT, TB, DIV>), grid, block, 0, stream, tensors, numel, offset, ntensors, \
                     bufs, a, count)
#define HVDX_SMALL_D(TT, TB) \
  if (divmode == DIV_NONE) { HVDX_SMALL(TT, TB, DIV_NONE); } \
  else if (divmode == DIV_POW2) { HVDX_SMALL(TT, TB, DIV_POW2); } \
  else { HVDX_SMALL(TT, TB, DIV_TRUE); }
  if (tensor_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32) {
    HVDX_SMALL_D(float, float)
  } else if (tensor_dtype == HVDX_FLOAT32) {
    HVDX_SMALL_D(float, _Float16)
  } else {
    HVDX_SMALL_D(_Float16, _Float16)
  }
#undef HVDX_SMALL_D
#undef HVDX_SMALL
  return hipGetLastError();
}

hipError_t launch_pack_tiles(const TiledCopy& k, int src_dtype, int buf_dtype, int nranks, int64_t blocks,
                             hipStream_t stream) {
  if (blocks < 1 || blocks > 0x7fffffff || nranks < 2) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks, (unsigned)(nranks - 1));
  if (src_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((pack_tiles_kernel<float, float, HVDX_TILE_U32>), grid, dim3(kTileLanes), 0, stream, k, nranks);
  else if (src_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((pack_tiles_kernel<float, _Float16, HVDX_TILE_U16>), grid, dim3(kTileLanes), 0, stream, k, nranks);
  else
    HVDX_LAUNCH((pack_tiles_kernel<_Float16, _Float16, HVDX_TILE_UH>), grid, dim3(kTileLanes), 0, stream, k, nranks);
  return hipGetLastError();
}

hipError_t launch_unpack_tiles(const TiledCopy& k, int buf_dtype, int dst_dtype, int nranks, int64_t blocks,
                               hipStream_t stream) {
  if (blocks < 1 || blocks > 0x7fffffff || nranks < 1) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks, (unsigned)nranks);
  if (dst_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((unpack_tiles_kernel<float, float, HVDX_TILE_U32>), grid, dim3(kTileLanes), 0, stream, k, nranks);
  else if (dst_dtype == HVDX_FLOAT32)
    HVDX_LAUNCH((unpack_tiles_kernel<float, _Float16, HVDX_TILE_U16>), grid, dim3(kTileLanes), 0, stream, k, nranks);
  else
    HVDX_LAUNCH((unpack_tiles_kernel<_Float16, _Float16, HVDX_TILE_UH>), grid, dim3(kTileLanes), 0, stream, k,
                nranks);
  return hipGetLastError();
}

static int64_t ring_tiles(const TiledRing& k) { return k.nbuckets > 0 ? k.end[k.nbuckets - 1] : 0; }

static bool ring_ok(const TiledRing& k) {
  const int64_t n = ring_tiles(k);
  return k.nbuckets >= 1 && k.nbuckets <= kRingBuckets && k.nranks >= 3 &&
         (int64_t)k.nbuckets * k.nranks <= kRingBufPtrs && n >= 1 && n <= 0x7fffffff;
}

hipError_t launch_rs_ag_tiles(const TiledRing& k, const RingArgs& a, int tensor_dtype, int buf_dtype, int divmode,
                              bool own_in_tensors, hipStream_t stream) {
  if (!ring_ok(k) || a.n != k.nranks) return hipErrorInvalidValue;
  const dim3 grid((unsigned)ring_tiles(k));
  const dim3 block(kTileLanes);
#define HVDX_RSAG_T(TT, TB, U, OWN)                                                                       \
  do {                                                                                                   \
    if (divmode == DIV_NONE)                                                                             \
      HVDX_LAUNCH((rs_ag_tiles_kernel<TT, TB, DIV_NONE, OWN, U>), grid, block, 0, stream, k, a);         \
    else if (divmode == DIV_POW2)                                                                        \
      HVDX_LAUNCH((rs_ag_tiles_kernel<TT, TB, DIV_POW2, OWN, U>), grid, block, 0, stream, k, a);         \
    else HVDX_LAUNCH((rs_ag_tiles_kernel<TT, TB, DIV_TRUE, OWN, U>), grid, block, 0, stream, k, a);      \
  } while (0)
  if (tensor_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32) {
    if (own_in_tensors) HVDX_RSAG_T(float, float, HVDX_TILE_U32, true);
    else HVDX_RSAG_T(float, float, HVDX_TILE_U32, false);
  } else if (tensor_dtype == HVDX_FLOAT32) {
    if (own_in_tensors) HVDX_RSAG_T(float, _Float16, HVDX_TILE_U16, true);
    else HVDX_RSAG_T(float, _Float16, HVDX_TILE_U16, false);
  } else {
    if (own_in_tensors) HVDX_RSAG_T(_Float16, _Float16, HVDX_TILE_UH, true);
    else HVDX_RSAG_T(_Float16, _Float16, HVDX_TILE_UH, false);
  }
#undef HVDX_RSAG_T
  return hipGetLastError();
}

hipError_t launch_add_tiles(const TiledRing& k, int tensor_dtype, int buf_dtype, int step, hipStream_t stream) {
  if (!ring_ok(k) || step < 0 || step > k.nranks - 3) return hipErrorInvalidValue;
  constexpr int TPB = HVDX_ADDT_TPB;
  const int64_t ntiles = ring_tiles(k);
  const dim3 grid((unsigned)((ntiles + TPB - 1) / TPB));
  const dim3 block(kTileLanes);
#define HVDX_ADD_T(TT, TB, U)                                                                              \
  do {                                                                                                    \
    if (step == 0) HVDX_LAUNCH((add_tiles_kernel<TT, TB, true, TPB, U>), grid, block, 0, stream, k, step, ntiles); \
    else HVDX_LAUNCH((add_tiles_kernel<TT, TB, false, TPB, U>), grid, block, 0, stream, k, step, ntiles);        \
  } while (0)
  if (tensor_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32) HVDX_ADD_T(float, float, HVDX_TILE_U32);
  else if (tensor_dtype == HVDX_FLOAT32) HVDX_ADD_T(float, _Float16, HVDX_TILE_U16);
  else HVDX_ADD_T(_Float16, _Float16, HVDX_TILE_UH);
#undef HVDX_ADD_T
  return hipGetLastError();
}

hipError_t launch_ag_tiles(const TiledRing& k, int tensor_dtype, int buf_dtype, int step, hipStream_t stream) {
  if (!ring_ok(k) || step < 1 || step > k.nranks - 2) return hipErrorInvalidValue;
  constexpr int TPB = HVDX_AGT_TPB;
  const int64_t ntiles = ring_tiles(k);
  const dim3 grid((unsigned)((ntiles + TPB - 1) / TPB));
  const dim3 block(kTileLanes);
  const bool last = step == k.nranks - 2;
  // the tensors' own type; the tiles hold what tile_vectors(tensor, buffer) vectors per lane cover
#define HVDX_AG_T(T, U)                                                                                  \
  do {                                                                                                  \
    if (last) HVDX_LAUNCH((ag_tiles_kernel<T, true, TPB, U>), grid, block, 0, stream, k, step, ntiles);  \
    else HVDX_LAUNCH((ag_tiles_kernel<T, false, TPB, U>), grid, block, 0, stream, k, step, ntiles);      \
  } while (0)
  if (tensor_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32) HVDX_AG_T(float, HVDX_TILE_U32);
  else if (tensor_dtype == HVDX_FLOAT32) HVDX_AG_T(float, HVDX_TILE_U16);
  else HVDX_AG_T(_Float16, HVDX_TILE_UH);
#undef HVDX_AG_T
  return hipGetLastError();
}

hipError_t launch_bcast_tensors_step(const BcastTensorsArgs& a, hipStream_t stream) {
  const int64_t tile = (int64_t)BcastCfg::kTileVecs * 16;
  const int64_t longest = (a.q + (a.rem ? 1 : 0)) * 16;  // bytes of the longest chunk
  int64_t bx = (longest + tile - 1) / tile;
  if (bx < 1) bx = 1;
  if (bx > 0x7fffffff) return hipErrorInvalidValue;  // one tile per block: no block may be dropped
  HVDX_LAUNCH(bcast_tensors_step_kernel, dim3((unsigned)bx, (unsigned)(a.n - 1)), dim3(BcastCfg::BS), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_unpack(const RankPtrs& bufs, int64_t count, int buf_dtype, void* const* dsts,
                         const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                         bool ring, hipStream_t stream) {
  if (buf_dtype == HVDX_FLOAT32) {
    if (ring)
      unpack_with<UnpackCfg, true>(bufs, count, buf_dtype, dsts, numel, offset, ntensors, dst_dtype, nranks, stream);
    else
      unpack_with<UnpackCfg, false>(bufs, count, buf_dtype, dsts, numel, offset, ntensors, dst_dtype, nranks, stream);
  } else {
    if (ring)
      unpack_with<Unpack16Cfg, true>(bufs, count, buf_dtype, dsts, numel, offset, ntensors, dst_dtype, nranks,
                                     stream);
    else
      unpack_with<Unpack16Cfg, false>(bufs, count, buf_dtype, dsts, numel, offset, ntensors, dst_dtype, nranks,
                                      stream);
  }
  return hipGetLastError();
}

}  // namespace hvdx
