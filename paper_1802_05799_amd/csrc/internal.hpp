// Internal declarations shared by the library's translation units (not installed).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "hvdx.h"

namespace hvdx {

// Events that a timeline record hands to this thread's next kernel launch, which then
// runs through hipExtLaunchKernel: the dispatch itself stamps them with the kernel's
// start and end, with no extra commands in the stream.  Empty when nothing waits.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& pending_launch_events();

// Every rank's base pointer travels in the kernel arguments (1 KiB).
struct RankPtrs {
  void* p[HVDX_MAX_RANKS];
};

// Ring partition and step, identical for every block of one launch.
struct RingArgs {
  int n;          // ranks
  int step;       // 0 .. n-2
  int64_t q;      // count / n
  int64_t rem;    // count % n
  float nf;       // (float) n
  float inv;      // 1 / n, used only when n is a power of two
  int64_t wire_stride;  // elements per rank in the fp16 wire workspace
};

// The same step of two rings (two fusion buffers of one call) in one launch.
struct RingPair {
  RankPtrs bufs[2];
  RingArgs a[2];  // same n and step, each ring its own count
};

// The fused copy-in or copy-out of two fusion buffers in one launch.
struct CopyPair {
  void* const* t[2];  // DEVICE tables of tensor pointers, rank-major
  const int64_t* numel[2];
  const int64_t* offset[2];
  int ntensors[2];
  RankPtrs bufs[2];
  int64_t count[2], q[2], rem[2];  // buffer elements and their ring partition
};

// The fused copies of one or two fusion buffers driven by tile tables (hvdx_copy_tile):
// blocks [0, x0) take bucket 0's tiles, the rest bucket 1's.  A tile is at most
// kTileLanes * tile_vectors(...) vectors of tile_vec_elems(...) elements: the host cuts
// the tables and the kernels move them with the same constants.
constexpr int kTileLanes = 256;
#ifndef HVDX_TILE_U32
#define HVDX_TILE_U32 1  // binary32 tensors and buffers
#endif
#ifndef HVDX_TILE_U16  // binary32 tensors, binary16 buffers: one vector per lane.  Two make the copies of
#define HVDX_TILE_U16 1  // the paper's mode 3 points faster; the ring on the tensors is 1% faster with one
#endif
#ifndef HVDX_TILE_UH
#define HVDX_TILE_UH 1  // binary16 tensors and buffers
#endif
inline int tile_vec_elems(int tensor_dtype, int buf_dtype) {
  return tensor_dtype == HVDX_FLOAT32 || buf_dtype == HVDX_FLOAT32 ? 4 : 8;
}
inline int tile_vectors(int tensor_dtype, int buf_dtype) {
  if (tensor_dtype == HVDX_FLOAT32 && buf_dtype == HVDX_FLOAT32) return HVDX_TILE_U32;
  if (tensor_dtype == HVDX_FLOAT32) return HVDX_TILE_U16;
  return HVDX_TILE_UH;
}
struct TiledCopy {
  CopyPair m;  // tensors and buffers of the buckets (the partition fields are not used)
  const hvdx_copy_tile* tiles[2];
  int64_t x0;
};

// How the last adding step finishes an AVERAGE.
enum DivMode { DIV_NONE = 0, DIV_POW2 = 1, DIV_TRUE = 2 };

constexpr int kBlock = 256;

// Launchers (ring_kernels.hip).  Arguments are already validated; return a hipError_t.
hipError_t launch_rs_step(const RankPtrs& bufs, const RingArgs& a, int dtype, int divmode, bool vector_ok,
                          hipStream_t stream);
hipError_t launch_ag_step(const RankPtrs& bufs, const RingArgs& a, int dtype, bool vector_ok, hipStream_t stream);
hipError_t launch_rs_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, int divmode, bool vector_ok,
                              hipStream_t stream);
hipError_t launch_ag_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, bool vector_ok, hipStream_t stream);
hipError_t launch_roundtrip_c16(void* x, int64_t count, hipStream_t stream);
// Adding step N-2 and replacing step 0 in one launch.
hipError_t launch_rs_ag_step(const RankPtrs& bufs, const RingArgs& a, int dtype, int divmode, bool vector_ok,
                             hipStream_t stream);
hipError_t launch_rs_ag_step_c16(const RankPtrs& x, void* wire, const RingArgs& a, int divmode, bool vector_ok,
                                 hipStream_t stream);
// One step of two rings at once (binary32 or binary16 buffers, both 16-byte aligned):
// an adding step, adding step N-2 fused with replacing step 0, a replacing step.
hipError_t launch_rs_step_pair(const RingPair& m, int dtype, int divmode, hipStream_t stream);
hipError_t launch_rs_ag_step_pair(const RingPair& m, int dtype, int divmode, hipStream_t stream);
hipError_t launch_ag_step_pair(const RingPair& m, int dtype, hipStream_t stream);
// The copy-in fused with adding step 0 (no sender storing its own sent chunk), and
// replacing step N-2 fused with the copy-out, for two fusion buffers at once.
hipError_t launch_pack_pair(const CopyPair& m, int src_dtype, int buf_dtype, int nranks, hipStream_t stream);
hipError_t launch_unpack_pair(const CopyPair& m, int buf_dtype, int dst_dtype, int nranks, hipStream_t stream);
// The same two fused copies driven by tile tables, for one or two buckets: `blocks` tiles in
// all, each block one tile and one rank.
hipError_t launch_pack_tiles(const TiledCopy& k, int src_dtype, int buf_dtype, int nranks, int64_t blocks,
                             hipStream_t stream);
hipError_t launch_unpack_tiles(const TiledCopy& k, int buf_dtype, int dst_dtype, int nranks, int64_t blocks,
                               hipStream_t stream);
// The ring on the tensors of one to kRingBuckets fusion buffers, every launch serving
// all of them: the launch's tiles [end[i-1], end[i]) are bucket i's (from tiles[i]),
// bucket i's tensor pointer table is the DEVICE table t[i] (rank-major, ntensors[i] per
// rank), and its rank r fusion buffer is bufs[i * nranks + r].
constexpr int kRingBuckets = 4;
constexpr int kRingBufPtrs = 256;  // nbuckets * nranks at most
struct TiledRing {
  const hvdx_copy_tile* tiles[kRingBuckets];
  int64_t end[kRingBuckets];
  void* const* t[kRingBuckets];
  int64_t ntensors[kRingBuckets];
  int nbuckets;
  int nranks;
  void* bufs[kRingBufPtrs];
};

// Replacing steps that deliver into the tensors, over the copy-out's tiles: adding step
// N-2 with replacing step 0 (own_in_tensors: the owner's value from its tensors), and
// replacing step s between the tensors.
hipError_t launch_rs_ag_tiles(const TiledRing& k, const RingArgs& a, int tensor_dtype, int buf_dtype, int divmode,
                              bool own_in_tensors, hipStream_t stream);
hipError_t launch_ag_tiles(const TiledRing& k, int tensor_dtype, int buf_dtype, int step, hipStream_t stream);
// Adding step s (0 .. N-3) reading every receiver's own values from its tensors (and at
// s = 0 the sender's too), over the copy-in's tiles.
hipError_t launch_add_tiles(const TiledRing& k, int tensor_dtype, int buf_dtype, int step, hipStream_t stream);
// A small ring in one launch: each thread runs every step for its elements.
hipError_t launch_chain(const RankPtrs& bufs, const RingArgs& a, int64_t count, int dtype, int divmode,
                        bool vector_ok, hipStream_t stream);
// A small fusion buffer's copy-in, ring and copy-out in one launch.
hipError_t launch_small_cycle(const void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                              int tensor_dtype, const RankPtrs& bufs, const RingArgs& a, int64_t count, int buf_dtype,
                              int divmode, hipStream_t stream);
// The ring's per-element fold in one pass (same bits, no per-step messages).
hipError_t launch_fold(const RankPtrs& bufs, const RingArgs& a, int64_t count, int dtype, int compress, int divmode,
                       bool vector_ok, hipStream_t stream);

// Broadcast chain step (broadcast_kernels.hip).
struct BcastArgs {
  int n, root, step;
  int64_t nbytes;
  int64_t q, rem;  // 16-byte units per chunk: q, the first rem chunks one more
};
hipError_t launch_bcast_step(const RankPtrs& bufs, const BcastArgs& a, bool vector_ok, hipStream_t stream);

// One chain step of a broadcast of many tensors (fusion_kernels.hip): the chain runs over
// a virtual byte space in which tensor t occupies [voff[t], voff[t] + nbytes[t]).
struct BcastTensorsArgs {
  const void* const* ptrs;  // DEVICE table of tensor pointers, rank-major [n * ntensors]
  const int64_t* nbytes;    // DEVICE [ntensors]
  const int64_t* voff;      // DEVICE [ntensors], ascending multiples of 16, disjoint extents
  int ntensors;
  int n, root, step;
  int64_t total;            // bytes of the virtual space
  int64_t q, rem;           // 16-byte units per chunk: q, the first rem chunks one more
};
hipError_t launch_bcast_tensors_step(const BcastTensorsArgs& a, hipStream_t stream);

// Launchers (fusion_kernels.hip).  With `ring` (nranks >= 3), the copy-in also does
// the ring's adding step 0 (and with `skip_sender` leaves out each chunk's sender's
// own copy, which the fused cycle never reads) and the copy-out its replacing step N-2.
hipError_t launch_pack(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                       int src_dtype, const RankPtrs& bufs, int64_t count, int buf_dtype, int nranks, bool ring,
                       bool skip_sender, hipStream_t stream);
hipError_t launch_unpack(const RankPtrs& bufs, int64_t count, int buf_dtype, void* const* dsts,
                         const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                         bool ring, hipStream_t stream);

}  // namespace hvdx

// Every kernel launch of the library goes through this.
#define HVDX_LAUNCH(kernel, grid, block, shmem, stream, ...)                                                \
  do {                                                                                                      \
    ::hvdx::LaunchEvents& hvdx_ev_ = ::hvdx::pending_launch_events();                                       \
    if (hvdx_ev_.start) {                                                                                   \
      const ::hvdx::LaunchEvents hvdx_take_ = hvdx_ev_;                                                     \
      hvdx_ev_ = ::hvdx::LaunchEvents{};                                                                    \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, hvdx_take_.start, hvdx_take_.stop, 0,       \
                            __VA_ARGS__);                                                                   \
    } else {                                                                                                \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                                  \
    }                                                                                                       \
  } while (0)
