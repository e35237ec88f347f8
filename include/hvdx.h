/*
 * hvdx -- the data-parallel hot path of Horovod (Sergeev & Del Balso, "Horovod:
 * fast and easy distributed deep learning in TensorFlow", 2018) for AMD MI355X.
 *
 * The library averages N workers' gradient tensors with Tensor Fusion (paper
 * section 7) and the ring-allreduce (paper section 3).  The N ranks' buffers live
 * side by side in one GPU's memory and every rank's per-step work runs there; a
 * ring step is one kernel that performs all N ranks' transfers of that step.
 *
 * Conventions for every entry point
 *   - "device" pointers address GPU memory, "host" pointers CPU memory.  Arrays
 *     of device pointers are host arrays unless the comment says "device array".
 *   - The caller owns all memory.  The library allocates and frees nothing.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Launches are
 *     asynchronous and ordered on that stream; calls return before the GPU work
 *     is done.  Faults inside kernels surface at the caller's next stream sync.
 *   - Arguments are checked before anything is launched.  A negative return
 *     value is an error code (HVDX_ERR_*); nothing has been enqueued then.
 *     hvdx_last_error() gives a message for the calling thread's last error.
 *   - Entry points keep no state between calls; concurrent calls on different
 *     streams are safe when they touch disjoint memory.
 */
#ifndef HVDX_H
#define HVDX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HVDX_VERSION 1

/* element types */
#define HVDX_FLOAT32 0
#define HVDX_FLOAT16 1

/* reduction: SUM, or AVERAGE = SUM divided by nranks (paper section 3, the step of
 * the data-parallel recipe that averages the gradients; section 5, the optimizer
 * wrapper that averages gradients) */
#define HVDX_SUM 0
#define HVDX_AVERAGE 1

/* compression of the values that travel around the ring */
#define HVDX_COMPRESS_NONE 0
#define HVDX_COMPRESS_FP16 1

/* status codes */
#define HVDX_OK 0
#define HVDX_ERR_INVALID (-1)     /* null pointer, bad size, bad enum value */
#define HVDX_ERR_ALIAS (-2)       /* rank buffers or workspace overlap */
#define HVDX_ERR_WORKSPACE (-3)   /* workspace missing or too small */
#define HVDX_ERR_HIP (-4)         /* a HIP call failed; see hvdx_last_error() */
#define HVDX_ERR_UNSUPPORTED (-5) /* valid request this build does not handle */

#define HVDX_MAX_RANKS 128                          /* simulated ranks per call */
#define HVDX_DEFAULT_FUSION_THRESHOLD (64LL << 20)  /* bytes (paper section 7: 64 MB) */
#define HVDX_DEFAULT_FUSION_ALIGN 16                /* bytes */

/* ring phases for hvdx_ring_step */
#define HVDX_PHASE_REDUCE_SCATTER 0
#define HVDX_PHASE_ALLGATHER 1

/*
 * hvdx_fuse_plan -- group tensors into fusion buffers (paper section 7, steps 1,
 * 2 and 6: a leading run of the ready tensors whose total fits the buffer forms
 * one buffer, and so on until every tensor has one).  Host only; touches no GPU
 * state.
 *
 *   numel[ntensors]        host, elements of each tensor in ready order (>= 0)
 *   buf_dtype              HVDX_FLOAT32 or HVDX_FLOAT16: element type of the
 *                          buffer; sizes are counted in its bytes
 *   threshold_bytes        buffer capacity (>= 0); HVDX_DEFAULT_FUSION_THRESHOLD
 *   align_bytes            each tensor starts at a multiple of this many bytes;
 *                          a power of two, at least the element size
 *   bucket_of[ntensors]    out, host: buffer index of each tensor
 *   offset[ntensors]       out, host: element offset of each tensor in its buffer
 *   bucket_count[ntensors] out, host: element count of each buffer (only the
 *                          first *nbuckets entries are written)
 *   bucket_direct[ntensors] out, host: 1 if the buffer is a single tensor larger
 *                          than threshold_bytes, reduced in place without a copy
 *   nbuckets               out, host: number of buffers
 *
 * Buffers take a contiguous run of the list; a tensor fits while the aligned
 * end of the run stays <= threshold_bytes (equality fits).  Gaps before aligned
 * offsets are padding.  A buffer's count is the end of its last tensor.
 * Errors: HVDX_ERR_INVALID for a null pointer, ntensors < 0, a negative numel,
 * an unknown dtype, or a bad threshold/alignment.
 */
int hvdx_fuse_plan(const int64_t* numel, int ntensors, int buf_dtype, int64_t threshold_bytes,
                   int64_t align_bytes, int32_t* bucket_of, int64_t* offset, int64_t* bucket_count,
                   int32_t* bucket_direct, int32_t* nbuckets);

/*
 * hvdx_fuse_pack -- copy every rank's tensors into its fusion buffer (paper
 * section 7, step 3), one launch for all ranks and tensors.  Padding positions are
 * written with zero.  With src_dtype FLOAT32 and buf_dtype FLOAT16 each value is
 * rounded to nearest even (gradual underflow, overflow to infinity); FLOAT16 to
 * FLOAT32 is exact.
 *
 *   srcs[nranks*ntensors]  DEVICE array of device pointers, rank-major
 *                          (entry r*ntensors + t is rank r's tensor t), each
 *                          numel[t] elements of src_dtype
 *   numel[ntensors]        DEVICE array of int64, elements per tensor
 *   offset[ntensors]       DEVICE array of int64, element offsets in the buffer,
 *                          ascending, with offset[t] + numel[t] <= offset[t+1]
 *                          and <= buf_count (as produced by hvdx_fuse_plan)
 *   bufs[nranks]           host array of device pointers, each buf_count
 *                          elements of buf_dtype; must not overlap
 *   nranks                 1 .. HVDX_MAX_RANKS
 *
 * Every buffer element [0, buf_count) is written exactly once; tensor t of rank
 * r is read only at [0, numel[t]).  Descriptor contents are the caller's
 * responsibility (they are device data and are not checked).
 * Errors: HVDX_ERR_INVALID (null pointers, sizes, dtypes), HVDX_ERR_ALIAS
 * (overlapping buffers), HVDX_ERR_HIP (launch failure).
 */
int hvdx_fuse_pack(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                   int src_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks,
                   void* stream);

/*
 * hvdx_fuse_unpack -- copy every rank's reduced buffer out to its tensors (paper
 * section 7, step 5), one launch for all ranks and tensors.  Padding is not
 * copied.  Conversions as in hvdx_fuse_pack.
 *
 *   bufs[nranks]           host array of device pointers (buf_count of buf_dtype)
 *   dsts[nranks*ntensors]  DEVICE array of device pointers, rank-major, each
 *                          numel[t] elements of dst_dtype; written only at
 *                          [0, numel[t])
 *   numel, offset          DEVICE arrays as for hvdx_fuse_pack
 * Errors: as hvdx_fuse_pack.
 */
int hvdx_fuse_unpack(const void* const* bufs, int64_t buf_count, int buf_dtype, void* const* dsts,
                     const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                     void* stream);

/*
 * hvdx_fuse_pack_rs -- hvdx_fuse_pack and the ring's adding step 0 (paper section 3,
 * the first iteration whose received values are added) in one launch: the buffers
 * end exactly as hvdx_fuse_pack followed by hvdx_ring_step(REDUCE_SCATTER, step 0)
 * on buf_dtype leaves them (chunk c of rank c+1 holds rank c+1's packed values
 * plus rank c's, added in buf_dtype), without reading any buffer back.  Needs
 * nranks >= 3, so that step 0 is not the step that divides for AVERAGE.
 * Arguments as hvdx_fuse_pack.
 * Errors: as hvdx_fuse_pack; HVDX_ERR_UNSUPPORTED for nranks < 3.
 */
int hvdx_fuse_pack_rs(const void* const* srcs, const int64_t* numel, const int64_t* offset, int ntensors,
                      int src_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks, void* stream);

/*
 * hvdx_fuse_ag_unpack -- the ring's last replacing step (step N-2) and
 * hvdx_fuse_unpack in one launch: every tensor receives what hvdx_ring_step
 * (ALLGATHER, step N-2) followed by hvdx_fuse_unpack would give it.  In chunk c
 * that step hands rank c-3's values to rank c-2 (mod N); here rank c-2 copies them
 * out of rank c-3's buffer directly, so rank c-2's buffer keeps that chunk's
 * previous contents (the buffers are left as before the step).  Needs
 * nranks >= 3 (for fewer ranks the last replacing step is step 0).
 * Arguments as hvdx_fuse_unpack.
 * Errors: as hvdx_fuse_unpack; HVDX_ERR_UNSUPPORTED for nranks < 3.
 */
int hvdx_fuse_ag_unpack(const void* const* bufs, int64_t buf_count, int buf_dtype, void* const* dsts,
                        const int64_t* numel, const int64_t* offset, int ntensors, int dst_dtype, int nranks,
                        void* stream);

/*
 * hvdx_fuse_allreduce -- one fusion buffer's whole cycle (paper section 7, steps 3
 * to 5, around the ring-allreduce of section 3), in place on the tensors: their
 * values end exactly as hvdx_fuse_pack, hvdx_ring_allreduce (buf_dtype, no
 * compression) and hvdx_fuse_unpack would leave them.  For nranks >= 3 it launches
 * the copy-in fused with adding step 0 (as hvdx_fuse_pack_rs, except that no rank
 * stores its copy of the chunk it sends in that step: nothing reads it before
 * replacing step 0 overwrites it), adding steps 1..N-3, the fused adding step N-2 /
 * replacing step 0, replacing steps 1..N-3, and hvdx_fuse_ag_unpack: 2N-3 launches
 * and five buffer passes fewer than the separate calls.  For nranks <= 2 it makes
 * the separate calls.  The fusion buffers are scratch: their contents afterwards
 * are unspecified.
 *
 *   tensors[nranks*ntensors]  DEVICE array of device pointers, rank-major, read
 *                             and then written at [0, numel[t]), tensor_dtype
 *   numel, offset, bufs       as for hvdx_fuse_pack; tensors must not overlap bufs
 *                             (not checked: the table is device data)
 *   op                        HVDX_SUM or HVDX_AVERAGE
 * Errors: as hvdx_fuse_pack, and HVDX_ERR_INVALID for an unknown op.
 */
int hvdx_fuse_allreduce(void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                        int tensor_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks, int op,
                        void* stream);

/*
 * hvdx_fuse_allreduce_pair -- two fusion buffers' whole cycles (paper section 7,
 * steps 3 to 5, for two buffers of one call) with each launch serving both buffers:
 * the copy-ins fused with adding step 0, adding steps 1..N-3, the fused adding step
 * N-2 / replacing step 0, replacing steps 1..N-3, and replacing step N-2 fused with
 * the copy-outs: 2N-3 launches instead of 2(2N-3).  The tensors end exactly as after
 * hvdx_fuse_allreduce on b0 and then on b1 (the two rings share no data, and each
 * element's additions keep its own ring's order).  For callers with several fusion
 * buffers ready at once; each buffer keeps its own plan and its own fusion buffers.
 *
 *   b0, b1         host pointers to bucket descriptors (fields as the arguments of
 *                  hvdx_fuse_allreduce: tensors, numel, offset, ntensors, bufs,
 *                  buf_count)
 *   tensor_dtype, buf_dtype, nranks, op   shared by both buckets
 * All 2*nranks fusion buffers must be pairwise disjoint (checked); the buckets'
 * tensors must be disjoint from each other and from every fusion buffer (not
 * checked: device data).
 * Errors: as hvdx_fuse_allreduce for each bucket; HVDX_ERR_INVALID for a NULL
 * descriptor, HVDX_ERR_ALIAS when fusion buffers of the two buckets overlap,
 * HVDX_ERR_UNSUPPORTED for nranks < 3.  A bucket with buf_count 0 is skipped (the
 * other runs as hvdx_fuse_allreduce).
 */
typedef struct hvdx_bucket {
  void* const* tensors;   /* DEVICE array [nranks*ntensors] of device pointers */
  const int64_t* numel;   /* DEVICE array [ntensors] */
  const int64_t* offset;  /* DEVICE array [ntensors] */
  int ntensors;
  void* const* bufs;      /* host array [nranks] of device pointers, buf_count elements each */
  int64_t buf_count;
} hvdx_bucket;

int hvdx_fuse_allreduce_pair(const hvdx_bucket* b0, const hvdx_bucket* b1, int tensor_dtype, int buf_dtype,
                             int nranks, int op, void* stream);

/*
 * Tile tables for the fused copies (paper section 7, steps 3 and 5, fused with the
 * ring's first and last step as in hvdx_fuse_allreduce).  A fusion buffer's copy can be
 * cut, once, into tiles that each lie inside one tensor (or one run of padding) and one
 * ring chunk; a kernel then needs no search for the tensors of its stretch of the buffer:
 * each block reads its tile and moves it for one rank, one 16-byte vector per lane.
 *
 * hvdx_fuse_copy_tiles -- host only, pure: the tiles of one direction for a buffer
 * described as for hvdx_fuse_allreduce (numel, offset: HOST arrays here).
 *   direction  HVDX_COPY_IN: every buffer position, padding included, cut at tensor
 *              ends, chunk ends and multiples of the tile length in buffer positions (the
 *              copy-in writes the buffer: its stores start on the buffer's tile bounds);
 *              HVDX_COPY_OUT: every tensor element, cut at tensor ends, chunk ends and
 *              multiples of the tile length inside each tensor (the copy-out writes the
 *              tensors: its stores start on the tensors' own tile bounds).  After a chunk
 *              boundary that is not on a vector boundary, a short tile reaches the next one.
 *   tiles      host array of `capacity` entries, or NULL to count them
 * Returns the number of tiles (written when tiles is not NULL and capacity suffices),
 * or a negative HVDX_ERR_* (HVDX_ERR_WORKSPACE when capacity is too small).  A tile holds
 * at most hvdx_fuse_tile_elems(tensor_dtype, buf_dtype) elements: what one 256-thread
 * block moves (1024 for binary32 buffers, 2048 for binary16 buffers).
 */
#define HVDX_COPY_IN 0
#define HVDX_COPY_OUT 1
typedef struct hvdx_copy_tile {
  int64_t pos;     /* buffer position of the tile's first element */
  int64_t li;      /* that element's index in its tensor (0 for padding) */
  int32_t tensor;  /* tensor index, -1 for a run of padding (HVDX_COPY_IN only) */
  int32_t len;     /* elements in the tile, 1 .. hvdx_fuse_tile_elems(...) */
  int32_t chunk;   /* ring chunk holding every element of the tile */
  int32_t reserved;
} hvdx_copy_tile;
int64_t hvdx_fuse_copy_tiles(const int64_t* numel, const int64_t* offset, int ntensors, int64_t buf_count,
                             int tensor_dtype, int buf_dtype, int nranks, int direction, hvdx_copy_tile* tiles,
                             int64_t capacity);
/* The most elements a tile holds for these types (0 for an unsupported pair). */
int64_t hvdx_fuse_tile_elems(int tensor_dtype, int buf_dtype);

/*
 * hvdx_fuse_allreduce_tiled -- the Tensor Fusion cycle of 1 to HVDX_TILED_MAX_BUCKETS
 * fusion buffers, every launch serving all of them, with the fused copies driven by tile
 * tables: the same result, bit for bit, as hvdx_fuse_allreduce on each bucket.
 *   buckets[nbuckets]  host array of bucket descriptors, each as for
 *                      hvdx_fuse_allreduce_pair, plus
 *     in_tiles         DEVICE array of n_in tiles from hvdx_fuse_copy_tiles(HVDX_COPY_IN)
 *     out_tiles        DEVICE array of n_out tiles from hvdx_fuse_copy_tiles(HVDX_COPY_OUT)
 *                      for exactly this bucket (numel, offset, buf_count, both types and
 *                      nranks): the tables are device memory and are not checked; other
 *                      tables make the kernels read or write outside the buffers and
 *                      tensors.  All buckets' fusion buffers must be pairwise disjoint
 *                      (checked), and every rank's tensors of all buckets disjoint from one
 *                      another and from the buffers (not checked: the tables are device
 *                      memory; overlapping tensors give results that depend on block order).
 *                      More than two buckets (with something to reduce) need both tensor
 *                      flags; with HVDX_TILED_REPLACE_IN_TENSORS, buckets x nranks <= 256.
 *   flags              0 (HVDX_TILED_BUFFERS): the fusion buffers as in paper section 7 --
 *                      the copy-in fused with adding step 0, the ring in the buffers
 *                      (step 4), the copy-out fused with the last replacing step (step 5);
 *                      the same launches as the untiled calls, and the fusion buffers end
 *                      holding the result.  Or a combination of:
 *     HVDX_TILED_REPLACE_IN_TENSORS  the replacing steps (paper section 3) store the chunk
 *                      each one delivers in the receiver's output tensors, from which the
 *                      next step forwards it (the finished sum goes from adding step N-2 to
 *                      the owner's and the next rank's tensors): no copy-out;
 *     HVDX_TILED_ADD_FROM_TENSORS  (with REPLACE_IN_TENSORS) each adding step reads the
 *                      receiver's own elements of its chunk from its tensors (and in step 0
 *                      the sender's too), where the copy-in would have put them: no copy-in;
 *                      the buffers then only ever hold received partial sums.
 *                      Every message of the ring moves in its order with either flag, and
 *                      with either the fusion buffers are scratch afterwards.  With binary32
 *                      tensors and binary16 buffers (compression) these are the compressed
 *                      ring's steps: elements rounded to binary16 where first read, binary16
 *                      partial sums, and replacing steps that copy the binary32 values
 *                      holding the binary16 results exactly (twice the binary16 width).
 * Errors as hvdx_fuse_allreduce_pair, HVDX_ERR_INVALID for a missing table, a negative
 * tile count, an unknown flag or a bucket count out of range, HVDX_ERR_UNSUPPORTED for
 * more buckets than the flags allow.
 */
#define HVDX_TILED_MAX_BUCKETS 4
#define HVDX_TILED_BUFFERS 0
#define HVDX_TILED_REPLACE_IN_TENSORS 1
#define HVDX_TILED_ADD_FROM_TENSORS 2
typedef struct hvdx_tiled_bucket {
  hvdx_bucket b;
  const hvdx_copy_tile* in_tiles;
  int64_t n_in;
  const hvdx_copy_tile* out_tiles;
  int64_t n_out;
} hvdx_tiled_bucket;
int hvdx_fuse_allreduce_tiled(const hvdx_tiled_bucket* buckets, int nbuckets, int tensor_dtype, int buf_dtype,
                              int nranks, int op, int flags, void* stream);

/*
 * hvdx_fuse_allreduce_small -- hvdx_fuse_allreduce for small fusion buffers: the same
 * result, bit for bit, in one kernel launch instead of 2N-1.  Each thread takes a
 * 16-byte stretch of the buffer (element by element where it meets a tensor edge)
 * through the copy-in for every rank (paper section 7, step 3), all 2(N-1) steps of
 * the ring of paper section 3 in their order -- each step reading the sender's
 * buffer and writing the receiver's -- and the copy-out (step 5).  An element's ring
 * never involves another element, so its steps need not wait for the rest of the
 * buffer.  Intended for buffers of at most HVDX_SMALL_BUCKET_BYTES per rank, where
 * the per-step launches cost more than their data; any size works.
 * Arguments, ownership and errors as hvdx_fuse_allreduce (any nranks >= 1); the
 * fusion buffers are scratch afterwards (padding is not written).
 */
int hvdx_fuse_allreduce_small(void* const* tensors, const int64_t* numel, const int64_t* offset, int ntensors,
                              int tensor_dtype, void* const* bufs, int64_t buf_count, int buf_dtype, int nranks,
                              int op, void* stream);

/* Per-rank buffer bytes at or below which a fusion buffer's (or a tensor's) whole ring
 * costs less in one launch (hvdx_fuse_allreduce_small, hvdx_ring_allreduce_small) than
 * in one launch per step on MI355X: below it a step's messages take less time than
 * launching the step.  A recommendation for callers; the library does not switch. */
#define HVDX_SMALL_BUCKET_BYTES (4 << 20)

/*
 * hvdx_ring_allreduce -- the ring-allreduce of paper section 3: N-1 steps in which
 * every rank adds the chunk received from its left neighbour into its own buffer,
 * then N-1 steps in which the received chunk replaces its own.  In place on all
 * nranks buffers; afterwards every buffer holds the same result.
 *
 *   bufs[nranks]     host array of device pointers, each count elements of
 *                    dtype, pairwise non-overlapping
 *   count            elements per rank buffer (>= 0; 0 is a no-op)
 *   dtype            HVDX_FLOAT32 or HVDX_FLOAT16
 *   op               HVDX_SUM or HVDX_AVERAGE
 *   compress         HVDX_COMPRESS_NONE, or HVDX_COMPRESS_FP16 (dtype FLOAT32
 *                    only): values are rounded to binary16 when first sent,
 *                    added and averaged in binary16, and widened back into the
 *                    binary32 buffers by the replacing steps (the first one
 *                    widens the owner's binary16 result; the later ones forward
 *                    it as the binary32 value that holds it exactly)
 *   workspace        device memory of at least hvdx_ring_workspace_bytes(...)
 *                    bytes, 256-byte aligned, disjoint from bufs; only used with
 *                    compression (may be NULL otherwise); contents afterwards
 *                    are unspecified
 *
 * Schedule: chunk c (of N near-equal contiguous chunks, the first count mod N
 * one element longer) moves from rank (c+s) mod N to (c+s+1) mod N in adding
 * step s and from rank (c-1+s) mod N to (c+s) mod N in replacing step s, so the
 * sum of chunk c is formed in ring order starting at rank c.  (Adding step N-2
 * and replacing step 0 run as one kernel here; the buffers end the same.)  Each addition is
 * rounded to nearest even in dtype (binary16 when compressed); AVERAGE divides
 * the complete sum by nranks once, correctly rounded, at the last adding step.
 * Errors: HVDX_ERR_INVALID, HVDX_ERR_ALIAS, HVDX_ERR_WORKSPACE, HVDX_ERR_HIP.
 */
int hvdx_ring_allreduce(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * hvdx_ring_allreduce_small -- hvdx_ring_allreduce without compression, in one
 * launch: each thread runs all 2(N-1) steps (same schedule, same order of additions,
 * each step reading the sender's buffer and writing the receiver's) for one 16-byte
 * vector of every rank buffer, or element by element where a vector crosses a chunk
 * edge or a buffer is not 16-byte aligned.  Same result, bit for bit.  Intended for
 * buffers of at most HVDX_SMALL_BUCKET_BYTES; any size works.
 * Arguments and errors as hvdx_ring_allreduce with compress = HVDX_COMPRESS_NONE.
 */
int hvdx_ring_allreduce_small(void* const* bufs, int nranks, int64_t count, int dtype, int op, void* stream);

/*
 * hvdx_ring_allreduce_noalloc -- hvdx_ring_allreduce for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same kernels, the same result bit for bit, but the
 * compression workspace is a static array inside the library instead of an argument.
 * The call allocates nothing (no hipMalloc, hipFree or allocating library routine).
 *
 *   bufs, nranks, count, dtype, op, compress, stream   as hvdx_ring_allreduce
 *
 * Limit: hvdx_ring_workspace_bytes(nranks, count, dtype, compress) must not exceed
 * hvdx_ring_noalloc_max_bytes() (64 MiB: e.g. 8 ranks of up to 4,194,304 binary32
 * elements compressed); larger requests return HVDX_ERR_WORKSPACE before any HIP
 * call.  Without compression no workspace is used and any size works.
 * The static array is held by every GPU the library runs on until the process ends;
 * its device address is looked up on the first call per device (the stream's device,
 * or the current device for the null stream).  Nothing in it needs to start at zero
 * (every wire element a step reads was written by an earlier step of the same call),
 * and it keeps the last call's contents.  All calls on one GPU share the array:
 * calls that overlap in time on one GPU (on different streams, or from different
 * threads) race; serialize them on one stream.
 * Errors: as hvdx_ring_allreduce; HVDX_ERR_WORKSPACE beyond the limit;
 * HVDX_ERR_UNSUPPORTED on a device index of 64 or more.
 */
int hvdx_ring_allreduce_noalloc(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                                void* stream);
/* Bytes of the static compression workspace behind hvdx_ring_allreduce_noalloc. */
size_t hvdx_ring_noalloc_max_bytes(void);

/*
 * hvdx_ring_reduce_scatter / hvdx_ring_allgather -- the two halves of
 * hvdx_ring_allreduce (paper section 3: the N-1 adding iterations, then the N-1
 * replacing iterations), each one call.  Running the first and then the second
 * with the same arguments and workspace is hvdx_ring_allreduce.
 *
 * After the reduce-scatter half, rank (c-1) mod N holds chunk c of the reduced
 * result (with AVERAGE already divided) -- in its buffer, or, when compressing,
 * in its binary16 wire copy inside `workspace`, which the all-gather half then
 * needs unchanged.  The other chunks of every rank hold intermediate values.
 * The all-gather half copies each such chunk around the ring so every rank ends
 * with all of them; used on its own (no compression) it gathers rank r's chunk
 * (r+1) mod N into every rank.  With nranks = 1 both are no-ops, except that the
 * compressed reduce-scatter rounds the buffer through binary16.
 * Arguments and errors as hvdx_ring_allreduce.
 */
int hvdx_ring_reduce_scatter(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                             void* workspace, size_t workspace_bytes, void* stream);
int hvdx_ring_allgather(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * hvdx_ring_step -- one step of hvdx_ring_allreduce (all N transfers of adding or
 * replacing step `step`, 0 <= step < nranks-1), for tracing and for checking
 * intermediate states.  Running phase REDUCE_SCATTER steps 0..N-2 then
 * ALLGATHER steps 0..N-2 in order, with the same arguments and workspace, is
 * hvdx_ring_allreduce for nranks >= 2.  Arguments as hvdx_ring_allreduce.
 */
int hvdx_ring_step(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, int phase,
                   int step, void* workspace, size_t workspace_bytes, void* stream);

/*
 * hvdx_broadcast -- copy rank `root`'s buffer into every other rank's buffer (paper
 * section 4, the broadcast that gives every worker the same initial model;
 * section 5, broadcasting the variables from the first process to all others).
 * The bytes travel as a pipelined chain along the ring: the buffer is cut into N
 * chunks of whole 16-byte units (the first (units mod N) chunks one unit longer;
 * the last unit may be short), and in step s rank root+k forwards chunk s-k to rank
 * root+k+1 (k = 0..N-2, when 0 <= s-k < N): 2N-2 steps.  Bytes are copied, not
 * interpreted, so any element type works.
 *
 *   bufs[nranks]  host array of device pointers, each nbytes long, pairwise
 *                 non-overlapping (16-byte alignment of all of them enables the
 *                 vector path)
 *   nbytes        >= 0 (0 is a no-op); root in 0..nranks-1
 * hvdx_broadcast_step runs step `step` (0 <= step < 2*nranks-2) alone.
 * Errors: HVDX_ERR_INVALID, HVDX_ERR_ALIAS, HVDX_ERR_HIP.
 */
int hvdx_broadcast(void* const* bufs, int nranks, int64_t nbytes, int root, void* stream);
int hvdx_broadcast_step(void* const* bufs, int nranks, int64_t nbytes, int root, int step, void* stream);

/*
 * hvdx_broadcast_tensors -- hvdx_broadcast for many tensors in one call (paper
 * sections 4 and 5: every variable broadcast from the root at start-up), 2N-2 launches
 * in all instead of 2N-2 per tensor.  The tensors are laid end to end in a virtual
 * byte space, tensor t at [voffset[t], voffset[t] + nbytes[t]), and the chain of
 * hvdx_broadcast runs over that space as over one buffer of total_bytes bytes: chunk j
 * is the j-th run of whole 16-byte units, and in step s rank root+k forwards chunk s-k
 * to rank root+k+1.  Bytes of the space that belong to no tensor are not moved.  Every
 * rank ends with the root's bytes of every tensor.
 *
 *   ptrs[nranks*ntensors]  DEVICE array of tensor pointers, rank-major (rank r's tensor t
 *                          at r*ntensors + t); the tensors must not overlap (not
 *                          checked: the table is in device memory); 16-byte aligned
 *                          copies move as vectors, others byte by byte
 *   nbytes[ntensors]       DEVICE array, bytes of each tensor (>= 0)
 *   voffset[ntensors]      DEVICE array, ascending multiples of 16 with
 *                          voffset[t] >= voffset[t-1] + nbytes[t-1]
 *   total_bytes            >= voffset[T-1] + nbytes[T-1]; 0 (or ntensors 0) is a no-op
 *   root                   0..nranks-1
 * hvdx_broadcast_layout (host) computes the densest layout: each tensor at the first
 * multiple of 16 at or after the previous one's end; total_bytes = the last one's end.
 * hvdx_broadcast_tensors_step runs step `step` (0 <= step < 2*nranks-2) alone.
 * Errors: HVDX_ERR_INVALID (host-side arguments), HVDX_ERR_HIP.
 */
int hvdx_broadcast_layout(const int64_t* nbytes, int ntensors, int64_t* voffset, int64_t* total_bytes);
int hvdx_broadcast_tensors(const void* const* ptrs, const int64_t* nbytes, const int64_t* voffset, int ntensors,
                           int64_t total_bytes, int nranks, int root, void* stream);
int hvdx_broadcast_tensors_step(const void* const* ptrs, const int64_t* nbytes, const int64_t* voffset, int ntensors,
                                int64_t total_bytes, int nranks, int root, int step, void* stream);

/*
 * hvdx_fold_allreduce -- the same result as hvdx_ring_allreduce, bit for bit,
 * computed without the ring's messages: each element's N values are read once and
 * added in the ring's order (starting at the rank whose chunk holds the element,
 * paper section 3), divided once for AVERAGE, and written to all N buffers.  It
 * moves 2N elements per element instead of the ring's 5(N-1), so it bounds what a
 * one-GPU schedule can do; it is not a simulation of the ring's transport.
 * Arguments as hvdx_ring_allreduce; compression needs no workspace here.
 */
int hvdx_fold_allreduce(void* const* bufs, int nranks, int64_t count, int dtype, int op, int compress, void* stream);

/* Workspace bytes hvdx_ring_allreduce needs: 0 unless compressing binary32 data,
 * then nranks * (count rounded up to 128) * 2.  Host only. */
size_t hvdx_ring_workspace_bytes(int nranks, int64_t count, int dtype, int compress);

/* Chunk c of the ring partition of `count` elements over `nranks` ranks:
 * start = c*q + min(c, r), len = q + (c < r) with q, r = count / nranks,
 * count % nranks.  Host only.  HVDX_ERR_INVALID for bad arguments. */
int hvdx_ring_chunk(int64_t count, int nranks, int c, int64_t* start, int64_t* len);

/*
 * Timeline (paper section 6: a per-node record of what the collective did at each
 * step, viewable in Chrome's about:tracing).  Between hvdx_timeline_begin and
 * hvdx_timeline_end the library brackets its kernel launches, from any thread and
 * on any stream, with pairs of HIP events it owns; no device memory is allocated.
 *
 *   hvdx_timeline_begin(capacity, per_phase)  start recording up to `capacity`
 *       (>= 1) records; records past that are counted as dropped.  per_phase = 0
 *       records every launch, its events stamped by the kernel's own dispatch
 *       (hipExtLaunchKernel), so a record's duration is the kernel's run time;
 *       per_phase = 1 records each run of launches of one kernel inside one call
 *       (e.g. the N-2 plain adding steps of a ring) as one record whose `launches`
 *       says how many, with event records in the stream around the run.  Either
 *       way the records cost GPU time (a few microseconds per launch or per run).
 *       Returns HVDX_ERR_INVALID if a
 *       timeline is already recording or capacity < 1, HVDX_ERR_HIP if the events
 *       cannot be created.
 *   hvdx_timeline_end(out, capacity, nrecords, ndropped)  wait for the recorded
 *       work to finish, write up to `capacity` records to the host array `out` in
 *       launch order, set *nrecords and *ndropped, stop recording and release the
 *       events.  Times are microseconds from the start of the first record.
 *       HVDX_ERR_INVALID if no timeline is recording.  Call it when no other
 *       thread is launching library work.
 */
#define HVDX_KERNEL_PACK 0
#define HVDX_KERNEL_REDUCE_SCATTER 1
#define HVDX_KERNEL_ALLGATHER 2
#define HVDX_KERNEL_UNPACK 3
#define HVDX_KERNEL_ROUNDTRIP 4 /* one-rank compressed ring: round to binary16 and back */
#define HVDX_KERNEL_BROADCAST 5 /* one step of hvdx_broadcast */
#define HVDX_KERNEL_RS_AG 6     /* last adding step and first replacing step in one launch */
#define HVDX_KERNEL_FOLD 7      /* hvdx_fold_allreduce */
#define HVDX_KERNEL_PACK_RS 8   /* copy-in with adding step 0 (step = 0) */
#define HVDX_KERNEL_AG_UNPACK 9 /* replacing step N-2 with copy-out (step = N-2) */
#define HVDX_KERNEL_RING_SMALL 10  /* hvdx_ring_allreduce_small: every step in one launch */
#define HVDX_KERNEL_CYCLE_SMALL 11 /* hvdx_fuse_allreduce_small: copy-in, ring, copy-out in one launch */

typedef struct hvdx_trace_record {
  int32_t kind;     /* HVDX_KERNEL_* */
  int32_t step;     /* first ring or broadcast step of the record, else -1 */
  int32_t launches; /* kernel launches the record covers */
  int32_t nranks;
  int32_t dtype;    /* buffer element type (-1 for a broadcast, which copies bytes) */
  int32_t compress; /* HVDX_COMPRESS_* of the ring */
  int32_t root;     /* broadcast root, else -1 */
  int32_t reserved;
  int64_t count;    /* buffer elements per rank (bytes for a broadcast) */
  double start_us;
  double duration_us;
} hvdx_trace_record;

int hvdx_timeline_begin(int capacity, int per_phase);
int hvdx_timeline_end(hvdx_trace_record* out, int capacity, int* nrecords, int* ndropped);

/* Text for a status code (static storage). */
const char* hvdx_strerror(int status);

/* Detail of the calling thread's last failed call ("" if none). */
const char* hvdx_last_error(void);

/* HVDX_VERSION of the built library. */
int hvdx_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HVDX_H */
