/*
 * Plain C oracle of Horovod's data-parallel hot path: Tensor Fusion plus the
 * ring-allreduce, simulated over N rank buffers in host memory.
 *
 * TEST INFRASTRUCTURE.  Only tests/, the smoke check and bench.py's CPU baseline
 * load this library (through oracle/native.py).  It shares no code with the GPU
 * library.  It computes exactly what the numpy oracle in this package computes,
 * in the same order, and is pinned against it and against the golden files; it
 * exists so that the host can run the method at full workload size, with one
 * thread or with OpenMP threads over the elements of each chunk.
 *
 * What it follows:
 *   - section 7, the six-step list (Tensor Fusion): a leading run of the ready
 *     tensors whose total fits the fusion buffer is copied in, the buffer is
 *     allreduced, the results are copied out, and so on until none is left;
 *   - section 3, the paragraph after the ring-allreduce figure: N-1 iterations in
 *     which a received chunk is added to the local one, then N-1 in which it
 *     replaces it;
 *   - section 5: the optimizer wrapper averages the gradients.
 * The readings where the paper is silent are those of the numpy oracle: rank r
 * sends to r+1; in adding step s chunk c goes from rank (c+s) mod N to
 * (c+s+1) mod N, in replacing step s from (c-1+s) mod N to (c+s) mod N; chunk c
 * starts at c*q + min(c, rem) and holds q+1 elements for c < rem, else q
 * (q, rem = count / N, count % N); the complete sum is divided by N once, in the
 * buffer's precision, at the last adding step; tensors start at byte offsets that
 * are multiples of the alignment, padding is zero; a tensor larger than the
 * threshold is reduced on its own at offset 0; with fp16 compression the buffers
 * hold binary16 and the ring adds and divides in binary16.
 *
 * Build: gcc -O2 -std=c11 -fno-fast-math -ffp-contract=off -fopenmp -shared -fPIC.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_F32 0
#define OR_F16 1
#define OR_SUM 0
#define OR_AVERAGE 1

static char last_error[256];

static int fail(const char* msg) {
  snprintf(last_error, sizeof last_error, "%s", msg);
  return -1;
}

const char* oracle_last_error(void) { return last_error; }

/* ---------------------------------------------------------------------------
 * binary16 <-> binary32, written from the IEEE 754 encodings.
 * ------------------------------------------------------------------------- */

static float bits_to_float(uint32_t u) {
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static uint32_t float_to_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return u;
}

/* Exact widening: every binary16 value is a binary32 value. */
uint32_t oracle_f16_to_f32_bits(uint16_t h) {
  uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
  uint32_t e = (h >> 10) & 0x1fu;
  uint32_t m = h & 0x3ffu;
  if (e == 0x1fu) return sign | 0x7f800000u | (m << 13); /* infinity, NaN (payload kept) */
  if (e == 0) {
    if (m == 0) return sign; /* signed zero */
    /* subnormal: m * 2^-24; shift the leading one up to the implicit position */
    int ue = -14;
    while (!(m & 0x400u)) {
      m <<= 1;
      --ue;
    }
    return sign | ((uint32_t)(ue + 127) << 23) | ((m & 0x3ffu) << 13);
  }
  return sign | ((e - 15 + 127) << 23) | (m << 13);
}

/* Round to the nearest binary16, ties to even; gradual underflow; overflow gives
 * infinity; a NaN stays a NaN (quiet, top payload bits kept). */
uint16_t oracle_f32_bits_to_f16(uint32_t x) {
  uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
  int e = (int)((x >> 23) & 0xffu);
  uint32_t m = x & 0x7fffffu;
  if (e == 0xff) return (uint16_t)(sign | (m ? 0x7e00u | (m >> 13) : 0x7c00u));
  int ue = e - 127; /* unbiased exponent (fp32 subnormals land far below the binary16 range) */
  if (ue >= 16) return (uint16_t)(sign | 0x7c00u);
  if (ue >= -14) {
    /* normal range: keep 10 of the 23 fraction bits, round on the other 13 */
    uint32_t h = ((uint32_t)(ue + 15) << 10) | (m >> 13);
    uint32_t rest = m & 0x1fffu;
    if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) ++h; /* a carry may reach infinity: correct */
    return (uint16_t)(sign | h);
  }
  if (ue < -25) return sign; /* below half the smallest subnormal: rounds to zero */
  /* subnormal range: the value is (m | 2^23) * 2^(ue-23), in units of 2^-24 that is
   * (m | 2^23) >> (-ue - 1) with the shifted-out bits deciding the rounding */
  uint32_t full = m | 0x800000u;
  int shift = -ue - 1; /* 14 .. 24 */
  uint32_t h = full >> shift;
  uint32_t rest = full & ((1u << shift) - 1u);
  uint32_t half = 1u << (shift - 1);
  if (rest > half || (rest == half && (h & 1u))) ++h; /* may become the smallest normal: correct */
  return (uint16_t)(sign | h);
}

static float h2f(uint16_t h) { return bits_to_float(oracle_f16_to_f32_bits(h)); }
static uint16_t f2h(float f) { return oracle_f32_bits_to_f16(float_to_bits(f)); }

/* Bulk forms for the tests. */
void oracle_f32_to_f16_array(const float* src, uint16_t* dst, int64_t n) {
  for (int64_t i = 0; i < n; ++i) dst[i] = f2h(src[i]);
}

void oracle_f16_to_f32_array(const uint16_t* src, float* dst, int64_t n) {
  for (int64_t i = 0; i < n; ++i) dst[i] = h2f(src[i]);
}

/* ---------------------------------------------------------------------------
 * Section 7, steps 1, 2 and 6: which tensors share a fusion buffer.
 * ------------------------------------------------------------------------- */

/* bucket_of[t]: the buffer of tensor t; offset[t]: its element offset there;
 * direct[b]: buffer b is one oversize tensor; count[b]: buffer b's length in
 * elements.  All arrays have room for ntensors entries. */
int oracle_fuse_plan(const int64_t* numel, int ntensors, int esize, int64_t threshold, int64_t align,
                     int32_t* bucket_of, int64_t* offset, int32_t* direct, int64_t* count, int* nbuckets) {
  if (ntensors < 0 || (ntensors > 0 && (!numel || !bucket_of || !offset || !direct || !count)) || !nbuckets)
    return fail("fuse_plan: bad arguments");
  if (esize != 2 && esize != 4) return fail("fuse_plan: element size must be 2 or 4");
  if (align <= 0 || (align & (align - 1)) || align % esize) return fail("fuse_plan: bad alignment");
  if (threshold < 0) return fail("fuse_plan: negative threshold");
  int nb = 0;
  int open = 0; /* a buffer is being filled */
  int open_ntensors = 0;
  for (int t = 0; t < ntensors; ++t) {
    if (numel[t] < 0) return fail("fuse_plan: negative tensor size");
    int64_t bytes = numel[t] * esize;
    if (bytes > threshold) { /* larger than the whole buffer: reduced on its own */
      if (open) ++nb;
      open = 0;
      bucket_of[t] = nb;
      offset[t] = 0;
      direct[nb] = 1;
      count[nb] = numel[t];
      ++nb;
      continue;
    }
    if (!open) {
      open = 1;
      open_ntensors = 0;
      direct[nb] = 0;
      count[nb] = 0;
    }
    int64_t start_bytes = (count[nb] * esize + align - 1) / align * align;
    if (open_ntensors > 0 && start_bytes + bytes > threshold) { /* does not fit: close, open the next */
      ++nb;
      direct[nb] = 0;
      count[nb] = 0;
      open_ntensors = 0;
      start_bytes = 0;
    }
    bucket_of[t] = nb;
    offset[t] = start_bytes / esize;
    count[nb] = offset[t] + numel[t];
    ++open_ntensors;
  }
  if (open) ++nb;
  *nbuckets = nb;
  return 0;
}

/* ---------------------------------------------------------------------------
 * Section 3: the ring, in place on N buffers of `count` elements.
 * ------------------------------------------------------------------------- */

static void chunk(int64_t count, int n, int c, int64_t* start, int64_t* len) {
  int64_t q = count / n, rem = count % n;
  *start = c * q + (c < rem ? c : rem);
  *len = q + (c < rem ? 1 : 0);
}

/* dtype OR_F32: float buffers; OR_F16: uint16_t buffers holding binary16. */
int oracle_ring(void* const* bufs, int n, int64_t count, int dtype, int op, int nthreads) {
  if (n < 1 || count < 0 || !bufs) return fail("ring: bad arguments");
  if (dtype != OR_F32 && dtype != OR_F16) return fail("ring: bad dtype");
  if (op != OR_SUM && op != OR_AVERAGE) return fail("ring: bad op");
  if (nthreads < 1) nthreads = 1;
  (void)nthreads;
  const int avg = op == OR_AVERAGE;

  /* first N-1 iterations: the received chunk is added to the local one */
  for (int s = 0; s < n - 1; ++s) {
    const int last = s == n - 2;
    for (int c = 0; c < n; ++c) {
      const int snd = (c + s) % n, rcv = (c + s + 1) % n;
      int64_t start, len;
      chunk(count, n, c, &start, &len);
      if (dtype == OR_F32) {
        const float* x = (const float*)bufs[snd] + start;
        float* y = (float*)bufs[rcv] + start;
#pragma omp parallel for schedule(static) num_threads(nthreads)
        for (int64_t i = 0; i < len; ++i) {
          float v = y[i] + x[i];
          if (avg && last) v = v / (float)n;
          y[i] = v;
        }
      } else {
        const uint16_t* x = (const uint16_t*)bufs[snd] + start;
        uint16_t* y = (uint16_t*)bufs[rcv] + start;
#pragma omp parallel for schedule(static) num_threads(nthreads)
        for (int64_t i = 0; i < len; ++i) {
          uint16_t v = f2h(h2f(y[i]) + h2f(x[i])); /* one binary16 rounding of the exact sum */
          if (avg && last) v = f2h(h2f(v) / (float)n);
          y[i] = v;
        }
      }
    }
  }
  if (avg && n == 1) { /* the single rank divides by one */
    if (dtype == OR_F32) {
      float* y = (float*)bufs[0];
      for (int64_t i = 0; i < count; ++i) y[i] = y[i] / 1.0f;
    } else {
      uint16_t* y = (uint16_t*)bufs[0];
      for (int64_t i = 0; i < count; ++i) y[i] = f2h(h2f(y[i]) / 1.0f);
    }
  }

  /* second N-1 iterations: the received chunk replaces the local one */
  const size_t esize = dtype == OR_F32 ? 4 : 2;
  for (int s = 0; s < n - 1; ++s) {
    for (int c = 0; c < n; ++c) {
      const int snd = (c - 1 + s + n) % n, rcv = (c + s) % n;
      int64_t start, len;
      chunk(count, n, c, &start, &len);
      memcpy((char*)bufs[rcv] + start * esize, (const char*)bufs[snd] + start * esize, (size_t)len * esize);
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Sections 5 and 7 composed: one allreduce over every rank's tensors.
 * ------------------------------------------------------------------------- */

/* Bytes of fusion buffers (all N ranks, the largest buffer of the plan) that
 * oracle_allreduce can take instead of allocating them; -1 on bad arguments. */
int64_t oracle_workspace_bytes(const int64_t* numel, int ntensors, int n, int src_dtype, int compress,
                               int64_t threshold, int64_t align) {
  const int esize = (compress || src_dtype == OR_F16) ? 2 : 4;
  if (n < 1 || ntensors < 0 || (ntensors > 0 && !numel)) return fail("workspace_bytes: bad arguments");
  if (ntensors == 0) return 0;
  int32_t* bucket_of = malloc(sizeof(int32_t) * ntensors);
  int64_t* offset = malloc(sizeof(int64_t) * ntensors);
  int32_t* direct = malloc(sizeof(int32_t) * ntensors);
  int64_t* count = malloc(sizeof(int64_t) * ntensors);
  int nb = 0;
  int64_t most = -1;
  if (bucket_of && offset && direct && count &&
      oracle_fuse_plan(numel, ntensors, esize, threshold, align, bucket_of, offset, direct, count, &nb) == 0) {
    most = 0;
    for (int b = 0; b < nb; ++b)
      if (count[b] > most) most = count[b];
    most *= (int64_t)n * esize;
  } else if (!(bucket_of && offset && direct && count)) {
    fail("workspace_bytes: out of host memory");
  }
  free(bucket_of);
  free(offset);
  free(direct);
  free(count);
  return most;
}

/* x[r * ntensors + t]: rank r's tensor t (src_dtype); y likewise, same dtype.
 * Compression (binary32 tensors only) rounds the copies in to binary16; the
 * buffers then hold binary16 and the threshold counts binary16 bytes.
 * workspace: NULL, or at least oracle_workspace_bytes() bytes that hold the N
 * fusion buffers (allocated once by the caller, as section 7's step 2 allocates
 * the fusion buffer once); otherwise every buffer is allocated here. */
int oracle_allreduce(const void* const* x, const int64_t* numel, int ntensors, int n, int src_dtype, int op,
                     int compress, int64_t threshold, int64_t align, void* const* y, void* workspace,
                     int64_t workspace_bytes, int nthreads) {
  if (n < 1 || ntensors < 0 || (ntensors > 0 && (!x || !y || !numel))) return fail("allreduce: bad arguments");
  if (src_dtype != OR_F32 && src_dtype != OR_F16) return fail("allreduce: bad dtype");
  if (compress && src_dtype != OR_F32) return fail("allreduce: compression applies to binary32 tensors");
  if (nthreads < 1) nthreads = 1;
  const int buf_dtype = compress ? OR_F16 : src_dtype;
  const int esize = buf_dtype == OR_F32 ? 4 : 2;
  if (ntensors == 0) return 0;
  if (workspace) {
    int64_t need = oracle_workspace_bytes(numel, ntensors, n, src_dtype, compress, threshold, align);
    if (need < 0) return -1;
    if (workspace_bytes < need) return fail("allreduce: workspace too small");
  }

  int32_t* bucket_of = malloc(sizeof(int32_t) * ntensors);
  int64_t* offset = malloc(sizeof(int64_t) * ntensors);
  int32_t* direct = malloc(sizeof(int32_t) * ntensors);
  int64_t* count = malloc(sizeof(int64_t) * ntensors);
  void** bufs = malloc(sizeof(void*) * n);
  int nb = 0, rc = 0;
  if (!bucket_of || !offset || !direct || !count || !bufs) {
    rc = fail("allreduce: out of host memory");
    goto done;
  }
  rc = oracle_fuse_plan(numel, ntensors, esize, threshold, align, bucket_of, offset, direct, count, &nb);
  if (rc) goto done;

  for (int b = 0; b < nb; ++b) {
    /* step 3: every rank's selected tensors copied into its zeroed buffer */
    for (int r = 0; r < n; ++r) bufs[r] = NULL;
    for (int r = 0; r < n && workspace; ++r) {
      bufs[r] = (char*)workspace + (size_t)r * (size_t)count[b] * (size_t)esize;
      memset(bufs[r], 0, (size_t)count[b] * (size_t)esize);
    }
    for (int r = 0; r < n && !workspace; ++r) {
      bufs[r] = calloc((size_t)(count[b] > 0 ? count[b] : 1), (size_t)esize);
      if (!bufs[r]) {
        rc = fail("allreduce: out of host memory");
        break;
      }
    }
    if (rc == 0) {
      for (int r = 0; r < n; ++r) {
        for (int t = 0; t < ntensors; ++t) {
          if (bucket_of[t] != b) continue;
          const int64_t m = numel[t];
          if (buf_dtype == OR_F32) {
            const float* src = (const float*)x[(int64_t)r * ntensors + t];
            float* dst = (float*)bufs[r] + offset[t];
#pragma omp parallel for schedule(static) num_threads(nthreads)
            for (int64_t i = 0; i < m; ++i) dst[i] = src[i];
          } else if (src_dtype == OR_F16) {
            const uint16_t* src = (const uint16_t*)x[(int64_t)r * ntensors + t];
            uint16_t* dst = (uint16_t*)bufs[r] + offset[t];
#pragma omp parallel for schedule(static) num_threads(nthreads)
            for (int64_t i = 0; i < m; ++i) dst[i] = src[i];
          } else { /* compression: binary32 rounded to binary16 */
            const float* src = (const float*)x[(int64_t)r * ntensors + t];
            uint16_t* dst = (uint16_t*)bufs[r] + offset[t];
#pragma omp parallel for schedule(static) num_threads(nthreads)
            for (int64_t i = 0; i < m; ++i) dst[i] = f2h(src[i]);
          }
        }
      }
      /* step 4: the ring on the buffers */
      rc = oracle_ring(bufs, n, count[b], buf_dtype, op, nthreads);
    }
    if (rc == 0) {
      /* step 5: the results copied out to every rank's output tensors */
      for (int r = 0; r < n; ++r) {
        for (int t = 0; t < ntensors; ++t) {
          if (bucket_of[t] != b) continue;
          const int64_t m = numel[t];
          if (buf_dtype == OR_F32) {
            const float* src = (const float*)bufs[r] + offset[t];
            float* dst = (float*)y[(int64_t)r * ntensors + t];
#pragma omp parallel for schedule(static) num_threads(nthreads)
            for (int64_t i = 0; i < m; ++i) dst[i] = src[i];
          } else if (src_dtype == OR_F16) {
            const uint16_t* src = (const uint16_t*)bufs[r] + offset[t];
            uint16_t* dst = (uint16_t*)y[(int64_t)r * ntensors + t];
#pragma omp parallel for schedule(static) num_threads(nthreads)
            for (int64_t i = 0; i < m; ++i) dst[i] = src[i];
          } else { /* compression: binary16 widened exactly */
            const uint16_t* src = (const uint16_t*)bufs[r] + offset[t];
            float* dst = (float*)y[(int64_t)r * ntensors + t];
#pragma omp parallel for schedule(static) num_threads(nthreads)
            for (int64_t i = 0; i < m; ++i) dst[i] = h2f(src[i]);
          }
        }
      }
    }
    if (!workspace)
      for (int r = 0; r < n; ++r) free(bufs[r]);
    if (rc) break;
  }

done:
  free(bucket_of);
  free(offset);
  free(direct);
  free(count);
  free(bufs);
  return rc;
}

/* Threads an OpenMP region would use by default (1 without OpenMP). */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
