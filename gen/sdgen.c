/*
 * Seeded synthetic inputs for SpMM tests and benchmarks.
 *
 * This file builds input matrices and dense operands only.  It holds none of
 * the SpMM arithmetic: it never multiplies A by B, never converts formats and
 * never partitions work.  Both the CPU oracle and the GPU library receive the
 * arrays produced here.
 *
 * Random numbers: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014) used in counter mode.  The
 * i-th draw of a stream with key K is mix64(K + (i + 1) * GAMMA), where GAMMA
 * is the 64-bit golden-ratio increment and mix64 is SplitMix64's finaliser.
 * A stream key is key(seed, stream) = mix64(mix64(seed) + stream).  Because
 * every draw is addressed by its counter, the output does not depend on the
 * number of threads.
 *
 * Derived variates:
 *   u01      = (x >> 11) * 2^-53                       in [0, 1)
 *   U[-1,1)  = ((x >> 40) - 2^23) / 2^23               exact in fp32
 *   N(0,1)   = Box-Muller in fp64 on a counter pair, rounded to fp32
 *   int[0,R) = ((x >> 32) * R) >> 32                   (multiply-shift)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GAMMA 0x9e3779b97f4a7c15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

uint64_t sdg_key(uint64_t seed, uint64_t stream) { return mix64(mix64(seed) + stream); }

static inline uint64_t draw(uint64_t key, uint64_t ctr) { return mix64(key + (ctr + 1) * GAMMA); }

static inline double u01(uint64_t key, uint64_t ctr) { return (double)(draw(key, ctr) >> 11) * 0x1.0p-53; }

static inline float usym(uint64_t key, uint64_t ctr) {
  int32_t u = (int32_t)(draw(key, ctr) >> 40) - (1 << 23);
  return (float)u * 0x1.0p-23f;
}

static inline uint32_t below(uint64_t key, uint64_t ctr, uint32_t range) {
  return (uint32_t)(((draw(key, ctr) >> 32) * (uint64_t)range) >> 32);
}

uint64_t sdg_draw(uint64_t key, uint64_t ctr) { return draw(key, ctr); }

/* Dense operands ---------------------------------------------------------- */

void sdg_dense_uniform(uint64_t seed, uint64_t stream, int64_t count, float *out) {
  uint64_t key = sdg_key(seed, stream);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < count; ++i) out[i] = usym(key, (uint64_t)i);
}

void sdg_dense_normal(uint64_t seed, uint64_t stream, int64_t count, float *out) {
  uint64_t key = sdg_key(seed, stream);
  int64_t pairs = (count + 1) / 2;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < pairs; ++t) {
    /* u1 in (0, 1] so that log(u1) is finite */
    double u1 = (double)((draw(key, 2 * (uint64_t)t) >> 11) + 1) * 0x1.0p-53;
    double u2 = (double)(draw(key, 2 * (uint64_t)t + 1) >> 11) * 0x1.0p-53;
    double r = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586476925286766559 * u2;
    out[2 * t] = (float)(r * cos(ang));
    if (2 * t + 1 < count) out[2 * t + 1] = (float)(r * sin(ang));
  }
}

/* CSR result handle -------------------------------------------------------- */

typedef struct {
  int32_t m, k;
  int64_t nnz;
  int32_t *rowptr;
  int32_t *colidx;
  float *vals;
} sdg_csr;

int64_t sdg_csr_nnz(const sdg_csr *h) { return h->nnz; }
int32_t sdg_csr_m(const sdg_csr *h) { return h->m; }
int32_t sdg_csr_k(const sdg_csr *h) { return h->k; }

void sdg_csr_copy(const sdg_csr *h, int32_t *rowptr, int32_t *colidx, float *vals) {
  memcpy(rowptr, h->rowptr, sizeof(int32_t) * ((size_t)h->m + 1));
  if (h->nnz) {
    memcpy(colidx, h->colidx, sizeof(int32_t) * (size_t)h->nnz);
    memcpy(vals, h->vals, sizeof(float) * (size_t)h->nnz);
  }
}

void sdg_csr_free(sdg_csr *h) {
  if (!h) return;
  free(h->rowptr);
  free(h->colidx);
  free(h->vals);
  free(h);
}

static sdg_csr *csr_alloc(int32_t m, int32_t k, int64_t nnz) {
  sdg_csr *h = (sdg_csr *)calloc(1, sizeof(sdg_csr));
  h->m = m;
  h->k = k;
  h->nnz = nnz;
  h->rowptr = (int32_t *)calloc((size_t)m + 1, sizeof(int32_t));
  h->colidx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz > 0 ? nnz : 1));
  h->vals = (float *)malloc(sizeof(float) * (size_t)(nnz > 0 ? nnz : 1));
  return h;
}

static int cmp_i32(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

/* Draw `cnt` distinct integers of [lo, lo+range) into out[], sorted.  Draws
 * come in rounds: each round tops the list up with fresh draws (counters
 * ctr0, ctr0+1, ... in order), then sorts it and drops repeats.  After
 * `budget` draws the remaining values are the smallest absent ones (never
 * reached for the densities used here; it keeps the routine total).  When
 * more than half of the range is wanted, a partial Fisher-Yates shuffle over
 * the whole range is used instead. */
static void distinct_sorted(uint64_t key, uint64_t ctr0, uint64_t budget, int32_t lo, uint32_t range,
                            int32_t cnt, int32_t *out) {
  if ((uint32_t)cnt * 2u > range) {
    int32_t *pool = (int32_t *)malloc(sizeof(int32_t) * range);
    for (uint32_t i = 0; i < range; ++i) pool[i] = lo + (int32_t)i;
    for (int32_t i = 0; i < cnt; ++i) {
      uint32_t j = (uint32_t)i + below(key, ctr0 + (uint64_t)i, range - (uint32_t)i);
      int32_t tmp = pool[i];
      pool[i] = pool[j];
      pool[j] = tmp;
      out[i] = pool[i];
    }
    free(pool);
    qsort(out, (size_t)cnt, sizeof(int32_t), cmp_i32);
    return;
  }
  int32_t have = 0;
  uint64_t t = 0;
  while (have < cnt && t < budget) {
    while (have < cnt && t < budget) out[have++] = lo + (int32_t)below(key, ctr0 + t++, range);
    qsort(out, (size_t)have, sizeof(int32_t), cmp_i32);
    int32_t w = 0;
    for (int32_t q = 0; q < have; ++q)
      if (w == 0 || out[w - 1] != out[q]) out[w++] = out[q];
    have = w;
  }
  if (have < cnt) {
    int32_t c = lo;
    for (int32_t q = 0; have < cnt; ++c) {
      while (q < have && out[q] < c) ++q;
      if (q < have && out[q] == c) continue;
      out[have++] = c;
    }
    qsort(out, (size_t)cnt, sizeof(int32_t), cmp_i32);
  }
}

/* Uniform rows: every row has exactly `per_row` distinct columns drawn
 * uniformly from [0, k); values U[-1,1).  Streams: seed/0 columns,
 * seed/1 values (indexed by CSR position). */
sdg_csr *sdg_uniform_rows(int32_t m, int32_t k, int32_t per_row, uint64_t seed) {
  if (per_row > k) per_row = k;
  sdg_csr *h = csr_alloc(m, k, (int64_t)m * per_row);
  uint64_t kc = sdg_key(seed, 0), kv = sdg_key(seed, 1);
  for (int32_t i = 0; i <= m; ++i) h->rowptr[i] = i * per_row;
#pragma omp parallel for schedule(static)
  for (int32_t i = 0; i < m; ++i)
    distinct_sorted(kc, (uint64_t)i << 20, 1u << 20, 0, (uint32_t)k, per_row, h->colidx + (int64_t)i * per_row);
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < h->nnz; ++p) h->vals[p] = usym(kv, (uint64_t)p);
  return h;
}

/* Rows of caller-chosen lengths with distinct uniform columns; values
 * U[-1,1).  Used for edge cases (empty rows, one giant row, ragged tails). */
sdg_csr *sdg_random_rows(int32_t m, int32_t k, const int32_t *lengths, uint64_t seed) {
  int64_t nnz = 0;
  for (int32_t i = 0; i < m; ++i) nnz += lengths[i] < k ? lengths[i] : k;
  sdg_csr *h = csr_alloc(m, k, nnz);
  uint64_t kc = sdg_key(seed, 0), kv = sdg_key(seed, 1);
  int64_t p = 0;
  for (int32_t i = 0; i < m; ++i) {
    int32_t r = lengths[i] < k ? lengths[i] : k;
    h->rowptr[i] = (int32_t)p;
    p += r;
  }
  h->rowptr[m] = (int32_t)p;
#pragma omp parallel for schedule(dynamic, 64)
  for (int32_t i = 0; i < m; ++i) {
    int32_t r = h->rowptr[i + 1] - h->rowptr[i];
    if (r > 0) distinct_sorted(kc, (uint64_t)i << 32, 1ull << 31, 0, (uint32_t)k, r, h->colidx + h->rowptr[i]);
  }
#pragma omp parallel for schedule(static)
  for (int64_t q = 0; q < nnz; ++q) h->vals[q] = usym(kv, (uint64_t)q);
  return h;
}

/* 7-point Laplacian on an nx*ny*nz grid, natural order idx = x + nx*(y + ny*z),
 * Dirichlet boundary (neighbours outside the grid are dropped), diagonal 6,
 * neighbours -1, columns ascending. */
sdg_csr *sdg_laplacian3d(int32_t nx, int32_t ny, int32_t nz) {
  int32_t n = nx * ny * nz;
  int64_t nnz = 0;
  for (int32_t z = 0; z < nz; ++z)
    for (int32_t y = 0; y < ny; ++y)
      for (int32_t x = 0; x < nx; ++x)
        nnz += 1 + (x > 0) + (x < nx - 1) + (y > 0) + (y < ny - 1) + (z > 0) + (z < nz - 1);
  sdg_csr *h = csr_alloc(n, n, nnz);
  int64_t p = 0;
  for (int32_t z = 0; z < nz; ++z)
    for (int32_t y = 0; y < ny; ++y)
      for (int32_t x = 0; x < nx; ++x) {
        int32_t i = x + nx * (y + ny * z);
        h->rowptr[i] = (int32_t)p;
        /* ascending column order: -z, -y, -x, self, +x, +y, +z */
        if (z > 0) { h->colidx[p] = i - nx * ny; h->vals[p++] = -1.0f; }
        if (y > 0) { h->colidx[p] = i - nx; h->vals[p++] = -1.0f; }
        if (x > 0) { h->colidx[p] = i - 1; h->vals[p++] = -1.0f; }
        h->colidx[p] = i; h->vals[p++] = 6.0f;
        if (x < nx - 1) { h->colidx[p] = i + 1; h->vals[p++] = -1.0f; }
        if (y < ny - 1) { h->colidx[p] = i + nx; h->vals[p++] = -1.0f; }
        if (z < nz - 1) { h->colidx[p] = i + nx * ny; h->vals[p++] = -1.0f; }
      }
  h->rowptr[n] = (int32_t)p;
  return h;
}

/* Sort each row's columns, drop duplicates, optionally insert the diagonal.
 * Input: per-row unsorted lists in cols[rowptr_in[i] .. rowptr_in[i+1]).
 * Output compacted into a fresh handle (values left unset). */
static sdg_csr *canonicalise(int32_t m, int32_t k, const int64_t *rowptr_in, int32_t *cols, int add_diag) {
  int32_t *distinct = (int32_t *)malloc(sizeof(int32_t) * (size_t)(m > 0 ? m : 1));
  int32_t *cnt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(m > 0 ? m : 1));
#pragma omp parallel for schedule(dynamic, 256)
  for (int32_t i = 0; i < m; ++i) {
    int32_t *c = cols + rowptr_in[i];
    int64_t r = rowptr_in[i + 1] - rowptr_in[i];
    qsort(c, (size_t)r, sizeof(int32_t), cmp_i32);
    int64_t w = 0;
    for (int64_t q = 0; q < r; ++q)
      if (w == 0 || c[w - 1] != c[q]) c[w++] = c[q];
    int has_diag = 0;
    for (int64_t q = 0; q < w; ++q)
      if (c[q] == i) { has_diag = 1; break; }
    distinct[i] = (int32_t)w;
    cnt[i] = (int32_t)w + ((add_diag && i < k && !has_diag) ? 1 : 0);
  }
  int64_t nnz = 0;
  for (int32_t i = 0; i < m; ++i) nnz += cnt[i];
  sdg_csr *h = csr_alloc(m, k, nnz);
  int64_t p = 0;
  for (int32_t i = 0; i < m; ++i) {
    h->rowptr[i] = (int32_t)p;
    p += cnt[i];
  }
  h->rowptr[m] = (int32_t)p;
#pragma omp parallel for schedule(dynamic, 256)
  for (int32_t i = 0; i < m; ++i) {
    const int32_t *c = cols + rowptr_in[i];
    int32_t *dst = h->colidx + h->rowptr[i];
    int inserted = (cnt[i] == distinct[i]); /* nothing to insert */
    int32_t out = 0;
    for (int32_t q = 0; q < distinct[i]; ++q) {
      if (!inserted && c[q] > i) { dst[out++] = i; inserted = 1; }
      dst[out++] = c[q];
    }
    if (!inserted) dst[out++] = i;
  }
  free(cnt);
  free(distinct);
  return h;
}

/* GCN normalisation: val(u, v) = 1 / sqrt(d_u * d_v) in fp64, rounded to
 * fp32, with d = row nonzero count of the (already self-looped) matrix. */
static void gcn_values(sdg_csr *h) {
#pragma omp parallel for schedule(dynamic, 256)
  for (int32_t i = 0; i < h->m; ++i) {
    double du = (double)(h->rowptr[i + 1] - h->rowptr[i]);
    for (int32_t p = h->rowptr[i]; p < h->rowptr[i + 1]; ++p) {
      int32_t v = h->colidx[p];
      double dv = (v < h->m) ? (double)(h->rowptr[v + 1] - h->rowptr[v]) : 1.0;
      h->vals[p] = (float)(1.0 / sqrt(du * dv));
    }
  }
}

/* R-MAT edges.  Attempt e draws `scale` fp64 uniforms at counters
 * e*scale + l (l = 0 is the most significant bit).  Quadrant choice per
 * level: x < a -> (0,0); x < a+b -> (0,1); x < a+b+c -> (1,0); else (1,1),
 * first coordinate = row bit.  Attempts with an endpoint >= nmax are
 * rejected; the first `edges` accepted attempts are kept, in attempt order.
 * Duplicates are merged, self-loops added (merged if present), values are
 * the GCN normalisation above. */
sdg_csr *sdg_rmat(int32_t scale, int64_t edges, int32_t nmax, double a, double b, double c, uint64_t seed) {
  uint64_t key = sdg_key(seed, 0);
  int32_t *eu = (int32_t *)malloc(sizeof(int32_t) * (size_t)edges);
  int32_t *ev = (int32_t *)malloc(sizeof(int32_t) * (size_t)edges);
  const double ab = a + b, abc = a + b + c;
  int64_t accepted = 0;
  uint64_t next = 0;
  const int64_t batch = 1 << 22;
  int32_t *bu = (int32_t *)malloc(sizeof(int32_t) * batch);
  int32_t *bv = (int32_t *)malloc(sizeof(int32_t) * batch);
  while (accepted < edges) {
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < batch; ++t) {
      uint64_t e = next + (uint64_t)t;
      uint32_t u = 0, v = 0;
      for (int32_t l = 0; l < scale; ++l) {
        double x = u01(key, e * (uint64_t)scale + (uint64_t)l);
        uint32_t rb = (x >= ab) ? 1u : 0u;
        uint32_t cb = (x >= a && x < ab) || (x >= abc) ? 1u : 0u;
        u = (u << 1) | rb;
        v = (v << 1) | cb;
      }
      bu[t] = (int32_t)u;
      bv[t] = (int32_t)v;
    }
    for (int64_t t = 0; t < batch && accepted < edges; ++t) {
      if (bu[t] < nmax && bv[t] < nmax) {
        eu[accepted] = bu[t];
        ev[accepted] = bv[t];
        ++accepted;
      }
    }
    next += (uint64_t)batch;
  }
  free(bu);
  free(bv);
  /* bucket by row (stable by attempt order; order is irrelevant after sort) */
  int64_t *rp = (int64_t *)calloc((size_t)nmax + 1, sizeof(int64_t));
  for (int64_t e = 0; e < edges; ++e) rp[eu[e] + 1]++;
  for (int32_t i = 0; i < nmax; ++i) rp[i + 1] += rp[i];
  int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)nmax);
  memcpy(fill, rp, sizeof(int64_t) * (size_t)nmax);
  int32_t *cols = (int32_t *)malloc(sizeof(int32_t) * (size_t)edges);
  for (int64_t e = 0; e < edges; ++e) cols[fill[eu[e]]++] = ev[e];
  free(fill);
  free(eu);
  free(ev);
  sdg_csr *h = canonicalise(nmax, nmax, rp, cols, 1);
  free(rp);
  free(cols);
  gcn_values(h);
  return h;
}

/* Block-structured matrix built from b*b dense blocks.  Block-row br draws
 * `per_row` distinct block-columns uniformly from
 * [max(0, br-window), min(nbc-1, br+window)] (stream 0, counters br<<20 + t),
 * sorted.  Entry (rr, cc) of the j-th block of block-row br, counter
 * ((br*per_row + j)*b + rr)*b + cc, is kept when a stream-1 fp64 uniform is
 * below `fill`; kept entries take a stream-2 U[-1,1) value at the same
 * counter.  Dropped entries are absent from the CSR. */
sdg_csr *sdg_block(int32_t nbr, int32_t nbc, int32_t b, int32_t per_row, int32_t window, double fill, uint64_t seed) {
  uint64_t kc = sdg_key(seed, 0), kk = sdg_key(seed, 1), kv = sdg_key(seed, 2);
  int32_t *bcols = (int32_t *)malloc(sizeof(int32_t) * (size_t)nbr * per_row);
#pragma omp parallel for schedule(static)
  for (int32_t br = 0; br < nbr; ++br) {
    int32_t lo = br - window < 0 ? 0 : br - window;
    int32_t hi = br + window > nbc - 1 ? nbc - 1 : br + window;
    uint32_t range = (uint32_t)(hi - lo + 1);
    int32_t cnt = per_row < (int32_t)range ? per_row : (int32_t)range;
    distinct_sorted(kc, (uint64_t)br << 20, 1u << 20, lo, range, cnt, bcols + (int64_t)br * per_row);
    for (int32_t j = cnt; j < per_row; ++j) bcols[(int64_t)br * per_row + j] = -1;
  }
  int32_t m = nbr * b, k = nbc * b;
  int32_t *rowcnt = (int32_t *)calloc((size_t)m, sizeof(int32_t));
#pragma omp parallel for schedule(static)
  for (int32_t br = 0; br < nbr; ++br)
    for (int32_t rr = 0; rr < b; ++rr) {
      int32_t cnt = 0;
      for (int32_t j = 0; j < per_row; ++j) {
        if (bcols[(int64_t)br * per_row + j] < 0) continue;
        for (int32_t cc = 0; cc < b; ++cc) {
          uint64_t ctr = (((uint64_t)br * per_row + j) * b + rr) * b + cc;
          if (u01(kk, ctr) < fill) cnt++;
        }
      }
      rowcnt[br * b + rr] = cnt;
    }
  int64_t nnz = 0;
  for (int32_t i = 0; i < m; ++i) nnz += rowcnt[i];
  sdg_csr *h = csr_alloc(m, k, nnz);
  int64_t p = 0;
  for (int32_t i = 0; i < m; ++i) {
    h->rowptr[i] = (int32_t)p;
    p += rowcnt[i];
  }
  h->rowptr[m] = (int32_t)p;
  free(rowcnt);
#pragma omp parallel for schedule(static)
  for (int32_t br = 0; br < nbr; ++br)
    for (int32_t rr = 0; rr < b; ++rr) {
      int64_t q = h->rowptr[br * b + rr];
      for (int32_t j = 0; j < per_row; ++j) {
        int32_t bc = bcols[(int64_t)br * per_row + j];
        if (bc < 0) continue;
        for (int32_t cc = 0; cc < b; ++cc) {
          uint64_t ctr = (((uint64_t)br * per_row + j) * b + rr) * b + cc;
          if (u01(kk, ctr) < fill) {
            h->colidx[q] = bc * b + cc;
            h->vals[q] = usym(kv, ctr);
            ++q;
          }
        }
      }
    }
  free(bcols);
  return h;
}
