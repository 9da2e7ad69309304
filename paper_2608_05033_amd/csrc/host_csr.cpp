// Host-side CSR validation, structural analysis and transpose.
//
// The analysis follows Sec. "Structural Features and Overhead Modeling":
// intrinsic pattern features (size, density, row-length mean/max/CV,
// quartiles, empty rows, column degrees, row span and normalised span, mean
// column gap, diagonal share, 16x16 tile coverage and dense-tile share) and
// the representation-expansion factors of Eq. format-expansion
// (rho_ELL, rho_SELL(c) for c in {16, 32, 512}, rho_BSR(b) for b in
// {4, 8, 16}; the eighth factor is read as Blocked-ELL(16)).  All counts are
// exact; every fp64 field is one fixed formula over exact integer sums, so
// the result does not depend on evaluation order.  Block occupancy uses a
// stamp array over block-columns per block-row, O(nnz + m + k) overall.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>

#include "sd_internal.h"

namespace sd {

int validate_csr(const sd_csr_t *A, CsrView *out) {
  if (!A || !out) return SD_ERR_INVALID_VALUE;
  if (A->m < 0 || A->k < 0 || A->nnz < 0) return SD_ERR_INVALID_CSR;
  if (A->nnz > INT32_MAX) return SD_ERR_OVERFLOW;
  if (!A->rowptr) return SD_ERR_INVALID_VALUE;
  if (A->nnz > 0 && (!A->colidx || !A->values)) return SD_ERR_INVALID_VALUE;
  const int32_t *rp = A->rowptr;
  if (rp[0] != 0 || (int64_t)rp[A->m] != A->nnz) return SD_ERR_INVALID_CSR;
  for (int32_t i = 0; i < A->m; ++i) {
    if (rp[i + 1] < rp[i]) return SD_ERR_INVALID_CSR;
    int32_t prev = -1;
    for (int32_t p = rp[i]; p < rp[i + 1]; ++p) {
      int32_t c = A->colidx[p];
      if (c <= prev || c >= A->k) return SD_ERR_INVALID_CSR;
      prev = c;
    }
  }
  out->m = A->m;
  out->k = A->k;
  out->nnz = A->nnz;
  out->rowptr = A->rowptr;
  out->colidx = A->colidx;
  out->values = A->values;
  return SD_OK;
}

namespace {

double cv_from_sums(int64_t sum, int64_t sumsq, int64_t count) {
  if (count <= 0 || sum <= 0) return 0.0;
  double mean = (double)sum / (double)count;
  double var = (double)sumsq / (double)count - mean * mean;
  return var > 0.0 ? std::sqrt(var) / mean : 0.0;
}

int log2_bin(int64_t r) {
  int t = 0;
  while (t < 32 && r >= ((int64_t)1 << t)) ++t;
  return t;
}

}  // namespace

// k-th smallest (0-based) of a histogram of values 0..H-1
int64_t kth_from_hist(const std::vector<int64_t> &hist, int64_t kth) {
  int64_t seen = 0;
  for (size_t v = 0; v < hist.size(); ++v) {
    seen += hist[v];
    if (seen > kth) return (int64_t)v;
  }
  return hist.empty() ? 0 : (int64_t)hist.size() - 1;
}

void finish_stats(const StatsSums &sum, sd_stats_t *out) {
  sd_stats_t &st = *out;
  const int64_t m = st.m, k = st.k, nnz = st.nnz;
  if (m > 0) {
    st.row_mean = (double)nnz / (double)m;
    st.row_cv = cv_from_sums(nnz, sum.row_sumsq, m);
    st.empty_row_frac = (double)st.empty_rows / (double)m;
  }
  if (m > 0 && k > 0) st.density = (double)nnz / ((double)m * (double)k);
  if (k > 0) {
    st.col_deg_mean = (double)nnz / (double)k;
    st.col_deg_cv = cv_from_sums(nnz, sum.col_sumsq, k);
  }
  if (sum.nonempty > 0) {
    st.row_span_mean = (double)sum.span_sum / (double)sum.nonempty;
    if (k > 0) st.row_span_norm = st.row_span_mean / (double)k;
  }
  if (sum.gap_den > 0) st.col_gap_mean = (double)sum.gap_num / (double)sum.gap_den;
  const int64_t mn = std::min(m, k);
  if (mn > 0) st.diag_frac = (double)st.diag_nnz / (double)mn;
  if (m > 0 && k > 0)
    st.tile16_coverage = (double)st.nnzb16 / ((double)((m + 15) / 16) * (double)((k + 15) / 16));
  if (st.nnzb16 > 0) {
    st.dense_tile_frac = (double)st.dense_tiles16 / (double)st.nnzb16;
    st.nnz_per_tile16 = (double)nnz / (double)st.nnzb16;
  }
  if (nnz > 0) st.dense_tile_nnz_frac = (double)st.dense_tile_nnz16 / (double)nnz;

  // ---- expansion factors, Eq. format-expansion
  if (nnz > 0) {
    st.rho_ell = (double)(m * st.row_max) / (double)nnz;
    st.rho_sell16 = (double)st.sell16_slots / (double)nnz;
    st.rho_sell32 = (double)st.sell32_slots / (double)nnz;
    st.rho_sell512 = (double)st.sell512_slots / (double)nnz;
    st.rho_bsr4 = (double)(16 * st.nnzb4) / (double)nnz;
    st.rho_bsr8 = (double)(64 * st.nnzb8) / (double)nnz;
    st.rho_bsr16 = (double)(256 * st.nnzb16) / (double)nnz;
    st.rho_bell16 = (double)(256 * st.bell16_width * ((m + 15) / 16)) / (double)nnz;
  }

  // ---- shape class: a heuristic reading (the paper names five classes
  // without thresholds).  Bimodal: two local maxima of the log2 row-length
  // histogram at least two bins apart, each holding >= 10 % of the rows.
  {
    int bimodal = 0;
    const int64_t *h = st.row_hist;
    auto is_peak = [&](int a) {
      bool left = (a == 0) || h[a] > h[a - 1];
      bool right = (a == 32) || h[a] >= h[a + 1];
      return left && right && 10 * h[a] >= m;
    };
    for (int a = 0; a < 33 && !bimodal; ++a) {
      if (!is_peak(a)) continue;
      for (int c = a + 2; c < 33; ++c)
        if (c > 0 && is_peak(c)) {
          bimodal = 1;
          break;
        }
    }
    const double cv = st.row_cv;
    if (nnz == 0 || cv < 0.1) st.shape_class = 0;
    else if (bimodal) st.shape_class = 4;
    else if (cv < 0.5) st.shape_class = 1;
    else if (cv >= 1.0 && (double)st.row_max >= 50.0 * st.row_mean) st.shape_class = 3;
    else st.shape_class = 2;
  }
}

int analyze(const CsrView &A, int32_t dense_threshold, sd_stats_t *out) {
  if (!out) return SD_ERR_INVALID_VALUE;
  if (dense_threshold == 0) dense_threshold = 128;
  if (dense_threshold < 1 || dense_threshold > 256) return SD_ERR_INVALID_VALUE;
  sd_stats_t st;
  std::memset(&st, 0, sizeof(st));
  StatsSums sum;
  const int32_t m = A.m, k = A.k;
  const int64_t nnz = A.nnz;
  st.m = m;
  st.k = k;
  st.nnz = nnz;
  st.dense_threshold = dense_threshold;
  try {
    // ---- rows: lengths, histogram, quartiles via counting
    int64_t rmax = 0, rmin = m > 0 ? INT64_MAX : 0, empty = 0;
    for (int32_t i = 0; i < m; ++i) {
      int64_t r = A.rowptr[i + 1] - A.rowptr[i];
      rmax = std::max(rmax, r);
      rmin = std::min(rmin, r);
      sum.row_sumsq += r * r;
      empty += (r == 0);
      st.row_hist[log2_bin(r)]++;
    }
    st.row_min = rmin;
    st.row_max = rmax;
    st.empty_rows = empty;
    if (m > 0) {
      std::vector<int64_t> lhist((size_t)rmax + 1, 0);
      for (int32_t i = 0; i < m; ++i) lhist[A.rowptr[i + 1] - A.rowptr[i]]++;
      st.row_q25 = kth_from_hist(lhist, (int64_t)(m - 1) / 4);
      st.row_q50 = kth_from_hist(lhist, (int64_t)(m - 1) / 2);
      st.row_q75 = kth_from_hist(lhist, 3 * (int64_t)(m - 1) / 4);
    }

    // ---- columns
    {
      std::vector<int64_t> deg((size_t)k, 0);
      for (int64_t p = 0; p < nnz; ++p) deg[A.colidx[p]]++;
      int64_t dmax = 0;
      for (int32_t j = 0; j < k; ++j) {
        dmax = std::max(dmax, deg[j]);
        sum.col_sumsq += deg[j] * deg[j];
      }
      st.col_deg_max = dmax;
    }

    // ---- spans (median through a counting pass over span values), gaps, diagonal
    {
      int64_t diag = 0, smax = 0;
      for (int32_t i = 0; i < m; ++i) {
        int32_t p0 = A.rowptr[i], p1 = A.rowptr[i + 1];
        if (p1 == p0) continue;
        int64_t span = (int64_t)A.colidx[p1 - 1] - A.colidx[p0] + 1;
        ++sum.nonempty;
        sum.span_sum += span;
        smax = std::max(smax, span);
        if (p1 - p0 >= 2) {
          sum.gap_num += span - 1;
          sum.gap_den += p1 - p0 - 1;
        }
        if (i < k) {
          // columns ascending: binary search for the diagonal
          const int32_t *lo = A.colidx + p0, *hi = A.colidx + p1;
          const int32_t *f = std::lower_bound(lo, hi, i);
          diag += (f != hi && *f == i);
        }
      }
      if (sum.nonempty > 0) {
        std::vector<int64_t> shist((size_t)smax + 1, 0);
        for (int32_t i = 0; i < m; ++i) {
          int32_t p0 = A.rowptr[i], p1 = A.rowptr[i + 1];
          if (p1 > p0) shist[(int64_t)A.colidx[p1 - 1] - A.colidx[p0] + 1]++;
        }
        st.row_span_median = kth_from_hist(shist, (sum.nonempty - 1) / 2);
      }
      st.diag_nnz = diag;
    }

    // ---- block occupancy for b in {4, 8, 16}; tile fills for b = 16
    {
      const int32_t bs[3] = {4, 8, 16};
      int64_t nnzb[3] = {0, 0, 0};
      for (int t = 0; t < 3; ++t) {
        const int32_t b = bs[t];
        const int32_t kb = (k + b - 1) / b, mb = (m + b - 1) / b;
        std::vector<int32_t> stamp((size_t)kb, -1);
        std::vector<int32_t> count(b == 16 ? (size_t)kb : 0, 0);
        std::vector<int32_t> touched;
        int64_t width = 0, dense_tiles = 0, dense_nnz = 0;
        for (int32_t br = 0; br < mb; ++br) {
          const int32_t r0 = br * b, r1 = std::min(m, r0 + b);
          int64_t here = 0;
          touched.clear();
          for (int64_t p = A.rowptr[r0]; p < A.rowptr[r1]; ++p) {
            const int32_t bc = A.colidx[p] / b;
            if (stamp[bc] != br) {
              stamp[bc] = br;
              ++here;
              if (b == 16) {
                count[bc] = 0;
                touched.push_back(bc);
              }
            }
            if (b == 16) count[bc]++;
          }
          nnzb[t] += here;
          if (b == 16) {
            width = std::max(width, here);
            for (int32_t bc : touched) {
              const int32_t f = count[bc];
              st.fill16_hist[(f - 1) / 32]++;
              if (f >= dense_threshold) {
                ++dense_tiles;
                dense_nnz += f;
              }
            }
          }
        }
        if (b == 16) {
          st.bell16_width = width;
          st.dense_tiles16 = dense_tiles;
          st.dense_tile_nnz16 = dense_nnz;
        }
      }
      st.nnzb4 = nnzb[0];
      st.nnzb8 = nnzb[1];
      st.nnzb16 = nnzb[2];
    }

    // ---- SELL-c slots
    {
      const int32_t cs[3] = {16, 32, 512};
      int64_t *slots[3] = {&st.sell16_slots, &st.sell32_slots, &st.sell512_slots};
      for (int t = 0; t < 3; ++t) {
        int64_t s = 0;
        for (int32_t s0 = 0; s0 < m; s0 += cs[t]) {
          const int32_t s1 = std::min(m, s0 + cs[t]);
          int32_t mx = 0;
          for (int32_t i = s0; i < s1; ++i) mx = std::max(mx, A.rowptr[i + 1] - A.rowptr[i]);
          s += (int64_t)(s1 - s0) * mx;
        }
        *slots[t] = s;
      }
    }
  } catch (const std::bad_alloc &) {
    return SD_ERR_OUT_OF_MEMORY;
  }
  finish_stats(sum, &st);
  *out = st;
  return SD_OK;
}

int transpose(const CsrView &A, CsrOwned *out) {
  try {
    out->m = A.k;
    out->k = A.m;
    out->rowptr.assign((size_t)A.k + 1, 0);
    out->colidx.resize((size_t)A.nnz);
    out->values.resize((size_t)A.nnz);
    for (int64_t p = 0; p < A.nnz; ++p) out->rowptr[A.colidx[p] + 1]++;
    for (int32_t j = 0; j < A.k; ++j) out->rowptr[j + 1] += out->rowptr[j];
    std::vector<int32_t> cursor(out->rowptr.begin(), out->rowptr.end() - 1);
    for (int32_t i = 0; i < A.m; ++i)
      for (int32_t p = A.rowptr[i]; p < A.rowptr[i + 1]; ++p) {
        const int32_t q = cursor[A.colidx[p]]++;
        out->colidx[q] = i;
        std::memcpy(&out->values[q], &A.values[p], sizeof(float));
      }
  } catch (const std::bad_alloc &) {
    return SD_ERR_OUT_OF_MEMORY;
  }
  return SD_OK;
}

}  // namespace sd
