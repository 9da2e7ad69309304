// Host-side plan construction: representation conversions, work partitions
// and the planner's family rules.
//
// Conversions (Eq. format-expansion; Appendix "Compilation-Plan Design
// Space", SpMM row): BSR and Blocked-ELL with 16x16 blocks, block-columns
// ascending within a block-row, values row-major within a block, zero fill.
// Partitions: the heavy-row split of the SpMM web-graph case study
// (Appendix "Case Studies") and the merge-path decomposition (equal pieces of
// the merged row-end / nonzero sequence, Merrill and Garland, cited in
// Sec. "Background and Motivation").
#include <algorithm>
#include <cstdlib>
#include <cstring>

#include "sd_internal.h"

namespace sd {

void heavy_split(const CsrView &A, int32_t T, int32_t c, int32_t order, std::vector<int32_t> *light,
                 std::vector<int32_t> *chunks, std::vector<int32_t> *heavy_rows,
                 std::vector<int32_t> *heavy_ptr) {
  light->clear();
  chunks->clear();
  heavy_rows->clear();
  heavy_ptr->assign(1, 0);
  for (int32_t i = 0; i < A.m; ++i) {
    const int32_t p0 = A.rowptr[i], p1 = A.rowptr[i + 1];
    if (p1 - p0 < T) {
      light->push_back(i);
      continue;
    }
    heavy_rows->push_back(i);
    const int32_t pieces = (int32_t)(((int64_t)(p1 - p0) + c - 1) / c);
    for (int32_t q = 0; q < pieces; ++q) {
      const int32_t b = p0 + q * c;
      chunks->push_back(i);
      chunks->push_back(b);
      chunks->push_back(std::min(p1, b + c));
    }
    heavy_ptr->push_back((int32_t)(chunks->size() / 3));
  }
  if (order == 2) {  // by the column of the last nonzero, ties by row, empty rows last
    auto key = [&](int32_t r) { return A.rowptr[r + 1] > A.rowptr[r] ? A.colidx[A.rowptr[r + 1] - 1] : A.k; };
    std::stable_sort(light->begin(), light->end(), [&](int32_t a, int32_t b) { return key(a) < key(b); });
  }
}

void chunk_order(const std::vector<int32_t> &colidx, const std::vector<int32_t> &chunks, int32_t order,
                 std::vector<int32_t> *corder) {
  const size_t nch = chunks.size() / 3;
  corder->resize(nch);
  for (size_t q = 0; q < nch; ++q) (*corder)[q] = (int32_t)q;
  if (order != 2) return;
  auto key = [&](int32_t q) {
    const int64_t b = chunks[3 * (size_t)q + 1], e = chunks[3 * (size_t)q + 2];
    return colidx[(size_t)((b + e) / 2)];
  };
  std::stable_sort(corder->begin(), corder->end(), [&](int32_t a, int32_t b) { return key(a) < key(b); });
}

void split_layout(const CsrView &A, int32_t T, int32_t c, const std::vector<int32_t> &light,
                  std::vector<int32_t> *lptr, std::vector<int32_t> *colidx, std::vector<float> *vals,
                  std::vector<int32_t> *chunks) {
  lptr->assign(light.size() + 1, 0);
  colidx->resize((size_t)A.nnz);
  vals->resize((size_t)A.nnz);
  chunks->clear();
  int64_t pos = 0;
  auto copy_row = [&](int32_t r) {
    for (int32_t p = A.rowptr[r]; p < A.rowptr[r + 1]; ++p, ++pos) {
      (*colidx)[(size_t)pos] = A.colidx[p];
      (*vals)[(size_t)pos] = A.values[p];
    }
  };
  for (size_t i = 0; i < light.size(); ++i) {
    (*lptr)[i] = (int32_t)pos;
    copy_row(light[i]);
  }
  (*lptr)[light.size()] = (int32_t)pos;
  for (int32_t r = 0; r < A.m; ++r) {
    if (A.rowptr[r + 1] - A.rowptr[r] < T) continue;
    const int64_t start = pos;
    copy_row(r);
    for (int64_t b = start; b < pos; b += c) {
      chunks->push_back(r);
      chunks->push_back((int32_t)b);
      chunks->push_back((int32_t)std::min<int64_t>(pos, b + c));
    }
  }
}

// Unit u starts at path position d = min(u L, m + nnz).  The row ends taken
// by then are the rows i with rowptr[i+1] + i < d (row end i is the
// (rowptr[i+1] + i + 1)-th step of the path), a prefix because
// rowptr[i+1] + i is strictly increasing: binary search for its length.
void merge_split(const CsrView &A, int32_t U, std::vector<int32_t> *coords, int64_t *L_out) {
  const int64_t total = (int64_t)A.m + A.nnz;
  int64_t L = (total + U - 1) / U;
  if (L < 1) L = 1;
  coords->resize(2 * ((size_t)U + 1));
  for (int32_t u = 0; u <= U; ++u) {
    const int64_t d = std::min<int64_t>((int64_t)u * L, total);
    int64_t lo = std::max<int64_t>(0, d - A.nnz), hi = std::min<int64_t>(d, A.m);
    while (lo < hi) {
      const int64_t mid = (lo + hi) / 2;
      if ((int64_t)A.rowptr[mid + 1] + mid >= d) hi = mid;
      else lo = mid + 1;
    }
    (*coords)[2 * u] = (int32_t)lo;
    (*coords)[2 * u + 1] = (int32_t)(d - lo);
  }
  *L_out = L;
}

void block_convert(const CsrView &A, int32_t b, bool ell, std::vector<int32_t> *bptr,
                   std::vector<int32_t> *bcol, std::vector<float> *bval, int32_t *width) {
  const int32_t mb = (A.m + b - 1) / b, kb = (A.k + b - 1) / b;
  std::vector<int32_t> stamp((size_t)kb, -1), slot((size_t)kb, 0);
  // pass 1: distinct block-columns per block-row
  std::vector<int32_t> counts((size_t)mb, 0);
  for (int32_t br = 0; br < mb; ++br) {
    const int32_t r1 = std::min(A.m, (br + 1) * b);
    for (int32_t p = A.rowptr[br * b]; p < A.rowptr[r1]; ++p) {
      const int32_t bc = A.colidx[p] / b;
      if (stamp[bc] != br) {
        stamp[bc] = br;
        counts[br]++;
      }
    }
  }
  int32_t w = 0;
  for (int32_t br = 0; br < mb; ++br) w = std::max(w, counts[br]);
  *width = w;
  bptr->assign((size_t)mb + 1, 0);
  if (ell) {
    for (int32_t br = 0; br <= mb; ++br) (*bptr)[br] = br * w;
  } else {
    for (int32_t br = 0; br < mb; ++br) (*bptr)[br + 1] = (*bptr)[br] + counts[br];
  }
  const int64_t slots = (int64_t)(*bptr)[mb];
  bcol->assign((size_t)slots, -1);
  bval->assign((size_t)slots * b * b, 0.0f);
  std::fill(stamp.begin(), stamp.end(), -1);
  std::vector<int32_t> list;
  // pass 2: sorted block-columns, slot map, scatter of values
  for (int32_t br = 0; br < mb; ++br) {
    const int32_t r0 = br * b, r1 = std::min(A.m, r0 + b);
    list.clear();
    for (int32_t p = A.rowptr[r0]; p < A.rowptr[r1]; ++p) {
      const int32_t bc = A.colidx[p] / b;
      if (stamp[bc] != br) {
        stamp[bc] = br;
        list.push_back(bc);
      }
    }
    std::sort(list.begin(), list.end());
    const int64_t base = (*bptr)[br];
    for (size_t t = 0; t < list.size(); ++t) {
      slot[list[t]] = (int32_t)t;
      (*bcol)[base + (int64_t)t] = list[t];
    }
    for (int32_t i = r0; i < r1; ++i)
      for (int32_t p = A.rowptr[i]; p < A.rowptr[i + 1]; ++p) {
        const int32_t col = A.colidx[p];
        const int64_t q = base + slot[col / b];
        std::memcpy(&(*bval)[(q * b + (i - r0)) * b + col % b], &A.values[p], sizeof(float));
      }
  }
}

void ell_convert(const CsrView &A, std::vector<int32_t> *ecol, std::vector<float> *eval, int32_t *width) {
  int32_t w = 0;
  for (int32_t i = 0; i < A.m; ++i) w = std::max(w, A.rowptr[i + 1] - A.rowptr[i]);
  *width = w;
  ecol->assign((size_t)A.m * w, -1);
  eval->assign((size_t)A.m * w, 0.0f);
  for (int32_t i = 0; i < A.m; ++i) {
    const int64_t base = (int64_t)i * w;
    const int32_t r = A.rowptr[i + 1] - A.rowptr[i];
    std::memcpy(ecol->data() + base, A.colidx + A.rowptr[i], sizeof(int32_t) * (size_t)r);
    std::memcpy(eval->data() + base, A.values + A.rowptr[i], sizeof(float) * (size_t)r);
  }
}

void sell_convert(const CsrView &A, int32_t C, int32_t sigma, std::vector<int32_t> *perm,
                  std::vector<int64_t> *slice_ptr, std::vector<int32_t> *col, std::vector<float> *val) {
  perm->resize((size_t)A.m);
  for (int32_t i = 0; i < A.m; ++i) (*perm)[i] = i;
  auto len = [&](int32_t r) { return A.rowptr[r + 1] - A.rowptr[r]; };
  for (int64_t b = 0; b < A.m; b += sigma) {
    const int64_t e = std::min<int64_t>(A.m, b + sigma);
    std::stable_sort(perm->begin() + b, perm->begin() + e, [&](int32_t x, int32_t y) { return len(x) > len(y); });
  }
  const int64_t ns = ((int64_t)A.m + C - 1) / C;
  slice_ptr->assign((size_t)ns + 1, 0);
  int64_t total = 0;
  for (int64_t sl = 0; sl < ns; ++sl) {
    const int64_t r0 = sl * C, r1 = std::min<int64_t>(A.m, r0 + C);
    int32_t w = 0;
    for (int64_t i = r0; i < r1; ++i) w = std::max(w, len((*perm)[i]));
    (*slice_ptr)[sl] = total;
    total += (r1 - r0) * w;
  }
  (*slice_ptr)[ns] = total;
  col->assign((size_t)total, -1);
  val->assign((size_t)total, 0.0f);
  for (int64_t sl = 0; sl < ns; ++sl) {
    const int64_t r0 = sl * C, r1 = std::min<int64_t>(A.m, r0 + C);
    const int64_t w = ((*slice_ptr)[sl + 1] - (*slice_ptr)[sl]) / std::max<int64_t>(1, r1 - r0);
    for (int64_t i = r0; i < r1; ++i) {
      const int32_t r = (*perm)[i];
      const int64_t base = (*slice_ptr)[sl] + (i - r0) * w;
      std::memcpy(col->data() + base, A.colidx + A.rowptr[r], sizeof(int32_t) * (size_t)len(r));
      std::memcpy(val->data() + base, A.values + A.rowptr[r], sizeof(float) * (size_t)len(r));
    }
  }
}

void split_windows(int32_t k, const std::vector<int32_t> &lptr, int64_t n_light, std::vector<int32_t> *colidx,
                   int32_t R, int32_t cap, std::vector<int32_t> *wptr, std::vector<int32_t> *wcols, int32_t *wmax,
                   int64_t *staged_uses) {
  const int64_t nw = (n_light + R - 1) / R;
  wptr->assign((size_t)nw + 1, 0);
  wcols->clear();
  // per-column use count in the current window and staged position, reset
  // after each window (columns of a row are distinct, so uses count rows)
  std::vector<int32_t> uses((size_t)std::max(1, k), 0), pos((size_t)std::max(1, k), -1), seen, pick;
  int32_t dmax = 0;
  int64_t su = 0;
  for (int64_t w = 0; w < nw; ++w) {
    const int64_t t0 = w * R, t1 = std::min<int64_t>(n_light, (w + 1) * R);
    const int32_t p0 = lptr[(size_t)t0], p1 = lptr[(size_t)t1];
    seen.clear();
    for (int32_t p = p0; p < p1; ++p)
      if (uses[(size_t)(*colidx)[(size_t)p]]++ == 0) seen.push_back((*colidx)[(size_t)p]);
    pick.clear();
    for (int32_t c : seen)
      if (uses[(size_t)c] >= 2) pick.push_back(c);
    if ((int64_t)pick.size() > cap) {  // keep the most used, ties to the smaller column
      std::nth_element(pick.begin(), pick.begin() + cap, pick.end(), [&](int32_t a, int32_t b) {
        return uses[(size_t)a] != uses[(size_t)b] ? uses[(size_t)a] > uses[(size_t)b] : a < b;
      });
      pick.resize((size_t)cap);
    }
    std::sort(pick.begin(), pick.end());
    (*wptr)[(size_t)w] = (int32_t)wcols->size();
    for (size_t q = 0; q < pick.size(); ++q) {
      pos[(size_t)pick[q]] = (int32_t)q;
      wcols->push_back(pick[q]);
    }
    dmax = std::max<int32_t>(dmax, (int32_t)pick.size());
    for (int32_t p = p0; p < p1; ++p) {
      int32_t &c = (*colidx)[(size_t)p];
      if (pos[(size_t)c] >= 0) {
        c = -2 - pos[(size_t)c];
        ++su;
      }
    }
    for (int32_t c : seen) uses[(size_t)c] = 0;
    for (int32_t c : pick) pos[(size_t)c] = -1;
  }
  (*wptr)[(size_t)nw] = (int32_t)wcols->size();
  *wmax = dmax;
  *staged_uses = su;
}

void tag_cold_columns(const CsrView &A, int64_t budget_rows, std::vector<int32_t> *tagged, int64_t *hot_cols,
                      int64_t *hot_nnz) {
  std::vector<int32_t> deg((size_t)A.k, 0);
  for (int64_t p = 0; p < A.nnz; ++p) deg[A.colidx[p]]++;
  int32_t dmax = 0;
  for (int32_t d : deg) dmax = std::max(dmax, d);
  std::vector<int64_t> hist((size_t)dmax + 2, 0);
  for (int32_t d : deg) hist[d]++;
  // smallest D >= 2 with #{deg >= D} <= budget_rows
  int64_t above = 0;
  int32_t D = dmax + 1;
  for (int32_t d = dmax; d >= 2; --d) {
    if (above + hist[d] > budget_rows) break;
    above += hist[d];
    D = d;
  }
  tagged->resize((size_t)A.nnz);
  int64_t hn = 0;
  for (int64_t p = 0; p < A.nnz; ++p) {
    const int32_t c = A.colidx[p];
    const bool hot = deg[c] >= D;
    hn += hot;
    (*tagged)[p] = hot ? c : (int32_t)((uint32_t)c | 0x80000000u);
  }
  *hot_cols = above;
  *hot_nnz = hn;
}

// Planner rules.  The paper ranks templates with a learned energy model whose
// weights are not available; these rules encode the structural evidence it
// relies on instead (Sec. "Sensitivity to Sparsity Patterns"): block formats
// pay only when occupied tiles are nearly full (low rho_BSR), padding and
// serial long rows hurt under row-length imbalance, and a plain row schedule
// is best when rows are regular.  The thresholds were set by measuring every
// family on every workload.
PlanChoice choose_plan(const sd_stats_t &st, int32_t n, int32_t cu_count, int32_t G, const sd_plan_opts_t &o) {
  PlanChoice pc;
  // Heavy rows from 128 nonzeros, cut into chunks of 64 (128 at narrow widths,
  // where a chunk takes a whole wave), run in order of their middle column
  // (chunk_order 2): chunks of different heavy rows that cover the same
  // columns then share their B rows in L2, and shorter chunks cover narrower
  // stretches of columns.  Measured with B streamed from HBM (ms per SpMM):
  //   the four GCN products on R-MAT 2.4 M: 9.75 against 10.3 with T = 256,
  //   c = 128 and 10.6 with T = c = 128 (ordered, the same fix-up), and 13.9
  //   with the earlier T = 512, c = 2048 in row order;
  //   R-MAT 2^20 at N = 128: 0.93 against 1.03 (T = 512, c = 2048 ordered);
  //   at N = 1, 8, 32: 0.099, 0.150, 0.284 with c = 128 against 0.110, 0.165,
  //   0.297 with c = 64 and 0.097, 0.159, 0.315 with T = 512, c = 2048.
  // The fix-up sums a row's partials with a whole wave, so many short chunks
  // cost little there.  The family rule keeps its threshold of 512.
  pc.T = o.heavy_threshold > 0 ? o.heavy_threshold : 128;
  pc.c = o.chunk_nnz > 0 ? o.chunk_nnz : (G > 8 ? 64 : 128);
  const int32_t split_from = o.heavy_threshold > 0 ? o.heavy_threshold : 512;
  if (o.units > 0) {
    pc.U = o.units;
  } else {
    // Merge-path pieces: enough lane groups for ~32 waves per compute unit,
    // and at least 64 path steps per piece.
    const int64_t total = st.m + st.nnz;
    const int64_t groups = (int64_t)std::max(1, cu_count) * 32 * (64 / std::max(1, G));
    const int64_t per_unit = std::max<int64_t>(64, (total + groups - 1) / groups);
    int64_t U = (total + per_unit - 1) / per_unit;
    pc.U = (int32_t)std::max<int64_t>(1, std::min<int64_t>(U, INT32_MAX / 4));
  }
  pc.engine = o.engine;
  pc.policy = o.cache_policy > 0 ? o.cache_policy : 1;
  if (o.force != SD_FMT_AUTO) {
    pc.family = o.force;
  } else if (st.m >= 16 && st.nnz > 0 && st.rho_bsr16 <= 1.3) {
    pc.family = SD_FMT_BSR;
  } else if (st.nnz > 0 && st.rho_ell <= 1.2 && st.row_max <= 64 && n > 1) {
    // near-uniform short rows: ELL drops the row-pointer hop (padding <= 20 %).
    // Not at N = 1, where one lane per row walks its ELL slots alone and rows
    // shared by two lanes run faster (7-point Laplacian: 5.0 against 5.9 us).
    pc.family = SD_FMT_ELL;
  } else if (st.row_max >= split_from) {
    // long rows: cut into chunks (measured faster than merge-path pieces on the
    // power-law workloads: 1.60 vs 2.17 ms at 2^20 vertices, N = 128)
    pc.family = SD_FMT_CSR_SPLIT;
  } else {
    pc.family = SD_FMT_CSR_ROW;
  }
  if ((pc.family == SD_FMT_BSR || pc.family == SD_FMT_BELL) && pc.engine == SD_ENGINE_AUTO)
    pc.engine = SD_ENGINE_MFMA;
  // Workgroup order over the XCDs, measured with B streamed from HBM: the
  // row and merge kernels run faster when all XCDs sweep one band of rows
  // (a B row one XCD fetches, the others find in the Infinity Cache:
  // Laplacian ELL 37 vs 43 us, power-law merge 1.55 vs 1.85 ms); the block
  // kernels run faster with one contiguous range of block-rows per XCD, whose
  // L2 then keeps the B tiles that neighbouring block-rows share (144 vs 155 us).
  // build_plan refines the row families' order to chunked round-robin when the
  // rows' reach fits whole rounds of chunks (chunk_for_reach).
  pc.wg_order = (pc.family == SD_FMT_BSR || pc.family == SD_FMT_BELL) ? 1 : 2;
  return pc;
}

int64_t median_row_reach(const CsrView &A) {
  std::vector<int64_t> reach;
  reach.reserve((size_t)A.m);
  for (int32_t i = 0; i < A.m; ++i) {
    const int32_t p0 = A.rowptr[i], p1 = A.rowptr[i + 1];
    if (p0 == p1) continue;
    // columns ascend, so the farthest column is the first or the last
    const int64_t a = std::llabs((int64_t)A.colidx[p0] - i), b = std::llabs((int64_t)A.colidx[p1 - 1] - i);
    reach.push_back(std::max(a, b));
  }
  if (reach.empty()) return 0;
  const size_t mid = (reach.size() - 1) / 2;  // lower median
  std::nth_element(reach.begin(), reach.begin() + (long)mid, reach.end());
  return reach[mid];
}

int32_t chunk_for_reach(int64_t reach, int64_t rows_per_wg) {
  if (reach <= 0 || rows_per_wg <= 0 || reach % rows_per_wg != 0) return 0;
  const int64_t wgs = reach / rows_per_wg;  // workgroups between a row and its farthest neighbour
  for (int32_t S = 64; S >= 8; S /= 2)
    if (wgs % (8 * (int64_t)S) == 0) return S;
  return 0;
}

// Defaults measured on MI355X (Laplacian, uniform and block workloads): one
// row per lane group with 8 gathers in flight; batching rows per group raises
// register use and lowers occupancy by more than it adds parallelism.
void row_batch_for(const sd_stats_t &st, int64_t rows, int32_t G, int32_t cu_count, int32_t req_J,
                   int32_t req_unr, int32_t *J, int32_t *unr) {
  int32_t u = req_unr > 0 ? req_unr : (st.row_q75 <= 4 ? 4 : 8);
  u = std::min<int32_t>(u, std::max(1, G));
  const int64_t rpw = 64 / std::max(1, G);
  int32_t j = req_J > 0 ? req_J : 1;
  while (j > 1 && (j > G || j * u > 16 || (req_J <= 0 && (rows + rpw * j - 1) / (rpw * j) < 32ll * cu_count)))
    j /= 2;
  *J = j;
  *unr = u;
}

int32_t slices_for(const sd_stats_t &st, int32_t family, int32_t n, int32_t G) {
  (void)n;
  if ((family != SD_FMT_CSR_ROW && family != SD_FMT_CSR_SPLIT) || G > 8) return 1;
  // Heavy split: light rows of 8 lanes (16 at G = 8), measured on the
  // power-law workloads (R-MAT 2^20: 0.105 ms at N = 1 with 8 slices against
  // 0.19 without; 0.17 ms at N = 8 with 4 against 0.26; 0.35 ms at N = 32 with
  // 2 against 0.39; the GCN products agree at N = 8 and 32).
  if (family == SD_FMT_CSR_SPLIT) return std::max(2, 8 / G);
  // Row kernel: the power of two nearest a mean row's rounds of kSliceRound
  // nonzeros, at most 8 lanes per row (7-point Laplacian at N = 1: 5.0 us with
  // 2 slices against 6.1 without and 8.9 with 8; at N = 32 one group per row
  // is fastest).
  const double rounds = st.row_mean / kSliceRound;
  int32_t S = 1;
  while (2 * S <= 8 / G && 1.5 * S < rounds) S *= 2;
  return S;
}

}  // namespace sd
