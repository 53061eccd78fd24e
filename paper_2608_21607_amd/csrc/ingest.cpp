// Host-only parts of libnmd: schedule, partition, CSR validation, per-block arrangement of S.

#include "ingest.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>

namespace nmd {

namespace {

// ------------------------------------------------------------------------------ schedule --
// SplitMix64 (Steele, Lea and Flood 2014), Lemire's bounded integers (2019), Fisher-Yates
// (Durstenfeld order), and a proportional merge of column-block and row-block steps.
struct SplitMix64 {
  uint64_t s;
  uint64_t next() {
    s += 0x9E3779B97F4A7C15ULL;
    uint64_t z = s;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
  }
};

uint64_t bounded(SplitMix64& g, uint64_t k) {
  unsigned __int128 prod = (unsigned __int128)g.next() * k;
  uint64_t low = (uint64_t)prod;
  if (low < k) {
    const uint64_t thresh = (0 - k) % k;  // (2^64 - k) mod k
    while (low < thresh) {
      prod = (unsigned __int128)g.next() * k;
      low = (uint64_t)prod;
    }
  }
  return (uint64_t)(prod >> 64);
}

std::vector<int32_t> permutation(SplitMix64& g, int32_t k) {
  std::vector<int32_t> a(k);
  for (int32_t i = 0; i < k; ++i) a[i] = i;
  for (int32_t i = k - 1; i > 0; --i) {
    const int32_t j = (int32_t)bounded(g, (uint64_t)i + 1);
    std::swap(a[i], a[j]);
  }
  return a;
}

}  // namespace

std::vector<int32_t> make_schedule(uint64_t seed, int64_t t, int32_t R, int32_t C,
                                   bool stochastic) {
  std::vector<int32_t> out;
  out.reserve((size_t)R + C);
  if (!stochastic) {
    for (int32_t k = 0; k < C; ++k) out.push_back(k + 1);
    for (int32_t k = 0; k < R; ++k) out.push_back(-(k + 1));
    return out;
  }
  SplitMix64 g{seed ^ ((uint64_t)t * 0x9E3779B97F4A7C15ULL)};
  const std::vector<int32_t> sigma = permutation(g, C);
  const std::vector<int32_t> pi = permutation(g, R);
  int64_t w = 0, h = 0;
  while (w < C || h < R) {
    if (h == R || (w < C && (2 * w + 1) * (int64_t)R <= (2 * h + 1) * (int64_t)C)) {
      out.push_back(sigma[w] + 1);
      ++w;
    } else {
      out.push_back(-(pi[h] + 1));
      ++h;
    }
  }
  return out;
}

std::vector<int64_t> balanced_bounds(int64_t size, int64_t block) {
  const int64_t K = (size + block - 1) / block;
  std::vector<int64_t> b(K + 1);
  for (int64_t k = 0; k <= K; ++k) b[k] = (int64_t)(((__int128)k * size) / K);
  return b;
}

// ptr/idx/val: the rows of this side in compressed form (entries sorted within a row).
void build_side(SideHost& sd, int64_t rows, int64_t other, const std::vector<int64_t>& bounds,
                const int64_t* ptr, const int32_t* idx, const float* val) {
  sd.rows = rows;
  sd.other = other;
  sd.bounds = bounds;
  const int32_t nb = sd.nblk();
  std::vector<int32_t> blk_of(other);
  for (int32_t b = 0; b < nb; ++b)
    for (int64_t j = bounds[b]; j < bounds[b + 1]; ++j) blk_of[j] = b;
  std::vector<int64_t> cnt(nb, 0);
  const int64_t nnz = ptr[rows];
  for (int64_t e = 0; e < nnz; ++e) ++cnt[blk_of[idx[e]]];
  sd.entry_off.assign(nb + 1, 0);
  for (int32_t b = 0; b < nb; ++b) sd.entry_off[b + 1] = sd.entry_off[b] + cnt[b];
  sd.idx.resize(nnz);
  sd.val.resize(nnz);
  std::vector<int64_t> cur(sd.entry_off.begin(), sd.entry_off.end() - 1);
  std::vector<std::vector<Item>> items(nb);
  std::vector<std::vector<Split>> splits(nb);
  std::vector<int32_t> slots(nb, 0);
  sd.rowptr.assign((size_t)nb * (rows + 1), 0);
  for (int32_t b = 0; b < nb; ++b) sd.rowptr[(size_t)b * (rows + 1)] = sd.entry_off[b];
  for (int64_t i = 0; i < rows; ++i) {
    int64_t e = ptr[i];
    const int64_t e1 = ptr[i + 1];
    while (e < e1) {
      const int32_t b = blk_of[idx[e]];
      int64_t f = e;
      while (f < e1 && idx[f] < bounds[b + 1]) ++f;
      const int64_t count = f - e;
      const int64_t base = cur[b];
      std::memcpy(&sd.idx[base], idx + e, count * sizeof(int32_t));
      std::memcpy(&sd.val[base], val + e, count * sizeof(float));
      cur[b] += count;
      if (count <= kItemChunk) {
        items[b].push_back(Item{base, (int32_t)count, (int32_t)i, -1, 0});
      } else {
        const int32_t pieces = (int32_t)((count + kItemChunk - 1) / kItemChunk);
        splits[b].push_back(Split{(int32_t)i, slots[b], pieces, 0});
        for (int32_t p = 0; p < pieces; ++p) {
          const int64_t s0 = (int64_t)p * kItemChunk;
          const int64_t c = std::min<int64_t>(kItemChunk, count - s0);
          items[b].push_back(Item{base + s0, (int32_t)c, (int32_t)i, slots[b] + p, 0});
        }
        slots[b] += pieces;
      }
      e = f;
    }
    for (int32_t b = 0; b < nb; ++b) sd.rowptr[(size_t)b * (rows + 1) + i + 1] = cur[b];
  }
  sd.item_off.assign(nb + 1, 0);
  sd.split_off.assign(nb + 1, 0);
  sd.items.clear();
  sd.splits.clear();
  sd.max_slots = 0;
  for (int32_t b = 0; b < nb; ++b) {
    sd.item_off[b + 1] = sd.item_off[b] + (int64_t)items[b].size();
    sd.split_off[b + 1] = sd.split_off[b] + (int64_t)splits[b].size();
    sd.items.insert(sd.items.end(), items[b].begin(), items[b].end());
    sd.splits.insert(sd.splits.end(), splits[b].begin(), splits[b].end());
    sd.max_slots = std::max<int64_t>(sd.max_slots, slots[b]);
  }
}


std::string ingest_csr(int64_t m, int64_t n, int64_t nnz, const int64_t* row_ptr,
                       const int32_t* col_idx, const float* values, Compressed& rows,
                       Compressed& cols, double* s2) {
  char buf[256];
  if (row_ptr[0] != 0) {
    snprintf(buf, sizeof buf, "row_ptr[0] = %lld, expected 0", (long long)row_ptr[0]);
    return buf;
  }
  for (int64_t i = 0; i < m; ++i)
    if (row_ptr[i + 1] < row_ptr[i]) {
      snprintf(buf, sizeof buf, "row_ptr decreases at row %lld", (long long)i);
      return buf;
    }
  if (row_ptr[m] != nnz) {
    snprintf(buf, sizeof buf, "row_ptr[m] = %lld differs from nnz = %lld", (long long)row_ptr[m],
             (long long)nnz);
    return buf;
  }
  for (int64_t i = 0; i < m; ++i) {
    for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
      const int32_t j = col_idx[e];
      if (j < 0 || j >= n) {
        snprintf(buf, sizeof buf, "column index %d out of range in row %lld", j, (long long)i);
        return buf;
      }
      if (e > row_ptr[i] && j <= col_idx[e - 1]) {
        snprintf(buf, sizeof buf, "column indices not strictly increasing in row %lld",
                 (long long)i);
        return buf;
      }
      const float v = values[e];
      if (!std::isfinite(v) || v < 0.0f) {
        snprintf(buf, sizeof buf, "value at row %lld, column %d is negative or not finite",
                 (long long)i, j);
        return buf;
      }
    }
  }
  // keep the positive entries only (the mask of the Z-update is S_ij > 0)
  rows.ptr.assign(m + 1, 0);
  rows.idx.clear();
  rows.val.clear();
  rows.idx.reserve(nnz);
  rows.val.reserve(nnz);
  double sum2 = 0.0;
  for (int64_t i = 0; i < m; ++i) {
    for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
      if (values[e] > 0.0f) {
        rows.idx.push_back(col_idx[e]);
        rows.val.push_back(values[e]);
        sum2 += (double)values[e] * values[e];
      }
    }
    rows.ptr[i + 1] = (int64_t)rows.idx.size();
  }
  const int64_t nz = (int64_t)rows.idx.size();
  if (nz == 0) return "S has no positive entry";
  // column-compressed copy for the H side (rows ascending inside each column)
  cols.ptr.assign(n + 1, 0);
  for (int64_t e = 0; e < nz; ++e) ++cols.ptr[rows.idx[e] + 1];
  for (int64_t j = 0; j < n; ++j) cols.ptr[j + 1] += cols.ptr[j];
  cols.idx.assign(nz, 0);
  cols.val.assign(nz, 0.0f);
  std::vector<int64_t> cur(cols.ptr.begin(), cols.ptr.end() - 1);
  for (int64_t i = 0; i < m; ++i)
    for (int64_t e = rows.ptr[i]; e < rows.ptr[i + 1]; ++e) {
      const int64_t d = cur[rows.idx[e]]++;
      cols.idx[d] = (int32_t)i;
      cols.val[d] = rows.val[e];
    }
  *s2 = sum2;
  return std::string();
}

}  // namespace nmd
