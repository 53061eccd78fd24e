// Checks the host-only ingest code of libnmd (csrc/ingest.cpp) outside the GPU library, built
// with g++ and the address and undefined-behaviour sanitizers by tests/test_native_ingest.py.
//
//   ingest_check <input.bin>    input: int64 m, n, nnz, block_m, block_n, then row_ptr (m+1
//                               int64), col (nnz int32), val (nnz float32)
//   ingest_check --schedule seed t R C
//
// Prints one JSON object: the rejection reason, or the per-block entry counts of both sides
// and the item and split counts after checking every structural invariant (exit status 1 and
// a FAIL line on the first violation).

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../paper_2608_21607_amd/csrc/ingest.h"

namespace {

void fail(const char* what, long long a = 0, long long b = 0) {
  std::printf("FAIL %s %lld %lld\n", what, a, b);
  std::exit(1);
}

// Every invariant the GPU kernels rely on.
void check_side(const nmd::SideHost& sd, const nmd::Compressed& src) {
  const int32_t nb = sd.nblk();
  const int64_t nz = (int64_t)src.idx.size();
  if ((int64_t)sd.idx.size() != nz || (int64_t)sd.val.size() != nz) fail("entry count");
  if (sd.entry_off.size() != (size_t)nb + 1 || sd.entry_off[0] != 0 || sd.entry_off[nb] != nz)
    fail("entry_off ends");
  std::vector<char> seen_slot;
  for (int32_t b = 0; b < nb; ++b) {
    const int64_t e0 = sd.entry_off[b], e1 = sd.entry_off[b + 1];
    if (e1 < e0) fail("entry_off order", b);
    // row pointers of the block cover its entries in row order, each in the block's range
    const int64_t* rp = &sd.rowptr[(size_t)b * (sd.rows + 1)];
    if (rp[0] != e0 || rp[sd.rows] != e1) fail("rowptr ends", b);
    for (int64_t i = 0; i < sd.rows; ++i) {
      if (rp[i + 1] < rp[i]) fail("rowptr order", b, i);
      for (int64_t e = rp[i]; e < rp[i + 1]; ++e) {
        const int32_t j = sd.idx[e];
        if (j < sd.bounds[b] || j >= sd.bounds[b + 1]) fail("index outside block", b, e);
        if (e > rp[i] && j <= sd.idx[e - 1]) fail("indices not increasing", b, e);
        if (!(sd.val[e] > 0.0f)) fail("non-positive value", b, e);
      }
    }
    // items cover the block's entries exactly once, in order, at most kItemChunk each
    int64_t next = e0;
    for (int64_t k = sd.item_off[b]; k < sd.item_off[b + 1]; ++k) {
      const nmd::Item& it = sd.items[k];
      if (it.begin != next || it.count < 1 || it.count > nmd::kItemChunk) fail("item", b, k);
      if (it.row < 0 || it.row >= sd.rows) fail("item row", b, k);
      if (it.begin < rp[it.row] || it.begin + it.count > rp[it.row + 1]) fail("item span", b, k);
      if (it.slot >= sd.max_slots) fail("item slot", b, k);
      next += it.count;
    }
    if (next != e1) fail("items do not cover the block", b);
    // split rows: their items carry consecutive slots first .. first + nslots - 1
    seen_slot.assign((size_t)sd.max_slots + 1, 0);
    for (int64_t s = sd.split_off[b]; s < sd.split_off[b + 1]; ++s) {
      const nmd::Split& sp = sd.splits[s];
      if (sp.nslots < 2 || sp.first < 0 || sp.first + sp.nslots > sd.max_slots) fail("split", b, s);
      if (rp[sp.row + 1] - rp[sp.row] <= nmd::kItemChunk) fail("split of a short row", b, s);
      for (int32_t q = 0; q < sp.nslots; ++q) {
        if (seen_slot[sp.first + q]) fail("slot used twice", b, s);
        seen_slot[sp.first + q] = 1;
      }
    }
    for (int64_t k = sd.item_off[b]; k < sd.item_off[b + 1]; ++k) {
      const nmd::Item& it = sd.items[k];
      const int64_t len = rp[it.row + 1] - rp[it.row];
      if ((len > nmd::kItemChunk) != (it.slot >= 0)) fail("slot of a row", b, k);
      if (it.slot >= 0 && !seen_slot[it.slot]) fail("slot without split", b, k);
    }
  }
}

void print_counts(const char* name, const nmd::SideHost& sd) {
  std::printf("\"%s\": {\"nnz\": [", name);
  for (int32_t b = 0; b < sd.nblk(); ++b)
    std::printf("%s%lld", b ? ", " : "", (long long)(sd.entry_off[b + 1] - sd.entry_off[b]));
  std::printf("], \"items\": %zu, \"splits\": %zu, \"max_slots\": %lld}", sd.items.size(),
              sd.splits.size(), (long long)sd.max_slots);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc == 6 && std::strcmp(argv[1], "--schedule") == 0) {
    const std::vector<int32_t> s =
        nmd::make_schedule(std::strtoull(argv[2], nullptr, 10), std::atoll(argv[3]),
                           std::atoi(argv[4]), std::atoi(argv[5]), true);
    std::printf("{\"schedule\": [");
    for (size_t k = 0; k < s.size(); ++k) std::printf("%s%d", k ? ", " : "", s[k]);
    std::printf("]}\n");
    return 0;
  }
  if (argc != 2) return 2;
  FILE* f = std::fopen(argv[1], "rb");
  if (!f) return 2;
  int64_t hdr[5];
  if (std::fread(hdr, sizeof(int64_t), 5, f) != 5) return 2;
  const int64_t m = hdr[0], n = hdr[1], nnz = hdr[2], bm = hdr[3], bn = hdr[4];
  std::vector<int64_t> row_ptr(m + 1);
  std::vector<int32_t> col(nnz);
  std::vector<float> val(nnz);
  if (std::fread(row_ptr.data(), sizeof(int64_t), m + 1, f) != (size_t)(m + 1) ||
      std::fread(col.data(), sizeof(int32_t), nnz, f) != (size_t)nnz ||
      std::fread(val.data(), sizeof(float), nnz, f) != (size_t)nnz)
    return 2;
  std::fclose(f);
  nmd::Compressed rows, cols;
  double s2 = 0.0;
  const std::string why = nmd::ingest_csr(m, n, nnz, row_ptr.data(), col.data(), val.data(), rows,
                                          cols, &s2);
  if (!why.empty()) {
    std::printf("{\"error\": \"%s\"}\n", why.c_str());
    return 0;
  }
  const std::vector<int64_t> rb = nmd::balanced_bounds(m, bm), cb = nmd::balanced_bounds(n, bn);
  nmd::SideHost ws, hs;
  nmd::build_side(ws, m, n, cb, rows.ptr.data(), rows.idx.data(), rows.val.data());
  nmd::build_side(hs, n, m, rb, cols.ptr.data(), cols.idx.data(), cols.val.data());
  check_side(ws, rows);
  check_side(hs, cols);
  std::printf("{\"s2\": %.17g, ", s2);
  print_counts("w", ws);
  std::printf(", ");
  print_counts("h", hs);
  std::printf("}\n");
  return 0;
}
