// Host-only parts of libnmd that involve no device: the seeded block schedule, the balanced
// partition, CSR validation and the arrangement of S per block.  Plain C++17 (no HIP headers),
// so that it also builds with g++ under the address and undefined-behaviour sanitizers.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace nmd {

constexpr int kItemChunk = 128;  // entries per sparse work item

// One unit of sparse work: `count` consecutive entries (begin .. begin+count) of one row of a
// block.  slot < 0: the row has a single item and its result is added to Y directly; else the
// partial result goes to scratch row `slot` and a fix-up pass adds the row's slots in order.
struct Item {
  int64_t begin;
  int32_t count;
  int32_t row;
  int32_t slot;
  int32_t pad;
};

// A row whose entries were split over several items: slots first .. first+nslots-1.
struct Split {
  int32_t row;
  int32_t first;
  int32_t nslots;
  int32_t pad;
};

// Per-sweep block order: +(k+1) = W-step on column block k, -(k+1) = H-step on row block k.
std::vector<int32_t> make_schedule(uint64_t seed, int64_t t, int32_t R, int32_t C,
                                   bool stochastic);
// Bounds of the K = ceil(size / block) balanced blocks [floor(k size / K), floor((k+1) size / K)).
std::vector<int64_t> balanced_bounds(int64_t size, int64_t block);

// The entries of S arranged for the updates of one factor.  For the W side the "rows" are the
// m rows of S and the blocks split the n columns; for the H side the rows are the n columns of S
// and the blocks split its m rows (the transposed problem).
struct SideHost {
  int64_t rows = 0, other = 0;
  std::vector<int64_t> bounds;     // block bounds over `other`
  std::vector<int64_t> entry_off;  // entries of block b: [entry_off[b], entry_off[b+1])
  std::vector<int32_t> idx;        // index into `other`
  std::vector<float> val;
  std::vector<int64_t> item_off;   // items of block b
  std::vector<Item> items;
  std::vector<int64_t> split_off;  // split rows of block b
  std::vector<Split> splits;
  std::vector<int64_t> rowptr;     // block b, row i: entries [rowptr[b(rows+1)+i], ..+1])
  int64_t max_slots = 0;

  int32_t nblk() const { return (int32_t)bounds.size() - 1; }
};

// ptr/idx/val: the rows of this side in compressed form (entries sorted within a row).
void build_side(SideHost& sd, int64_t rows, int64_t other, const std::vector<int64_t>& bounds,
                const int64_t* ptr, const int32_t* idx, const float* val);

// A compressed matrix: rows (or columns) i hold entries ptr[i] .. ptr[i+1].
struct Compressed {
  std::vector<int64_t> ptr;
  std::vector<int32_t> idx;
  std::vector<float> val;
};

// Validates an m x n CSR matrix (row_ptr[0] = 0, non-decreasing, row_ptr[m] = nnz; columns in
// range and strictly increasing within a row; values finite and >= 0), keeps its positive
// entries in `rows` (CSR) and `cols` (CSC, rows ascending within a column) and their sum of
// squares in *s2.  Returns an empty string, or the reason the matrix was rejected (then the
// outputs are unspecified).  Throws std::bad_alloc when memory runs out.
std::string ingest_csr(int64_t m, int64_t n, int64_t nnz, const int64_t* row_ptr,
                       const int32_t* col_idx, const float* values, Compressed& rows,
                       Compressed& cols, double* s2);

}  // namespace nmd
