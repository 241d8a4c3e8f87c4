// Internal declarations shared by the host encoder/upload code and the device code.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "toc.h"

// One encoded mini-batch: (I, D) of Algorithm 1 plus counts of its prefix tree,
// gathered while encoding (the tree itself is not kept: C' is rebuilt from (I, D)
// by Algorithm 2 at upload time).
struct toc_enc {
  int32_t n_rows = 0, n_cols = 0;
  int64_t nnz = 0;
  std::vector<int32_t> I_col;
  std::vector<uint32_t> I_bits;
  std::vector<int64_t> D_rowptr;  // n_rows + 1
  std::vector<uint32_t> D_codes;  // paper numbering, 1..n_nodes-1
  int64_t n_nodes = 1;            // including the root
  int64_t n_live = 0, n_deep_live = 0;
  int32_t max_depth_live = 0, max_depth_all = 0;
  int64_t n_deep_all = 0;
  int64_t n_int1_live = 0, n_int1_all = 0;  // depth-1 codes with (live / any) children
};

struct toc_dev {
  void *buf = nullptr;
  size_t bytes = 0;
  bool host = false;
  int device = -1;
  uint32_t flags = 0;
  toc_layout layout{};
  toc_dev_info info{};
  std::vector<toc_batch> batches;  // host copy of the batch table
  int32_t max_rows = 0, max_codes = 0, max_levels = 0;
  int32_t max_ucols = 0;           // most distinct key columns of a batch (after build)
  int64_t max_keylinks = 0;        // most keys plus deep links of a batch (after build)
  int64_t max_deep = 0, max_tree = 0, max_d = 0;
  // most deep codes of two batches b, b + 8 with b / 8 even (the batch pairs of
  // the right product's tiled kernel)
  int64_t max_pair_deep = 0;
  int64_t total_deep = 0, total_tree = 0;
  std::vector<int64_t> dtile_base;  // first decode tile of each batch
  int64_t n_dtiles = 0;
  int64_t tot_levels = 0;           // level entries over all batches
  // image planned from physical bytes on the device and not yet built (the
  // per-batch counts of those bytes, kept for the build)
  bool pending = false;
  std::vector<toc_phys_info> phys;
};

namespace toc {

// Entries of D per decode tile (one independent workgroup each).
constexpr int64_t kDecodeTile = 1024;

// Marks a tree code in the column entries (centry) of the image; leaf
// occurrence words there hold a row below 2^30 and the first-occurrence bit.
constexpr uint32_t kTreeEntry = 0x40000000u;
constexpr int64_t kMaxBatchDim = (int64_t)1 << 30;   // rows and codes per batch

// Records a message for toc_last_error() and returns s.
toc_status fail(toc_status s, const char *fmt, ...);
void clear_error();

// Builds the upload image into `dst` (host memory of layout.end bytes).
toc_status build_image(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                       toc_dev *dev, uint8_t *dst);
// Writes the arrays of batches b0 .. b1-1 (host threads) at the offsets of layout
// L from dst: with L shifted per array, into a staging area holding only those
// batches' slices.  The batch table is not written.
toc_status write_batches(const toc_enc *const *encs, int64_t b0, int64_t b1, uint32_t flags,
                         const toc_layout &L, toc_dev *dev, uint8_t *dst);
// After every batch is written: maxima only the build computes.
void finish_image(toc_dev *dev);
// Element index at which batch b's slice of each per-batch array starts (b equal
// to the batch count: the arrays' ends).
struct ArrStarts {
  int64_t level, code, deep, span, d, tree, dtile, cols, b;
};
ArrStarts arr_starts(const toc_dev *dev, int64_t b);
// Computes layout and totals only.
toc_status plan_image(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                      toc_dev *dev);
// The counts of one batch that the layout depends on: tuples, stored codes, depth
// of the deepest stored code, |D|, stored codes of depth >= 2, depth-1 codes with
// children, nonzeros, and the canonical bytes (toc_dev_info.canon_bytes).
struct BatchCounts {
  int64_t rows, codes, levels, d, deep, int1, nnz, canon;
};
// Layout, batch table bases and totals from per-batch counts (the tables' n_lvl1
// and n_ucols are left to the writer).
toc_status plan_layout(const BatchCounts *bc, int64_t n_batches, int32_t n_cols, uint32_t flags,
                       toc_dev *dev);

}  // namespace toc
