// Host side of libtoc: sparse + logical encoding (Algorithm 1), sizes, and the
// upload image (Algorithm 2, live codes, level order).  Plain C++17, no HIP calls.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <thread>

#include "toc_internal.h"

namespace toc {

static thread_local std::string g_err;

toc_status fail(toc_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

void clear_error() { g_err.clear(); }

// ---------------------------------------------------------------------------
// Prefix tree C of section 3.1.1.  GetIndex(n, key) / AddNode(n, key) are served
// by one open-addressing table keyed by (node, column, value bits): the per-node
// child maps of the paper folded into a single hash table.
// ---------------------------------------------------------------------------
static_assert(sizeof(toc_key) == 8 && sizeof(toc_link) == 8, "toc_key and toc_link are 8 bytes");

namespace {

struct Slot {
  uint32_t node, col, bits, child;  // child == 0 marks an empty slot
};

class Trie {
 public:
  void reset(int64_t max_nodes) {
    size_t cap = 16;
    while (cap < (size_t)(2 * max_nodes + 16)) cap <<= 1;
    if (slots_.size() < cap) slots_.assign(cap, Slot{0, 0, 0, 0});
    else std::memset(slots_.data(), 0, cap * sizeof(Slot));
    mask_ = cap - 1;
  }
  // GetIndex: child index, or 0 when absent (0 is never a child).
  uint32_t get(uint32_t node, uint32_t col, uint32_t bits) const {
    size_t h = hash(node, col, bits) & mask_;
    for (;;) {
      const Slot &s = slots_[h];
      if (s.child == 0) return 0;
      if (s.node == node && s.col == col && s.bits == bits) return s.child;
      h = (h + 1) & mask_;
    }
  }
  // AddNode with a known-absent key.
  void add(uint32_t node, uint32_t col, uint32_t bits, uint32_t child) {
    size_t h = hash(node, col, bits) & mask_;
    while (slots_[h].child != 0) h = (h + 1) & mask_;
    slots_[h] = Slot{node, col, bits, child};
  }

 private:
  static size_t hash(uint32_t node, uint32_t col, uint32_t bits) {
    uint64_t x = (uint64_t)node * 0x9E3779B97F4A7C15ull;
    x ^= ((uint64_t)col << 32 | bits) * 0xC2B2AE3D27D4EB4Full;
    x ^= x >> 31;
    x *= 0xBF58476D1CE4E5B9ull;
    x ^= x >> 29;
    return (size_t)x;
  }
  std::vector<Slot> slots_;
  size_t mask_ = 0;
};

// Per-thread scratch reused across batches.
struct EncScratch {
  Trie trie;
  std::vector<uint32_t> rcol, rbits;   // kept pairs of the batch (zeros dropped)
  std::vector<int64_t> rptr;
  std::vector<uint32_t> parent;        // encoder-side parent of each node
  std::vector<int32_t> depth;
  std::vector<uint8_t> live;
};

inline bool is_finite_bits(uint32_t b) { return (b & 0x7F800000u) != 0x7F800000u; }

toc_status encode_one(int32_t n_rows, int32_t n_cols, const int64_t *rowptr,
                      const int32_t *col, const float *val, EncScratch &S,
                      toc_enc *e) {
  if (n_rows < 0 || n_cols < 0) return fail(TOC_EINVAL, "negative shape");
  if (!rowptr) return fail(TOC_EINVAL, "rowptr is NULL");
  if (rowptr[0] != 0) return fail(TOC_EINVAL, "rowptr[0] must be 0");
  const int64_t total = rowptr[n_rows];
  if (total < 0) return fail(TOC_EINVAL, "rowptr[n_rows] negative");
  if (total > 0 && (!col || !val)) return fail(TOC_EINVAL, "col/val is NULL");
  // --- validation + sparse encoding (drop zeros) ---
  S.rcol.clear();
  S.rbits.clear();
  S.rptr.assign((size_t)n_rows + 1, 0);
  for (int32_t i = 0; i < n_rows; ++i) {
    const int64_t a = rowptr[i], b = rowptr[i + 1];
    if (b < a || b > total) return fail(TOC_EINVAL, "rowptr not non-decreasing at row %d", i);
    int64_t prev = -1;
    for (int64_t p = a; p < b; ++p) {
      const int32_t c = col[p];
      if (c < 0 || c >= n_cols) return fail(TOC_EINVAL, "column %d out of range at row %d", c, i);
      if (c <= prev) return fail(TOC_EINVAL, "columns not strictly increasing at row %d", i);
      prev = c;
      uint32_t bits;
      std::memcpy(&bits, &val[p], 4);
      if (!is_finite_bits(bits)) return fail(TOC_EINVAL, "non-finite value at row %d", i);
      if ((bits & 0x7FFFFFFFu) == 0) continue;  // +0.0 / -0.0 are not stored
      S.rcol.push_back((uint32_t)c);
      S.rbits.push_back(bits);
    }
    S.rptr[i + 1] = (int64_t)S.rcol.size();
  }
  const int64_t nnz = (int64_t)S.rcol.size();
  if (2 * nnz + 1 > INT32_MAX) return fail(TOC_EUNSUPPORTED, "batch too large for 32-bit codes");
  e->n_rows = n_rows;
  e->n_cols = n_cols;
  e->nnz = nnz;
  S.trie.reset(2 * nnz + 1);
  S.parent.assign(1, 0);
  S.depth.assign(1, 0);
  uint32_t next = 1;  // sequence number of the next node; the root is node 0
  // --- phase I: distinct pairs under the root, first appearance first ---
  e->I_col.clear();
  e->I_bits.clear();
  for (int64_t p = 0; p < nnz; ++p) {
    if (S.trie.get(0, S.rcol[p], S.rbits[p]) == 0) {
      S.trie.add(0, S.rcol[p], S.rbits[p], next++);
      e->I_col.push_back((int32_t)S.rcol[p]);
      e->I_bits.push_back(S.rbits[p]);
      S.parent.push_back(0);
      S.depth.push_back(1);
    }
  }
  // --- phase II: greedy longest matches; one new node after each non-final match
  e->D_rowptr.assign((size_t)n_rows + 1, 0);
  e->D_codes.clear();
  e->D_codes.reserve((size_t)nnz);
  for (int32_t i = 0; i < n_rows; ++i) {
    const int64_t end = S.rptr[i + 1];
    int64_t j = S.rptr[i];
    while (j < end) {
      // LongestMatchFromTree: the first pair always matches (phase I).
      uint32_t n = S.trie.get(0, S.rcol[j], S.rbits[j]);
      ++j;
      while (j < end) {
        const uint32_t nx = S.trie.get(n, S.rcol[j], S.rbits[j]);
        if (nx == 0) break;
        n = nx;
        ++j;
      }
      e->D_codes.push_back(n);
      if (j < end) {
        S.trie.add(n, S.rcol[j], S.rbits[j], next++);
        S.parent.push_back(n);
        S.depth.push_back(S.depth[n] + 1);
      }
    }
    e->D_rowptr[i + 1] = (int64_t)e->D_codes.size();
  }
  e->n_nodes = next;
  // --- counts of the tree: live codes are those referenced by D and their
  // ancestors; parents always have smaller indices than their children.
  // flags: 1 live, 2 has a live child, 4 has a child
  S.live.assign(next, 0);
  for (uint32_t c : e->D_codes) S.live[c] = 1;
  int64_t n_live = 0, n_deep_live = 0, n_deep_all = 0;
  int32_t md_live = 0, md_all = 0;
  for (int64_t c = (int64_t)next - 1; c >= 1; --c) {
    md_all = std::max(md_all, S.depth[c]);
    if (S.depth[c] >= 2) ++n_deep_all;
    S.live[S.parent[c]] |= 4;
    if (!(S.live[c] & 1)) continue;
    ++n_live;
    if (S.depth[c] >= 2) ++n_deep_live;
    md_live = std::max(md_live, S.depth[c]);
    S.live[S.parent[c]] |= 1 | 2;
  }
  int64_t ni_live = 0, ni_all = 0;
  for (int64_t c = 1; c < (int64_t)next && S.depth[c] == 1; ++c) {
    ni_live += (S.live[c] & 2) != 0;
    ni_all += (S.live[c] & 4) != 0;
  }
  e->n_int1_live = ni_live;
  e->n_int1_all = ni_all;
  e->n_live = n_live;
  e->n_deep_live = n_deep_live;
  e->n_deep_all = n_deep_all;
  e->max_depth_live = md_live;
  e->max_depth_all = md_all;
  return TOC_OK;
}

// Bit packing of section 3.3: ceil(log2(max+1)/8) bytes per integer (at least 1)
// plus a 5-byte header (u32 count, u8 bytes per integer).
int64_t packed_bytes(uint64_t max_value, int64_t count) {
  int width = 1;
  if (max_value > 0) {
    int bits = 0;
    while (bits < 64 && (max_value >> bits) != 0) ++bits;  // = ceil(log2(max+1))
    width = std::max(1, (bits + 7) / 8);
  }
  return 5 + (int64_t)width * count;
}

int64_t physical_size(const toc_enc *e) {
  std::vector<uint32_t> u(e->I_bits);
  std::sort(u.begin(), u.end());
  u.erase(std::unique(u.begin(), u.end()), u.end());
  uint64_t max_col = 0, max_vi = u.empty() ? 0 : u.size() - 1, max_code = 0;
  for (int32_t c : e->I_col) max_col = std::max<uint64_t>(max_col, (uint64_t)c);
  for (uint32_t c : e->D_codes) max_code = std::max<uint64_t>(max_code, c);
  const int64_t nI = (int64_t)e->I_col.size();
  int64_t s = packed_bytes(max_col, nI);
  s += 5 + 4 * (int64_t)u.size();
  s += packed_bytes(max_vi, nI);
  s += packed_bytes(max_code, (int64_t)e->D_codes.size());
  s += packed_bytes((uint64_t)e->D_codes.size(), (int64_t)e->n_rows + 1);
  return s;
}

}  // namespace
}  // namespace toc

using namespace toc;

extern "C" {

const char *toc_last_error(void) { return g_err.c_str(); }

toc_status toc_encode(int32_t n_rows, int32_t n_cols, const int64_t *rowptr,
                      const int32_t *col, const float *val, toc_enc **out) {
  if (!out) return fail(TOC_EINVAL, "out is NULL");
  *out = nullptr;
  toc_enc *e = new (std::nothrow) toc_enc;
  if (!e) return fail(TOC_ENOMEM, "out of host memory");
  try {
    EncScratch S;
    toc_status st = encode_one(n_rows, n_cols, rowptr, col, val, S, e);
    if (st != TOC_OK) {
      delete e;
      return st;
    }
  } catch (const std::bad_alloc &) {
    delete e;
    return fail(TOC_ENOMEM, "out of host memory");
  }
  *out = e;
  return TOC_OK;
}

toc_status toc_encode_batches(int64_t n_batches, const int32_t *n_rows, int32_t n_cols,
                              const int64_t *rowptr, const int32_t *col,
                              const float *val, int32_t n_threads, toc_enc **out) {
  if (!out) return fail(TOC_EINVAL, "out is NULL");
  if (n_batches < 0) return fail(TOC_EINVAL, "n_batches < 0");
  if (n_batches == 0) return TOC_OK;
  if (!n_rows || !rowptr) return fail(TOC_EINVAL, "NULL pointer");
  std::vector<int64_t> row_off((size_t)n_batches + 1, 0);
  for (int64_t b = 0; b < n_batches; ++b) {
    out[b] = nullptr;
    if (n_rows[b] < 0) return fail(TOC_EINVAL, "n_rows[%lld] < 0", (long long)b);
    row_off[b + 1] = row_off[b] + n_rows[b];
  }
  if (rowptr[0] != 0) return fail(TOC_EINVAL, "rowptr[0] must be 0");
  int nt = n_threads > 0 ? n_threads : (int)std::max(1u, std::thread::hardware_concurrency());
  nt = (int)std::min<int64_t>(nt, n_batches);
  std::atomic<int64_t> next{0};
  std::atomic<int> first_err{0};
  std::vector<std::string> errs((size_t)nt);
  auto work = [&](int tid) {
    EncScratch S;
    for (;;) {
      const int64_t b = next.fetch_add(1);
      if (b >= n_batches || first_err.load() != 0) return;
      toc_enc *e = new (std::nothrow) toc_enc;
      toc_status st = e ? TOC_OK : TOC_ENOMEM;
      if (e) {
        try {
          const int64_t *rp = rowptr + row_off[b];
          const int64_t base = rp[0];
          // rebase this batch's rowptr to start at 0
          std::vector<int64_t> local((size_t)n_rows[b] + 1);
          for (int32_t i = 0; i <= n_rows[b]; ++i) local[i] = rp[i] - base;
          if (base < 0) st = fail(TOC_EINVAL, "rowptr decreasing");
          else
            st = encode_one(n_rows[b], n_cols, local.data(), col ? col + base : nullptr,
                            val ? val + base : nullptr, S, e);
        } catch (const std::bad_alloc &) {
          st = fail(TOC_ENOMEM, "out of host memory");
        }
      }
      if (st != TOC_OK) {
        int expect = 0;
        if (first_err.compare_exchange_strong(expect, (int)st))
          errs[tid] = std::string("batch ") + std::to_string(b) + ": " + g_err;
        delete e;
        return;
      }
      out[b] = e;
    }
  };
  std::vector<std::thread> th;
  for (int t = 1; t < nt; ++t) th.emplace_back(work, t);
  work(0);
  for (auto &t : th) t.join();
  if (first_err.load() != 0) {
    for (int64_t b = 0; b < n_batches; ++b) {
      delete out[b];
      out[b] = nullptr;
    }
    std::string msg;
    for (auto &s : errs)
      if (!s.empty()) msg = s;
    return fail((toc_status)first_err.load(), "%s", msg.c_str());
  }
  return TOC_OK;
}

toc_status toc_enc_info_get(const toc_enc *e, toc_enc_info *info) {
  if (!e || !info) return fail(TOC_EINVAL, "NULL pointer");
  toc_enc_info r{};
  r.n_rows = e->n_rows;
  r.n_cols = e->n_cols;
  r.nnz = e->nnz;
  r.n_first = (int64_t)e->I_col.size();
  r.n_codes = (int64_t)e->D_codes.size();
  r.n_nodes = e->n_nodes;
  r.n_live = e->n_live;
  r.n_deep = e->n_deep_live;
  r.max_depth = e->max_depth_live;
  r.phys_bytes = physical_size(e);
  r.canon_bytes = 4 * r.n_codes + 4 * ((int64_t)e->n_rows + 1) + 10 * e->n_live +
                  4 * ((int64_t)e->max_depth_live + 1);
  *info = r;
  return TOC_OK;
}

toc_status toc_enc_export(const toc_enc *e, int32_t *I_col, float *I_val,
                          int64_t *D_rowptr, uint32_t *D_codes) {
  if (!e) return fail(TOC_EINVAL, "NULL handle");
  if (I_col) std::memcpy(I_col, e->I_col.data(), e->I_col.size() * 4);
  if (I_val) std::memcpy(I_val, e->I_bits.data(), e->I_bits.size() * 4);
  if (D_rowptr) std::memcpy(D_rowptr, e->D_rowptr.data(), e->D_rowptr.size() * 8);
  if (D_codes) std::memcpy(D_codes, e->D_codes.data(), e->D_codes.size() * 4);
  return TOC_OK;
}

void toc_enc_free(toc_enc *e) { delete e; }

}  // extern "C"

// ---------------------------------------------------------------------------
// Upload image.
// ---------------------------------------------------------------------------
namespace toc {
namespace {

inline int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

struct Counts {
  int64_t codes, levels, rows, d;
};

Counts counts_of(const toc_enc *e, uint32_t flags) {
  const bool keep = flags & TOC_UPLOAD_KEEP_DEAD;
  Counts c;
  c.codes = keep ? e->n_nodes - 1 : e->n_live;
  c.levels = keep ? e->max_depth_all : e->max_depth_live;
  c.rows = e->n_rows;
  c.d = (int64_t)e->D_codes.size();
  return c;
}

struct ImgScratch {
  std::vector<uint32_t> parent, first, depth, newidx, bucket, fill, fpos, lpos, at_lpos, poff, prow;
  std::vector<uint8_t> live, has_child;
  std::vector<int64_t> cnt, bucket_off;
  std::vector<uint64_t> keys;
};

// Algorithm 2 on (I, D), then live marking and the depth-ordered renumbering;
// writes the batch's arrays at its offsets.  Returns the per-batch counts through bt.
toc_status write_batch(const toc_enc *e, int64_t b, uint32_t flags, const toc_layout &L,
                       uint8_t *dst, toc_batch &bt, int64_t dtile_base, ImgScratch &S) {
  const bool keep = flags & TOC_UPLOAD_KEEP_DEAD;
  const int64_t nI = (int64_t)e->I_col.size();
  const int64_t N = e->n_nodes;
  S.parent.assign((size_t)N, 0);
  S.first.assign((size_t)N, 0);
  S.depth.assign((size_t)N, 0);
  // phase I: nodes 1..|I| from I
  for (int64_t i = 1; i <= nI; ++i) {
    S.parent[i] = 0;
    S.first[i] = (uint32_t)i;  // F[i] = I[i-1], kept as the index of that I entry
    S.depth[i] = 1;
  }
  // phase II: replay the node creations from D
  int64_t idx = nI + 1;
  for (int32_t r = 0; r < e->n_rows; ++r) {
    const int64_t a = e->D_rowptr[r], b = e->D_rowptr[r + 1];
    for (int64_t j = a; j + 1 < b; ++j) {
      const uint32_t p = e->D_codes[j];
      if (idx >= N || p == 0 || (int64_t)p >= idx)
        return fail(TOC_EINVAL, "corrupt encoding (code %u)", p);
      S.parent[idx] = p;
      S.first[idx] = S.first[p];
      const uint32_t q = e->D_codes[j + 1];
      if (q == 0 || (int64_t)q > idx) return fail(TOC_EINVAL, "corrupt encoding (code %u)", q);
      // key of the new node = first pair of the next code's sequence
      S.depth[idx] = S.depth[p] + 1;
      ++idx;
    }
  }
  if (idx != N) return fail(TOC_EINVAL, "corrupt encoding (node count)");
  // live marking (parents precede children)
  S.live.assign((size_t)N, keep ? 1 : 0);
  S.has_child.assign((size_t)N, 0);
  for (uint32_t c : e->D_codes) {
    if (c == 0 || (int64_t)c >= N) return fail(TOC_EINVAL, "corrupt encoding (code %u)", c);
    S.live[c] = 1;
  }
  int32_t levels = 0;
  int64_t n_codes = 0;
  for (int64_t c = N - 1; c >= 1; --c) {
    if (!S.live[c]) continue;
    ++n_codes;
    levels = std::max<int32_t>(levels, (int32_t)S.depth[c]);
    S.live[S.parent[c]] = 1;
    if (S.parent[c] != 0) S.has_child[S.parent[c]] = 1;
  }
  const Counts want = counts_of(e, flags);
  if (n_codes != want.codes || levels != want.levels)
    return fail(TOC_EINVAL, "corrupt encoding (tree counts disagree)");
  // Order of the stored codes (every order with parents before children is valid
  // for the scans of section 4; this one serves the kernels):
  //   depth 1: codes with children (node order), then leaves in order of their
  //   first entry in D (the entries of a tuple then read nearby keys),
  //   depth d >= 2: sorted by parent, so the children of a node are contiguous.
  S.cnt.assign((size_t)levels + 2, 0);
  int64_t n_int1 = 0;
  for (int64_t c = 1; c < N; ++c) {
    if (!S.live[c]) continue;
    S.cnt[S.depth[c]]++;
    if (S.depth[c] == 1 && S.has_child[c]) ++n_int1;
  }
  if (n_int1 != bt.n_int1) return fail(TOC_EINVAL, "corrupt encoding (tree counts disagree)");
  uint32_t *level = (uint32_t *)(dst + L.level) + bt.lvl_base;
  level[0] = 0;
  for (int32_t d = 1; d <= levels; ++d) level[d] = level[d - 1] + (uint32_t)S.cnt[d];
  S.newidx.assign((size_t)N, 0xFFFFFFFFu);
  {
    // bucket live codes by depth, node order inside each bucket
    S.bucket_off.assign((size_t)levels + 3, 0);
    for (int32_t d = 1; d <= levels; ++d) S.bucket_off[d + 1] = S.bucket_off[d] + S.cnt[d];
    S.bucket.assign((size_t)n_codes, 0);
    std::vector<int64_t> fill(S.bucket_off.begin(), S.bucket_off.end());
    for (int64_t c = 1; c < N; ++c)
      if (S.live[c]) S.bucket[fill[S.depth[c]]++] = (uint32_t)c;
    int64_t pos_int = 0;
    S.keys.clear();
    S.fpos.assign((size_t)N, 0xFFFFFFFFu);
    for (size_t j = e->D_codes.size(); j-- > 0;) S.fpos[e->D_codes[j]] = (uint32_t)j;
    for (int64_t i = S.bucket_off[1]; i < S.bucket_off[2]; ++i) {
      const uint32_t c = S.bucket[i];
      if (S.has_child[c]) S.newidx[c] = (uint32_t)pos_int++;
      else S.keys.push_back(((uint64_t)S.fpos[c] << 32) | c);   // a leaf is in D
    }
    std::sort(S.keys.begin(), S.keys.end());
    int64_t at = n_int1;
    for (uint64_t kc : S.keys) S.newidx[(uint32_t)kc] = (uint32_t)at++;
    for (int32_t d = 2; d <= levels; ++d) {
      S.keys.clear();
      for (int64_t i = S.bucket_off[d]; i < S.bucket_off[d + 1]; ++i) {
        const uint32_t c = S.bucket[i];
        S.keys.push_back(((uint64_t)S.newidx[S.parent[c]] << 32) | c);
      }
      std::sort(S.keys.begin(), S.keys.end());
      at = level[d - 1];
      for (uint64_t kc : S.keys) S.newidx[(uint32_t)kc] = (uint32_t)at++;
    }
  }
  // links of the codes of depth >= 2 (a depth-1 code has no parent), by code - n1
  const int64_t n1 = levels >= 1 ? S.cnt[1] : 0;
  toc_key *node = (toc_key *)(dst + L.key) + bt.code_base;
  toc_link *link = (toc_link *)(dst + L.link) + bt.deep_base;
  for (int64_t c = 1; c < N; ++c) {
    if (!S.live[c] || S.depth[c] == 1) continue;
    const uint32_t at = S.newidx[c];
    link[at - n1].parent = S.newidx[S.parent[c]];
    link[at - n1].depth = S.depth[c];
  }
  auto parent_of = [&](int64_t c) -> uint32_t { return c < n1 ? 0xFFFFFFFFu : link[c - n1].parent; };
  auto depth_of = [&](int64_t c) -> uint32_t { return c < n1 ? 1u : link[c - n1].depth; };
  // keys: node c <= |I| has key I[c-1]; node idx > |I| has the first pair of the
  // code that follows its parent in D (Algorithm 2).
  auto set_key = [&](uint32_t at, uint32_t fi) {
    node[at].col = (uint32_t)e->I_col[fi - 1];
    std::memcpy(&node[at].val, &e->I_bits[fi - 1], sizeof(float));
  };
  for (int64_t c = 1; c <= nI; ++c)
    if (S.live[c]) set_key(S.newidx[c], (uint32_t)c);
  idx = nI + 1;
  for (int32_t r = 0; r < e->n_rows; ++r) {
    const int64_t a = e->D_rowptr[r], b = e->D_rowptr[r + 1];
    for (int64_t j = a; j + 1 < b; ++j, ++idx) {
      if (!S.live[idx]) continue;
      set_key(S.newidx[idx], S.first[e->D_codes[j + 1]]);   // index into I, 1-based
    }
  }
  // spans and renumbered D
  uint32_t *span = (uint32_t *)(dst + L.span) + bt.span_base;
  uint32_t *dcodes = (uint32_t *)(dst + L.dcodes) + bt.d_base;
  for (int32_t r = 0; r <= e->n_rows; ++r) span[r] = (uint32_t)e->D_rowptr[r];
  for (size_t j = 0; j < e->D_codes.size(); ++j) dcodes[j] = S.newidx[e->D_codes[j]];
  // Positions of the left multiplication: depth-1 leaves sorted by (column,
  // code), so that the leaves of a column are contiguous; every other code is at
  // its own index.  The column index and the column stretches follow them.
  S.lpos.resize((size_t)n_codes);
  S.at_lpos.resize((size_t)n_codes);
  for (int64_t c = 0; c < n_codes; ++c) S.lpos[c] = (uint32_t)c;
  S.keys.clear();
  for (int64_t c = n_int1; c < n1; ++c) S.keys.push_back(((uint64_t)node[c].col << 32) | (uint64_t)c);
  std::sort(S.keys.begin(), S.keys.end());
  for (size_t i = 0; i < S.keys.size(); ++i) S.lpos[(uint32_t)S.keys[i]] = (uint32_t)(n_int1 + (int64_t)i);
  for (int64_t c = 0; c < n_codes; ++c) S.at_lpos[S.lpos[c]] = (uint32_t)c;
  auto val_bits = [&](int64_t c) {
    uint32_t v;
    std::memcpy(&v, &node[c].val, 4);
    return v;
  };
  // D inverted (scratch): the rows of the entries of D equal to the code at each
  // position, ascending, grouped by position; bit 31 marks the first of each.
  // This is the index set of the sum that defines G(x) in Theorem 2.
  std::vector<uint32_t> &poff = S.poff, &prow = S.prow;
  poff.assign((size_t)n_codes + 1, 0u);
  prow.assign(e->D_codes.size(), 0u);
  for (size_t j = 0; j < e->D_codes.size(); ++j) poff[S.lpos[dcodes[j]] + 1]++;
  for (int64_t c = 0; c < n_codes; ++c) poff[c + 1] += poff[c];
  S.fill.assign(poff.begin(), poff.begin() + n_codes);
  for (int32_t r = 0; r < e->n_rows; ++r)
    for (int64_t j = e->D_rowptr[r]; j < e->D_rowptr[r + 1]; ++j)
      prow[S.fill[S.lpos[dcodes[j]]]++] = (uint32_t)r;
  for (int64_t c = 0; c < n_codes; ++c)
    if (poff[c] < poff[c + 1]) prow[poff[c]] |= 0x80000000u;
  // codes with an H row in the left multiplication (children or depth >= 2),
  // listed by column
  uint32_t *tlist = (uint32_t *)(dst + L.tlist) + bt.tree_base;
  S.keys.clear();
  for (int64_t c = 0; c < n_codes; ++c)
    if (c < n_int1 || c >= n1) S.keys.push_back(((uint64_t)node[c].col << 32) | (uint64_t)c);
  std::sort(S.keys.begin(), S.keys.end());
  for (size_t t = 0; t < S.keys.size(); ++t) tlist[t] = (uint32_t)S.keys[t];
  const int64_t n_tree = (int64_t)S.keys.size();
  // column index of the left multiplication (out row j sums over the codes of key
  // column j): per column the first position of a leaf (depth 1, no children) of
  // a column >= j, the leaf occurrences before it, the first tree-list entry of a
  // column >= j, and the columns ordered by number of entries (leaf occurrences +
  // tree codes), most first
  {
    const int64_t m = e->n_cols;
    uint32_t *cx = (uint32_t *)(dst + L.cols) + (int64_t)b * 4 * (m + 1);
    uint32_t *c_code = cx, *c_occ = cx + (m + 1), *c_tree = cx + 2 * (m + 1), *c_ord = cx + 3 * (m + 1);
    int64_t i = n_int1, t = 0;
    for (int64_t j = 0; j <= m; ++j) {
      while (i < n1 && (int64_t)node[S.at_lpos[i]].col < j) ++i;
      while (t < n_tree && (int64_t)node[tlist[t]].col < j) ++t;
      c_code[j] = (uint32_t)i;
      c_occ[j] = poff[i] - poff[n_int1];
      c_tree[j] = (uint32_t)t;
    }
    S.keys.clear();
    for (int64_t j = 0; j < m; ++j) {
      const uint64_t cnt = (uint64_t)(c_occ[j + 1] - c_occ[j]) + (c_tree[j + 1] - c_tree[j]);
      S.keys.push_back(((0xFFFFFFFFull - cnt) << 32) | (uint64_t)j);
    }
    std::sort(S.keys.begin(), S.keys.end());
    for (int64_t k = 0; k < m; ++k) c_ord[k] = (uint32_t)S.keys[k];
    c_ord[m] = 0;
    // columns that are the key column of some stored code (a leaf or a tree code)
    int32_t u = 0;
    for (int64_t j = 0; j < m; ++j)
      u += (c_code[j + 1] > c_code[j] || c_tree[j + 1] > c_tree[j]) ? 1 : 0;
    bt.n_ucols = u;
    // the left multiplication's entries, in three parts: the leaf occurrences by
    // position (so those of a column are one stretch, from c_occ[j]), the tree
    // codes by column marked with kTreeEntry (column j's from n_lo + c_tree[j]),
    // then the tree codes' own occurrences by tree row (plain tuple indexes).
    // cval beside each: the key value of the entry's code (0 in the third part).
    // occ_off: the start of each leaf position's occurrences (n_int1 .. n1-1,
    // then the end), then of each tree row's (and the end).
    uint32_t *ce = (uint32_t *)(dst + L.centry) + bt.d_base + bt.tree_base;
    uint32_t *cv = (uint32_t *)(dst + L.cval) + bt.d_base + bt.tree_base;
    uint32_t *lo = (uint32_t *)(dst + L.occ_off) + bt.code_base + 2 * b;
    uint32_t *to = lo + (n1 - n_int1) + 1;
    int64_t o = 0;
    for (int64_t p = n_int1; p < n1; ++p) {
      lo[p - n_int1] = (uint32_t)o;
      for (uint32_t q = poff[p]; q < poff[p + 1]; ++q) {
        ce[o] = prow[q];
        cv[o++] = val_bits(S.at_lpos[p]);
      }
    }
    lo[n1 - n_int1] = (uint32_t)o;
    for (int64_t t = 0; t < n_tree; ++t) {
      ce[o] = tlist[t] | kTreeEntry;
      cv[o++] = val_bits(tlist[t]);
    }
    for (int64_t h = 0; h < n_tree; ++h) {
      const int64_t c = h < n_int1 ? h : h - n_int1 + n1;   // tree row h's code (and position)
      to[h] = (uint32_t)o;
      for (uint32_t q = poff[c]; q < poff[c + 1]; ++q) ce[o++] = prow[q] & 0x7FFFFFFFu;
    }
    to[n_tree] = (uint32_t)o;
  }
  // children of each tree code (their H rows are added to its H in the left
  // multiplication): code h's children are codes tchild[h] .. tchild[h+1]-1, h
  // numbering the tree codes as in tlist's row order (depth-1 codes with children,
  // then deeper codes)
  {
    uint32_t *tch = (uint32_t *)(dst + L.tchild) + bt.tree_base + b;
    auto hrow = [&](uint32_t c) -> int64_t { return c < n_int1 ? c : (int64_t)c - n1 + n_int1; };
    int64_t c = n1;
    for (int64_t h = 0; h <= n_tree; ++h) {
      while (c < n_codes && hrow(parent_of(c)) < h) ++c;
      tch[h] = (uint32_t)c;
    }
  }
  // decode tiles: for every kDecodeTile entries of D, the batch, the first entry,
  // the number of pairs before it in the batch and the first row starting in it
  {
    uint32_t *dt = (uint32_t *)(dst + L.dtiles) + 4 * dtile_base;
    const int64_t nd = (int64_t)e->D_codes.size();
    const int64_t ntiles = std::max<int64_t>(1, (nd + kDecodeTile - 1) / kDecodeTile);
    uint64_t pairs = 0;
    int64_t row = 0;
    for (int64_t t = 0; t < ntiles; ++t) {
      const int64_t es = t * kDecodeTile;
      while (row < e->n_rows && e->D_rowptr[row] < es) ++row;
      dt[4 * t + 0] = (uint32_t)b;
      dt[4 * t + 1] = (uint32_t)es;
      dt[4 * t + 2] = (uint32_t)pairs;
      dt[4 * t + 3] = (uint32_t)row;
      for (int64_t j = es; j < std::min(nd, es + kDecodeTile); ++j) pairs += depth_of(dcodes[j]);
    }
  }
  bt.n_codes = (int32_t)n_codes;
  bt.n_lvl1 = (int32_t)n1;
  bt.n_levels = levels;
  return TOC_OK;
}

}  // namespace

toc_status plan_image(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                      toc_dev *dev) {
  if (n_batches < 0) return fail(TOC_EINVAL, "n_batches < 0");
  if (n_batches > 0 && !encs) return fail(TOC_EINVAL, "encs is NULL");
  if (flags & ~(TOC_UPLOAD_KEEP_DEAD | TOC_UPLOAD_HOST)) return fail(TOC_EINVAL, "unknown flag");
  int32_t n_cols = -1;
  std::vector<BatchCounts> bc((size_t)n_batches);
  const bool keep = flags & TOC_UPLOAD_KEEP_DEAD;
  for (int64_t b = 0; b < n_batches; ++b) {
    const toc_enc *e = encs[b];
    if (!e) return fail(TOC_EINVAL, "encs[%lld] is NULL", (long long)b);
    if (n_cols < 0) n_cols = e->n_cols;
    if (e->n_cols != n_cols) return fail(TOC_EINVAL, "batches differ in n_cols");
    const Counts c = counts_of(e, flags);
    BatchCounts &k = bc[(size_t)b];
    k.rows = c.rows;
    k.codes = c.codes;
    k.levels = c.levels;
    k.d = c.d;
    k.deep = keep ? e->n_deep_all : e->n_deep_live;
    k.int1 = keep ? e->n_int1_all : e->n_int1_live;
    k.nnz = e->nnz;
    k.canon = 4 * c.d + 4 * (c.rows + 1) + 10 * e->n_live + 4 * ((int64_t)e->max_depth_live + 1);
  }
  return plan_layout(bc.data(), n_batches, n_cols, flags, dev);
}

toc_status plan_layout(const BatchCounts *bc, int64_t n_batches, int32_t n_cols, uint32_t flags,
                       toc_dev *dev) {
  int64_t codes = 0, levels = 0, rows = 0, d = 0, spans = 0, nnz = 0, canon = 0, deep = 0,
          tree = 0;
  int32_t max_depth = 0;
  dev->batches.assign((size_t)n_batches, toc_batch{});
  dev->max_rows = dev->max_codes = dev->max_levels = 0;
  dev->max_d = dev->max_deep = dev->max_tree = dev->max_pair_deep = 0;
  dev->dtile_base.assign((size_t)n_batches, 0);
  int64_t dtiles = 0;
  for (int64_t b = 0; b < n_batches; ++b) {
    const BatchCounts &c = bc[b];
    if (c.codes >= kMaxBatchDim || c.d > INT32_MAX || c.rows >= kMaxBatchDim)
      return fail(TOC_EUNSUPPORTED, "batch too large");
    toc_batch &bt = dev->batches[b];
    bt.code_base = codes;
    bt.d_base = d;
    bt.row_base = rows;
    bt.span_base = spans;
    bt.nnz_base = nnz;
    bt.lvl_base = levels;
    bt.n_rows = (int32_t)c.rows;
    bt.n_codes = (int32_t)c.codes;
    bt.n_levels = (int32_t)c.levels;
    bt.n_d = (int32_t)c.d;
    const int64_t nd = c.deep;
    const int64_t ni = c.int1;
    bt.n_int1 = (int32_t)ni;
    bt.deep_base = deep;
    bt.tree_base = tree;
    dev->max_deep = std::max(dev->max_deep, nd);
    dev->max_tree = std::max(dev->max_tree, nd + ni);
    tree += nd + ni;
    dev->dtile_base[b] = dtiles;
    dtiles += std::max<int64_t>(1, (c.d + kDecodeTile - 1) / kDecodeTile);
    codes += c.codes;
    levels += c.levels + 1;
    rows += c.rows;
    spans += c.rows + 1;
    d += c.d;
    nnz += c.nnz;
    deep += nd;
    canon += c.canon;
    max_depth = std::max<int32_t>(max_depth, (int32_t)c.levels);
    dev->max_rows = std::max<int32_t>(dev->max_rows, (int32_t)c.rows);
    dev->max_codes = std::max<int32_t>(dev->max_codes, (int32_t)c.codes);
    dev->max_levels = std::max<int32_t>(dev->max_levels, (int32_t)c.levels);
    dev->max_d = std::max<int64_t>(dev->max_d, c.d);
  }
  toc_layout &L = dev->layout;
  int64_t off = 0;
  L.batches = off; off = align256(off + (int64_t)sizeof(toc_batch) * n_batches);
  L.level = off;   off = align256(off + 4 * levels);
  L.key = off;     off = align256(off + (int64_t)sizeof(toc_key) * codes);
  L.link = off;    off = align256(off + (int64_t)sizeof(toc_link) * deep);
  L.span = off;    off = align256(off + 4 * spans);
  L.dcodes = off;  off = align256(off + 4 * d);
  L.occ_off = off; off = align256(off + 4 * (codes + 2 * n_batches));
  L.tlist = off;   off = align256(off + 4 * tree);
  L.dtiles = off;  off = align256(off + 16 * dtiles);
  L.cols = off;    off = align256(off + 16 * n_batches * ((int64_t)std::max(n_cols, 0) + 1));
  L.tchild = off;  off = align256(off + 4 * (tree + n_batches));
  L.centry = off;  off = align256(off + 4 * (d + tree));
  L.cval = off;    off = align256(off + 4 * (d + tree));
  dev->n_dtiles = dtiles;
  dev->tot_levels = levels;
  L.end = std::max<int64_t>(off, 256);
  dev->total_deep = deep;
  dev->total_tree = tree;
  dev->max_pair_deep = 0;
  for (int64_t b = 0; b < n_batches; ++b) {
    auto nd = [&](int64_t i) {
      return (i + 1 < n_batches ? dev->batches[i + 1].deep_base : deep) - dev->batches[i].deep_base;
    };
    const bool first = (b / 8) % 2 == 0 && b + 8 < n_batches;
    dev->max_pair_deep = std::max(dev->max_pair_deep, nd(b) + (first ? nd(b + 8) : 0));
  }
  toc_dev_info &I = dev->info;
  I = toc_dev_info{};
  I.n_batches = n_batches;
  I.n_rows = rows;
  I.n_cols = n_cols < 0 ? 0 : n_cols;
  I.max_depth = max_depth;
  I.nnz = nnz;
  I.n_codes = d;
  I.n_stored = codes;
  I.n_deep = deep;
  I.canon_bytes = canon;
  I.image_bytes = L.end;
  dev->flags = flags;
  return TOC_OK;
}

toc_status write_batches(const toc_enc *const *encs, int64_t b0, int64_t b1, uint32_t flags,
                         const toc_layout &L, toc_dev *dev, uint8_t *dst) {
  const int nt = (int)std::min<int64_t>(std::max(1u, std::thread::hardware_concurrency()),
                                        std::max<int64_t>(b1 - b0, 1));
  std::atomic<int64_t> next{b0};
  std::atomic<int> first_err{0};
  std::string err_msg;
  std::atomic<int> err_taken{0};
  auto work = [&]() {
    ImgScratch S;
    for (;;) {
      const int64_t b = next.fetch_add(1);
      if (b >= b1 || first_err.load() != 0) return;
      toc_status st;
      try {
        st = write_batch(encs[b], b, flags, L, dst, dev->batches[b], dev->dtile_base[b], S);
      } catch (const std::bad_alloc &) {
        st = fail(TOC_ENOMEM, "out of host memory");
      }
      if (st != TOC_OK) {
        int expect = 0;
        if (first_err.compare_exchange_strong(expect, (int)st)) {
          err_msg = g_err;
          err_taken = 1;
        }
        return;
      }
    }
  };
  std::vector<std::thread> th;
  for (int t = 1; t < nt; ++t) th.emplace_back(work);
  work();
  for (auto &t : th) t.join();
  if (first_err.load() != 0) return fail((toc_status)first_err.load(), "%s", err_msg.c_str());
  return TOC_OK;
}

void finish_image(toc_dev *dev) {
  dev->max_ucols = 0;
  dev->max_keylinks = 0;
  for (const toc_batch &bt : dev->batches) {
    dev->max_ucols = std::max(dev->max_ucols, bt.n_ucols);
    dev->max_keylinks = std::max<int64_t>(dev->max_keylinks, 2 * (int64_t)bt.n_codes - bt.n_lvl1);
  }
}

toc_status build_image(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                       toc_dev *dev, uint8_t *dst) {
  const toc_layout &L = dev->layout;
  std::memset(dst, 0, (size_t)L.end);
  toc_status st = write_batches(encs, 0, n_batches, flags, L, dev, dst);
  if (st != TOC_OK) return st;
  finish_image(dev);
  std::memcpy(dst + L.batches, dev->batches.data(), sizeof(toc_batch) * dev->batches.size());
  return TOC_OK;
}

ArrStarts arr_starts(const toc_dev *dev, int64_t b) {
  ArrStarts a;
  const int64_t n = (int64_t)dev->batches.size();
  const int64_t m1 = 4 * ((int64_t)std::max(dev->info.n_cols, 0) + 1);
  if (b < n) {
    const toc_batch &t = dev->batches[b];
    a.level = t.lvl_base;
    a.code = t.code_base;
    a.deep = t.deep_base;
    a.span = t.span_base;
    a.d = t.d_base;
    a.tree = t.tree_base;
    a.dtile = dev->dtile_base[b];
  } else {
    a.level = dev->tot_levels;
    a.code = dev->info.n_stored;
    a.deep = dev->total_deep;
    a.span = dev->info.n_rows + n;
    a.d = dev->info.n_codes;
    a.tree = dev->total_tree;
    a.dtile = dev->n_dtiles;
  }
  a.cols = b * m1;
  a.b = b;
  return a;
}

}  // namespace toc
