// Mini-batch gradient descent on the uploaded image (section 2.1's update rule)
// for the linear models of Table 1: per batch, the right product r = A.h
// (Theorem 1, Algorithm 4), the loss gradient g_i at r_i, the left product g^T.A
// (Theorem 2, Algorithm 5) and the update of h, all in one workgroup with H in
// LDS.  The batches are consecutive steps of one launch: each step reads the
// model the previous one wrote.  A step's reads of the image do not depend on the
// model, so helper workgroups on the stepping workgroup's XCD read the next
// batches' arrays ahead of it, and its loads find them in that XCD's L2.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>

#include "toc_internal.h"

namespace {

constexpr int kMgBlock = 1024;
constexpr int kMgLanes = 8;                    // lanes per tuple in the right product
constexpr int kMgTup = 24;                     // a lane's codes of a tuple loaded at once
constexpr uint32_t kMgFirst = 0x80000000u;     // first-occurrence bit of a leaf occurrence
constexpr size_t kMgLdsMax = 160 * 1024;
constexpr int kMgXcds = 8;                     // workgroups are dealt to the XCDs in turn
constexpr int kMgHelpers = 1;                  // workgroups reading ahead of the steps (more
                                               // measured slower: the XCD's L2 overflows)
constexpr int64_t kMgAheadMax = (int64_t)1280 << 10;   // larger batches are not read ahead
constexpr uint32_t kMgSpinMax = 1u << 20;      // a helper's wait for the steps is bounded

// The step the stepping workgroup of the latest launch works on: the launch's tag
// in the upper half, the batch (from b0) in the lower.  Only the helpers read it,
// to stay at most kMgHelpers batches ahead; a stale or foreign value only moves
// their reads in time.
__device__ uint64_t mgd_progress;

struct MgImg {
  const toc_batch *batches;
  const uint32_t *level;
  const toc_key *key;
  const toc_link *link;
  const uint32_t *span, *dcodes, *occ_off, *tlist, *cols, *tchild, *centry, *cval;
};

// d loss / d r of one tuple: squared 1/2 (y - r)^2, logistic log(1 + exp(-y r)),
// hinge max(0, 1 - y r) (subgradient 0 at the kink)
__device__ inline float dloss(int loss, float r, float y) {
  if (loss == TOC_MGD_LINEAR) return r - y;
  if (loss == TOC_MGD_LOGISTIC) return -y / (1.0f + expf(y * r));
  return y * r < 1.0f ? -y : 0.0f;
}

// A helper: reads the batches b0 + role - 1 + i * kMgHelpers of the launch, each
// once the steps are at most kMgHelpers batches behind it, touching one word of
// every 128-byte line of the arrays the step reads.
__device__ void mgd_read_ahead(const MgImg &im, int64_t b0, int64_t nb, int32_t m,
                               const float *y, int role, uint32_t tag) {
  __shared__ int s_go;
  uint32_t acc = 0;
  for (int64_t rt = role - 1; rt < nb; rt += kMgHelpers) {
    if (threadIdx.x == 0) {
      uint32_t spins = 0;
      for (; spins < kMgSpinMax; ++spins) {
        const uint64_t v = __hip_atomic_load(&mgd_progress, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((uint32_t)(v >> 32) == tag && (int64_t)(uint32_t)v + kMgHelpers >= rt) break;
        __builtin_amdgcn_s_sleep(8);
      }
      s_go = spins < kMgSpinMax;
    }
    __syncthreads();
    const bool go = s_go;
    __syncthreads();
    if (!go) return;                // the steps went quiet: leave them alone
    const int64_t b = b0 + rt;
    const toc_batch bt = im.batches[b];
    const int64_t nc = bt.n_codes, n1 = bt.n_lvl1, nd = bt.n_d, nr = bt.n_rows;
    const int64_t nt = bt.n_int1 + nc - n1;
    struct Range { const void *p; int64_t bytes; };
    const Range r[] = {
        {im.dcodes + bt.d_base, 4 * nd},
        {im.key + bt.code_base, 8 * nc},
        {im.link + bt.deep_base, 8 * (nc - n1)},
        {im.span + bt.span_base, 4 * (nr + 1)},
        {im.occ_off + bt.code_base + 2 * b, 4 * (nc + 2)},
        {im.centry + bt.d_base + bt.tree_base, 4 * (nd + nt)},
        {im.cval + bt.d_base + bt.tree_base, 4 * (nd + nt)},
        {im.cols + b * 4 * (int64_t)(m + 1), 4 * 3 * (int64_t)(m + 1)},
        {im.tlist + bt.tree_base, 4 * nt},
        {im.tchild + bt.tree_base + b, 4 * (nt + 1)},
        {im.level + bt.lvl_base, 4 * ((int64_t)bt.n_levels + 1)},
        {y + bt.row_base, 4 * nr},
    };
    int64_t total = 0;
    for (const Range &x : r) total += x.bytes;
    if (total > kMgAheadMax) continue;
    for (const Range &x : r)
      for (int64_t o = (int64_t)threadIdx.x * 128; o < x.bytes; o += (int64_t)kMgBlock * 128)
        acc += *(const uint32_t *)((const char *)x.p + o);
  }
  asm volatile("" : : "v"(acc));    // the loads are the point: keep them
}

// HL: the model h is kept in LDS for the whole launch (read at the start, written
// back at the end), else every step reads and writes it in memory
template <bool HL>
__global__ __launch_bounds__(kMgBlock) void mgd_kernel(MgImg im, int64_t b0, int64_t nb, int32_t m,
                                                       int32_t max_rows, int32_t max_codes,
                                                       int loss, float lr,
                                                       const float *__restrict__ y,
                                                       float *__restrict__ hg, uint32_t tag) {
  // workgroup 0 steps; workgroups kMgXcds, 2 kMgXcds, ... (on its XCD) read ahead;
  // the others have nothing to do
  if (blockIdx.x % kMgXcds != 0) return;
  if (blockIdx.x != 0) {
    mgd_read_ahead(im, b0, nb, m, y, (int)(blockIdx.x / kMgXcds), tag);
    return;
  }
  extern __shared__ float sm[];
  float *Gs = sm;                  // per tuple: d loss / d r
  float *H = sm + max_rows;        // per code (right), then per left position (left)
  float *h = HL ? H + max_codes : hg;
  if (HL) {
    for (int j = threadIdx.x; j < m; j += kMgBlock) h[j] = hg[j];
    __syncthreads();
  }
  for (int64_t b = b0; b < b0 + nb; ++b) {
    if (threadIdx.x == 0)
      __hip_atomic_store(&mgd_progress, ((uint64_t)tag << 32) | (uint32_t)(b - b0), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    const toc_batch bt = im.batches[b];
    const int nr = bt.n_rows;
    if (nr == 0) continue;          // no tuple: the step leaves h unchanged
    const uint32_t nc = (uint32_t)bt.n_codes, n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1;
    const uint32_t *lvl = im.level + bt.lvl_base;
    const toc_key *key = im.key + bt.code_base;
    const toc_link *link = im.link + (bt.deep_base - (int64_t)bt.n_lvl1);   // depth >= 2 only
    // right: H[c] = H[parent] + val * h[col], level by level
    for (int d = 1; d <= bt.n_levels; ++d) {
      const uint32_t a = lvl[d - 1], e = lvl[d];
#pragma unroll 8
      for (uint32_t c = a + threadIdx.x; c < e; c += kMgBlock) {
        const toc_key k = key[c];
        const float base = d > 1 ? H[link[c].parent] : 0.0f;
        H[c] = fmaf(k.val, h[k.col], base);
      }
      __syncthreads();
    }
    // r_i = sum of H over the tuple's codes; then the loss gradient at r_i
    {
      const uint32_t *span = im.span + bt.span_base;
      const uint32_t *dc = im.dcodes + bt.d_base;
      const bool long_tuples = bt.n_d >= (int64_t)kMgLanes * 8 * nr;   // 8 codes a lane on average
      const int lane = threadIdx.x % kMgLanes, grp = threadIdx.x / kMgLanes;
      for (int r = grp; r < nr; r += kMgBlock / kMgLanes) {
        const uint32_t s = span[r], e = span[r + 1];
        // long tuples (image-like batches): a lane's codes of the tuple (up to
        // kMgTup of them) are loaded together and summed as one block; short ones
        // (categorical batches) a few at a time
        float acc = 0.0f;
        if (!long_tuples) {
#pragma unroll 4
          for (uint32_t j = s + lane; j < e; j += kMgLanes) acc += H[dc[j]];
        } else
        for (uint32_t j0 = s + lane; j0 < e; j0 += kMgLanes * kMgTup) {
          uint32_t cc[kMgTup];
#pragma unroll
          for (int q = 0; q < kMgTup; ++q) {
            const uint32_t j = j0 + (uint32_t)(q * kMgLanes);
            cc[q] = j < e ? dc[j] : 0xFFFFFFFFu;
          }
          float part = 0.0f;
#pragma unroll
          for (int q = 0; q < kMgTup; ++q)
            if (cc[q] != 0xFFFFFFFFu) part += H[cc[q]];
          acc += part;
        }
#pragma unroll
        for (int o = kMgLanes / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, kMgLanes);
        if (lane == 0) Gs[r] = dloss(loss, acc, y[bt.row_base + r]);
      }
    }
    __syncthreads();
    // left, by pulling: H at each left position = the gradients of the tuples
    // holding its code, then children added into parents, deepest first
    // a leaf position p's tuples: entries lo[p - ni] .. of the batch's entry array
    // (its value beside the first); a tree code's: entries to[tree row] ..
    const uint32_t *lo = im.occ_off + bt.code_base + 2 * b, *to = lo + (n1 - ni) + 1;
    const uint32_t *ce = im.centry + bt.d_base + bt.tree_base;
    const uint32_t *cv = im.cval + bt.d_base + bt.tree_base;
    auto occ = [&](uint32_t p, uint32_t &o0, uint32_t &o1) {
      const bool leaf = p >= ni && p < n1;
      const uint32_t hr = p < ni ? p : p - n1 + ni;
      o0 = leaf ? lo[p - ni] : to[hr];
      o1 = leaf ? lo[p - ni + 1] : to[hr + 1];
    };
#pragma unroll 2
    for (uint32_t p = threadIdx.x; p < nc; p += kMgBlock) {
      float s = 0.0f;
      uint32_t o0, o1;
      occ(p, o0, o1);
      // a leaf's sum times its value (beside its first occurrence) right away: it
      // has no children to add first
      const bool lv = p >= ni && p < n1 && o1 > o0;
      const float v = lv ? __uint_as_float(cv[o0]) : 1.0f;
#pragma unroll 4
      for (uint32_t o = o0; o < o1; ++o) s += Gs[ce[o] & ~kMgFirst];
      H[p] = lv ? v * s : s;
    }
    __syncthreads();
    const uint32_t *tch = im.tchild + bt.tree_base + b;
    for (int d = bt.n_levels - 1; d >= 1; --d) {
      const uint32_t a = d == 1 ? 0u : lvl[d - 1], e = d == 1 ? ni : lvl[d];
      for (uint32_t c = a + threadIdx.x; c < e; c += kMgBlock) {
        const uint32_t hr = c < ni ? c : c - n1 + ni;
        float s = H[c];
        const uint32_t c1 = tch[hr + 1];
        for (uint32_t ch = tch[hr]; ch < c1; ++ch) s += H[ch];
        H[c] = s;
      }
      __syncthreads();
    }
    // each key column once: its gradient is the sum of val * H over the column's
    // leaves (a position range) and tree codes (a tree-list range); the step is
    // h_j -= lr / |B| * gradient_j
    const uint32_t *cx = im.cols + b * 4 * (int64_t)(m + 1);
    const uint32_t *Loff = cx, *Toff = cx + 2 * (m + 1);
    const uint32_t *tl = im.tlist + bt.tree_base;
    const float step = lr / (float)nr;
    for (int j = threadIdx.x; j < m; j += kMgBlock) {
      float s = 0.0f;
      const uint32_t l1 = Loff[j + 1], t1 = Toff[j + 1];
#pragma unroll 4
      for (uint32_t p = Loff[j]; p < l1; ++p) s += H[p];      // leaves: val * H already
#pragma unroll 4
      for (uint32_t t = Toff[j]; t < t1; ++t) {
        const uint32_t c = tl[t];
        s = fmaf(key[c].val, H[c], s);
      }
      h[j] = fmaf(-step, s, h[j]);
    }
    __syncthreads();                // the next step's right product reads the new h
  }
  if (HL)
    for (int j = threadIdx.x; j < m; j += kMgBlock) hg[j] = h[j];
}

// ---------------------------------------------------------------------------
// The same steps split over many workgroups, two launches per step (the stream
// orders them: a step's update is seen by the next step's forward pass):
//  * mgds_fwd_kernel: a 16-lane group per tuple sums val * h[col] over the pairs
//    of its codes (a deeper code walks its chain to the root: its sequence's
//    pairs), kMsCodes of a lane's codes and then their keys loaded together, and
//    writes the tuple's loss derivative g to the workspace; the model is staged in
//    LDS when the matrix has at most kMsHlds columns;
//  * mgds_bwd_kernel: every workgroup stages g, sums each tree code's own
//    occurrences (its tree row) and adds children into parents deepest level
//    first in LDS (a thread holds the ranges of its first kMbRows rows), then
//    takes 64 of the batch's used columns (a 16-lane group per column): the
//    gradient of column j sums val * g over its leaf occurrences and
//    val * (tree row) over its tree codes, the multipliers beside the entries,
//    and h_j -= lr / |B| * gradient.
// Each launch has kMgXcds more workgroups (one per XCD) that read ahead, so
// neither launch starts on arrays found in HBM only.  Every sum has a fixed
// order, so one call over many batches equals the batches one call each, bit for
// bit.
// ---------------------------------------------------------------------------
constexpr int kMsBlock = 256;
constexpr int kMsLanes = 16;                   // lanes per tuple or column
constexpr int kMsGroups = kMsBlock / kMsLanes;
constexpr int kMsCodes = 8;                    // a lane's codes (or entries) loaded together
constexpr int kMsHlds = 8192;                  // most columns whose model the forward pass stages
constexpr int kMbBlock = 1024;                 // backward workgroup
constexpr int kMbGroups = kMbBlock / kMsLanes; // its columns: one per 16-lane group
constexpr int kMbRows = 4;                     // tree rows per thread whose ranges it holds
constexpr uint32_t kMsNone = 0xFFFFFFFFu;

// Reads one word of every 128-byte line of the arrays of batch b that one side of
// a split step reads (fwd: the forward launch's, else the backward launch's), so
// that the launch finds them in this XCD's L2; the extra workgroups of each launch
// (one per XCD) run it beside the launch's work.
template <int NT>
__device__ void mgds_touch(const MgImg &im, int64_t b, int32_t m, const float *y, bool fwd) {
  const toc_batch bt = im.batches[b];
  const int64_t nc = bt.n_codes, n1 = bt.n_lvl1, nd = bt.n_d, nr = bt.n_rows;
  const int64_t nt = bt.n_int1 + nc - n1;
  struct Range { const void *p; int64_t bytes; };
  const Range rf[] = {
      {im.dcodes + bt.d_base, 4 * nd},
      {im.key + bt.code_base, 8 * nc},
      {im.link + bt.deep_base, 8 * (nc - n1)},
      {im.span + bt.span_base, 4 * (nr + 1)},
      {y + bt.row_base, 4 * nr},
  };
  const Range rb[] = {
      {im.occ_off + bt.code_base + 2 * b + (n1 - bt.n_int1) + 1, 4 * (nt + 1)},
      {im.centry + bt.d_base + bt.tree_base, 4 * (nd + nt)},
      {im.cval + bt.d_base + bt.tree_base, 4 * (nd + nt)},
      {im.cols + b * 4 * (int64_t)(m + 1) + (m + 1), 4 * 3 * (int64_t)(m + 1)},
      {im.tchild + bt.tree_base + b, 4 * (nt + 1)},
      {im.level + bt.lvl_base, 4 * ((int64_t)bt.n_levels + 1)},
  };
  uint32_t acc = 0;
  const Range *r = fwd ? rf : rb;
  const int n = fwd ? 5 : 6;
  for (int i = 0; i < n; ++i)
    for (int64_t o0 = (int64_t)threadIdx.x * 128; o0 < r[i].bytes; o0 += (int64_t)kMsCodes * NT * 128) {
      uint32_t t[kMsCodes];
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) {
        const int64_t o = o0 + (int64_t)q * NT * 128;
        t[q] = o < r[i].bytes ? *(const uint32_t *)((const char *)r[i].p + o) : 0u;
      }
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) acc += t[q];
    }
  asm volatile("" : : "v"(acc));    // the loads are the point: keep them
}

template <bool HLDS>
__global__ __launch_bounds__(kMsBlock) void mgds_fwd_kernel(MgImg im, int64_t b, int32_t m, int loss,
                                                            const float *__restrict__ y,
                                                            const float *__restrict__ hg,
                                                            float *__restrict__ g, int n_work) {
  // the workgroups past n_work read the backward launch's arrays of this batch
  if ((int)blockIdx.x >= n_work) {
    mgds_touch<kMsBlock>(im, b, m, y, false);
    return;
  }
  __shared__ float hs[HLDS ? kMsHlds : 1];
  const toc_batch bt = im.batches[b];
  if (HLDS) {
    for (int j0 = threadIdx.x; j0 < m; j0 += kMsCodes * kMsBlock) {
      float t[kMsCodes];
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) {
        const int j = j0 + q * kMsBlock;
        t[q] = j < m ? hg[j] : 0.0f;
      }
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) {
        const int j = j0 + q * kMsBlock;
        if (j < m) hs[j] = t[q];
      }
    }
    __syncthreads();
  }
  const float *h = HLDS ? hs : hg;
  const int lane = threadIdx.x % kMsLanes, grp = threadIdx.x / kMsLanes;
  const int r = (int)blockIdx.x * kMsGroups + grp;
  const uint32_t n1 = (uint32_t)bt.n_lvl1;
  const toc_key *key = im.key + bt.code_base;
  const toc_link *link = im.link + (bt.deep_base - (int64_t)bt.n_lvl1);   // depth >= 2 only
  float acc = 0.0f;
  if (r < bt.n_rows) {
    const uint32_t *span = im.span + bt.span_base;
    const uint32_t *dc = im.dcodes + bt.d_base;
    const uint32_t s = span[r], e = span[r + 1];
    for (uint32_t j0 = s + lane; j0 < e; j0 += kMsLanes * kMsCodes) {
      uint32_t c[kMsCodes];
      toc_key k[kMsCodes];
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) {
        const uint32_t j = j0 + (uint32_t)(q * kMsLanes);
        c[q] = j < e ? dc[j] : kMsNone;
      }
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) k[q] = c[q] != kMsNone ? key[c[q]] : toc_key{0u, 0.0f};
      float part = 0.0f;
#pragma unroll
      for (int q = 0; q < kMsCodes; ++q) {
        if (c[q] == kMsNone) continue;
        float v = k[q].val * h[k[q].col];
        for (uint32_t x = c[q]; x >= n1;) {        // a deeper code: the rest of its chain
          x = link[x].parent;
          const toc_key kp = key[x];
          v = fmaf(kp.val, h[kp.col], v);
        }
        part += v;
      }
      acc += part;
    }
  }
#pragma unroll
  for (int o = kMsLanes / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o, kMsLanes);
  if (r < bt.n_rows && lane == 0) g[r] = dloss(loss, acc, y[bt.row_base + r]);
}

__global__ __launch_bounds__(kMbBlock) void mgds_bwd_kernel(MgImg im, int64_t b, int32_t m,
                                                            int32_t max_rows, float lr,
                                                            const float *__restrict__ g,
                                                            float *__restrict__ h, int n_work,
                                                            int64_t next,
                                                            const float *__restrict__ y) {
  // the workgroups past n_work read the next step's forward arrays
  if ((int)blockIdx.x >= n_work) {
    if (next >= 0) mgds_touch<kMbBlock>(im, next, m, y, true);
    return;
  }
  extern __shared__ float sm[];
  float *Gs = sm;                  // per tuple: d loss / d r
  float *Ht = sm + max_rows;       // per tree row (tree code c: row c < ni ? c : c - n1 + ni)
  const toc_batch bt = im.batches[b];
  const int nr = bt.n_rows;
  const uint32_t nc = (uint32_t)bt.n_codes, n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1;
  const uint32_t n_tree = ni + (nc - n1);
  const uint32_t *to = im.occ_off + bt.code_base + 2 * b + (n1 - ni) + 1;
  const uint32_t *ce = im.centry + bt.d_base + bt.tree_base;
  const uint32_t *cv = im.cval + bt.d_base + bt.tree_base;
  const uint32_t *tch = im.tchild + bt.tree_base + b;
  auto row_code = [&](uint32_t t) { return t < ni ? t : t - ni + n1; };
  // this thread's first kMbRows tree rows: their occurrence and children ranges,
  // loaded while g is staged
  uint32_t o0[kMbRows], o1[kMbRows], k0[kMbRows], k1[kMbRows];
#pragma unroll
  for (int i = 0; i < kMbRows; ++i) {
    const uint32_t t = threadIdx.x + (uint32_t)(i * kMbBlock);
    o0[i] = o1[i] = k0[i] = k1[i] = 0u;
    if (t < n_tree) {
      o0[i] = to[t];
      o1[i] = to[t + 1];
      k0[i] = tch[t];
      k1[i] = tch[t + 1];
    }
  }
  for (int r0 = threadIdx.x; r0 < nr; r0 += kMsCodes * kMbBlock) {
    float t[kMsCodes];
#pragma unroll
    for (int q = 0; q < kMsCodes; ++q) {
      const int r = r0 + q * kMbBlock;
      t[q] = r < nr ? g[r] : 0.0f;
    }
#pragma unroll
    for (int q = 0; q < kMsCodes; ++q) {
      const int r = r0 + q * kMbBlock;
      if (r < nr) Gs[r] = t[q];
    }
  }
  __syncthreads();
  // tree rows: the gradients of the tuples holding the code (the first
  // occurrences of a thread's rows loaded together)
  {
    uint32_t w0[kMbRows];
#pragma unroll
    for (int i = 0; i < kMbRows; ++i) w0[i] = o1[i] > o0[i] ? ce[o0[i]] : 0u;
#pragma unroll
    for (int i = 0; i < kMbRows; ++i) {
      const uint32_t t = threadIdx.x + (uint32_t)(i * kMbBlock);
      if (t >= n_tree) continue;
      float s = 0.0f;
      if (o1[i] > o0[i]) s += Gs[w0[i] & ~kMgFirst];
      for (uint32_t o = o0[i] + 1; o < o1[i]; ++o) s += Gs[ce[o] & ~kMgFirst];
      Ht[t] = s;
    }
    for (uint32_t t = threadIdx.x + (uint32_t)(kMbRows * kMbBlock); t < n_tree; t += kMbBlock) {
      const uint32_t e1 = to[t + 1];
      float s = 0.0f;
      for (uint32_t o = to[t]; o < e1; ++o) s += Gs[ce[o] & ~kMgFirst];
      Ht[t] = s;
    }
  }
  __syncthreads();
  // children added into parents, deepest level first (a thread's first rows from
  // the ranges it holds, the others from memory)
  const uint32_t *lvl = im.level + bt.lvl_base;
  for (int d = bt.n_levels - 1; d >= 1; --d) {
    const uint32_t a = d == 1 ? 0u : lvl[d - 1], e = d == 1 ? ni : lvl[d];
#pragma unroll
    for (int i = 0; i < kMbRows; ++i) {
      const uint32_t t = threadIdx.x + (uint32_t)(i * kMbBlock);
      const uint32_t c = row_code(t);
      if (t < n_tree && c >= a && c < e) {
        float s = Ht[t];
        for (uint32_t ch = k0[i]; ch < k1[i]; ++ch) s += Ht[ch - n1 + ni];
        Ht[t] = s;
      }
    }
    for (uint32_t t = threadIdx.x + (uint32_t)(kMbRows * kMbBlock); t < n_tree; t += kMbBlock) {
      const uint32_t c = row_code(t);
      if (c < a || c >= e) continue;
      float s = Ht[t];
      const uint32_t c1 = tch[t + 1];
      for (uint32_t ch = tch[t]; ch < c1; ++ch) s += Ht[ch - n1 + ni];
      Ht[t] = s;
    }
    __syncthreads();
  }
  // this workgroup's used columns, a 16-lane group per column
  const uint32_t *cx = im.cols + b * 4 * (int64_t)(m + 1);
  const uint32_t *Ost = cx + (m + 1), *Toff = cx + 2 * (m + 1), *Ord = cx + 3 * (m + 1);
  const uint32_t n_lo = Ost[m];      // leaf occurrences; the tree entries follow them
  const int n_used = bt.n_ucols;
  const float step = lr / (float)nr;
  const int lane = threadIdx.x % kMsLanes, grp = threadIdx.x / kMsLanes;
  const int u = (int)blockIdx.x * kMbGroups + grp;
  uint32_t j = 0, lst = 0, tst = 0, nl = 0, nt = 0;
  if (u < n_used) {
    j = Ord[u];
    lst = Ost[j];
    nl = Ost[j + 1] - lst;
    tst = n_lo + Toff[j];
    nt = Toff[j + 1] - Toff[j];
  }
  float s = 0.0f;
  for (uint32_t q0 = lane; q0 < nl + nt; q0 += kMsLanes * kMsCodes) {
    uint32_t w[kMsCodes];
    float v[kMsCodes];
#pragma unroll
    for (int i = 0; i < kMsCodes; ++i) {
      const uint32_t q = q0 + (uint32_t)(i * kMsLanes);
      const uint32_t at = q < nl ? lst + q : tst + (q - nl);
      w[i] = q < nl + nt ? ce[at] : 0u;
      v[i] = q < nl + nt ? __uint_as_float(cv[at]) : 0.0f;
    }
    float part = 0.0f;
#pragma unroll
    for (int i = 0; i < kMsCodes; ++i) {
      const uint32_t q = q0 + (uint32_t)(i * kMsLanes);
      if (q < nl) {
        part = fmaf(v[i], Gs[w[i] & ~kMgFirst], part);
      } else if (q < nl + nt) {
        const uint32_t c = w[i] & ~toc::kTreeEntry;
        part = fmaf(v[i], Ht[c < ni ? c : c - n1 + ni], part);
      }
    }
    s += part;
  }
#pragma unroll
  for (int o = kMsLanes / 2; o > 0; o >>= 1) s += __shfl_xor(s, o, kMsLanes);
  if (u < n_used && lane == 0) h[j] = fmaf(-step, s, h[j]);
}

}  // namespace

using namespace toc;

namespace {

// Argument checks shared by the two entry points; *done is set when there is
// nothing to do.
toc_status mgd_check(const toc_dev *d, int64_t b0, int64_t n_batches, int32_t loss, float lr,
                     const float *y, const float *h, bool *done) {
  *done = false;
  if (!d) return fail(TOC_EINVAL, "dev is NULL");
  if (d->pending) return fail(TOC_EINVAL, "image planned but not built");
  if (d->host) return fail(TOC_EINVAL, "image was uploaded to host memory");
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return fail(TOC_EDEVICE, "hipGetDevice failed");
  if (cur != d->device) return fail(TOC_EINVAL, "current device %d differs from upload device %d", cur, d->device);
  const int64_t nb = d->info.n_batches;
  if (b0 < 0 || n_batches < 0 || b0 > nb || n_batches > nb - b0)
    return fail(TOC_EINVAL, "batches %lld..%lld outside 0..%lld", (long long)b0,
                (long long)(b0 + n_batches), (long long)nb);
  if (loss != TOC_MGD_LINEAR && loss != TOC_MGD_LOGISTIC && loss != TOC_MGD_HINGE)
    return fail(TOC_EINVAL, "unknown loss %d", loss);
  if (!std::isfinite(lr)) return fail(TOC_EINVAL, "learning rate not finite");
  if (n_batches == 0) {
    *done = true;
    return TOC_OK;
  }
  if (!h || (!y && d->info.n_rows > 0)) return fail(TOC_EINVAL, "NULL pointer");
  return TOC_OK;
}

MgImg mgd_image(const toc_dev *d) {
  const uint8_t *base = (const uint8_t *)d->buf;
  const toc_layout &L = d->layout;
  return MgImg{(const toc_batch *)(base + L.batches), (const uint32_t *)(base + L.level),
               (const toc_key *)(base + L.key), (const toc_link *)(base + L.link),
               (const uint32_t *)(base + L.span), (const uint32_t *)(base + L.dcodes),
               (const uint32_t *)(base + L.occ_off), (const uint32_t *)(base + L.tlist),
               (const uint32_t *)(base + L.cols), (const uint32_t *)(base + L.tchild),
               (const uint32_t *)(base + L.centry), (const uint32_t *)(base + L.cval)};
}

}  // namespace

extern "C" {

toc_status toc_mgd_epoch(const toc_dev *d, int64_t b0, int64_t n_batches, int32_t loss, float lr,
                         const float *y, float *h, void *stream) {
  clear_error();
  bool done = false;
  const toc_status st = mgd_check(d, b0, n_batches, loss, lr, y, h, &done);
  if (st != TOC_OK || done) return st;
  const size_t lds0 = 4 * ((size_t)d->max_rows + (size_t)d->max_codes);
  if (lds0 > kMgLdsMax)
    return fail(TOC_EUNSUPPORTED, "a batch needs %zu bytes of LDS (max %zu)", lds0, kMgLdsMax);
  // the model in LDS too when it fits
  const bool hl = lds0 + 4 * (size_t)d->info.n_cols <= kMgLdsMax;
  const size_t lds = hl ? lds0 + 4 * (size_t)d->info.n_cols : lds0;
  const void *fn = hl ? (const void *)mgd_kernel<true> : (const void *)mgd_kernel<false>;
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  const MgImg im = mgd_image(d);
  static std::atomic<uint32_t> launches{0};
  const uint32_t tag = launches.fetch_add(1) + 1;
  if (hl)
    hipLaunchKernelGGL(mgd_kernel<true>, dim3(kMgXcds * (1 + kMgHelpers)), dim3(kMgBlock), lds,
                       (hipStream_t)stream, im, b0, n_batches, d->info.n_cols, d->max_rows,
                       d->max_codes, (int)loss, lr, y, h, tag);
  else
    hipLaunchKernelGGL(mgd_kernel<false>, dim3(kMgXcds * (1 + kMgHelpers)), dim3(kMgBlock), lds,
                       (hipStream_t)stream, im, b0, n_batches, d->info.n_cols, d->max_rows,
                       d->max_codes, (int)loss, lr, y, h, tag);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "mgd_kernel: %s", hipGetErrorString(e));
  return TOC_OK;
}

toc_status toc_mgd_workspace_size(const toc_dev *d, size_t *bytes) {
  clear_error();
  if (!d || !bytes) return fail(TOC_EINVAL, "NULL pointer");
  *bytes = 4 * (size_t)std::max<int32_t>(d->max_rows, 1);
  return TOC_OK;
}

toc_status toc_mgd_epoch_split(const toc_dev *d, int64_t b0, int64_t n_batches, int32_t loss,
                               float lr, const float *y, float *h, void *ws, size_t ws_bytes,
                               void *stream) {
  clear_error();
  bool done = false;
  const toc_status st = mgd_check(d, b0, n_batches, loss, lr, y, h, &done);
  if (st != TOC_OK || done) return st;
  const size_t need = 4 * (size_t)std::max<int32_t>(d->max_rows, 1);
  if (!ws) return fail(TOC_EINVAL, "workspace is NULL");
  if (ws_bytes < need) return fail(TOC_ESIZE, "workspace of %zu bytes below the %zu needed", ws_bytes, need);
  const size_t lds = 4 * ((size_t)d->max_rows + (size_t)d->max_tree + 1);
  if (lds > kMgLdsMax)
    return fail(TOC_EUNSUPPORTED, "a batch needs %zu bytes of LDS (max %zu)", lds, kMgLdsMax);
  if (lds > 64 * 1024 && hipFuncSetAttribute((const void *)mgds_bwd_kernel,
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)lds) != hipSuccess)
    return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  const MgImg im = mgd_image(d);
  const int32_t m = d->info.n_cols;
  const bool hl = m <= kMsHlds;
  float *g = (float *)ws;
  hipStream_t s = (hipStream_t)stream;
  // each launch has kMgXcds more workgroups, one per XCD, that read ahead: the
  // forward launch the backward launch's arrays, the backward launch the next
  // step's forward arrays
  int64_t b = b0;
  while (b < b0 + n_batches && d->batches[(size_t)b].n_rows == 0) ++b;
  while (b < b0 + n_batches) {
    const toc_batch &bt = d->batches[(size_t)b];
    int64_t next = b + 1;                     // the next batch with tuples, or -1
    while (next < b0 + n_batches && d->batches[(size_t)next].n_rows == 0) ++next;
    const int gf = (bt.n_rows + kMsGroups - 1) / kMsGroups;
    if (hl)
      hipLaunchKernelGGL(mgds_fwd_kernel<true>, dim3(gf + kMgXcds), dim3(kMsBlock), 0, s, im, b, m,
                         (int)loss, y, (const float *)h, g, gf);
    else
      hipLaunchKernelGGL(mgds_fwd_kernel<false>, dim3(gf + kMgXcds), dim3(kMsBlock), 0, s, im, b, m,
                         (int)loss, y, (const float *)h, g, gf);
    // (a batch without used columns changes no entry of h: its launch only reads ahead)
    const int gb = (bt.n_ucols + kMbGroups - 1) / kMbGroups;
    hipLaunchKernelGGL(mgds_bwd_kernel, dim3(gb + kMgXcds), dim3(kMbBlock), lds, s, im, b, m,
                       d->max_rows, lr, (const float *)g, h, gb,
                       next < b0 + n_batches ? next : (int64_t)-1, y);
    b = next;
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "mgds kernels: %s", hipGetErrorString(e));
  return TOC_OK;
}

}  // extern "C"
