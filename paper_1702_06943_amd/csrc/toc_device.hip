// Device side of libtoc for gfx950: upload copy, the right/left products run on
// the compressed image, and decode to CSR.
//
// Image (built on the host by Algorithm 2 + level order): per batch, codes are
// numbered 0..n_codes-1 by depth; depth-1 codes with children come first.  H, the
// dictionary table of Theorems 1 and 2, exists only inside these kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <type_traits>
#include <utility>
#include <vector>

#include "toc_internal.h"

using toc::fail;

// Workspace of toc_left_mul_noalloc: one copy on each GPU the library runs on,
// held until the process ends.  Host code never passes this name to a kernel (on
// the host it is a stand-in, not a device address): the address comes from
// hipGetSymbolAddress, once per device (scratch_address below).
static __device__ __align__(256) float scratch[TOC_NOALLOC_SCRATCH_BYTES / sizeof(float)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on the first call
// on each device, with that device current).
toc_status scratch_address(int device, void **ptr) {
  if (device < 0 || device >= kMaxDevices)
    return fail(TOC_EUNSUPPORTED, "device %d beyond the %d this build tracks", device, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(TOC_EDEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", device,
                  hipGetErrorString(e));
    g_scratch_ptr[device] = p;
  }
  *ptr = g_scratch_ptr[device];
  return TOC_OK;
}

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWaves = kBlock / kWave;
constexpr int kMaxKpl = 8;                    // wide kernels: up to 8 columns per lane
constexpr int kKTile = kWave * kMaxKpl;       // 512 columns per pass
constexpr size_t kLdsMax = 160 * 1024;        // gfx950 LDS per workgroup

struct Img {
  const toc_batch *batches;
  const uint32_t *level;
  const toc_key *key;
  const toc_link *link;
  const uint32_t *span;
  const uint32_t *dcodes;
  const uint32_t *centry;   // left-product entries: leaf occurrences, tree codes, tree occurrences
  const uint32_t *cval;     // key value bits of each centry entry's code
};

Img image_of(const toc_dev *d) {
  const uint8_t *b = (const uint8_t *)d->buf;
  const toc_layout &L = d->layout;
  return Img{(const toc_batch *)(b + L.batches), (const uint32_t *)(b + L.level),
             (const toc_key *)(b + L.key), (const toc_link *)(b + L.link),
             (const uint32_t *)(b + L.span), (const uint32_t *)(b + L.dcodes),
             (const uint32_t *)(b + L.centry), (const uint32_t *)(b + L.cval)};
}

// Views of one field of a batch's node records, indexed by local code.
struct NodeCol {
  const toc_key *n;
  __device__ uint32_t operator[](int64_t c) const { return n[c].col; }
};
struct NodeVal {
  const toc_key *n;
  __device__ float operator[](int64_t c) const { return n[c].val; }
};
struct NodePar {
  const toc_link *n;
  __device__ uint32_t operator[](int64_t c) const { return n[c].parent; }
};

// The links of a batch's codes of depth >= 2 (the image stores none for depth-1
// codes), as a view indexed by local code: valid for codes n_lvl1 .. n_codes-1.
__device__ inline const toc_link *deep_links(const toc_link *all, const toc_batch &bt) {
  return all + (bt.deep_base - (int64_t)bt.n_lvl1);
}

// Index of the calling wave in its workgroup, as a wave-uniform (scalar) value.
__device__ inline int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

template <int W>
__device__ inline float group_sum(float x) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, W);
  return x;
}

__device__ inline uint32_t wave_incl_scan(uint32_t x, int lane) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  return x;
}

// A batch record read into wave-uniform (scalar) registers, so that pointers and
// buffer descriptors derived from it stay scalar.
__device__ inline int64_t uniform64(int64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ inline toc_batch uniform_batch(const toc_batch *p) {
  toc_batch t = *p;
  t.code_base = uniform64(t.code_base);
  t.d_base = uniform64(t.d_base);
  t.row_base = uniform64(t.row_base);
  t.span_base = uniform64(t.span_base);
  t.nnz_base = uniform64(t.nnz_base);
  t.deep_base = uniform64(t.deep_base);
  t.tree_base = uniform64(t.tree_base);
  t.lvl_base = uniform64(t.lvl_base);
  t.n_rows = __builtin_amdgcn_readfirstlane(t.n_rows);
  t.n_codes = __builtin_amdgcn_readfirstlane(t.n_codes);
  t.n_lvl1 = __builtin_amdgcn_readfirstlane(t.n_lvl1);
  t.n_int1 = __builtin_amdgcn_readfirstlane(t.n_int1);
  t.n_levels = __builtin_amdgcn_readfirstlane(t.n_levels);
  t.n_d = __builtin_amdgcn_readfirstlane(t.n_d);
  return t;
}

// Maximum of v over the wave, as a wave-uniform value.
__device__ inline uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, kWave));
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

// Blocked summation of f(i) over i = a, a + step, ... < e: every kBlk terms form
// a partial sum that then joins the running sum, so no serial chain of fp32
// additions is longer than kBlk or the number of blocks.
constexpr uint32_t kBlk = 16;

// load(i) fetches the index of term i (issued IN at a time, before any of them
// is used); use(x) gives the term for that index.
template <uint32_t IN = 4, typename L, typename U>
__device__ inline float blocked_sum(uint32_t a, uint32_t e, uint32_t step, L load, U use) {
  constexpr uint32_t kIn = IN;     // loads in flight together
  static_assert(kBlk % kIn == 0, "a block is a whole number of load groups");
  float acc = 0.0f;
  for (uint32_t b = a; b < e; b += kBlk * step) {
    float p = 0.0f;
    for (uint32_t u0 = 0; u0 < kBlk; u0 += kIn) {
      const uint32_t i0 = b + u0 * step;
      if (i0 >= e) break;
      uint32_t x[kIn];
#pragma unroll
      for (uint32_t u = 0; u < kIn; ++u) {
        const uint32_t i = i0 + u * step;
        x[u] = i < e ? load(i) : 0u;
      }
#pragma unroll
      for (uint32_t u = 0; u < kIn; ++u)
        if (i0 + u * step < e) p += use(x[u]);
    }
    acc += p;
  }
  return acc;
}

// ===========================================================================
// k = 1, H resident in LDS, one workgroup per batch.
// ===========================================================================

// Right multiplication (Theorem 1, Algorithm 4): H level by level, then one
// group of LPR lanes per tuple sums H over the tuple's codes.
constexpr int kK1RegCodes = 12;  // codes per thread held in registers by the k = 1 right product

template <int LPR, int BLK>
__global__ __launch_bounds__(BLK) void right_k1_kernel(Img im, int64_t b0,
                                                          const float *__restrict__ W,
                                                          int64_t ldw, float *__restrict__ R,
                                                          int64_t ldr) {
  extern __shared__ float H[];
  const toc_batch bt = im.batches[b0 + blockIdx.x];
  const uint32_t *lvl = im.level + bt.lvl_base;
  const NodePar par{deep_links(im.link, bt)};
  const NodeCol col{im.key + bt.code_base};
  const NodeVal val{im.key + bt.code_base};
  const uint32_t nc = (uint32_t)bt.n_codes, n1 = (uint32_t)bt.n_lvl1;
  if (nc <= (uint32_t)(kK1RegCodes * BLK)) {
    // every code's key, W entry and parent are loaded at once (thread t holds
    // codes t, t + BLK, ...); depth-1 codes' H is written right away, and each
    // deeper level then needs only LDS: H[c] = H[parent] + val * W[col]
    float v[kK1RegCodes], w[kK1RegCodes];
    uint32_t pr[kK1RegCodes];
#pragma unroll
    for (int i = 0; i < kK1RegCodes; ++i) {
      const uint32_t c = threadIdx.x + (uint32_t)(i * BLK);
      v[i] = 0.0f;
      w[i] = 0.0f;
      pr[i] = 0u;
      if (c < nc) {
        v[i] = val[c];
        w[i] = W[(int64_t)col[c] * ldw];
        if (c >= n1) pr[i] = par[c];
      }
    }
#pragma unroll
    for (int i = 0; i < kK1RegCodes; ++i) {
      const uint32_t c = threadIdx.x + (uint32_t)(i * BLK);
      if (c < n1) H[c] = fmaf(v[i], w[i], 0.0f);
    }
    __syncthreads();
    for (int d = 2; d <= bt.n_levels; ++d) {
      const uint32_t a = lvl[d - 1], e = lvl[d];
#pragma unroll
      for (int i = 0; i < kK1RegCodes; ++i) {
        const uint32_t c = threadIdx.x + (uint32_t)(i * BLK);
        if (c >= a && c < e) H[c] = fmaf(v[i], w[i], H[pr[i]]);
      }
      __syncthreads();
    }
  } else {
    for (int d = 1; d <= bt.n_levels; ++d) {
      const uint32_t a = lvl[d - 1], e = lvl[d];
#pragma unroll 4
      for (uint32_t c = a + threadIdx.x; c < e; c += BLK) {
        const float base = d > 1 ? H[par[c]] : 0.0f;
        H[c] = fmaf(val[c], W[(int64_t)col[c] * ldw], base);
      }
      __syncthreads();
    }
  }
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % LPR, grp = threadIdx.x / LPR;
  for (int r = grp; r < bt.n_rows; r += BLK / LPR) {
    const uint32_t s = span[r], e = span[r + 1];
    // (a whole block's codes loaded at once: 10 % faster on categorical batches
    // than 4 at a time)
    float acc = blocked_sum<kBlk>(s + lane, e, LPR, [&](uint32_t j) { return dc[j]; },
                                  [&](uint32_t c) { return H[c]; });
    acc = group_sum<LPR>(acc);
    if (lane == 0) R[(bt.row_base + r) * ldr] = acc;
  }
}

// Left multiplication (Theorem 2, Algorithm 5) without atomics, over the
// image's left positions (a leaf's position orders it by column; every other
// code is at its own index): H[p] = G(x) is pulled from the inverted index (the
// sum over the entries of D equal to the code x at p, whose tuples are listed in
// the batch's entry array; a thread takes 4 positions at a time and loads their
// occurrence rows together), each code then adds its children's H (children are
// contiguous: levels are sorted by parent), deepest level first; finally a thread
// per key column writes it once, summing val * H over the column's leaves (a
// contiguous range of positions) and tree codes (a contiguous stretch of the tree
// list), both read from the image's column index.
constexpr uint32_t kFirstOccK1 = 0x80000000u;
// Workgroup of the k = 1 right product: small, so that many batches (each a chain
// of dependent loads and barriers) are in flight on a CU at once.
constexpr int kK1RightBlock = 256;
constexpr int kK1Codes = 4;      // codes per thread and pass
constexpr int kK1Occ = 4;        // occurrences per code loaded together
// output columns per thread and pass: 4 or 8 (template argument NCOL of
// left_k1_kernel: 8 only for wide matrices, as 4 keeps the kernel at 50 VGPRs and
// 8 waves per SIMD, 8 needs 82)
constexpr int kK1Tree = 4;       // tree-list entries per column loaded together

// Where a batch's left positions find their occurrences: a leaf position p
// (n_int1 <= p < n_lvl1) at entries lo[p - n_int1] .. lo[p - n_int1 + 1]-1 of the
// batch's entry array, a tree code (its own position) at to[h] .. to[h+1]-1, h its
// tree row; a leaf's value beside its first occurrence, a tree code's in its key.
struct OccIndex {
  const uint32_t *lo, *to, *ce, *cv;
  const toc_key *key;
  uint32_t ni, n1;
  __device__ uint32_t hrow(uint32_t c) const { return c < ni ? c : c - n1 + ni; }
  __device__ bool leaf(uint32_t p) const { return p >= ni && p < n1; }
  __device__ uint32_t start(uint32_t p) const { return leaf(p) ? lo[p - ni] : to[hrow(p)]; }
  __device__ uint32_t end(uint32_t p) const { return leaf(p) ? lo[p - ni + 1] : to[hrow(p) + 1]; }
  // (0 for a leaf without occurrences, a kept dead code, whose sum is 0 anyway)
  __device__ float val(uint32_t p) const {
    if (!leaf(p)) return key[p].val;
    const uint32_t o = lo[p - ni];
    return o < lo[p - ni + 1] ? __uint_as_float(cv[o]) : 0.0f;
  }
};

__device__ inline OccIndex occ_index(const Img &im, const uint32_t *occ_off_all, const toc_batch &bt,
                                     int64_t b) {
  OccIndex x;
  x.ni = (uint32_t)bt.n_int1;
  x.n1 = (uint32_t)bt.n_lvl1;
  x.lo = occ_off_all + bt.code_base + 2 * b;
  x.to = x.lo + (x.n1 - x.ni) + 1;
  x.ce = im.centry + bt.d_base + bt.tree_base;
  x.cv = im.cval + bt.d_base + bt.tree_base;
  x.key = im.key + bt.code_base;
  return x;
}

template <int NCOL>
__global__ __launch_bounds__(kBlock) void left_k1_kernel(
    Img im, const uint32_t *__restrict__ occ_off_all, const uint32_t *__restrict__ tlist_all,
    const uint32_t *__restrict__ cols_all, const uint32_t *__restrict__ tchild_all, int64_t b0,
    int32_t m, int32_t max_rows, int32_t max_codes, const float *__restrict__ G, int64_t ldg,
    float *__restrict__ out, int64_t ldo, int accumulate) {
  extern __shared__ float sm[];
  const int64_t b = b0 + blockIdx.x;
  const toc_batch bt = uniform_batch(im.batches + b);
  const uint32_t *lvl = im.level + bt.lvl_base;
  const OccIndex ox = occ_index(im, occ_off_all, bt, b);
  const uint32_t *tl = tlist_all + bt.tree_base;
  const uint32_t *tch = tchild_all + bt.tree_base + b;
  const uint32_t *cx = cols_all + b * 4 * (int64_t)(m + 1);   // Loff, Ost, Toff, Ord
  const uint32_t nc = (uint32_t)bt.n_codes, ni = (uint32_t)bt.n_int1;
  float *Gs = sm;                                     // max_rows
  float *H = sm + max_rows;                           // max_codes
  auto hrow = [&](uint32_t c) -> uint32_t { return ox.hrow(c); };
  float *ob = out + b * (int64_t)m * ldo;
  // G(c) for every code; a leaf's times its value (read beside its first
  // occurrence), since a leaf has no children to add first.  A pass loads the
  // occurrence ranges and first entries of kK1Codes codes per thread; the first
  // pass's loads are issued before the G rows are staged, as they need none
  uint32_t o0[kK1Codes], o1[kK1Codes], vb[kK1Codes], w[kK1Codes][kK1Occ];
  auto load_pass = [&](uint32_t c0) {
#pragma unroll
    for (int u = 0; u < kK1Codes; ++u) {
      const uint32_t c = c0 + u * kBlock;
      o0[u] = c < nc ? ox.start(c) : 0u;
      o1[u] = c < nc ? ox.end(c) : 0u;
    }
#pragma unroll
    for (int u = 0; u < kK1Codes; ++u) {
      const uint32_t c = c0 + u * kBlock;
      // 1.0 for a tree code; a leaf without occurrences (kept dead code) sums to 0
      vb[u] = c < nc && ox.leaf(c) && o1[u] > o0[u] ? ox.cv[o0[u]] : 0x3F800000u;
#pragma unroll
      for (int v = 0; v < kK1Occ; ++v) w[u][v] = o0[u] + v < o1[u] ? ox.ce[o0[u] + v] : 0xFFFFFFFFu;
    }
  };
  load_pass(threadIdx.x);
  for (int r = threadIdx.x; r < bt.n_rows; r += kBlock) Gs[r] = G[(bt.row_base + r) * ldg];
  __syncthreads();
  for (uint32_t c0 = threadIdx.x; c0 < nc; c0 += kBlock * kK1Codes) {
    if (c0 != threadIdx.x) load_pass(c0);
    float s[kK1Codes];
#pragma unroll
    for (int u = 0; u < kK1Codes; ++u) {
      s[u] = 0.0f;
#pragma unroll
      for (int v = 0; v < kK1Occ; ++v)
        if (w[u][v] != 0xFFFFFFFFu) s[u] += Gs[w[u][v] & ~kFirstOccK1];
      if (o1[u] > o0[u] + kK1Occ)
        s[u] += blocked_sum<8>(o0[u] + kK1Occ, o1[u], 1u, [&](uint32_t o) { return ox.ce[o]; },
                            [&](uint32_t w) { return Gs[w & ~kFirstOccK1]; });
    }
#pragma unroll
    for (int u = 0; u < kK1Codes; ++u) {
      const uint32_t c = c0 + u * kBlock;
      if (c < nc) H[c] = ox.leaf(c) ? __uint_as_float(vb[u]) * s[u] : s[u];
    }
  }
  __syncthreads();
  // children into parents, deepest parent level first
  for (int d = bt.n_levels - 1; d >= 1; --d) {
    const uint32_t a = d == 1 ? 0 : lvl[d - 1], e = d == 1 ? ni : lvl[d];
    for (uint32_t c = a + threadIdx.x; c < e; c += kBlock) {
      const uint32_t h = hrow(c);
      H[c] += blocked_sum(tch[h], tch[h + 1], 1u, [&](uint32_t ch) { return ch; },
                          [&](uint32_t ch) { return H[ch]; });
    }
    __syncthreads();
  }
  // a tree code's H becomes val * H (the leaves' already are): a key column's
  // output is the plain sum of these over the column's codes
  const uint32_t n_tree = ni + (nc - ox.n1);
  for (uint32_t t0 = threadIdx.x; t0 < n_tree; t0 += kBlock * kK1Codes) {
    float v[kK1Codes];
#pragma unroll
    for (int u = 0; u < kK1Codes; ++u) {
      const uint32_t t = t0 + u * kBlock, c = t < ni ? t : t - ni + ox.n1;
      v[u] = t < n_tree ? ox.key[c].val : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kK1Codes; ++u) {
      const uint32_t t = t0 + u * kBlock, c = t < ni ? t : t - ni + ox.n1;
      if (t < n_tree) H[c] *= v[u];
    }
  }
  __syncthreads();
  // each key column once: its depth-1 leaves (a code range), then its tree
  // codes (a tree-list range); a thread has NCOL columns in flight and
  // loads the first kK1Tree tree-list entries of each before summing
  const uint32_t *Loff = cx, *Toff = cx + 2 * (m + 1);
  for (int j0 = 0; j0 < m; j0 += kBlock * NCOL) {
    uint32_t l0[NCOL], l1[NCOL], t0[NCOL], t1[NCOL];
#pragma unroll
    for (int u = 0; u < NCOL; ++u) {
      const int j = j0 + u * kBlock + threadIdx.x;
      const bool in = j < m;
      l0[u] = in ? Loff[j] : 0u;
      l1[u] = in ? Loff[j + 1] : 0u;
      t0[u] = in ? Toff[j] : 0u;
      t1[u] = in ? Toff[j + 1] : 0u;
    }
    uint32_t tc[NCOL][kK1Tree];
#pragma unroll
    for (int u = 0; u < NCOL; ++u)
#pragma unroll
      for (int v = 0; v < kK1Tree; ++v) tc[u][v] = t0[u] + v < t1[u] ? tl[t0[u] + v] : 0xFFFFFFFFu;
#pragma unroll
    for (int u = 0; u < NCOL; ++u) {
      const int j = j0 + u * kBlock + threadIdx.x;
      float sum = blocked_sum(l0[u], l1[u], 1u, [&](uint32_t c) { return c; },
                              [&](uint32_t c) { return H[c]; });
      float tsum = 0.0f;
#pragma unroll
      for (int v = 0; v < kK1Tree; ++v)
        if (tc[u][v] != 0xFFFFFFFFu) tsum += H[tc[u][v]];
      sum += tsum;
      if (t1[u] > t0[u] + kK1Tree)
        sum += blocked_sum(t0[u] + kK1Tree, t1[u], 1u, [&](uint32_t t) { return tl[t]; },
                           [&](uint32_t c) { return H[c]; });
      if (j < m) {
        float *p = ob + (int64_t)j * ldo;
        *p = accumulate ? *p + sum : sum;
      }
    }
  }
}

// ===========================================================================
// Any k: one workgroup per batch, one wave per code or tuple, lanes over up to
// kt = 64*KPL columns.  H rows of the codes that need one live in a workspace.
// ===========================================================================

// Right: H of depth >= 2 codes (depth-1 rows are val * W[col] and are formed where
// used), then per-tuple sums.  Algorithm 7 with the column loop innermost.
template <int KPL>
__global__ __launch_bounds__(kBlock) void right_wide_kernel(
    Img im, int64_t b0, int64_t ws_base, const float *__restrict__ W, int64_t ldw, int kt,
    float *__restrict__ R, int64_t ldr, float *__restrict__ ws) {
  const toc_batch bt = im.batches[b0 + blockIdx.x];
  const uint32_t *lvl = im.level + bt.lvl_base;
  const NodePar par{deep_links(im.link, bt)};
  const NodeCol col{im.key + bt.code_base};
  const NodeVal val{im.key + bt.code_base};
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const uint32_t n1 = (uint32_t)bt.n_lvl1;
  float *Hd = ws + (bt.deep_base - ws_base) * kt;
  for (int d = 2; d <= bt.n_levels; ++d) {
    const uint32_t a = lvl[d - 1], e = lvl[d];
    for (uint32_t c = a + wave; c < e; c += kWaves) {
      const uint32_t p = par[c];
      const float vc = val[c], vp = val[p];
      const float *wc = W + (int64_t)col[c] * ldw;
      const float *wp = W + (int64_t)col[p] * ldw;
      const float *hp = Hd + (int64_t)(p - n1) * kt;
      float *hc = Hd + (int64_t)(c - n1) * kt;
#pragma unroll
      for (int i = 0; i < KPL; ++i) {
        const int q = lane + kWave * i;
        if (q < kt) {
          const float base = p < n1 ? vp * wp[q] : hp[q];
          hc[q] = fmaf(vc, wc[q], base);
        }
      }
    }
    __syncthreads();
  }
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  for (int r = wave; r < bt.n_rows; r += kWaves) {
    float acc[KPL], part[KPL];
#pragma unroll
    for (int i = 0; i < KPL; ++i) acc[i] = 0.0f;
    const uint32_t s = span[r], e = span[r + 1];
    // blocked summation: kBlk entries per partial sum
    for (uint32_t j0 = s; j0 < e; j0 += kBlk) {
      const uint32_t je = min(e, j0 + kBlk);
#pragma unroll
      for (int i = 0; i < KPL; ++i) part[i] = 0.0f;
      for (uint32_t j = j0; j < je; ++j) {
        const uint32_t c = dc[j];
        if (c < n1) {
          const float v = val[c];
          const float *w = W + (int64_t)col[c] * ldw;
#pragma unroll
          for (int i = 0; i < KPL; ++i) {
            const int q = lane + kWave * i;
            if (q < kt) part[i] = fmaf(v, w[q], part[i]);
          }
        } else {
          const float *h = Hd + (int64_t)(c - n1) * kt;
#pragma unroll
          for (int i = 0; i < KPL; ++i) {
            const int q = lane + kWave * i;
            if (q < kt) part[i] += h[q];
          }
        }
      }
#pragma unroll
      for (int i = 0; i < KPL; ++i) acc[i] += part[i];
    }
    float *rr = R + (bt.row_base + r) * ldr;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int q = lane + kWave * i;
      if (q < kt) rr[q] = acc[i];
    }
  }
}

// Left by pulling (Theorem 2 read as a definition, the result of Algorithm 8),
// deterministic and without atomics: the H row of each tree code (a code with
// children or of depth >= 2) is the sum of the G rows of its occurrences (the
// inverted index of D) plus its children's H rows, deepest level first, a wave
// per code; then a wave per key column j sums val * G[row] over the occurrences
// of the column's depth-1 leaves and val * H over its tree codes, and writes
// out[j] once.  Column loop innermost (lanes over up to 64 * KPL columns); every
// sum is blocked (kBlk terms per partial sum).  H rows live in the workspace.
template <int KPL>
__global__ __launch_bounds__(kBlock) void left_wide_kernel(
    Img im, const uint32_t *__restrict__ occ_off_all,
    const uint32_t *__restrict__ tlist_all, const uint32_t *__restrict__ cols_all,
    const uint32_t *__restrict__ tchild_all, int64_t b0, int64_t ws_base, int32_t m,
    const float *__restrict__ G, int64_t ldg, int kt, float *__restrict__ out, int64_t ldo,
    int accumulate, float *__restrict__ ws) {
  constexpr uint32_t kFirst = 0x80000000u;
  const int64_t b = b0 + blockIdx.x;
  const toc_batch bt = uniform_batch(im.batches + b);
  const uint32_t *lvl = im.level + bt.lvl_base;
  const OccIndex ox = occ_index(im, occ_off_all, bt, b);
  const uint32_t *tl = tlist_all + bt.tree_base;
  const uint32_t *tch = tchild_all + bt.tree_base + b;
  const uint32_t *cx = cols_all + b * 4 * (int64_t)(m + 1);
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const uint32_t n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1;
  float *Ht = ws + (bt.tree_base - ws_base) * kt;
  const float *Gb = G + bt.row_base * ldg;
  auto hrow = [&](uint32_t c) -> int64_t { return c < ni ? c : (int64_t)c - n1 + ni; };
  float acc[KPL], part[KPL];
  uint32_t cnt = 0;
  auto start = [&]() {
#pragma unroll
    for (int i = 0; i < KPL; ++i) acc[i] = part[i] = 0.0f;
    cnt = 0;
  };
  // part += mul * row; every kBlk terms the partial sum joins acc
  auto add_term = [&](float mul, const float *row) {
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int q = lane + kWave * i;
      if (q < kt) part[i] = fmaf(mul, row[q], part[i]);
    }
    if (++cnt == kBlk) {
#pragma unroll
      for (int i = 0; i < KPL; ++i) {
        acc[i] += part[i];
        part[i] = 0.0f;
      }
      cnt = 0;
    }
  };
  auto finish = [&]() {
#pragma unroll
    for (int i = 0; i < KPL; ++i) acc[i] += part[i];
  };
  // tree codes, deepest level first (children are one level deeper)
  for (int d = bt.n_levels; d >= 1; --d) {
    const uint32_t a = d == 1 ? 0u : lvl[d - 1], e = d == 1 ? ni : lvl[d];
    for (uint32_t c = a + wave; c < e; c += kWaves) {
      const int64_t h = hrow(c);
      start();
      for (uint32_t o = ox.start(c), o1 = ox.end(c); o < o1; ++o)
        add_term(1.0f, Gb + (int64_t)(ox.ce[o] & ~kFirst) * ldg);
      for (uint32_t ch = tch[h], ch1 = tch[h + 1]; ch < ch1; ++ch)
        add_term(1.0f, Ht + hrow(ch) * kt);
      finish();
      float *hr = Ht + h * kt;
#pragma unroll
      for (int i = 0; i < KPL; ++i) {
        const int q = lane + kWave * i;
        if (q < kt) hr[q] = acc[i];
      }
    }
    __syncthreads();
  }
  // key columns: the leaves of column j are positions Loff[j] .. Loff[j+1]-1, its
  // tree codes tree-list entries Toff[j] .. Toff[j+1]-1
  const uint32_t *Loff = cx, *Toff = cx + 2 * (m + 1);
  float *ob = out + b * (int64_t)m * ldo;
  for (int j = wave; j < m; j += kWaves) {
    start();
    for (uint32_t p = Loff[j], p1 = Loff[j + 1]; p < p1; ++p) {
      const float v = ox.val(p);
      for (uint32_t o = ox.start(p), o1 = ox.end(p); o < o1; ++o)
        add_term(v, Gb + (int64_t)(ox.ce[o] & ~kFirst) * ldg);
    }
    for (uint32_t t = Toff[j], t1 = Toff[j + 1]; t < t1; ++t) {
      const uint32_t c = tl[t];
      add_term(ox.val(c), Ht + hrow(c) * kt);
    }
    finish();
    float *o = ob + (int64_t)j * ldo;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int q = lane + kWave * i;
      if (q < kt) o[q] = accumulate ? o[q] + acc[i] : acc[i];
    }
  }
}

// ===========================================================================
// ===========================================================================
// Tiled kernels for wide k.  Persistent workgroups, one per CU.  Blocks are dealt
// to the 8 XCDs round-robin; worker s of XCD x takes items s, s + spw, ... of its
// XCD's list, in which item i is column tile i % n_tiles of batch
// x + 8 * (i / n_tiles).  The tiles of a batch are consecutive items, so they run
// together on one XCD and share the batch's image in that XCD's L2.
// ===========================================================================
constexpr int kXcd = 8;
constexpr int kCuPerXcd = 32;

__device__ inline float4 f4fma(float s, float4 x, float4 a) {
  return make_float4(fmaf(s, x.x, a.x), fmaf(s, x.y, a.y), fmaf(s, x.z, a.z), fmaf(s, x.w, a.w));
}

__device__ inline void add4(float4 &a, const float4 &b) {
  a.x += b.x;
  a.y += b.y;
  a.z += b.z;
  a.w += b.w;
}

__device__ inline uint32_t rdlane(uint32_t v, uint32_t i) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)i);
}


// Raw buffer resource over n 32-bit elements: loads at an index >= n return 0
// instead of touching memory (the range check of buffer instructions).
using BufRes = __amdgpu_buffer_rsrc_t;
constexpr int kBufFlags = 0x00020000;   // dword 3 of a raw 32-bit buffer descriptor on gfx9

__device__ inline BufRes buf_res(const void *p, uint32_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)(n * 4u),
                                           kBufFlags);
}

__device__ inline uint32_t buf_load(BufRes r, uint32_t i) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, i * 4u, 0, 0);
}

// Buffer over n keys; key_load reads the key pair (col, val bits) of one.
__device__ inline BufRes key_res(const toc_key *p, uint32_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<toc_key *>(p), (short)0,
                                           (int)(n * (uint32_t)sizeof(toc_key)), kBufFlags);
}

__device__ inline uint2 key_load(BufRes r, uint32_t c) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, c * (uint32_t)sizeof(toc_key), 0, 0);
  return make_uint2(v[0], v[1]);
}

// Buffer over n links; link_load reads the (parent, depth) pair of one.
__device__ inline BufRes link_res(const toc_link *p, uint32_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<toc_link *>(p), (short)0,
                                           (int)(n * (uint32_t)sizeof(toc_link)), kBufFlags);
}

__device__ inline uint2 link_load(BufRes r, uint32_t c) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, c * (uint32_t)sizeof(toc_link), 0, 0);
  return make_uint2(v[0], v[1]);
}

// LDS reads through address-space-3 pointers (byte addresses in LDS): the
// compiler never merges such a read with a global one into a flat access.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;

__device__ inline uint32_t lds_base(float4 *smem) {
  return (uint32_t)(size_t)(__attribute__((address_space(3))) float4 *)smem;
}

__device__ inline float4 lds_load4(uint32_t byte) {
  const f32x4 v = *(const lds_f32x4 *)(size_t)byte;
  return make_float4(v[0], v[1], v[2], v[3]);
}

// ---------------------------------------------------------------------------
// Right multiplication (Theorem 1, Algorithm 7), tiled over the columns of W.
// Work items are (batch, 32-column tile) pairs.  The items of one batch are
// consecutive in the item order of one XCD, so the workers that take them run
// together there and share the batch's image in that XCD's L2.  A worker keeps
// the tile of W it last used in LDS (rows 0..m-1; row m is all zeros) and the H
// rows of the batch's depth >= 2 codes after it, built level by level.
// A 16-lane row of the wave owns one tuple (a lane holds 2 columns), so a wave
// sums 4 tuples at once and needs no cross-lane reduction of sums.  Lane l of a
// row loads the codes of entries l and l + 16 of its tuple's chunk two steps
// ahead, gathers their keys one step ahead and translates them to (LDS address
// of the H row, multiplier) in registers.  While a chunk is summed, the row
// broadcast of the DPP cross-lane operations hands entry t of every tuple to
// all 16 lanes of its row (the address through an add, the multiplier through
// the FMA itself), so the only LDS reads are the H rows.  Entries past the end
// of a tuple point at the zero row with multiplier 0.
// ---------------------------------------------------------------------------
constexpr int kRtKT = 32;
constexpr int kRtBlock = 1024;
constexpr int kRtWaves = kRtBlock / kWave;
constexpr int kRtLanes = 16;                      // lanes per tuple: one DPP row
constexpr int kRtGroups = kWave / kRtLanes;       // tuples per wave
constexpr int kRtPer = 2;                         // entries per lane and chunk
constexpr int kRtChunk = kRtPer * kRtLanes;       // entries per tuple per pipeline step
constexpr uint32_t kRtRowBytes = kRtKT * 4;
constexpr uint32_t kRtStaticBytes = 16;           // static LDS: two tuple-group counters
constexpr uint32_t kRtGlobal = 0x80000000u;       // row index flag: the H row lives in the workspace
constexpr int kRtDeepU = 2;                       // deep codes per 8-lane group and round

// The value v of lane T of the caller's 16-lane row, in every lane of the row.
template <int T>
__device__ inline uint32_t row_bcast(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x150 + T, 0xF, 0xF, true);
}

// f(std::integral_constant<int, I>{}) for I = 0 .. N-1, unrolled.
template <typename F, int... I>
__device__ inline void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ inline void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) f32x2 lds_f32x2;

__device__ inline float2 lds_load2(uint32_t byte) {
  const f32x2 v = *(const lds_f32x2 *)(size_t)byte;
  return make_float2(v[0], v[1]);
}

// acc += mu(lane L of the row) * x[i] for 8 entries, lanes L = T0 .. T0 + 7: the
// FMA reads the multiplier across lanes itself.  A cross-lane read of a register
// needs two wait states after a vector write of it; the s_nop provides them.
#define TOC_FMAC2(I, L)                                                                  \
  "v_fmac_f32_dpp %[ax], %[mu], %[x" #I "] row_newbcast:" #L                             \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"                                          \
  "v_fmac_f32_dpp %[ay], %[mu], %[y" #I "] row_newbcast:" #L                             \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
#define TOC_FMA8(L0, L1, L2, L3, L4, L5, L6, L7)                                         \
  asm volatile("s_nop 1\n\t" TOC_FMAC2(0, L0) TOC_FMAC2(1, L1) TOC_FMAC2(2, L2)          \
                   TOC_FMAC2(3, L3) TOC_FMAC2(4, L4) TOC_FMAC2(5, L5) TOC_FMAC2(6, L6)   \
                       TOC_FMAC2(7, L7)                                                   \
               : [ax] "+v"(acc.x), [ay] "+v"(acc.y)                                       \
               : [mu] "v"(mu), [x0] "v"(x[0].x), [y0] "v"(x[0].y), [x1] "v"(x[1].x),      \
                 [y1] "v"(x[1].y), [x2] "v"(x[2].x), [y2] "v"(x[2].y), [x3] "v"(x[3].x),  \
                 [y3] "v"(x[3].y), [x4] "v"(x[4].x), [y4] "v"(x[4].y), [x5] "v"(x[5].x),  \
                 [y5] "v"(x[5].y), [x6] "v"(x[6].x), [y6] "v"(x[6].y), [x7] "v"(x[7].x),  \
                 [y7] "v"(x[7].y))

template <int T0>
__device__ inline void fma8_bcast(float2 &acc, uint32_t mu, const float2 (&x)[8]) {
  static_assert(T0 == 0 || T0 == 8, "lanes 0..7 or 8..15 of a row");
  if constexpr (T0 == 0) {
    TOC_FMA8(0, 1, 2, 3, 4, 5, 6, 7);
  } else {
    TOC_FMA8(8, 9, 10, 11, 12, 13, 14, 15);
  }
}
#undef TOC_FMA8
#undef TOC_FMAC2

// The same for 4 columns per lane: acc += mu(lane L) * x[i] for 4 entries.
#define TOC_FMAC4(I, L)                                                                  \
  "v_fmac_f32_dpp %[ax], %[mu], %[x" #I "] row_newbcast:" #L                             \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"                                          \
  "v_fmac_f32_dpp %[ay], %[mu], %[y" #I "] row_newbcast:" #L                             \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"                                          \
  "v_fmac_f32_dpp %[az], %[mu], %[z" #I "] row_newbcast:" #L                             \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"                                          \
  "v_fmac_f32_dpp %[aw], %[mu], %[w" #I "] row_newbcast:" #L                             \
  " row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
#define TOC_X4(I) [x##I] "v"(x[I].x), [y##I] "v"(x[I].y), [z##I] "v"(x[I].z), [w##I] "v"(x[I].w)
#define TOC_FMA4X4(L0, L1, L2, L3)                                                       \
  asm volatile("s_nop 1\n\t" TOC_FMAC4(0, L0) TOC_FMAC4(1, L1) TOC_FMAC4(2, L2)          \
                   TOC_FMAC4(3, L3)                                                       \
               : [ax] "+v"(acc.x), [ay] "+v"(acc.y), [az] "+v"(acc.z), [aw] "+v"(acc.w)   \
               : [mu] "v"(mu), TOC_X4(0), TOC_X4(1), TOC_X4(2), TOC_X4(3))

template <int T0>
__device__ inline void fma4x4_bcast(float4 &acc, uint32_t mu, const float4 (&x)[4]) {
  static_assert(T0 % 4 == 0 && T0 < 16, "lanes T0 .. T0 + 3 of a row");
  if constexpr (T0 == 0) {
    TOC_FMA4X4(0, 1, 2, 3);
  } else if constexpr (T0 == 4) {
    TOC_FMA4X4(4, 5, 6, 7);
  } else if constexpr (T0 == 8) {
    TOC_FMA4X4(8, 9, 10, 11);
  } else {
    TOC_FMA4X4(12, 13, 14, 15);
  }
}
#undef TOC_FMA4X4
#undef TOC_X4
#undef TOC_FMAC4

// The H rows of entries T0 .. T0 + 7 of a half chunk (rb: the row address held
// by each lane, qoff: this lane's columns in a row).
template <int T0>
__device__ inline void load8_bcast(uint32_t rb, uint32_t qoff, float2 (&x)[8]) {
  static_for<8>([&](auto i) { x[i] = lds_load2(row_bcast<T0 + decltype(i)::value>(rb) + qoff); });
}

// The rows of entries T0 .. T0 + 3 with 4 columns per lane (16-byte reads).
template <int T0>
__device__ inline void load4x4_bcast(uint32_t rb, uint32_t qoff, float4 (&x)[4]) {
  static_for<4>([&](auto i) { x[i] = lds_load4(row_bcast<T0 + decltype(i)::value>(rb) + qoff); });
}

struct RtChunk {
  int tg;           // tuple group (tuples 4*tg .. 4*tg+3 of the batch); >= n_tg: none
  uint32_t steps;   // entries per tuple to process, rounded up to a multiple of 8
  bool last;        // last chunk of the tuple group
};

__global__ __launch_bounds__(kRtBlock) void right_tiled_kernel(
    Img im, int64_t nb, int n_tiles, int spw, int per, int m, const float *__restrict__ W,
    int64_t ldw, int k, float *__restrict__ R, int64_t ldr) {
  extern __shared__ float4 smem4[];
  const int x = (int)(blockIdx.x % kXcd), s = (int)(blockIdx.x / kXcd);
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const int grp = lane / kRtLanes, sub = lane % kRtLanes, q = 2 * sub;
  __shared__ uint32_t tg_next[2];                             // next free tuple group, by item parity
  float *Wt = (float *)smem4;                                 // (m + 1) x kRtKT, then deep rows
  const uint32_t wb = lds_base(smem4);                        // LDS address of row 0
  const uint32_t qoff = 4u * (uint32_t)q;                     // this lane's columns in a row
  const uint32_t zrow_b = wb + (uint32_t)m * kRtRowBytes;
  for (int e = threadIdx.x; e < kRtKT; e += kRtBlock) Wt[m * kRtKT + e] = 0.0f;
  if (threadIdx.x < 2) tg_next[threadIdx.x] = kRtWaves;
  // batches of this XCD, taken `per` (1 or 2) at a time
  const int64_t nbx = nb > x ? (nb - x + kXcd - 1) / kXcd : 0;
  const int64_t n_items = (nbx + per - 1) / per * n_tiles;
  int cur_tile = -1;
  uint32_t parity = 0;
  for (int64_t it = s; it < n_items; it += spw, parity ^= 1u) {
    const int64_t gj = uniform64(per * (it / n_tiles));
    const bool two = per == 2 && gj + 1 < nbx;               // a second batch B after A
    const int tile = __builtin_amdgcn_readfirstlane((int)(it % n_tiles));
    const int k0 = tile * kRtKT;
    const int kt = min(kRtKT, k - k0);
    const toc_batch ba = uniform_batch(im.batches + x + kXcd * gj);
    const toc_batch bb = uniform_batch(im.batches + x + kXcd * (two ? gj + 1 : gj));
    const uint32_t *lvl_a = im.level + ba.lvl_base, *lvl_b = im.level + bb.lvl_base;
    const uint32_t n1a = (uint32_t)ba.n_lvl1, n1b = (uint32_t)bb.n_lvl1;
    const int nrows_a = ba.n_rows, nrows_b = two ? bb.n_rows : 0;
    const int lev_a = ba.n_levels, lev_b = two ? bb.n_levels : 0;
    // H row of deep code c: db + c (A's deep rows first, then B's)
    const uint32_t db_a = (uint32_t)m + 1u - n1a;
    const uint32_t db_b = (uint32_t)m + 1u + ((uint32_t)ba.n_codes - n1a) - n1b;
    __syncthreads();   // the previous item no longer reads the W tile or the deep rows
    // the counter of the previous item is free again: ready for the next one
    if (threadIdx.x == 0) tg_next[parity ^ 1u] = kRtWaves;
    if (tile != cur_tile) {
      // all loads of a pass first, then the stores
      const int n4 = m * (kRtKT / 4);
      const bool vec = kt == kRtKT && (ldw % 4) == 0 && (((uintptr_t)(W + k0)) & 15u) == 0;
      for (int e0 = threadIdx.x; e0 < n4; e0 += 8 * kRtBlock) {
        float4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i * kRtBlock;
          v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (e < n4) {
            const int c = e / (kRtKT / 4), q4 = 4 * (e % (kRtKT / 4));
            const float *src = W + (int64_t)c * ldw + k0 + q4;
            if (vec) {
              v[i] = *(const float4 *)src;
            } else {
              if (q4 + 0 < kt) v[i].x = src[0];
              if (q4 + 1 < kt) v[i].y = src[1];
              if (q4 + 2 < kt) v[i].z = src[2];
              if (q4 + 3 < kt) v[i].w = src[3];
            }
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i * kRtBlock;
          if (e < n4) *(float4 *)&Wt[e * 4] = v[i];
        }
      }
      cur_tile = tile;
      __syncthreads();
    }
    // H of depth >= 2 codes, level by level, both batches together: 8 lanes per
    // code (4 columns each, 16-byte accesses), kRtDeepU codes per group and
    // round.  Every load is unconditional (indices are clamped to valid codes)
    // so that the loads of a round are all in flight together.
    {
      const toc_key *key_a = im.key + ba.code_base, *key_b = im.key + bb.code_base;
      const toc_link *link_a = deep_links(im.link, ba), *link_b = deep_links(im.link, bb);
      const uint32_t g8 = threadIdx.x / 8u, q4 = 4u * (threadIdx.x % 8u);
      constexpr uint32_t stride = kRtBlock / 8;
      const int n_lev = max(lev_a, lev_b);
      for (int d = 2; d <= n_lev; ++d) {
        // level d of A is codes [a0, a0 + na), of B [b0, b0 + (n - na))
        const uint32_t a0 = d <= lev_a ? lvl_a[d - 1] : 0u;
        const uint32_t na = d <= lev_a ? lvl_a[d] - a0 : 0u;
        const uint32_t b0 = d <= lev_b ? lvl_b[d - 1] : 0u;
        const uint32_t n = na + (d <= lev_b ? lvl_b[d] - b0 : 0u);
        for (uint32_t i0 = g8; i0 < n; i0 += kRtDeepU * stride) {
          uint32_t cs[kRtDeepU], p[kRtDeepU], n1[kRtDeepU], db[kRtDeepU];
          bool live[kRtDeepU];
          uint2 kc[kRtDeepU], kp[kRtDeepU];
          const toc_key *kb[kRtDeepU];
#pragma unroll
          for (int u = 0; u < kRtDeepU; ++u) {
            live[u] = i0 + u * stride < n;
            const uint32_t i = live[u] ? i0 + u * stride : i0;
            const bool in_b = i >= na;
            cs[u] = in_b ? b0 + (i - na) : a0 + i;
            kb[u] = in_b ? key_b : key_a;
            n1[u] = in_b ? n1b : n1a;
            db[u] = in_b ? db_b : db_a;
            p[u] = (in_b ? link_b : link_a)[cs[u]].parent;
            kc[u] = *(const uint2 *)(kb[u] + cs[u]);
          }
#pragma unroll
          for (int u = 0; u < kRtDeepU; ++u) kp[u] = *(const uint2 *)(kb[u] + (p[u] < n1[u] ? p[u] : 0u));
          float4 bl[kRtDeepU], w[kRtDeepU];
#pragma unroll
          for (int u = 0; u < kRtDeepU; ++u) {
            const uint32_t lrow = p[u] < n1[u] ? kp[u].x : db[u] + p[u];
            bl[u] = *(const float4 *)&Wt[lrow * kRtKT + q4];
            w[u] = *(const float4 *)&Wt[kc[u].x * kRtKT + q4];
          }
#pragma unroll
          for (int u = 0; u < kRtDeepU; ++u) {
            const float vp = p[u] < n1[u] ? __uint_as_float(kp[u].y) : 1.0f;
            const float vc = __uint_as_float(kc[u].y);
            const float4 h = make_float4(fmaf(vc, w[u].x, vp * bl[u].x), fmaf(vc, w[u].y, vp * bl[u].y),
                                         fmaf(vc, w[u].z, vp * bl[u].z), fmaf(vc, w[u].w, vp * bl[u].w));
            if (live[u]) *(float4 *)&Wt[(db[u] + cs[u]) * kRtKT + q4] = h;
          }
        }
        __syncthreads();
      }
    }
    // per-tuple sums.  Tuple groups 0 .. n_tga - 1 are A's, then B's.
    const int n_tga = (nrows_a + kRtGroups - 1) / kRtGroups;
    const int n_tg = n_tga + (nrows_b + kRtGroups - 1) / kRtGroups;
    const uint32_t *span_a = im.span + ba.span_base, *span_b = im.span + bb.span_base;
    // rows past the end read span[nrows] twice: an empty tuple
    auto spans_of = [&](int tg, uint32_t &st, uint32_t &en) {
      const bool in_b = tg >= n_tga;
      const uint32_t *span = in_b ? span_b : span_a;
      const int nr = in_b ? nrows_b : nrows_a;
      const int r = min((in_b ? tg - n_tga : tg) * kRtGroups + grp, nr);
      st = span[r];
      en = span[min(r + 1, nr)];
    };
    auto wave_max = [&](uint32_t v) -> uint32_t {
      v = max(v, (uint32_t)__shfl_xor((int)v, 16, kWave));
      v = max(v, (uint32_t)__shfl_xor((int)v, 32, kWave));
      return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
    };
    // Tuple groups: wave w starts with group w, then takes the next free group
    // from the item's counter, so waves that finish early take more groups.
    auto grab = [&]() -> int {
      uint32_t g = 0;
      if (lane == 0) g = atomicAdd(&tg_next[parity], 1u);
      return __builtin_amdgcn_readfirstlane((int)g);
    };
    // load stage: tuple group ltg, entries [lj, lj + kRtChunk) of each tuple;
    // ntg is the group after it, whose spans are in nst, nen
    int ltg = wave, ntg = n_tg;
    uint32_t lj = 0, lmax = 0, lst = 0, len = 0, nst = 0, nen = 0;
    if (ltg < n_tg) {
      spans_of(ltg, lst, len);
      lmax = wave_max(len - lst);
      ntg = grab();
    }
    spans_of(ntg, nst, nen);
    auto chunk_of_l = [&]() -> RtChunk {
      const uint32_t n = lmax > lj ? min((uint32_t)kRtChunk, lmax - lj) : 0u;
      return RtChunk{ltg, (n + 7u) & ~7u, lj + kRtChunk >= lmax};
    };
    // the next group's spans are reloaded on every step (cache hits), so that a
    // switch of group only moves values loaded a step earlier
    auto advance = [&]() {
      if (ltg < n_tg) {
        lj += kRtChunk;
        if (lj >= lmax) {
          ltg = ntg;
          lj = 0;
          lst = nst;
          len = nen;
          lmax = 0u;
          if (ltg < n_tg) {
            lmax = wave_max(len - lst);
            ntg = grab();
          }
        }
      }
      spans_of(ntg, nst, nen);
    };
    // Every load below is unconditional: the buffer range checks turn reads past
    // the batch's arrays into zeros, and entries past the end of a tuple are
    // marked in a wave mask and become (zero row, 0) when translated.
    const BufRes rs_dc_a = buf_res(im.dcodes + ba.d_base, (uint32_t)ba.n_d);
    const BufRes rs_dc_b = buf_res(im.dcodes + bb.d_base, (uint32_t)bb.n_d);
    const BufRes rs_node_a = key_res(im.key + ba.code_base, (uint32_t)ba.n_codes);
    const BufRes rs_node_b = key_res(im.key + bb.code_base, (uint32_t)bb.n_codes);
    // codes of entries sub + 16 h (h < kRtPer) of the load stage's chunk
    auto load_codes = [&](uint32_t (&d)[kRtPer], uint64_t (&ok)[kRtPer]) {
      const bool live = ltg < n_tg;
      const BufRes rs_dc = ltg >= n_tga ? rs_dc_b : rs_dc_a;
      static_for<kRtPer>([&](auto hc) {
        constexpr int h = decltype(hc)::value;
        const uint32_t j = lst + lj + (uint32_t)sub + (uint32_t)(h * kRtLanes);
        ok[h] = __ballot(live && j < len);
        d[h] = buf_load(rs_dc, j);
      });
    };
    // (H row, multiplier) of an entry: a depth-1 code's row is its column of W
    // times its value; a deeper code's row is its own H row, times 1
    auto translate = [&](uint32_t d, uint2 key, uint64_t ok, uint32_t n1, uint32_t db, uint32_t &rb,
                         uint32_t &mu) {
      if (d < n1) {
        rb = wb + key.x * kRtRowBytes;
        mu = key.y;
      } else {
        rb = wb + (db + d) * kRtRowBytes;
        mu = __float_as_uint(1.0f);
      }
      if (!__builtin_amdgcn_inverse_ballot_w64(ok)) {
        rb = zrow_b;
        mu = 0u;
      }
    };
    float2 acc = make_float2(0.f, 0.f);
    // Pipeline: codes of chunk L load while chunk G's keys are gathered and
    // chunk C, translated in registers, is summed; G is translated at the end of
    // the step.  Two register sets of codes alternate between the roles of G and
    // L, so no loaded value is ever copied.
    RtChunk G = chunk_of_l();
    RtChunk C{n_tg, 0u, false};
    uint32_t crb[kRtPer], cmu[kRtPer];
#pragma unroll
    for (int h = 0; h < kRtPer; ++h) {
      crb[h] = zrow_b;
      cmu[h] = 0u;
    }
    auto step = [&](const uint32_t (&gd)[kRtPer], const uint64_t (&gok)[kRtPer],
                    uint32_t (&ld)[kRtPer], uint64_t (&lok)[kRtPer]) {
      advance();
      const bool g_in_b = G.tg >= n_tga;
      const BufRes rs_node = g_in_b ? rs_node_b : rs_node_a;
      uint2 key[kRtPer];
      static_for<kRtPer>([&](auto hc) {
        constexpr int h = decltype(hc)::value;
        key[h] = key_load(rs_node, gd[h]);
      });
      const RtChunk L = chunk_of_l();
      load_codes(ld, lok);
      if (C.tg < n_tg) {
        // blocked summation: the chunk's entries go into a partial sum of their
        // own, which then joins the tuple's running sum, so no serial chain is
        // longer than a chunk (kRtChunk) or the tuple's number of chunks
        float2 part = make_float2(0.f, 0.f);
        if (C.steps == kRtChunk) {
          // each block's reads are issued before the previous block's FMAs
          float2 x0[8], x1[8];
          load8_bcast<0>(crb[0], qoff, x0);
          static_for<kRtPer>([&](auto hc) {
            constexpr int h = decltype(hc)::value;
            load8_bcast<8>(crb[h], qoff, x1);
            fma8_bcast<0>(part, cmu[h], x0);
            if constexpr (h + 1 < kRtPer) load8_bcast<0>(crb[h + 1], qoff, x0);
            fma8_bcast<8>(part, cmu[h], x1);
          });
        } else {
          static_for<kRtPer>([&](auto hc) {
            constexpr int h = decltype(hc)::value;
            if (C.steps > (uint32_t)(16 * h)) {
              float2 xr[8];
              load8_bcast<0>(crb[h], qoff, xr);
              fma8_bcast<0>(part, cmu[h], xr);
            }
            if (C.steps > (uint32_t)(16 * h + 8)) {
              float2 xr[8];
              load8_bcast<8>(crb[h], qoff, xr);
              fma8_bcast<8>(part, cmu[h], xr);
            }
          });
        }
        acc.x += part.x;
        acc.y += part.y;
        if (C.last) {
          const bool in_b = C.tg >= n_tga;
          const int r = (in_b ? C.tg - n_tga : C.tg) * kRtGroups + grp;
          if (r < (in_b ? nrows_b : nrows_a)) {
            float *rr = R + ((in_b ? bb.row_base : ba.row_base) + r) * ldr + k0 + q;
            if (q + 1 < kt) {
              rr[0] = acc.x;
              rr[1] = acc.y;
            } else if (q < kt) {
              rr[0] = acc.x;
            }
          }
          acc = make_float2(0.f, 0.f);
        }
      }
      // chunk G becomes chunk C
      static_for<kRtPer>([&](auto hc) {
        constexpr int h = decltype(hc)::value;
        translate(gd[h], key[h], gok[h], g_in_b ? n1b : n1a, g_in_b ? db_b : db_a, crb[h], cmu[h]);
      });
      C = G;
      G = L;
    };
    uint32_t dA[kRtPer], dB[kRtPer];
    uint64_t okA[kRtPer], okB[kRtPer];
    load_codes(dA, okA);
    while (G.tg < n_tg || C.tg < n_tg) {
      step(dA, okA, dB, okB);
      if (!(G.tg < n_tg || C.tg < n_tg)) break;
      step(dB, okB, dA, okA);
    }
  }
}

// ---------------------------------------------------------------------------
// Right multiplication, the same product for batches whose deep H rows do not
// fit in LDS next to the W tile: those rows live in the worker's workspace
// slot.  An 8-lane group owns one tuple (a lane holds 4 columns, so a workspace
// row is read with 16-byte loads), so a wave sums 8 tuples at once.  The codes
// of the wave's entries are loaded two chunks ahead and translated to (row,
// multiplier) one chunk ahead; a chunk (16 entries of each of the 8 tuples) is
// staged in the wave's part of LDS, where every lane of a group reads its
// tuple's entry by broadcast.  Entries past the end of a tuple point at the
// zero row.  Rows in the workspace are marked with kRtGlobal.
// ---------------------------------------------------------------------------
constexpr int kRsGroups = kWave / 8;              // tuples per wave
constexpr int kRsChunk = 16;                      // entries per tuple per pipeline step
constexpr uint32_t kRsStageBytes = kRtWaves * kRsChunk * kRsGroups * 8;

struct RsChunk {
  int tg;           // tuple group (tuples 8*tg .. 8*tg+7 of the batch); >= n_tg: none
  uint32_t steps;   // entries per tuple to process, rounded up to a multiple of 4
  bool last;        // last chunk of the tuple group
};

__global__ __launch_bounds__(kRtBlock) void right_staged_kernel(
    Img im, int64_t nb, int n_tiles, int spw, int m, const float *__restrict__ W,
    int64_t ldw, int k, float *__restrict__ R, int64_t ldr, float *__restrict__ ws,
    int64_t slot_floats) {
  extern __shared__ float4 smem4[];
  char *lds = (char *)smem4;
  const int x = (int)(blockIdx.x % kXcd), s = (int)(blockIdx.x / kXcd);
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const int grp = lane / 8, sub = lane % 8, q = 4 * sub;
  __shared__ uint32_t tg_next[2];                             // next free tuple group, by item parity
  uint2 *stage = (uint2 *)lds + wave * (kRsChunk * kRsGroups);
  float *Wt = (float *)(lds + kRsStageBytes);                 // (m + 1) x kRtKT, then deep rows
  const uint32_t qb = lds_base(smem4) + kRsStageBytes + 4u * (uint32_t)q;   // LDS address of this lane's columns
  const uint32_t zrow = (uint32_t)m;
  float *Hg = ws + blockIdx.x * slot_floats;
  for (int e = threadIdx.x; e < kRtKT; e += kRtBlock) Wt[m * kRtKT + e] = 0.0f;
  if (threadIdx.x < 2) tg_next[threadIdx.x] = kRtWaves;
  const int64_t nbx = nb > x ? (nb - x + kXcd - 1) / kXcd : 0;
  const int64_t n_items = nbx * n_tiles;
  int cur_tile = -1;
  uint32_t parity = 0;
  for (int64_t it = s; it < n_items; it += spw, parity ^= 1u) {
    const int64_t b = uniform64(x + kXcd * (it / n_tiles));
    const int tile = __builtin_amdgcn_readfirstlane((int)(it % n_tiles));
    const int k0 = tile * kRtKT;
    const int kt = min(kRtKT, k - k0);
    const toc_batch bt = uniform_batch(im.batches + b);
    const uint32_t *lvl = im.level + bt.lvl_base;
    const NodePar par{deep_links(im.link, bt)};
    const NodeCol col{im.key + bt.code_base};
    const NodeVal val{im.key + bt.code_base};
    const uint32_t *span = im.span + bt.span_base;
    const uint32_t *dc = im.dcodes + bt.d_base;
    const uint32_t n1 = (uint32_t)bt.n_lvl1;
    const int nrows = bt.n_rows;
    __syncthreads();   // the previous item no longer reads the W tile or the deep rows
    // the counter of the previous item is free again: ready for the next one
    if (threadIdx.x == 0) tg_next[parity ^ 1u] = kRtWaves;
    if (tile != cur_tile) {
      // all loads of a pass first, then the stores
      const int n4 = m * (kRtKT / 4);
      const bool vec = kt == kRtKT && (ldw % 4) == 0 && (((uintptr_t)(W + k0)) & 15u) == 0;
      for (int e0 = threadIdx.x; e0 < n4; e0 += 8 * kRtBlock) {
        float4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i * kRtBlock;
          v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (e < n4) {
            const int c = e / (kRtKT / 4), q4 = 4 * (e % (kRtKT / 4));
            const float *src = W + (int64_t)c * ldw + k0 + q4;
            if (vec) {
              v[i] = *(const float4 *)src;
            } else {
              if (q4 + 0 < kt) v[i].x = src[0];
              if (q4 + 1 < kt) v[i].y = src[1];
              if (q4 + 2 < kt) v[i].z = src[2];
              if (q4 + 3 < kt) v[i].w = src[3];
            }
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i * kRtBlock;
          if (e < n4) *(float4 *)&Wt[e * 4] = v[i];
        }
      }
      cur_tile = tile;
      __syncthreads();
    }
    // H of depth >= 2 codes, level by level; a group per code
    const int gidx = wave * kRsGroups + grp;
    for (int d = 2; d <= bt.n_levels; ++d) {
      const uint32_t a = lvl[d - 1], e = lvl[d];
      for (uint32_t c = a + gidx; c < e; c += kRtWaves * kRsGroups) {
        const uint32_t p = par[c];
        const uint32_t cc = col[c];
        const float vc = val[c];
        float4 base;
        if (p < n1) {
          const float vp = val[p];
          base = *(const float4 *)&Wt[col[p] * kRtKT + q];
          base = make_float4(vp * base.x, vp * base.y, vp * base.z, vp * base.w);
        } else {
          base = *(const float4 *)&Hg[(int64_t)(p - n1) * kRtKT + q];
        }
        const float4 h = f4fma(vc, *(const float4 *)&Wt[cc * kRtKT + q], base);
        *(float4 *)&Hg[(int64_t)(c - n1) * kRtKT + q] = h;
      }
      __syncthreads();
    }
    // per-tuple sums
    const int n_tg = (nrows + kRsGroups - 1) / kRsGroups;
    // rows past the end read span[nrows] twice: an empty tuple
    auto spans_of = [&](int tg, uint32_t &st, uint32_t &en) {
      const int r = min(tg * kRsGroups + grp, nrows);
      st = span[r];
      en = span[min(r + 1, nrows)];
    };
    auto wave_max = [&](uint32_t v) -> uint32_t {
      v = max(v, (uint32_t)__shfl_xor((int)v, 8, kWave));
      v = max(v, (uint32_t)__shfl_xor((int)v, 16, kWave));
      v = max(v, (uint32_t)__shfl_xor((int)v, 32, kWave));
      return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
    };
    // Tuple groups: wave w starts with group w, then takes the next free group
    // from the item's counter, so waves that finish early take more groups.
    auto grab = [&]() -> int {
      uint32_t g = 0;
      if (lane == 0) g = atomicAdd(&tg_next[parity], 1u);
      return __builtin_amdgcn_readfirstlane((int)g);
    };
    // load stage: tuple group ltg, entries [lj, lj + kRsChunk) of each tuple;
    // ntg is the group after it, whose spans are in nst, nen
    int ltg = wave, ntg = n_tg;
    uint32_t lj = 0, lmax = 0, lst = 0, len = 0, nst = 0, nen = 0;
    if (ltg < n_tg) {
      spans_of(ltg, lst, len);
      lmax = wave_max(len - lst);
      ntg = grab();
    }
    spans_of(ntg, nst, nen);
    auto chunk_of_l = [&]() -> RsChunk {
      const uint32_t n = lmax > lj ? min((uint32_t)kRsChunk, lmax - lj) : 0u;
      return RsChunk{ltg, (n + 3u) & ~3u, lj + kRsChunk >= lmax};
    };
    // the next group's spans are reloaded on every step (cache hits), so that a
    // switch of group only moves values loaded a step earlier
    auto advance = [&]() {
      if (ltg < n_tg) {
        lj += kRsChunk;
        if (lj >= lmax) {
          ltg = ntg;
          lj = 0;
          lst = nst;
          len = nen;
          lmax = 0u;
          if (ltg < n_tg) {
            lmax = wave_max(len - lst);
            ntg = grab();
          }
        }
      }
      spans_of(ntg, nst, nen);
    };
    // Every load below is unconditional: the buffer range checks turn reads past
    // the batch's arrays into zeros, and entries past the end of a tuple are
    // marked in a wave mask and become (zero row, 0) when staged.
    const BufRes rs_dc = buf_res(dc, (uint32_t)bt.n_d);
    const BufRes rs_node = key_res(im.key + bt.code_base, (uint32_t)bt.n_codes);
    auto load_codes = [&](uint32_t &d0, uint32_t &d1, uint64_t &ok0, uint64_t &ok1) {
      const uint32_t j0 = lst + lj + (uint32_t)sub, j1 = j0 + 8u;
      const bool live = ltg < n_tg;
      ok0 = __ballot(live && j0 < len);
      ok1 = __ballot(live && j1 < len);
      d0 = buf_load(rs_dc, j0);
      d1 = buf_load(rs_dc, j1);
    };
    auto entry = [&](uint32_t d, uint2 key, uint64_t ok) -> uint2 {
      uint2 g;
      if (d < n1) {
        g = key;
      } else {
        g.x = kRtGlobal | (d - n1);
        g.y = __float_as_uint(1.0f);
      }
      if (!__builtin_amdgcn_inverse_ballot_w64(ok)) g = make_uint2(zrow, 0u);
      return g;
    };
    // an H row in LDS or in the workspace; both loads are issued and the values
    // selected (a select of the two pointers would make a flat pointer)
    auto row_f4 = [&](uint32_t r) -> float4 {
      const bool g = (r & kRtGlobal) != 0;
      const float4 xl = lds_load4(qb + (g ? zrow : r) * (kRtKT * 4));
      float4 xg = make_float4(0.f, 0.f, 0.f, 0.f);
      if (g) xg = *(const float4 *)&Hg[(int64_t)(r & ~kRtGlobal) * kRtKT + q];
      return g ? xg : xl;
    };
    // Pipeline: codes of chunk L load while chunk G's codes are translated and
    // chunk C, staged in LDS, is summed.  Two register sets alternate between the
    // roles of G and L, so no loaded value is ever copied.
    RsChunk G = chunk_of_l();
    RsChunk C{n_tg, 0u, false};
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    auto step = [&](uint32_t gd0, uint32_t gd1, uint64_t gok0, uint64_t gok1, uint32_t &ld0,
                    uint32_t &ld1, uint64_t &lok0, uint64_t &lok1) {
      advance();
      const uint2 key0 = key_load(rs_node, gd0), key1 = key_load(rs_node, gd1);
      const RsChunk L = chunk_of_l();
      load_codes(ld0, ld1, lok0, lok1);
      bool done = false;
      // blocked summation: a chunk's entries form a partial sum that then joins
      // the tuple's running sum (serial chains of at most kRsChunk terms, and of
      // the tuple's number of chunks)
      float4 part = make_float4(0.f, 0.f, 0.f, 0.f);
      if (C.tg < n_tg && C.steps == kRsChunk) {
        // a full chunk: all staged entries first, then the rows, so that many
        // LDS reads are in flight (rows in the workspace take the loop below)
        uint2 e[kRsChunk];
#pragma unroll
        for (int t = 0; t < kRsChunk; ++t) e[t] = stage[t * kRsGroups + grp];
        uint32_t any = 0;
#pragma unroll
        for (int t = 0; t < kRsChunk; ++t) any |= e[t].x;
        if (!(any & kRtGlobal)) {
          // rows in blocks of 8 reads issued back to back
#pragma unroll
          for (int h = 0; h < kRsChunk; h += 8) {
            float4 xr[8];
#pragma unroll
            for (int t = 0; t < 8; ++t)
              xr[t] = lds_load4(qb + e[h + t].x * (kRtKT * 4));
#pragma unroll
            for (int t = 0; t < 8; ++t) part = f4fma(__uint_as_float(e[h + t].y), xr[t], part);
            __builtin_amdgcn_sched_barrier(0);
          }
          done = true;
        }
      }
      if (C.tg < n_tg && !done) {
        for (uint32_t t = 0; t < C.steps; t += 4) {
          const uint2 e0 = stage[(t + 0) * kRsGroups + grp], e1 = stage[(t + 1) * kRsGroups + grp];
          const uint2 e2 = stage[(t + 2) * kRsGroups + grp], e3 = stage[(t + 3) * kRsGroups + grp];
          float4 x0, x1, x2, x3;
          if ((e0.x | e1.x | e2.x | e3.x) & kRtGlobal) {
            x0 = row_f4(e0.x);
            x1 = row_f4(e1.x);
            x2 = row_f4(e2.x);
            x3 = row_f4(e3.x);
          } else {
            x0 = lds_load4(qb + e0.x * (kRtKT * 4));
            x1 = lds_load4(qb + e1.x * (kRtKT * 4));
            x2 = lds_load4(qb + e2.x * (kRtKT * 4));
            x3 = lds_load4(qb + e3.x * (kRtKT * 4));
          }
          part = f4fma(__uint_as_float(e0.y), x0, part);
          part = f4fma(__uint_as_float(e1.y), x1, part);
          part = f4fma(__uint_as_float(e2.y), x2, part);
          part = f4fma(__uint_as_float(e3.y), x3, part);
        }
      }
      if (C.tg < n_tg) {
        acc.x += part.x;
        acc.y += part.y;
        acc.z += part.z;
        acc.w += part.w;
        if (C.last) {
          const int r = C.tg * kRsGroups + grp;
          if (r < nrows) {
            float *rr = R + (bt.row_base + r) * ldr + k0 + q;
            if (q + 3 < kt) {
              rr[0] = acc.x;
              rr[1] = acc.y;
              rr[2] = acc.z;
              rr[3] = acc.w;
            } else {
              if (q + 0 < kt) rr[0] = acc.x;
              if (q + 1 < kt) rr[1] = acc.y;
              if (q + 2 < kt) rr[2] = acc.z;
            }
          }
          acc = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      // entries of chunk G: entry t of tuple grp goes to stage[t * 8 + grp]
      stage[(sub + 0) * kRsGroups + grp] = entry(gd0, key0, gok0);
      stage[(sub + 8) * kRsGroups + grp] = entry(gd1, key1, gok1);
      __builtin_amdgcn_wave_barrier();
      C = G;
      G = L;
    };
    uint32_t dA0, dA1, dB0, dB1;
    uint64_t okA0, okA1, okB0, okB1;
    load_codes(dA0, dA1, okA0, okA1);
    while (G.tg < n_tg || C.tg < n_tg) {
      step(dA0, dA1, okA0, okA1, dB0, dB1, okB0, okB1);
      if (!(G.tg < n_tg || C.tg < n_tg)) break;
      step(dB0, dB1, okB0, okB1, dA0, dA1, okA0, okA1);
    }
  }
}

// ---------------------------------------------------------------------------
// Right multiplication with a compact W tile: the tile holds only the rows of W
// whose column is the key column of some code of the batch (an image-like batch
// uses about two thirds of its columns), so a tile of kRcKT = 64 columns fits in
// LDS and each lane of a 16-lane row holds 4 columns: one 16-byte LDS read and
// one row-address broadcast serve 4 FMAs.  Rows are 256 bytes, so the 16 lanes of
// a row read 64 distinct banks (rows of 240 bytes measured 44 % bank-conflict
// cycles).  Work items are (batch, 64-column tile) pairs, dealt per XCD as in
// right_tiled_kernel.  Per item:
//  * the batch's used columns come from the column index of the image (a column
//    is used when it has a depth-1 leaf or a tree code): a ballot scan gives each
//    its row, kept in an LDS map column -> row, and the rows are gathered from W.
//    This is pipelined one item ahead: the map of the next item is built (into a
//    second map) while the current item starts, from column-index words loaded
//    one item earlier still, and a wave that has no tuples left loads its share
//    of the next item's rows of W into registers before it waits for the others;
//  * the H rows of the deep codes (depth >= 2) are built level by level into
//    the worker's workspace slot (H[c] = H[parent] + val * W[col]);
//  * tuple sums as in right_tiled_kernel (16 lanes per tuple, entries loaded two
//    steps ahead, translated one step ahead, broadcast along the DPP row); an
//    entry of a deep code counts as the zero row in the LDS pass and its H row
//    is added from the workspace after the chunk's FMAs (deep entries are rare:
//    about one in two hundred on image-like batches).
// ---------------------------------------------------------------------------
constexpr int kRcKT = 64;                         // columns per tile: 16 lanes x 4
constexpr uint32_t kRcRowBytes = kRcKT * 4;       // 256
constexpr int kRcHgRow = 64;                      // floats per deep row in the workspace
constexpr int kRcPer = 2;                         // entries per lane and chunk
constexpr int kRcChunk = kRcPer * kRtLanes;       // 32 entries per tuple per step
constexpr uint32_t kRcNone = 0xFFFFFFFFu;
constexpr int kRcWv = 10;                         // float4 of W rows per thread held across the barrier

// LDS bytes of the compact kernel: rows 0 .. umax-1 (W), row umax (zeros), two
// maps (u16 per column), two used-column lists (u16 per row) and 16 wave totals.
inline size_t rc_lds_bytes(int64_t umax, int64_t m) {
  const size_t rows = (size_t)(umax + 1) * kRcRowBytes;
  return rows + (size_t)4 * m + (size_t)4 * umax + 64 + 16;
}

__global__ __launch_bounds__(kRtBlock) void right_compact_kernel(
    Img im, const uint32_t *__restrict__ cols_all, int64_t nb, int n_tiles, int spw, int m,
    int cap, const float *__restrict__ W, int64_t ldw, int k, float *__restrict__ R, int64_t ldr,
    float *__restrict__ ws, int64_t slot_floats) {
  extern __shared__ float4 smem4[];
  char *lds = (char *)smem4;
  __shared__ uint32_t tg_next[2];
  const int x = (int)(blockIdx.x % kXcd), s = (int)(blockIdx.x / kXcd);
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const int grp = lane / kRtLanes, sub = lane % kRtLanes, q = 4 * sub;
  float *Wt = (float *)lds;                                       // rows of 64 floats
  const uint32_t wb = lds_base(smem4);
  const uint32_t qoff = 16u * (uint32_t)sub;
  const uint32_t zrow_b = wb + (uint32_t)cap * kRcRowBytes;
  uint16_t *maps = (uint16_t *)(lds + (size_t)(cap + 1) * kRcRowBytes);   // two maps of m
  uint16_t *ucols = maps + 2 * m;                                         // two lists of cap
  uint32_t *wsum = (uint32_t *)(((uintptr_t)(ucols + 2 * cap) + 3) & ~(uintptr_t)3);
  float *Hg = ws + blockIdx.x * slot_floats;
  // the zero row
  for (int e = threadIdx.x; e < kRcKT; e += kRtBlock) Wt[cap * kRcKT + e] = 0.0f;
  if (threadIdx.x < 2) tg_next[threadIdx.x] = kRtWaves;
  const int64_t nbx = nb > x ? (nb - x + kXcd - 1) / kXcd : 0;
  const int64_t n_items = nbx * n_tiles;
  auto batch_of = [&](int64_t it) -> int64_t { return uniform64(x + kXcd * (it / n_tiles)); };
  auto tile_of = [&](int64_t it) -> int {
    return __builtin_amdgcn_readfirstlane((int)(it % n_tiles)) * kRcKT;
  };
  // column-index words of column j = threadIdx.x of batch b (leaf positions and
  // tree-list entries of columns j and j + 1), loaded ahead of the map build
  auto load_cols = [&](int64_t b, uint32_t (&cw)[4]) {
    const uint32_t *Loff = cols_all + b * 4 * (int64_t)(m + 1);
    const uint32_t *Toff = Loff + 2 * (m + 1);
    const int j = (int)threadIdx.x;
    cw[0] = cw[1] = cw[2] = cw[3] = 0u;
    if (j < m) {
      cw[0] = Loff[j];
      cw[1] = Loff[j + 1];
      cw[2] = Toff[j];
      cw[3] = Toff[j + 1];
    }
  };
  // used columns: column j is used when it has a depth-1 leaf or a tree code; its
  // row is the number of used columns before it (at most cap: the host sized cap
  // for the batch with the most).  Columns from kRtBlock on (wide matrices) are
  // loaded here.  Returns the number of rows; the map and the list are complete
  // for every thread on return.
  auto build_map = [&](int64_t b, const uint32_t (&cw)[4], uint16_t *map, uint16_t *ucol) -> uint32_t {
    const uint32_t *Loff = cols_all + b * 4 * (int64_t)(m + 1);
    const uint32_t *Toff = Loff + 2 * (m + 1);
    uint32_t base = 0;
    for (int j0 = 0; j0 < m; j0 += kRtBlock) {
      const int j = j0 + (int)threadIdx.x;
      bool used;
      if (j0 == 0) {
        used = cw[1] > cw[0] || cw[3] > cw[2];
      } else {
        used = j < m && (Loff[j + 1] > Loff[j] || Toff[j + 1] > Toff[j]);
      }
      const uint64_t bal = __ballot(used);
      const uint32_t below = (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) wsum[wave] = (uint32_t)__popcll(bal);
      __syncthreads();
      uint32_t before = base, total = base;
#pragma unroll
      for (int w = 0; w < kRtWaves; ++w) {
        const uint32_t t = wsum[w];
        before += w < wave ? t : 0u;
        total += t;
      }
      const uint32_t row = before + below;
      if (used && row < (uint32_t)cap) {
        map[j] = (uint16_t)row;
        ucol[row] = (uint16_t)j;
      }
      base = total;
      __syncthreads();
    }
    return min(base, (uint32_t)cap);
  };
  // this thread's share of the item's rows of W (float4 e = threadIdx.x + i *
  // kRtBlock of the U rows of 16 float4); columns past kt are zeros
  auto w_at = [&](uint32_t e, int k0, int kt, bool vec, const uint16_t *ucol) -> float4 {
    const uint32_t r = e / (kRcKT / 4), q4 = 4 * (e % (kRcKT / 4));
    const float *src = W + (int64_t)ucol[r] * ldw + k0 + q4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (vec) {
      v = *(const float4 *)src;
    } else {
      if ((int)q4 + 0 < kt) v.x = src[0];
      if ((int)q4 + 1 < kt) v.y = src[1];
      if ((int)q4 + 2 < kt) v.z = src[2];
      if ((int)q4 + 3 < kt) v.w = src[3];
    }
    return v;
  };
  auto is_vec = [&](int k0, int kt) {
    return kt == kRcKT && (ldw % 4) == 0 && (((uintptr_t)(W + k0)) & 15u) == 0;
  };
  auto load_w = [&](uint32_t U, int k0, const uint16_t *ucol, float4 (&wv)[kRcWv]) {
    const int kt = min(kRcKT, k - k0);
    const bool vec = is_vec(k0, kt);
    const uint32_t n4 = U * (kRcKT / 4);
#pragma unroll
    for (int i = 0; i < kRcWv; ++i) {
      const uint32_t e = threadIdx.x + (uint32_t)(i * kRtBlock);
      wv[i] = e < n4 ? w_at(e, k0, kt, vec, ucol) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  // the held share into the tile, and rows past kRcWv * kRtBlock float4 (more
  // than 640 used columns) straight from W
  auto store_w = [&](uint32_t U, int k0, const uint16_t *ucol, const float4 (&wv)[kRcWv]) {
    const uint32_t n4 = U * (kRcKT / 4);
#pragma unroll
    for (int i = 0; i < kRcWv; ++i) {
      const uint32_t e = threadIdx.x + (uint32_t)(i * kRtBlock);
      if (e < n4) *(float4 *)&Wt[e * 4] = wv[i];
    }
    const int kt = min(kRcKT, k - k0);
    const bool vec = is_vec(k0, kt);
    for (uint32_t e = threadIdx.x + (uint32_t)(kRcWv * kRtBlock); e < n4; e += kRtBlock)
      *(float4 *)&Wt[e * 4] = w_at(e, k0, kt, vec, ucol);
  };
  // the first item's map and rows, and the column-index words of the second
  uint32_t cw[4];
  float4 wv[kRcWv];
  uint32_t U = 0;
  if (s < n_items) {
    load_cols(batch_of(s), cw);
    U = build_map(batch_of(s), cw, maps, ucols);
    if (s + spw < n_items) load_cols(batch_of(s + spw), cw);
    load_w(U, tile_of(s), ucols, wv);
  }
  uint32_t parity = 0;
  for (int64_t it = s; it < n_items; it += spw, parity ^= 1u) {
    const int64_t b = batch_of(it);
    const int k0 = tile_of(it);
    const int kt = min(kRcKT, k - k0);
    const toc_batch bt = uniform_batch(im.batches + b);
    const uint32_t n1 = (uint32_t)bt.n_lvl1;
    const int nrows = bt.n_rows;
    const uint16_t *map = maps + parity * (uint32_t)m;
    __syncthreads();   // the previous item no longer reads the tile, the other map or counters
    if (threadIdx.x == 0) tg_next[parity ^ 1u] = kRtWaves;
    store_w(U, k0, ucols + parity * (uint32_t)cap, wv);
    // the next item's map (its barriers also publish the tile), then the
    // column-index words of the item after it
    const int64_t itn = it + spw;
    uint32_t U_next = 0;
    if (itn < n_items) {
      U_next = build_map(batch_of(itn), cw, maps + (parity ^ 1u) * (uint32_t)m,
                         ucols + (parity ^ 1u) * (uint32_t)cap);
      if (itn + spw < n_items) load_cols(batch_of(itn + spw), cw);
    } else {
      __syncthreads();
    }
    // H rows of the deep codes into the workspace slot, level by level: a 16-lane
    // row per code (4 columns per lane)
    {
      const uint32_t *lvl = im.level + bt.lvl_base;
      const toc_key *key = im.key + bt.code_base;
      const toc_link *link = deep_links(im.link, bt);
      const uint32_t g16 = threadIdx.x / kRtLanes;
      constexpr uint32_t stride = kRtBlock / kRtLanes;
      for (int d = 2; d <= bt.n_levels; ++d) {
        const uint32_t a = lvl[d - 1], e = lvl[d];
        for (uint32_t c = a + g16; c < e; c += stride) {
          const uint32_t p = link[c].parent;
          const uint2 kc = *(const uint2 *)(key + c);
          const float4 wc = *(const float4 *)&Wt[map[kc.x] * kRcKT + q];
          float4 base;
          if (p < n1) {
            const uint2 kp = *(const uint2 *)(key + p);
            const float vp = __uint_as_float(kp.y);
            const float4 wp = *(const float4 *)&Wt[map[kp.x] * kRcKT + q];
            base = make_float4(vp * wp.x, vp * wp.y, vp * wp.z, vp * wp.w);
          } else {
            base = *(const float4 *)&Hg[(int64_t)(p - n1) * kRcHgRow + q];
          }
          *(float4 *)&Hg[(int64_t)(c - n1) * kRcHgRow + q] = f4fma(__uint_as_float(kc.y), wc, base);
        }
        __syncthreads();
      }
    }
    // per-tuple sums
    const int n_tg = (nrows + kRtGroups - 1) / kRtGroups;
    const uint32_t *span = im.span + bt.span_base;
    auto spans_of = [&](int tg, uint32_t &st, uint32_t &en) {
      const int r = min(tg * kRtGroups + grp, nrows);
      st = span[r];
      en = span[min(r + 1, nrows)];
    };
    auto wave_max = [&](uint32_t v) -> uint32_t {
      v = max(v, (uint32_t)__shfl_xor((int)v, 16, kWave));
      v = max(v, (uint32_t)__shfl_xor((int)v, 32, kWave));
      return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
    };
    auto grab = [&]() -> int {
      uint32_t g = 0;
      if (lane == 0) g = atomicAdd(&tg_next[parity], 1u);
      return __builtin_amdgcn_readfirstlane((int)g);
    };
    int ltg = wave, ntg = n_tg;
    uint32_t lj = 0, lmax = 0, lst = 0, len = 0, nst = 0, nen = 0;
    if (ltg < n_tg) {
      spans_of(ltg, lst, len);
      lmax = wave_max(len - lst);
      ntg = grab();
    }
    spans_of(ntg, nst, nen);
    auto chunk_of_l = [&]() -> RtChunk {
      const uint32_t n = lmax > lj ? min((uint32_t)kRcChunk, lmax - lj) : 0u;
      return RtChunk{ltg, (n + 3u) & ~3u, lj + kRcChunk >= lmax};
    };
    auto advance = [&]() {
      if (ltg < n_tg) {
        lj += kRcChunk;
        if (lj >= lmax) {
          ltg = ntg;
          lj = 0;
          lst = nst;
          len = nen;
          lmax = 0u;
          if (ltg < n_tg) {
            lmax = wave_max(len - lst);
            ntg = grab();
          }
          spans_of(ntg, nst, nen);
        }
      }
    };
    const BufRes rs_dc = buf_res(im.dcodes + bt.d_base, (uint32_t)bt.n_d);
    const BufRes rs_node = key_res(im.key + bt.code_base, (uint32_t)bt.n_codes);
    auto load_codes = [&](uint32_t (&d)[kRcPer], uint64_t (&ok)[kRcPer]) {
      const bool live = ltg < n_tg;
      static_for<kRcPer>([&](auto hc) {
        constexpr int h = decltype(hc)::value;
        const uint32_t j = lst + lj + (uint32_t)sub + (uint32_t)(h * kRtLanes);
        ok[h] = __ballot(live && j < len);
        d[h] = buf_load(rs_dc, j);
      });
    };
    // (LDS row address, multiplier, deep row) of an entry: a depth-1 code's row is
    // its column's row of the tile times its value; a deep code and an entry past
    // the end of its tuple take the zero row (the deep code's H row is added
    // after the chunk)
    auto translate = [&](uint32_t d, uint2 key, uint64_t ok, uint32_t &rb, uint32_t &mu,
                         uint32_t &dp) {
      const bool in = __builtin_amdgcn_inverse_ballot_w64(ok);
      const uint32_t row = map[min(key.x, (uint32_t)m - 1u)];
      const bool leaf = in && d < n1;
      rb = leaf ? wb + row * kRcRowBytes : zrow_b;
      mu = leaf ? key.y : 0u;
      dp = (in && d >= n1) ? d - n1 : kRcNone;
    };
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    RtChunk G = chunk_of_l();
    RtChunk C{n_tg, 0u, false};
    uint32_t crb[kRcPer], cmu[kRcPer], cdp[kRcPer];
#pragma unroll
    for (int h = 0; h < kRcPer; ++h) {
      crb[h] = zrow_b;
      cmu[h] = 0u;
      cdp[h] = kRcNone;
    }
    auto step = [&](const uint32_t (&gd)[kRcPer], const uint64_t (&gok)[kRcPer],
                    uint32_t (&ld)[kRcPer], uint64_t (&lok)[kRcPer]) {
      advance();
      uint2 key[kRcPer];
      static_for<kRcPer>([&](auto hc) {
        constexpr int h = decltype(hc)::value;
        key[h] = key_load(rs_node, gd[h]);
      });
      const RtChunk L = chunk_of_l();
      load_codes(ld, lok);
      if (C.tg < n_tg) {
        // blocked summation: the chunk's terms form a partial sum that then joins
        // the tuple's running sum
        float4 part = make_float4(0.f, 0.f, 0.f, 0.f);
        constexpr int NB = kRcChunk / 4;       // blocks of 4 entries
        if (C.steps == (uint32_t)kRcChunk) {
          // each block's reads are issued before the previous block's FMAs
          float4 xa[4], xb[4];
          load4x4_bcast<0>(crb[0], qoff, xa);
          static_for<NB>([&](auto bc) {
            constexpr int bk = decltype(bc)::value;
            if constexpr (bk + 1 < NB) {
              constexpr int nx = bk + 1;
              if constexpr (bk % 2 == 0) load4x4_bcast<4 * (nx % 4)>(crb[nx / 4], qoff, xb);
              else load4x4_bcast<4 * (nx % 4)>(crb[nx / 4], qoff, xa);
            }
            if constexpr (bk % 2 == 0) fma4x4_bcast<4 * (bk % 4)>(part, cmu[bk / 4], xa);
            else fma4x4_bcast<4 * (bk % 4)>(part, cmu[bk / 4], xb);
          });
        } else {
          static_for<NB>([&](auto bc) {
            constexpr int bk = decltype(bc)::value;
            if (C.steps > (uint32_t)(4 * bk)) {
              float4 xv[4];
              load4x4_bcast<4 * (bk % 4)>(crb[bk / 4], qoff, xv);
              fma4x4_bcast<4 * (bk % 4)>(part, cmu[bk / 4], xv);
            }
          });
        }
        // deep entries of the chunk: the H rows from the workspace, each row of
        // lanes taking the entry of its own tuple at each lane position t that
        // holds a deep entry in some tuple
#pragma unroll
        for (int h = 0; h < kRcPer; ++h) {
          const uint64_t dm = __ballot(cdp[h] != kRcNone);
          uint32_t pos = (uint32_t)((dm | (dm >> 16) | (dm >> 32) | (dm >> 48)) & 0xFFFFu);
          while (pos) {
            const int t = __builtin_ctz(pos);
            pos &= pos - 1u;
            const uint32_t r = (uint32_t)__shfl((int)cdp[h], grp * kRtLanes + t, kWave);
            if (r != kRcNone) add4(part, *(const float4 *)&Hg[(int64_t)r * kRcHgRow + q]);
          }
        }
        add4(acc, part);
        if (C.last) {
          const int r = C.tg * kRtGroups + grp;
          if (r < nrows) {
            float *rr = R + (bt.row_base + r) * ldr + k0 + q;
            if (q + 3 < kt) {
              rr[0] = acc.x;
              rr[1] = acc.y;
              rr[2] = acc.z;
              rr[3] = acc.w;
            } else {
              if (q + 0 < kt) rr[0] = acc.x;
              if (q + 1 < kt) rr[1] = acc.y;
              if (q + 2 < kt) rr[2] = acc.z;
            }
          }
          acc = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      // chunk G becomes chunk C
      static_for<kRcPer>([&](auto hc) {
        constexpr int h = decltype(hc)::value;
        translate(gd[h], key[h], gok[h], crb[h], cmu[h], cdp[h]);
      });
      C = G;
      G = L;
    };
    uint32_t dA[kRcPer], dB[kRcPer];
    uint64_t okA[kRcPer], okB[kRcPer];
    load_codes(dA, okA);
    while (G.tg < n_tg || C.tg < n_tg) {
      step(dA, okA, dB, okB);
      if (!(G.tg < n_tg || C.tg < n_tg)) break;
      step(dB, okB, dA, okA);
    }
    // no tuples left for this wave: its share of the next item's rows of W, held
    // until every wave is done with the tile
    // (none after the last item: U_next is 0 there)
    load_w(U_next, tile_of(itn), ucols + (parity ^ 1u) * (uint32_t)cap, wv);
    U = U_next;
  }
}

// ---------------------------------------------------------------------------
// Left multiplication by pulling (Theorem 2 read as a definition, Algorithm 8's
// result): H(x) is the sum of the G rows over the entries of D equal to x (the
// image lists each tree code's tuples after the column entries, where occ_off
// points) plus the H of x's children, and output row j is the sum of
// val(x) * H(x) over the codes x of key column j.  Work items are (batch,
// TW-column tile) pairs dealt per XCD as in the right product.  A worker loads the
// batch's G tile into LDS (row nrows_max is all zeros), then
//  * tree codes (codes with children or of depth >= 2), deepest level first, a
//    lane group per code: H = own occurrences + children's H (children of a code
//    are contiguous, levels being sorted by parent); H rows follow the G tile in
//    LDS, or go to the worker's workspace slot when they do not fit;
//  * output columns: a group of TW/4 lanes owns one column j (a lane holds 4 of
//    the tile's columns) and sums val * row over its entries: the occurrences of
//    the column's leaf codes (depth-1 codes without children, whose left
//    positions are ordered by column, so one contiguous stretch of the entry
//    array) and then its tree codes (a stretch after all leaf occurrences), the
//    multiplier loaded beside each entry.  Entries are loaded two chunks ahead
//    and translated to (LDS row, multiplier) one chunk ahead; a group of 16
//    lanes takes them from the lane that translated them by DPP row broadcast,
//    a group of 8 from a per-wave stage in LDS.  Groups of columns are handed
//    out from an LDS counter.
// ---------------------------------------------------------------------------
constexpr int kLtBlock = 1024;
constexpr int kLtWaves = kLtBlock / kWave;
constexpr uint32_t kFirstOcc = 0x80000000u;
constexpr uint32_t kLtStaticBytes = 16;           // static LDS: two column-group counters
constexpr int kLtU = 4;                           // tree codes per group at a time
constexpr uint32_t kLtBlk = 16;                   // children per block of a tree code's sum

// LDS bytes of the per-wave stages and of the column tables
// (groups of 16 lanes pass entries round with the DPP row broadcast: no stage)
template <int TW>
constexpr uint32_t lt_stage_bytes() {
  return TW / 4 == kRtLanes ? 0u : (uint32_t)kLtWaves * (TW / 4) * (kWave / (TW / 4)) * 8;
}

// LDS byte offset of the rows: stages, then the batch's column index (Loff, Ost,
// Toff, Ord: m + 1 entries each, as in the image), the children offsets Coff of
// the tree rows and, when toc is set, their occurrence offsets Toc (max_tree + 1
// each) and ocr words for the tree rows' occurrences themselves
template <int TW>
constexpr uint32_t lt_rows_offset(int64_t m, int64_t max_tree, bool toc, int64_t ocr) {
  return (uint32_t)((lt_stage_bytes<TW>() +
                     4 * (4 * (m + 1) + (toc ? 2 : 1) * (max_tree + 1) + (toc ? ocr : 0)) + 15) &
                    ~(int64_t)15);
}
constexpr int kLtOcr = 1024;   // LDS words for a batch's tree-row occurrences
constexpr int kLtCopy = 4;     // children (and occurrence) offsets per thread in flight

struct LtChunk {
  int cg;           // column group (columns GPW*cg .. GPW*cg+GPW-1); >= n_cg: none
  uint32_t steps;   // entries per column to process, rounded up to a multiple of 4
  uint32_t first;   // first entry of the chunk (0: a column starts)
  bool last;        // last chunk of the column group
  bool tree;        // the chunk holds tree entries
};

template <int TW, bool TREE_LDS>
__global__ __launch_bounds__(kLtBlock) void left_tiled_kernel(
    Img im, const uint32_t *__restrict__ occ_off_all, const uint32_t *__restrict__ tlist_all, const uint32_t *__restrict__ cols_all,
    const uint32_t *__restrict__ tchild_all, int64_t nb, int n_tiles, int spw, int max_rows,
    int max_tree, int tree_cap, int toc_lds, int ocr_cap, int m, const float *__restrict__ G,
    int64_t ldg, int k,
    float *__restrict__ out, int64_t ldo, int accumulate, float *__restrict__ ws,
    int64_t slot_floats) {
  // TREE_LDS: every tree row is in LDS; else the first tree_cap are and the others
  // are in the worker's workspace slot
  constexpr int LPG = TW / 4;                 // lanes per group (4 columns each)
  constexpr int GPW = kWave / LPG;            // groups (output columns) per wave
  constexpr int CH = LPG;                     // entries per column per chunk: one per lane
  constexpr uint32_t RB = TW * 4;             // bytes of an LDS row
  extern __shared__ float4 smem4[];
  __shared__ uint32_t cg_next[2];
  char *lds = (char *)smem4;
  const int x = (int)(blockIdx.x % kXcd), s = (int)(blockIdx.x / kXcd);
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const int grp = lane / LPG, sub = lane % LPG, q = 4 * sub;
  // LDS: stages | Loff, Ost, Toff, Ord (m + 1 each) | Coff (max_tree + 1) | rows
  uint2 *stage = (uint2 *)lds + wave * (CH * GPW);
  uint32_t *Loff = (uint32_t *)(lds + lt_stage_bytes<TW>());
  uint32_t *Ost = Loff + (m + 1);
  uint32_t *Toff = Ost + (m + 1);
  uint32_t *Ord = Toff + (m + 1);             // columns by decreasing number of entries
  uint32_t *Coff = Ord + (m + 1);
  uint32_t *Toc = Coff + (max_tree + 1);     // (toc_lds only)
  uint32_t *Ocr = Toc + (max_tree + 1);      // (toc_lds only: ocr_cap words)
  const uint32_t rows_b = lt_rows_offset<TW>(m, max_tree, toc_lds != 0, ocr_cap);
  float *Rw = (float *)(lds + rows_b);        // G rows, zero row, then tree rows
  const uint32_t qb = lds_base(smem4) + rows_b + 4u * (uint32_t)q;   // LDS address of this lane's columns
  constexpr bool DPP = LPG == kRtLanes;       // a group is one 16-lane row: entries by broadcast
  constexpr int PER = DPP ? 2 : 1;            // entries per lane and chunk (16-lane groups: 2,
                                              // 3 % faster on dense quantised batches)
  constexpr int CHK = PER * LPG;              // entries per column per chunk
  const uint32_t rb0 = lds_base(smem4) + rows_b;                      // LDS address of row 0
  const uint32_t qoff = 4u * (uint32_t)q;
  const uint32_t zrow = (uint32_t)max_rows;
  const uint32_t trow0 = zrow + 1u;
  float *Hg = ws + blockIdx.x * slot_floats;
  for (int e = threadIdx.x; e < TW; e += kLtBlock) Rw[zrow * TW + e] = 0.0f;
  if (threadIdx.x < 2) cg_next[threadIdx.x] = kLtWaves;
  const int64_t nbx = nb > x ? (nb - x + kXcd - 1) / kXcd : 0;
  const int64_t n_items = nbx * n_tiles;
  auto item_batch = [&](int64_t it) -> int64_t { return uniform64(x + kXcd * (it / n_tiles)); };
  auto item_k0 = [&](int64_t it) -> int {
    return __builtin_amdgcn_readfirstlane((int)(it % n_tiles)) * TW;
  };
  uint32_t parity = 0;
  for (int64_t it = s; it < n_items; it += spw, parity ^= 1u) {
    const int64_t b = item_batch(it);
    const int k0 = item_k0(it);
    const int kt = min(TW, k - k0);
    const toc_batch bt = uniform_batch(im.batches + b);
    const uint32_t *lvl = im.level + bt.lvl_base;
    const uint32_t nc = (uint32_t)bt.n_codes, n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1;
    // tree row h's occurrences: entries to[h] .. to[h+1]-1 of the batch's entry array
    // (copied to Toc in LDS when toc_lds is set)
    const uint32_t *to = occ_off_all + bt.code_base + 2 * b + (n1 - ni) + 1;
    auto occ_at = [&](uint32_t h) -> uint32_t {
      if (toc_lds) return Toc[h];
      return to[h];
    };
    const uint32_t *orow = im.centry + bt.d_base + bt.tree_base;
    const uint32_t n_tree = ni + (nc - n1);
    const int nrows = bt.n_rows;
    auto hrow = [&](uint32_t c) -> uint32_t { return c < ni ? c : c - n1 + ni; };
    // the tree rows' occurrences are the last entries of the batch's entry array,
    // from to[0]; they are copied to LDS when they fit in ocr_cap words
    const uint32_t p3 = toc_lds && ocr_cap ? (uint32_t)__builtin_amdgcn_readfirstlane((int)to[0]) : 0u;
    const uint32_t n_p3 = (uint32_t)bt.n_d + n_tree - p3;
    const bool use_ocr = toc_lds && ocr_cap && n_p3 <= (uint32_t)ocr_cap;
    auto occ_row = [&](uint32_t o) -> uint32_t {
      if (use_ocr) return Ocr[o - p3];
      return orow[o];
    };
    __syncthreads();   // the previous item no longer reads the LDS rows and tables
    if (threadIdx.x == 0) cg_next[parity ^ 1u] = kLtWaves;
    // the first pass of the column index and of the tree rows' occurrences is
    // loaded before the G tile and stored after it
    const uint4 *csrc = (const uint4 *)(cols_all + b * 4 * (int64_t)(m + 1));
    const uint32_t *tch = tchild_all + bt.tree_base + b;
    const uint4 cx0 = threadIdx.x < m + 1 ? csrc[threadIdx.x] : make_uint4(0u, 0u, 0u, 0u);
    const uint32_t oc0 = use_ocr && threadIdx.x < n_p3 ? orow[p3 + threadIdx.x] : 0u;
    // G tile: all loads of a pass first, then the stores
    {
      const int n4 = nrows * (TW / 4);
      const bool vec = kt == TW && (ldg % 4) == 0 && (k0 % 4) == 0 &&
                       ((((uintptr_t)G) & 15u) == 0);
      for (int e0 = threadIdx.x; e0 < n4; e0 += 8 * kLtBlock) {
        float4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i * kLtBlock;
          v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
          if (e < n4) {
            const int r = e / (TW / 4), q4 = 4 * (e % (TW / 4));
            const float *src = G + (bt.row_base + r) * ldg + k0 + q4;
            if (vec) {
              v[i] = *(const float4 *)src;
            } else {
              if (q4 + 0 < kt) v[i].x = src[0];
              if (q4 + 1 < kt) v[i].y = src[1];
              if (q4 + 2 < kt) v[i].z = src[2];
              if (q4 + 3 < kt) v[i].w = src[3];
            }
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i * kLtBlock;
          if (e < n4) *(float4 *)&Rw[e * 4] = v[i];
        }
      }
    }
    // the batch's column index, children ranges and (when they fit) occurrence
    // offsets, from the image
    {
      if (threadIdx.x < m + 1) ((uint4 *)Loff)[threadIdx.x] = cx0;
      for (int e = threadIdx.x + kLtBlock; e < m + 1; e += kLtBlock) ((uint4 *)Loff)[e] = csrc[e];
      // (a thread's loads of a pass, up to kLtCopy of each table, before its stores)
      for (uint32_t h0 = threadIdx.x; h0 <= n_tree; h0 += kLtCopy * kLtBlock) {
        uint32_t ct[kLtCopy], ot[kLtCopy];
#pragma unroll
        for (int q = 0; q < kLtCopy; ++q) {
          const uint32_t h = h0 + (uint32_t)(q * kLtBlock);
          ct[q] = h <= n_tree ? tch[h] : 0u;
          ot[q] = toc_lds && h <= n_tree ? to[h] : 0u;
        }
#pragma unroll
        for (int q = 0; q < kLtCopy; ++q) {
          const uint32_t h = h0 + (uint32_t)(q * kLtBlock);
          if (h <= n_tree) {
            Coff[h] = ct[q];
            if (toc_lds) Toc[h] = ot[q];
          }
        }
      }
      if (use_ocr) {
        if (threadIdx.x < n_p3) Ocr[threadIdx.x] = oc0;
        for (uint32_t t = threadIdx.x + kLtBlock; t < n_p3; t += kLtBlock) Ocr[t] = orow[p3 + t];
      }
    }
    __syncthreads();
    // Tree codes, deepest level first: H = own occurrences' G rows + children's
    // H rows.  A group takes kLtU codes at a time and issues their loads
    // together; a code's occurrence rows are broadcast along its group.
    // a tree row: in LDS (the first tree_cap) or in the workspace; both loads are
    // issued and the values selected (a select of the two pointers would make a
    // flat pointer)
    const uint32_t cap = TREE_LDS ? 0xFFFFFFFFu : (uint32_t)tree_cap;
    auto load_trow = [&](uint32_t h) -> float4 {
      const bool inl = h < cap;
      const float4 xl = lds_load4(qb + (inl ? trow0 + h : zrow) * RB);
      if (TREE_LDS) return xl;
      float4 xg = make_float4(0.f, 0.f, 0.f, 0.f);
      if (!inl) xg = *(const float4 *)&Hg[(int64_t)h * TW + q];
      return inl ? xl : xg;
    };
    auto store_trow = [&](uint32_t h, float4 v) {
      if (h < cap) *(float4 *)&Rw[(size_t)(trow0 + h) * TW + q] = v;
      else *(float4 *)&Hg[(int64_t)h * TW + q] = v;
    };
    // value v of lane i of the caller's group
    auto gbcast = [&](uint32_t v, auto ic) -> uint32_t {
      constexpr int i = decltype(ic)::value;
      if constexpr (LPG == kRtLanes) return row_bcast<i>(v);
      else return (uint32_t)__shfl((int)v, grp * LPG + i, kWave);
    };
    const int gidx = wave * GPW + grp;
    constexpr uint32_t NG = kLtWaves * GPW;
    for (int d = bt.n_levels; d >= 1; --d) {
      const uint32_t a = d == 1 ? 0u : lvl[d - 1], e = d == 1 ? ni : lvl[d];
      for (uint32_t c0 = a + gidx; c0 < e; c0 += kLtU * NG) {
        uint32_t h[kLtU], o0[kLtU], o1[kLtU], k0[kLtU], k1[kLtU], mine[kLtU];
        uint32_t nmax = 0, cmax = 0;
#pragma unroll
        for (int u = 0; u < kLtU; ++u) {
          const uint32_t c = c0 + u * NG;
          const bool in = c < e;
          const uint32_t cc = in ? c : c0;
          h[u] = hrow(cc);
          o0[u] = occ_at(h[u]);
          o1[u] = in ? occ_at(h[u] + 1) : o0[u];
          k0[u] = Coff[h[u]];
          k1[u] = in ? Coff[h[u] + 1] : k0[u];
        }
#pragma unroll
        for (int u = 0; u < kLtU; ++u) {
          mine[u] = o0[u] + sub < o1[u] ? occ_row(o0[u] + sub) & ~kFirstOcc : zrow;
          nmax = max(nmax, min(o1[u] - o0[u], (uint32_t)LPG));
          cmax = max(cmax, k1[u] - k0[u]);
        }
        nmax = wave_max_u32(nmax);
        cmax = wave_max_u32(cmax);
        // blocked summation: children and occurrences are summed in blocks of at
        // most kLtBlk (children) or LPG (occurrences) terms, each block's partial
        // sum then joining the code's running sum
        float4 acc[kLtU], part[kLtU];
#pragma unroll
        for (int u = 0; u < kLtU; ++u) acc[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        // children: one per code at a time, all codes' loads in flight
        for (uint32_t cb0 = 0; cb0 < cmax; cb0 += kLtBlk) {
          const uint32_t ce = min(cmax, cb0 + kLtBlk);
#pragma unroll
          for (int u = 0; u < kLtU; ++u) part[u] = make_float4(0.f, 0.f, 0.f, 0.f);
          for (uint32_t cb = cb0; cb < ce; ++cb) {
            float4 g[kLtU];
#pragma unroll
            for (int u = 0; u < kLtU; ++u) {
              g[u] = make_float4(0.f, 0.f, 0.f, 0.f);
              if (k0[u] + cb < k1[u]) g[u] = load_trow(hrow(k0[u] + cb));
            }
#pragma unroll
            for (int u = 0; u < kLtU; ++u) add4(part[u], g[u]);
          }
#pragma unroll
          for (int u = 0; u < kLtU; ++u) add4(acc[u], part[u]);
        }
        // occurrences: the first LPG of each code by broadcast
#pragma unroll
        for (int u = 0; u < kLtU; ++u) part[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        static_for<LPG>([&](auto ic) {
          if (nmax > (uint32_t)decltype(ic)::value) {
            float4 g[kLtU];
#pragma unroll
            for (int u = 0; u < kLtU; ++u) g[u] = lds_load4(qb + gbcast(mine[u], ic) * RB);
#pragma unroll
            for (int u = 0; u < kLtU; ++u) add4(part[u], g[u]);
          }
        });
#pragma unroll
        for (int u = 0; u < kLtU; ++u) {
          add4(acc[u], part[u]);
          // occurrences past the first LPG (rare): one at a time
          for (uint32_t ob = o0[u] + LPG; ob < o1[u]; ob += LPG) {
            const uint32_t mo = ob + sub < o1[u] ? occ_row(ob + sub) & ~kFirstOcc : zrow;
            const uint32_t n = min((uint32_t)LPG, o1[u] - ob);
            float4 pb = make_float4(0.f, 0.f, 0.f, 0.f);
            for (uint32_t i = 0; i < n; ++i) {
              const uint32_t r = (uint32_t)__shfl((int)mo, grp * LPG + (int)i, kWave);
              add4(pb, lds_load4(qb + r * RB));
            }
            add4(acc[u], pb);
          }
          if (c0 + u * NG < e) store_trow(h[u], acc[u]);
        }
      }
      __syncthreads();
    }
    // output columns.  The image orders a batch's columns by entries, most
    // first, so its n_ucols columns with entries come first: column groups cover
    // only those, and the output rows of the others are zero (written here once).
    const int n_used = bt.n_ucols;
    const int n_cg = (n_used + GPW - 1) / GPW;
    if (!accumulate) {
      const int n4 = (m - n_used) * (TW / 4);
      for (int e = threadIdx.x; e < n4; e += kLtBlock) {
        const int j = (int)Ord[n_used + e / (TW / 4)], q4 = 4 * (e % (TW / 4));
        float *o = out + (b * m + j) * ldo + k0 + q4;
        if (q4 + 3 < kt) {
          o[0] = 0.0f;
          o[1] = 0.0f;
          o[2] = 0.0f;
          o[3] = 0.0f;
        } else {
          for (int i = 0; i < kt - q4; ++i) o[i] = 0.0f;
        }
      }
    }
    auto grab = [&]() -> int {
      uint32_t g = 0;
      if (lane == 0) g = atomicAdd(&cg_next[parity], 1u);
      return __builtin_amdgcn_readfirstlane((int)g);
    };
    auto wave_max = [&](uint32_t v) -> uint32_t {
#pragma unroll
      for (int o = LPG; o < kWave; o <<= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, kWave));
      return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
    };
    // column j of group g of column group cg; past the last column: no entries.
    // Its entries (leaf occurrences, then tree codes) start at cst in centry.
    // Its leaf occurrences start at lst in centry, its tree codes at tst (after all
    // the batch's leaf occurrences).
    struct ColSpan { uint32_t lst, tst, nl, nt; };
    const uint32_t n_lo = Ost[m];
    auto col_of = [&](int cg) -> ColSpan {
      const int o = cg * GPW + grp;
      const int j = o < n_used ? (int)Ord[o] : m;
      const int j1 = min(j + 1, m);
      ColSpan c;
      const uint32_t ost = Ost[j], tof = Toff[j];
      c.lst = ost;
      c.tst = n_lo + tof;
      c.nl = Ost[j1] - ost;
      c.nt = Toff[j1] - tof;
      return c;
    };
    // load stage: column group lcg, entries [lj, lj + CHK) of each column
    int lcg = wave, ncg = n_cg;
    uint32_t lj = 0, lmax = 0;
    ColSpan lc{0u, 0u, 0u, 0u};
    if (lcg < n_cg) {
      lc = col_of(lcg);
      lmax = wave_max(lc.nl + lc.nt);
      ncg = grab();
    }
    auto chunk_of_l = [&]() -> LtChunk {
      const uint32_t n = lmax > lj ? min((uint32_t)CHK, lmax - lj) : 0u;
      bool tree = false;
#pragma unroll
      for (int h = 0; h < PER; ++h) {
        const uint32_t e = lj + (uint32_t)(sub + h * LPG);
        tree |= __ballot(e >= lc.nl && e < lc.nl + lc.nt) != 0;
      }
      return LtChunk{lcg, (n + 3u) & ~3u, lj, lj + CHK >= lmax, tree};
    };
    auto advance = [&]() {
      if (lcg < n_cg) {
        lj += CHK;
        if (lj >= lmax) {
          lcg = ncg;
          lj = 0;
          lmax = 0u;
          if (lcg < n_cg) {
            lc = col_of(lcg);
            lmax = wave_max(lc.nl + lc.nt);
            ncg = grab();
          }
        }
      }
    };
    const BufRes rs_cent = buf_res(im.centry + bt.d_base + bt.tree_base, (uint32_t)bt.n_d + n_tree);
    const BufRes rs_cval = buf_res(im.cval + bt.d_base + bt.tree_base, (uint32_t)bt.n_d + n_tree);
    // L: the entry words of each lane (entries sub + h * LPG of the chunk: the
    // tuple of a leaf occurrence, or a tree code marked kTreeEntry), the
    // value of the entry's code beside it, and the wave masks of lanes with an
    // entry.  A lane without one reads past the buffers: word and value 0.
    auto load_entry = [&](uint32_t (&w)[PER], uint32_t (&v)[PER], uint64_t (&ok)[PER]) {
      const bool live = lcg < n_cg;
#pragma unroll
      for (int h = 0; h < PER; ++h) {
        const uint32_t e = lj + (uint32_t)(sub + h * LPG);
        const bool in = live && e < lc.nl + lc.nt;
        ok[h] = __ballot(in);
        const uint32_t at = in ? e + (e < lc.nl ? lc.lst : lc.tst - lc.nl) : 0xFFFFFFFFu;
        w[h] = buf_load(rs_cent, at);
        v[h] = buf_load(rs_cval, at);
      }
    };
    auto row_f4 = [&](uint32_t r) -> float4 {
      if (TREE_LDS) return lds_load4(qb + r * RB);
      const bool g = (r & kRtGlobal) != 0;
      const float4 xl = lds_load4(qb + (g ? zrow : r) * RB);
      float4 xg = make_float4(0.f, 0.f, 0.f, 0.f);
      if (g) xg = *(const float4 *)&Hg[(int64_t)(r & ~kRtGlobal) * TW + q];
      return g ? xg : xl;
    };
    LtChunk G = chunk_of_l();
    LtChunk C{n_cg, 0u, 0u, false, false};
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    // 16-lane groups: chunk C's translated entries stay in registers (lane t
    // holds entries t + 16 h: LDS address of the row, or kRtGlobal | tree row in
    // the workspace, and the multiplier) and are broadcast along the row
    const uint32_t zaddr = rb0 + zrow * RB;
    uint32_t cra[PER], cmu[PER];
#pragma unroll
    for (int h = 0; h < PER; ++h) {
      cra[h] = zaddr;
      cmu[h] = 0u;
    }
    auto step = [&](const uint32_t (&gw)[PER], const uint32_t (&gv)[PER],
                    const uint64_t (&gok)[PER], uint32_t (&lw)[PER], uint32_t (&lv)[PER],
                    uint64_t (&lok)[PER]) {
      advance();
      // G: entries of the chunk loaded a step ago: a leaf occurrence reads the G
      // row of its tuple, a tree code its H row; the multiplier is the value
      // loaded beside the entry (0 for a lane without entry)
      uint32_t row[PER], pv[PER];
#pragma unroll
      for (int h = 0; h < PER; ++h) {
        const bool tree = (gw[h] & toc::kTreeEntry) != 0u;     // a lane without entry has word 0
        const bool leaf = __builtin_amdgcn_inverse_ballot_w64(gok[h]) && !tree;
        const uint32_t hr = hrow(gw[h] & ~toc::kTreeEntry);
        const uint32_t trow = hr < cap ? trow0 + hr : (kRtGlobal | hr);
        row[h] = leaf ? (gw[h] & ~kFirstOcc) : (tree ? trow : zrow);
        pv[h] = gv[h];
      }
      const LtChunk L = chunk_of_l();
      load_entry(lw, lv, lok);
      // blocked summation: a chunk's entries form a partial sum that then joins
      // the column's running sum (serial chains of at most CHK terms, and of the
      // column's number of chunks)
      float4 part = make_float4(0.f, 0.f, 0.f, 0.f);
      if constexpr (DPP) {
        constexpr int NB = CHK / 4;             // blocks of 4 entries
        // does an entry of chunk C read a tree row in the workspace?
        bool ws_chunk = false;
        if (!TREE_LDS && C.tree) {
#pragma unroll
          for (int h = 0; h < PER; ++h) ws_chunk |= __ballot((cra[h] & kRtGlobal) != 0) != 0;
        }
        if (C.cg < n_cg && !ws_chunk && C.steps == (uint32_t)CHK) {
          // a full chunk of leaf entries: LDS rows only, each block's reads
          // issued before the previous block's FMAs
          float4 xa[4], xb[4];
          load4x4_bcast<0>(cra[0], qoff, xa);
          static_for<NB>([&](auto bc) {
            constexpr int bk = decltype(bc)::value;
            if constexpr (bk + 1 < NB) {
              constexpr int nb = bk + 1;
              if constexpr (bk % 2 == 0) load4x4_bcast<4 * (nb % 4)>(cra[nb / 4], qoff, xb);
              else load4x4_bcast<4 * (nb % 4)>(cra[nb / 4], qoff, xa);
            }
            if constexpr (bk % 2 == 0) fma4x4_bcast<4 * (bk % 4)>(part, cmu[bk / 4], xa);
            else fma4x4_bcast<4 * (bk % 4)>(part, cmu[bk / 4], xb);
          });
        } else if (C.cg < n_cg && !ws_chunk) {
          // a partial chunk, rows in LDS: blocks of 4 entries
          static_for<NB>([&](auto bc) {
            constexpr int bk = decltype(bc)::value;
            if (C.steps > (uint32_t)(4 * bk)) {
              float4 xv[4];
              load4x4_bcast<4 * (bk % 4)>(cra[bk / 4], qoff, xv);
              fma4x4_bcast<4 * (bk % 4)>(part, cmu[bk / 4], xv);
            }
          });
        } else if (C.cg < n_cg) {
          // blocks of 4 entries; tree rows may be in the workspace: both loads
          // are issued and the values selected
          static_for<NB>([&](auto bc) {
            constexpr int bk = decltype(bc)::value;
            constexpr int t0 = 4 * (bk % 4), hh = bk / 4;
            if (C.steps > (uint32_t)(4 * bk)) {
              float4 xv[4];
              float mt[4];
              static_for<4>([&](auto ic) {
                constexpr int i = decltype(ic)::value;
                const uint32_t r = row_bcast<t0 + i>(cra[hh]);
                mt[i] = __uint_as_float(row_bcast<t0 + i>(cmu[hh]));
                const bool g = (r & kRtGlobal) != 0;
                const float4 xl = lds_load4((g ? zaddr : r) + qoff);
                float4 xg = make_float4(0.f, 0.f, 0.f, 0.f);
                if (g) xg = *(const float4 *)&Hg[(int64_t)(r & ~kRtGlobal) * TW + q];
                xv[i] = g ? xg : xl;
              });
              static_for<4>([&](auto ic) {
                constexpr int i = decltype(ic)::value;
                part = f4fma(mt[i], xv[i], part);
              });
            }
          });
        }
      } else {
        static_assert(DPP || PER == 1, "the staged path takes one entry per lane");
        // C: the staged chunk; a full chunk of leaf entries reads only LDS rows, 8
        // of them issued back to back
        if (C.cg < n_cg && !C.tree && C.steps == (uint32_t)CH) {
  #pragma unroll
          for (int h = 0; h < CH; h += 8) {
            uint2 e[8];
  #pragma unroll
            for (int t = 0; t < 8; ++t) e[t] = stage[(h + t) * GPW + grp];
            float4 xr[8];
  #pragma unroll
            for (int t = 0; t < 8; ++t) xr[t] = lds_load4(qb + e[t].x * RB);
  #pragma unroll
            for (int t = 0; t < 8; ++t) part = f4fma(__uint_as_float(e[t].y), xr[t], part);
            __builtin_amdgcn_sched_barrier(0);
          }
        } else if (C.cg < n_cg) {
          for (uint32_t t = 0; t < C.steps; t += 4) {
            const uint2 e0 = stage[(t + 0) * GPW + grp], e1 = stage[(t + 1) * GPW + grp];
            const uint2 e2 = stage[(t + 2) * GPW + grp], e3 = stage[(t + 3) * GPW + grp];
            float4 x0, x1, x2, x3;
            if (C.tree) {
              x0 = row_f4(e0.x);
              x1 = row_f4(e1.x);
              x2 = row_f4(e2.x);
              x3 = row_f4(e3.x);
            } else {
              x0 = lds_load4(qb + e0.x * RB);
              x1 = lds_load4(qb + e1.x * RB);
              x2 = lds_load4(qb + e2.x * RB);
              x3 = lds_load4(qb + e3.x * RB);
            }
            part = f4fma(__uint_as_float(e0.y), x0, part);
            part = f4fma(__uint_as_float(e1.y), x1, part);
            part = f4fma(__uint_as_float(e2.y), x2, part);
            part = f4fma(__uint_as_float(e3.y), x3, part);
          }
        }
            }
      if (C.cg < n_cg) {
        acc.x += part.x;
        acc.y += part.y;
        acc.z += part.z;
        acc.w += part.w;
        if (C.last) {
          const int o = C.cg * GPW + grp;
          if (o < n_used) {
            const int j = (int)Ord[o];
            float *o = out + (b * m + j) * ldo + k0 + q;
            if (accumulate) {
              if (q + 0 < kt) acc.x += o[0];
              if (q + 1 < kt) acc.y += o[1];
              if (q + 2 < kt) acc.z += o[2];
              if (q + 3 < kt) acc.w += o[3];
            }
            if (q + 3 < kt) {
              o[0] = acc.x;
              o[1] = acc.y;
              o[2] = acc.z;
              o[3] = acc.w;
            } else {
              if (q + 0 < kt) o[0] = acc.x;
              if (q + 1 < kt) o[1] = acc.y;
              if (q + 2 < kt) o[2] = acc.z;
            }
          }
          acc = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      if constexpr (DPP) {
        // entries of chunk G become chunk C
#pragma unroll
        for (int h = 0; h < PER; ++h) {
          cra[h] = (row[h] & kRtGlobal) ? row[h] : rb0 + row[h] * RB;
          cmu[h] = pv[h];
        }
      } else {
        // S: entry sub of column grp goes to stage[sub * GPW + grp]
        stage[sub * GPW + grp] = make_uint2(row[0], pv[0]);
        __builtin_amdgcn_wave_barrier();
      }
      C = G;
      G = L;
    };
    uint32_t wA[PER], wB[PER], vA[PER], vB[PER];
    uint64_t kA[PER], kB[PER];
    load_entry(wA, vA, kA);
    while (G.cg < n_cg || C.cg < n_cg) {
      step(wA, vA, kA, wB, vB, kB);
      if (!(G.cg < n_cg || C.cg < n_cg)) break;
      step(wB, vB, kB, wA, vA, kA);
    }
  }
}

// ===========================================================================
// Decode to CSR (the backtracking of Algorithm 6).  Rows are concatenated in D
// and in the CSR alike, so the output position of entry j of D is the number of
// pairs of the entries before it.  The upload recorded, for every run of
// kDecodeTile entries, that count at the run's start and the first row starting
// in it, so each run is an independent workgroup: an exclusive scan of the
// entries' depths inside the run gives every position (and rowptr at row
// starts), then each entry writes its sequence backwards while walking to the
// root.  Entries are dealt to threads with stride kDecBlock, so loads and
// depth-1 stores are coalesced; the scan takes each wave's part of every row of
// kDecBlock entries, then the row-and-wave totals in one wave.
// ===========================================================================
constexpr int kDecBlock = 256;
constexpr int kDecWaves = kDecBlock / kWave;
constexpr int kDecPer = (int)toc::kDecodeTile / kDecBlock;   // 4

__global__ __launch_bounds__(kDecBlock) void decode_kernel(Img im, const uint4 *__restrict__ dtiles,
                                                           int64_t t0, int64_t n_runs,
                                                           int64_t *__restrict__ rowptr,
                                                           int32_t *__restrict__ ocol,
                                                           uint32_t *__restrict__ oval) {
  __shared__ uint32_t sh[toc::kDecodeTile];
  __shared__ uint32_t wave_tot[kDecPer * kDecWaves];
  // blocks are dealt to the 8 XCDs round-robin; the grid is a multiple of 8 and
  // each XCD gets a contiguous range of runs, so the runs of a batch share its L2
  const int64_t per_xcd = (int64_t)gridDim.x / kXcd;
  const int64_t slot = (int64_t)(blockIdx.x % kXcd) * per_xcd + blockIdx.x / kXcd;
  if (slot >= n_runs) return;
  const int64_t t = t0 + slot;
  const uint4 dt = dtiles[t];                       // batch, first entry, pairs before, first row
  const toc_batch bt = im.batches[dt.x];
  const toc_key *key = im.key + bt.code_base;
  const toc_link *link = deep_links(im.link, bt);
  const uint32_t n1 = (uint32_t)bt.n_lvl1;
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const uint32_t nd = (uint32_t)bt.n_d, es = dt.y;
  const int64_t base = bt.nnz_base + dt.z;
  // every load is unconditional, so that all of a thread's gathers are in
  // flight together: entries past the batch's end take the code 0xFFFFFFFF,
  // whose key and link reads fall outside the buffers and return zeros (depth
  // 0); depth-1 codes (below n_lvl1) read no link either
  const BufRes rs_dc = buf_res(dc, nd);
  const BufRes rs_key = key_res(key, (uint32_t)bt.n_codes);
  const BufRes rs_link = link_res(link, (uint32_t)bt.n_codes);
  uint32_t c[kDecPer];
#pragma unroll
  for (int i = 0; i < kDecPer; ++i) {
    const uint32_t j = es + i * kDecBlock + threadIdx.x;
    c[i] = buf_load(rs_dc, j);
    if (j >= nd) c[i] = 0xFFFFFFFFu;
  }
  // the key pair of each entry's code and its link (parent, depth)
  uint2 kv[kDecPer];
  uint2 lk[kDecPer];
#pragma unroll
  for (int i = 0; i < kDecPer; ++i) {
    kv[i] = key_load(rs_key, c[i]);
    lk[i] = link_load(rs_link, c[i] < n1 ? 0xFFFFFFFFu : c[i]);
    if (c[i] < n1) lk[i].y = 1u;
  }
  // exclusive scan of the depths in entry order: entry i * kDecBlock + t is row
  // i, position t; each wave scans its 64 positions of every row, then the
  // (row, wave) totals, in entry order, are scanned across one wave
  uint32_t incl[kDecPer];
#pragma unroll
  for (int i = 0; i < kDecPer; ++i) {
    incl[i] = wave_incl_scan(lk[i].y, lane);
    if (lane == kWave - 1) wave_tot[i * kDecWaves + wave] = incl[i];
  }
  __syncthreads();
  const uint32_t wt = lane < kDecPer * kDecWaves ? wave_tot[lane] : 0u;
  const uint32_t wi = wave_incl_scan(wt, lane);
  const uint32_t total = (uint32_t)__shfl((int)wi, kDecPer * kDecWaves - 1, kWave);
  uint32_t pos[kDecPer];
#pragma unroll
  for (int i = 0; i < kDecPer; ++i) {
    pos[i] = (uint32_t)__shfl((int)(wi - wt), i * kDecWaves + wave, kWave) + incl[i] - lk[i].y;
    sh[i * kDecBlock + threadIdx.x] = pos[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kDecPer; ++i) {
    const uint32_t j = es + i * kDecBlock + threadIdx.x;
    if (j < nd) {
      uint2 kk = kv[i];
      uint32_t par = lk[i].x;
      const uint32_t d = lk[i].y;
      int64_t p = base + pos[i] + d - 1;
      for (uint32_t q = 0;;) {
        // ordinary stores: L2 merges the chains' partial lines (streaming stores
        // measured 1.9x slower on the categorical workload's deeper chains)
        ocol[p] = (int32_t)kk.x;
        oval[p] = kk.y;
        if (++q >= d) break;
        --p;
        kk = *(const uint2 *)(key + par);
        if (par >= n1) par = link[par].parent;
      }
    }
  }
  // rows starting in this run; the batch's last run also writes the rows that
  // start at the end of D and the end mark
  const bool last = (uint64_t)es + toc::kDecodeTile >= nd;
  const uint32_t r_end = last ? (uint32_t)bt.n_rows + 1 : dtiles[t + 1].w;
  for (uint32_t r = dt.w + threadIdx.x; r < r_end; r += kDecBlock) {
    const uint32_t sr = span[r];
    rowptr[bt.row_base + r] = sr < nd ? base + sh[sr - es] : base + total;
  }
}

// Decode of a batch whose keys and links fit in LDS: one workgroup per batch
// copies them (coalesced) into LDS, so every step of a walk to the root is an LDS
// read instead of a dependent gather from L2; the batch's entries of D then go
// through in runs of kDecodeTile as in decode_kernel (a scan of the depths gives
// each entry's output position, rowptr at tuple starts).  Writing the pairs in
// output order instead (a thread per pair, found by a binary search over the
// run's positions) measured slower on the categorical workload (5.8 -> 7.9 ms).
constexpr size_t kDecLdsMax = 64 * 1024;
constexpr int kDbBlock = 1024;                    // 16 waves: two or more workgroups per CU
constexpr int kDbWaves = kDbBlock / kWave;
constexpr int kDbPer = (int)toc::kDecodeTile / kDbBlock;   // 1
constexpr int kDbAhead = 8;                       // runs whose codes are loaded together
constexpr int kDbCopy = 4;                        // keys, links and tuple starts per thread in flight
static_assert(kDbPer == 1, "one entry per thread and run");

__global__ __launch_bounds__(kDbBlock) void decode_batch_kernel(Img im, int64_t b0,
                                                                 int64_t *__restrict__ rowptr,
                                                                 int32_t *__restrict__ ocol,
                                                                 uint32_t *__restrict__ oval,
                                                                 int64_t max_slots) {
  extern __shared__ uint2 kl[];                     // keys, then the links of deep codes
  __shared__ uint32_t sh[toc::kDecodeTile];       // positions of the run's entries
  __shared__ uint32_t wave_tot[kDbWaves];
  const int64_t b = b0 + blockIdx.x;
  const toc_batch bt = uniform_batch(im.batches + b);
  const uint32_t nc = (uint32_t)bt.n_codes, n1 = (uint32_t)bt.n_lvl1, nd = (uint32_t)bt.n_d;
  const uint32_t nr = (uint32_t)bt.n_rows;
  uint2 *lk = kl + nc;                              // link of code c >= n1 at lk[c - n1]
  uint32_t *sp = (uint32_t *)(kl + (size_t)max_slots);   // the tuple starts
  const uint2 *key = (const uint2 *)(im.key + bt.code_base);
  const uint2 *link = (const uint2 *)(im.link + bt.deep_base);
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  // keys, deep links and tuple starts into LDS: a thread's loads of a pass (up to
  // kDbCopy of each) are all issued before its stores
  const uint32_t nlk = nc - n1;
  for (uint32_t i0 = threadIdx.x; i0 < nc || i0 < nlk || i0 <= nr; i0 += kDbCopy * kDbBlock) {
    uint2 kt[kDbCopy], lt[kDbCopy];
    uint32_t st[kDbCopy];
#pragma unroll
    for (int q = 0; q < kDbCopy; ++q) {
      const uint32_t i = i0 + (uint32_t)(q * kDbBlock);
      kt[q] = i < nc ? key[i] : make_uint2(0u, 0u);
      lt[q] = i < nlk ? link[i] : make_uint2(0u, 0u);
      st[q] = i <= nr ? span[i] : 0u;
    }
#pragma unroll
    for (int q = 0; q < kDbCopy; ++q) {
      const uint32_t i = i0 + (uint32_t)(q * kDbBlock);
      if (i < nc) kl[i] = kt[q];
      if (i < nlk) lk[i] = lt[q];
      if (i <= nr) sp[i] = st[q];
    }
  }
  __syncthreads();
  const int lane = threadIdx.x % kWave, wave = wave_id();
  const int64_t base = bt.nnz_base;
  uint32_t carry = 0;                               // pairs of the runs before
  // the codes of kDbAhead runs are loaded at once, so one load latency serves them
  // (loading the first ones before the tables measured slower)
  uint32_t ahead[kDbAhead];
  for (uint32_t es = 0; es < nd; es += (uint32_t)toc::kDecodeTile) {
    const uint32_t r_in = (es / (uint32_t)toc::kDecodeTile) % kDbAhead;
    if (r_in == 0) {
#pragma unroll
      for (int a = 0; a < kDbAhead; ++a) {
        const uint32_t j = es + a * (uint32_t)toc::kDecodeTile + threadIdx.x;
        ahead[a] = j < nd ? dc[j] : 0xFFFFFFFFu;
      }
    }
    // thread t owns entry es + t of the run: its depth, then an exclusive scan
    // of the depths in entry order gives its output position
    uint32_t c = ahead[0];
#pragma unroll
    for (int a = 1; a < kDbAhead; ++a)
      if (r_in == (uint32_t)a) c = ahead[a];
    const uint32_t dd = c == 0xFFFFFFFFu ? 0u : (c < n1 ? 1u : lk[c - n1].y);
    const uint32_t incl = wave_incl_scan(dd, lane);
    if (lane == kWave - 1) wave_tot[wave] = incl;
    __syncthreads();
    // the waves' totals: lane w holds wave w's, scanned across the wave
    const uint32_t wt = lane < kDbWaves ? wave_tot[lane] : 0u;
    const uint32_t wi = wave_incl_scan(wt, lane);
    const uint32_t off = (uint32_t)__shfl((int)(wi - wt), wave, kWave);
    const uint32_t total = (uint32_t)__shfl((int)wi, kDbWaves - 1, kWave);
    const uint32_t pos = off + incl - dd;
    sh[threadIdx.x] = pos;
    // each entry writes its sequence backwards, walking to the root in LDS
    if (c != 0xFFFFFFFFu) {
      uint32_t x = c;
      int64_t p = base + carry + pos + dd - 1;
      for (;;) {
        const uint2 kk = kl[x];
        ocol[p] = (int32_t)kk.x;
        oval[p] = kk.y;
        if (x < n1) break;
        x = lk[x - n1].x;
        --p;
      }
    }
    // every position is in sh, and every wave has read wave_tot (the next run
    // writes wave_tot before its first barrier and sh only after it)
    __syncthreads();
    // tuples starting in this run
    for (uint32_t r = threadIdx.x; r <= nr; r += kDbBlock) {
      const uint32_t sr = sp[r];
      if (sr >= es && sr - es < (uint32_t)toc::kDecodeTile && sr < nd)
        rowptr[bt.row_base + r] = base + carry + sh[sr - es];
    }
    carry += total;
  }
  // tuples starting at the end of D, and the end mark
  for (uint32_t r = threadIdx.x; r <= nr; r += kDbBlock)
    if (sp[r] >= nd) rowptr[bt.row_base + r] = base + carry;
}

// ===========================================================================
// Sparse-safe element-wise operations (Algorithm 3): every key value of the
// image, and its copies beside the left multiplication's entries, changes alike.
// ===========================================================================
constexpr int kMapBlock = 256;

__global__ __launch_bounds__(kMapBlock) void map_values_kernel(toc_key *__restrict__ key, int64_t n,
                                                               uint32_t *__restrict__ cval,
                                                               int64_t n_cval, int op, float c) {
  const int64_t stride = (int64_t)gridDim.x * kMapBlock;
  for (int64_t i = (int64_t)blockIdx.x * kMapBlock + threadIdx.x; i < n; i += stride) {
    const float v = key[i].val;
    key[i].val = op == TOC_MAP_SCALE ? v * c : v * v;
  }
  // the copies beside the left multiplication's column entries
  for (int64_t i = (int64_t)blockIdx.x * kMapBlock + threadIdx.x; i < n_cval; i += stride) {
    const float w = __uint_as_float(cval[i]);
    cval[i] = __float_as_uint(op == TOC_MAP_SCALE ? w * c : w * w);
  }
}

// ===========================================================================
// Dense decode plus a scalar (Algorithm 9): one workgroup per batch, a wave per
// tuple.  When a row of the dense block fits (ROW_LDS: n_cols floats per wave in
// LDS), the wave fills its row in LDS with c, every entry of the tuple (a lane
// each) writes its sequence's pairs a_ij + c there while walking its chain to the
// root, and the row goes to HBM once with 16-byte stores.  Otherwise the rows are
// filled in HBM first, made visible (fence, barrier), then the pairs written.
// ===========================================================================
constexpr int kDnBlock = 1024;
constexpr int kDnWaves = kDnBlock / kWave;
constexpr int kDnPer = 4;        // a lane's entries of a tuple whose loads fly together

template <bool ROW_LDS>
__global__ __launch_bounds__(kDnBlock) void decode_dense_kernel(Img im, int64_t b0, int m,
                                                                float c, float *__restrict__ A,
                                                                int64_t lda) {
  extern __shared__ float dn_rows[];
  const int64_t b = b0 + blockIdx.x;
  const toc_batch bt = uniform_batch(im.batches + b);
  const int lane = threadIdx.x % kWave, wave = wave_id();
  float *Ab = A + bt.row_base * lda;
  const toc_key *key = im.key + bt.code_base;
  const toc_link *link = deep_links(im.link, bt);
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const uint32_t n1 = (uint32_t)bt.n_lvl1;
  // the wave's tuples' starts and ends, one tuple per lane (tuple wave + 16 i in
  // lane i), loaded once
  const int nrows = bt.n_rows;
  uint32_t ps = 0u, pe = 0u;
  {
    const int rl = wave + kDnWaves * lane;
    if (rl < nrows) {
      ps = span[rl];
      pe = span[rl + 1];
    }
  }
  // the pairs of the tuple r into row (LDS or HBM): kDnPer of a lane's entries at
  // a time, their codes and then their keys loaded together; deeper codes walk
  // the rest of their chain to the root
  auto scatter = [&](int r, float *row) {
    const int i = (r - wave) / kDnWaves;
    const uint32_t s0 = i < kWave ? (uint32_t)__shfl((int)ps, i, kWave) : span[r];
    const uint32_t e = i < kWave ? (uint32_t)__shfl((int)pe, i, kWave) : span[r + 1];
    for (uint32_t j0 = s0 + lane; j0 < e; j0 += kWave * kDnPer) {
      uint32_t x[kDnPer];
      toc_key kk[kDnPer];
#pragma unroll
      for (int q = 0; q < kDnPer; ++q) {
        const uint32_t j = j0 + (uint32_t)(q * kWave);
        x[q] = j < e ? dc[j] : 0xFFFFFFFFu;
      }
#pragma unroll
      for (int q = 0; q < kDnPer; ++q) kk[q] = x[q] != 0xFFFFFFFFu ? key[x[q]] : toc_key{0u, 0.0f};
#pragma unroll
      for (int q = 0; q < kDnPer; ++q) {
        if (x[q] == 0xFFFFFFFFu) continue;
        row[kk[q].col] = kk[q].val + c;
        uint32_t xx = x[q];
        while (xx >= n1) {   // depth 1 ends the chain
          xx = link[xx].parent;
          const toc_key k = key[xx];
          row[k.col] = k.val + c;
        }
      }
    }
  };
  if constexpr (ROW_LDS) {
    float *row = dn_rows + (size_t)wave * m;
    const bool vec = (m % 4) == 0 && (lda % 4) == 0 && (((uintptr_t)A) & 15u) == 0;
    for (int r = wave; r < nrows; r += kDnWaves) {
      for (int j = lane; j < m; j += kWave) row[j] = c;
      __builtin_amdgcn_wave_barrier();
      scatter(r, row);
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      float *dst = Ab + (int64_t)r * lda;
      // streaming stores: the block is written once and not read back here
      if (vec) {
        typedef float f4v __attribute__((ext_vector_type(4)));
        for (int j = 4 * lane; j < m; j += 4 * kWave)
          __builtin_nontemporal_store(*(const f4v *)&row[j], (f4v *)&dst[j]);
      } else {
        for (int j = lane; j < m; j += kWave) __builtin_nontemporal_store(row[j], &dst[j]);
      }
      __builtin_amdgcn_wave_barrier();
    }
  } else {
    for (int r = wave; r < bt.n_rows; r += kDnWaves) {
      float *row = Ab + (int64_t)r * lda;
      for (int j = lane; j < m; j += kWave) row[j] = c;
    }
    __threadfence();
    __syncthreads();
    for (int r = wave; r < nrows; r += kDnWaves) scatter(r, Ab + (int64_t)r * lda);
  }
}

// ===========================================================================
// Host helpers
// ===========================================================================
toc_status check_device(const toc_dev *d) {
  if (!d) return fail(TOC_EINVAL, "dev is NULL");
  if (d->pending) return fail(TOC_EINVAL, "image planned but not built");
  if (d->host) return fail(TOC_EINVAL, "image was uploaded to host memory");
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return fail(TOC_EDEVICE, "hipGetDevice failed");
  if (cur != d->device) return fail(TOC_EINVAL, "current device %d differs from upload device %d", cur, d->device);
  return TOC_OK;
}

toc_status launch_status(const char *what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "%s: %s", what, hipGetErrorString(e));
  return TOC_OK;
}

template <typename K>
toc_status allow_lds(K kernel, size_t bytes) {
  if (bytes > 64 * 1024) {
    if (hipFuncSetAttribute((const void *)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)bytes) != hipSuccess)
      return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", bytes);
  }
  return TOC_OK;
}

// Lanes that sum one tuple in the k = 1 right product: few, so that a workgroup
// sums many tuples at once and each lane has several independent code loads in
// flight (a tuple of c codes takes about c / lanes steps plus log2(lanes) for the
// reduction, and the tuples of a batch take rows / (256 / lanes) rounds).
int lanes_per_row(const toc_dev *d) {
  const double avg = d->info.n_rows ? (double)d->info.n_codes / (double)d->info.n_rows : 0.0;
  if (avg <= 40) return 4;
  if (avg <= 64) return 8;
  if (avg <= 160) return 16;
  if (avg <= 400) return 32;
  return 64;
}

// Whether the k = 1 kernels can keep a batch's H in LDS.
size_t k1_lds(const toc_dev *d, int op) {
  if (op == TOC_OP_RIGHT) return std::max<size_t>(16, (size_t)d->max_codes * 4);
  return ((size_t)d->max_rows + d->max_codes) * 4;
}

bool k1_fits(const toc_dev *d, int op) { return k1_lds(d, op) <= kLdsMax; }

// Execution plan of an op: which kernel family, its LDS bytes, and the workspace
// it needs (rows of row_floats floats per code that needs an H row in memory).
enum { kPathK1 = 0, kPathTiled = 1, kPathWide = 2 };

struct OpPlan {
  int path = kPathWide;
  int n_tiles = 1, tw = 0, spx = 1;
  bool deep_lds = false;
  size_t lds = 0;
  unsigned grid = 0;
  int64_t row_floats = 0;     // workspace floats per H row (0: no workspace)
  int64_t rows_max = 0, rows_total = 0;
  int64_t ws_floats = 0;      // tiled: whole workspace (one slot per worker)
  int64_t lds_rows = 0;       // tiled left: tree rows in LDS
  int per = 1;                // tiled right: batches per item
  bool compact = false;       // tiled right: the compact-tile kernel (64 columns)
  bool toc_lds = false;       // tiled left: tree rows' occurrence offsets in LDS
  int ocr_cap = 0;            // tiled left: LDS words for the tree rows' occurrences
};

OpPlan plan_op(const toc_dev *d, int op, int k) {
  OpPlan p;
  const int64_t m = d->info.n_cols;
  const bool right = op == TOC_OP_RIGHT;
  p.rows_max = right ? d->max_deep : d->max_tree;
  p.rows_total = right ? d->total_deep : d->total_tree;
  if (k == 1 && k1_fits(d, op)) {
    p.path = kPathK1;
    return p;
  }
  if (right && k >= kRcKT && m <= 65535 && d->max_ucols > 0 &&
      rc_lds_bytes(d->max_ucols, m) <= kLdsMax - kRtStaticBytes) {
    // the batch's used rows of W fit in LDS at 64 columns: right_compact_kernel,
    // deep rows in the workspace.  (Two batches per item, sharing one tile of
    // their used columns, measured slower: 128 VGPRs and scalar spills.)
    p.path = kPathTiled;
    p.compact = true;
    p.tw = kRcKT;
    p.n_tiles = (k + kRcKT - 1) / kRcKT;
    p.lds_rows = d->max_ucols;
    p.lds = rc_lds_bytes(d->max_ucols, m);
    p.per = 1;
    const int64_t per_xcd = (d->info.n_batches + kXcd - 1) / kXcd;
    const int64_t items = (per_xcd + p.per - 1) / p.per * p.n_tiles;
    p.spx = (int)std::min<int64_t>(kCuPerXcd, std::max<int64_t>(1, items));
    p.grid = (unsigned)(kXcd * p.spx);
    p.row_floats = kRcHgRow;
    const int64_t deep_rows = std::max<int64_t>(p.per == 2 ? d->max_pair_deep : d->max_deep, 1);
    p.ws_floats = (int64_t)p.grid * deep_rows * kRcHgRow;
    return p;
  }
  if (right) {
    // deep rows in LDS: right_tiled_kernel; else right_staged_kernel, with the
    // deep rows in the workspace and a per-wave stage in LDS
    const size_t tile = ((size_t)m + 1) * kRtKT * 4;
    const size_t lds_max = kLdsMax - kRtStaticBytes;
    const size_t with_deep = tile + (size_t)d->max_deep * kRtKT * 4;
    const size_t with_pair = tile + (size_t)d->max_pair_deep * kRtKT * 4;
    if (k >= 4 && (with_deep <= lds_max || kRsStageBytes + tile <= lds_max)) {
      p.path = kPathTiled;
      p.n_tiles = (k + kRtKT - 1) / kRtKT;
      p.tw = kRtKT;
      p.deep_lds = with_deep <= lds_max;
      // two batches per item when every pair's deep rows fit next to the tile
      p.per = p.deep_lds && with_pair <= lds_max ? 2 : 1;
      p.lds = p.deep_lds ? (p.per == 2 ? with_pair : with_deep) : kRsStageBytes + tile;
      // workers per XCD: one per CU, fewer when there are fewer items
      const int64_t per_xcd = (d->info.n_batches + kXcd - 1) / kXcd;
      const int64_t items = (per_xcd + p.per - 1) / p.per * p.n_tiles;
      p.spx = (int)std::min<int64_t>(kCuPerXcd, std::max<int64_t>(1, items));
      p.grid = (unsigned)(kXcd * p.spx);
      p.row_floats = p.deep_lds ? 0 : kRtKT;
      p.ws_floats = p.deep_lds ? 0 : (int64_t)p.grid * d->max_deep * kRtKT;
      return p;
    }
  } else if (k >= 2) {
    // widest tile first; tree rows in LDS when they fit, else in the workspace
    const size_t lds_max = kLdsMax - kLtStaticBytes;
    // widest tile first, then with the tree rows' occurrence offsets and (kLtOcr
    // words of) occurrences in LDS, then with the offsets only, then neither
    for (int cfg = 0; cfg < 6; ++cfg) {
      const int tw = cfg < 3 ? 64 : 32;
      const bool toc = cfg % 3 != 2;
      const int ocr = cfg % 3 == 0 ? kLtOcr : 0;
      const size_t head = tw == 64 ? lt_rows_offset<64>(m, d->max_tree, toc, ocr)
                                   : lt_rows_offset<32>(m, d->max_tree, toc, ocr);
      const size_t rows = ((size_t)d->max_rows + 1) * tw * 4;
      if (head + rows > lds_max) continue;
      p.path = kPathTiled;
      p.tw = tw;
      p.toc_lds = toc;
      p.ocr_cap = ocr;
      p.n_tiles = (k + tw - 1) / tw;
      // the tree rows that fit in LDS go there, the others to the workspace
      p.lds_rows = std::min<int64_t>(d->max_tree, (int64_t)((lds_max - head - rows) / ((size_t)tw * 4)));
      p.deep_lds = p.lds_rows == d->max_tree;
      p.lds = head + rows + (size_t)p.lds_rows * tw * 4;
      const int64_t items = (d->info.n_batches + kXcd - 1) / kXcd * p.n_tiles;
      p.spx = (int)std::min<int64_t>(kCuPerXcd, std::max<int64_t>(1, items));
      p.grid = (unsigned)(kXcd * p.spx);
      p.row_floats = p.deep_lds ? 0 : tw;
      p.ws_floats = p.deep_lds ? 0 : (int64_t)p.grid * d->max_tree * tw;
      return p;
    }
  }
  p.path = kPathWide;
  p.row_floats = std::min<int64_t>(k, kKTile);
  return p;
}

// Splits batches into passes whose workspace rows fit `cap_rows`; calls fn(b0, nb, base).
template <typename F>
toc_status for_each_pass(const toc_dev *d, int op, int64_t cap_rows, F fn) {
  const int64_t nb = (int64_t)d->batches.size();
  int64_t b0 = 0;
  const int64_t max_grid = 1 << 26;
  while (b0 < nb) {
    const toc_batch &first = d->batches[b0];
    const int64_t base = op == TOC_OP_RIGHT ? first.deep_base : first.tree_base;
    int64_t b1 = b0;
    while (b1 < nb && b1 - b0 < max_grid) {
      const toc_batch &x = d->batches[b1];
      const int64_t need = (op == TOC_OP_RIGHT ? x.deep_base + (x.n_codes - x.n_lvl1)
                                               : x.tree_base + (x.n_codes - x.n_lvl1) + x.n_int1) - base;
      if (need > cap_rows) break;
      ++b1;
    }
    if (b1 == b0) return fail(TOC_ESIZE, "workspace below the per-batch minimum");
    toc_status st = fn(b0, b1 - b0, base);
    if (st != TOC_OK) return st;
    b0 = b1;
  }
  return TOC_OK;
}

// Rows of the workspace available to a plan, or an error when below the minimum.
toc_status ws_capacity(const OpPlan &p, void *ws, size_t ws_bytes, int64_t &cap_rows) {
  cap_rows = INT64_MAX / 2;
  if (p.row_floats == 0 || p.rows_max == 0) return TOC_OK;
  cap_rows = (int64_t)(ws_bytes / 4) / p.row_floats;
  if (!ws || cap_rows < p.rows_max)
    return fail(TOC_ESIZE, "workspace of %zu bytes below the per-batch minimum of %lld", ws_bytes,
                (long long)(p.rows_max * p.row_floats * 4));
  return TOC_OK;
}

#define TOC_DISPATCH_KPL(kpl, KERNEL, ...)                           \
  switch (kpl) {                                                     \
    case 1: hipLaunchKernelGGL(KERNEL<1>, __VA_ARGS__); break;       \
    case 2: hipLaunchKernelGGL(KERNEL<2>, __VA_ARGS__); break;       \
    case 3: hipLaunchKernelGGL(KERNEL<3>, __VA_ARGS__); break;       \
    case 4: hipLaunchKernelGGL(KERNEL<4>, __VA_ARGS__); break;       \
    case 5: hipLaunchKernelGGL(KERNEL<5>, __VA_ARGS__); break;       \
    case 6: hipLaunchKernelGGL(KERNEL<6>, __VA_ARGS__); break;       \
    case 7: hipLaunchKernelGGL(KERNEL<7>, __VA_ARGS__); break;       \
    default: hipLaunchKernelGGL(KERNEL<8>, __VA_ARGS__); break;      \
  }

}  // namespace

extern "C" {

}  // extern "C"

namespace {

// The per-batch arrays of the image: offset in the layout, bytes per element and
// the element at which batch b's slice starts (slices are in batch order).
struct ImgArr {
  int64_t toc_layout::*off;
  int64_t elem;
  int64_t (*start)(const toc::ArrStarts &);
};

const ImgArr kImgArrs[] = {
    {&toc_layout::level, 4, [](const toc::ArrStarts &a) { return a.level; }},
    {&toc_layout::key, 8, [](const toc::ArrStarts &a) { return a.code; }},
    {&toc_layout::link, 8, [](const toc::ArrStarts &a) { return a.deep; }},
    {&toc_layout::span, 4, [](const toc::ArrStarts &a) { return a.span; }},
    {&toc_layout::dcodes, 4, [](const toc::ArrStarts &a) { return a.d; }},
    {&toc_layout::occ_off, 4, [](const toc::ArrStarts &a) { return a.code + 2 * a.b; }},
    {&toc_layout::tlist, 4, [](const toc::ArrStarts &a) { return a.tree; }},
    {&toc_layout::dtiles, 16, [](const toc::ArrStarts &a) { return a.dtile; }},
    {&toc_layout::cols, 4, [](const toc::ArrStarts &a) { return a.cols; }},
    {&toc_layout::tchild, 4, [](const toc::ArrStarts &a) { return a.tree + a.b; }},
    {&toc_layout::centry, 4, [](const toc::ArrStarts &a) { return a.d + a.tree; }},
    {&toc_layout::cval, 4, [](const toc::ArrStarts &a) { return a.d + a.tree; }},
};
constexpr int kNumImgArrs = (int)(sizeof(kImgArrs) / sizeof(kImgArrs[0]));
constexpr size_t kStageBytes = (size_t)256 << 20;   // each of the two pinned buffers

inline int64_t round256(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Builds the image batch range by batch range into two pinned host buffers in
// turn and copies each range's slices of every array to the device while the
// next range is built, so host memory holds two buffers, never the whole image.
toc_status upload_chunked(const toc_enc *const *encs, int64_t n, uint32_t flags, toc_dev *d,
                          uint8_t *dbuf, hipStream_t s) {
  std::vector<toc::ArrStarts> st((size_t)n + 1);
  for (int64_t b = 0; b <= n; ++b) st[(size_t)b] = toc::arr_starts(d, b);
  auto range_bytes = [&](int64_t b0, int64_t b1) {
    int64_t t = 0;
    for (const ImgArr &a : kImgArrs)
      t += round256((a.start(st[(size_t)b1]) - a.start(st[(size_t)b0])) * a.elem);
    return t;
  };
  size_t cap = kStageBytes;
  for (int64_t b = 0; b < n; ++b) cap = std::max(cap, (size_t)range_bytes(b, b + 1));
  uint8_t *stage[2] = {nullptr, nullptr};
  hipEvent_t done[2] = {nullptr, nullptr};
  toc_status ret = TOC_OK;
  for (int i = 0; i < 2 && ret == TOC_OK; ++i) {
    if (hipHostMalloc((void **)&stage[i], cap, hipHostMallocDefault) != hipSuccess)
      ret = fail(TOC_ENOMEM, "pinned staging buffer of %zu bytes failed", cap);
    else if (hipEventCreateWithFlags(&done[i], hipEventDisableTiming) != hipSuccess)
      ret = fail(TOC_EDEVICE, "hipEventCreate failed");
  }
  int64_t b0 = 0;
  for (int i = 0; ret == TOC_OK && b0 < n; ++i) {
    uint8_t *buf = stage[i % 2];
    if (i >= 2 && hipEventSynchronize(done[i % 2]) != hipSuccess) {
      ret = fail(TOC_EDEVICE, "staging copy failed");
      break;
    }
    int64_t b1 = b0 + 1;
    while (b1 < n && range_bytes(b0, b1 + 1) <= (int64_t)cap) ++b1;
    // each array's slice for batches b0 .. b1-1, packed; the layout shifted so
    // that the batch writer lands in those slices
    toc_layout Ls = d->layout;
    int64_t so = 0, at[kNumImgArrs], len[kNumImgArrs];
    for (int a = 0; a < kNumImgArrs; ++a) {
      const ImgArr &A = kImgArrs[a];
      const int64_t e0 = A.start(st[(size_t)b0]) * A.elem;
      len[a] = A.start(st[(size_t)b1]) * A.elem - e0;
      at[a] = so;
      Ls.*(A.off) = so - e0;
      so = round256(so + len[a]);
    }
    std::memset(buf, 0, (size_t)so);
    if ((ret = toc::write_batches(encs, b0, b1, flags, Ls, d, buf)) != TOC_OK) break;
    for (int a = 0; a < kNumImgArrs && ret == TOC_OK; ++a) {
      if (len[a] == 0) continue;
      const ImgArr &A = kImgArrs[a];
      uint8_t *dst = dbuf + d->layout.*(A.off) + A.start(st[(size_t)b0]) * A.elem;
      if (hipMemcpyAsync(dst, buf + at[a], (size_t)len[a], hipMemcpyHostToDevice, s) != hipSuccess)
        ret = fail(TOC_EDEVICE, "upload copy failed");
    }
    if (ret == TOC_OK && hipEventRecord(done[i % 2], s) != hipSuccess)
      ret = fail(TOC_EDEVICE, "hipEventRecord failed");
    b0 = b1;
  }
  if (ret == TOC_OK) {
    toc::finish_image(d);
    if (n > 0 && hipMemcpyAsync(dbuf + d->layout.batches, d->batches.data(),
                                sizeof(toc_batch) * (size_t)n, hipMemcpyHostToDevice, s) != hipSuccess)
      ret = fail(TOC_EDEVICE, "upload copy failed");
  }
  if (hipStreamSynchronize(s) != hipSuccess && ret == TOC_OK) ret = fail(TOC_EDEVICE, "upload copy failed");
  for (int i = 0; i < 2; ++i) {
    if (done[i]) hipEventDestroy(done[i]);
    if (stage[i]) hipHostFree(stage[i]);
  }
  return ret;
}

}  // namespace

extern "C" {

toc_status toc_upload_size(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                           size_t *bytes) {
  if (!bytes) return fail(TOC_EINVAL, "bytes is NULL");
  toc_dev tmp;
  try {
    toc_status st = toc::plan_image(encs, n_batches, flags, &tmp);
    if (st != TOC_OK) return st;
  } catch (const std::bad_alloc &) {
    return fail(TOC_ENOMEM, "out of host memory");
  }
  *bytes = (size_t)tmp.layout.end;
  return TOC_OK;
}

toc_status toc_upload(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                      void *buf, size_t bytes, void *stream, toc_dev **out) {
  if (!out) return fail(TOC_EINVAL, "out is NULL");
  *out = nullptr;
  if (!buf) return fail(TOC_EINVAL, "buf is NULL");
  toc_dev *d = new (std::nothrow) toc_dev;
  if (!d) return fail(TOC_ENOMEM, "out of host memory");
  try {
    toc_status st = toc::plan_image(encs, n_batches, flags, d);
    if (st != TOC_OK) {
      delete d;
      return st;
    }
    if ((int64_t)bytes < d->layout.end) {
      const long long need = (long long)d->layout.end;
      delete d;
      return fail(TOC_ESIZE, "buffer has %zu bytes, image needs %lld", bytes, need);
    }
    d->buf = buf;
    d->bytes = bytes;
    d->host = (flags & TOC_UPLOAD_HOST) != 0;
    if (d->host) {
      st = toc::build_image(encs, n_batches, flags, d, (uint8_t *)buf);
      if (st != TOC_OK) {
        delete d;
        return st;
      }
    } else {
      if (hipGetDevice(&d->device) != hipSuccess) {
        delete d;
        return fail(TOC_EDEVICE, "hipGetDevice failed");
      }
      st = upload_chunked(encs, n_batches, flags, d, (uint8_t *)buf, (hipStream_t)stream);
      if (st != TOC_OK) {
        delete d;
        return st;
      }
    }
  } catch (const std::bad_alloc &) {
    delete d;
    return fail(TOC_ENOMEM, "out of host memory");
  }
  *out = d;
  return TOC_OK;
}

void toc_dev_free(toc_dev *d) { delete d; }

toc_status toc_dev_info_get(const toc_dev *d, toc_dev_info *info) {
  if (!d || !info) return fail(TOC_EINVAL, "NULL pointer");
  *info = d->info;
  return TOC_OK;
}

toc_status toc_dev_layout_get(const toc_dev *d, toc_layout *layout) {
  if (!d || !layout) return fail(TOC_EINVAL, "NULL pointer");
  *layout = d->layout;
  return TOC_OK;
}

toc_status toc_workspace_size(const toc_dev *d, int32_t op, int32_t k, size_t *bytes,
                              size_t *min_bytes) {
  if (!d || !bytes) return fail(TOC_EINVAL, "NULL pointer");
  if (k < 1) return fail(TOC_EINVAL, "k must be >= 1");
  if (op != TOC_OP_RIGHT && op != TOC_OP_LEFT && op != TOC_OP_DECODE)
    return fail(TOC_EINVAL, "unknown op %d", op);
  size_t need = 0, minimum = 0;
  if (op != TOC_OP_DECODE) {
    const OpPlan p = plan_op(d, op, k);
    if (p.path == kPathTiled) {
      minimum = need = (size_t)p.ws_floats * 4;
    } else if (p.row_floats > 0 && p.rows_max > 0) {
      minimum = (size_t)(p.rows_max * p.row_floats * 4);
      need = std::max(minimum, (size_t)(p.rows_total * p.row_floats * 4));
    }
  }
  *bytes = need;
  if (min_bytes) *min_bytes = minimum;
  return TOC_OK;
}

toc_status toc_right_mul(const toc_dev *d, const float *W, int32_t k, int64_t ldw, float *R,
                         int64_t ldr, void *ws, size_t ws_bytes, void *stream) {
  toc_status st = check_device(d);
  if (st != TOC_OK) return st;
  if (k < 1) return fail(TOC_EINVAL, "k must be >= 1");
  if (ldw < k || ldr < k) return fail(TOC_EINVAL, "ldw and ldr must be >= k");
  if ((!W && d->info.n_cols > 0) || (!R && d->info.n_rows > 0))
    return fail(TOC_EINVAL, "W or R is NULL");
  const int64_t nb = d->info.n_batches;
  if (nb == 0) return TOC_OK;
  hipStream_t s = (hipStream_t)stream;
  const Img im = image_of(d);
  if (k == 1 && k1_fits(d, TOC_OP_RIGHT)) {
    const size_t lds = k1_lds(d, TOC_OP_RIGHT);
    const int lpr = lanes_per_row(d);
    for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
      const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
      switch (lpr) {
#define TOC_RK1(L)                                                                         \
  case L:                                                                                  \
    if ((st = allow_lds(right_k1_kernel<L, kK1RightBlock>, lds))) return st;               \
    hipLaunchKernelGGL((right_k1_kernel<L, kK1RightBlock>), dim3(g), dim3(kK1RightBlock), lds, s, \
                       im, b0, W, ldw, R, ldr);                                            \
    break;
        TOC_RK1(4)
        TOC_RK1(8)
        TOC_RK1(16)
        TOC_RK1(32)
        default: TOC_RK1(64)
#undef TOC_RK1
      }
      if ((st = launch_status("right_k1_kernel"))) return st;
    }
    return TOC_OK;
  }
  const OpPlan plan = plan_op(d, TOC_OP_RIGHT, k);
  if (plan.path == kPathTiled) {
    if (plan.ws_floats > 0 && (!ws || ws_bytes < (size_t)plan.ws_floats * 4))
      return fail(TOC_ESIZE, "workspace of %zu bytes below the %lld needed", ws_bytes,
                  (long long)plan.ws_floats * 4);
    const int m = d->info.n_cols;
    if (plan.compact) {
      if ((st = allow_lds(right_compact_kernel, plan.lds))) return st;
      const uint32_t *cols = (const uint32_t *)((const uint8_t *)d->buf + d->layout.cols);
      hipLaunchKernelGGL(right_compact_kernel, dim3(plan.grid), dim3(kRtBlock), plan.lds, s, im,
                         cols, nb, plan.n_tiles, plan.spx, m, (int)plan.lds_rows, W, ldw, k, R, ldr,
                         (float *)ws, plan.ws_floats / plan.grid);
      return launch_status("right_compact_kernel");
    }
    if (plan.deep_lds) {
      if ((st = allow_lds(right_tiled_kernel, plan.lds))) return st;
      hipLaunchKernelGGL(right_tiled_kernel, dim3(plan.grid), dim3(kRtBlock), plan.lds, s, im, nb,
                         plan.n_tiles, plan.spx, plan.per, m, W, ldw, k, R, ldr);
    } else {
      if ((st = allow_lds(right_staged_kernel, plan.lds))) return st;
      hipLaunchKernelGGL(right_staged_kernel, dim3(plan.grid), dim3(kRtBlock), plan.lds, s, im,
                         nb, plan.n_tiles, plan.spx, m, W, ldw, k, R, ldr, (float *)ws,
                         (int64_t)d->max_deep * kRtKT);
    }
    return launch_status("right_tiled_kernel");
  }
  int64_t cap_rows = 0;
  if ((st = ws_capacity(plan, ws, ws_bytes, cap_rows))) return st;
  for (int64_t k0 = 0; k0 < k; k0 += kKTile) {
    const int kt = (int)std::min<int64_t>(kKTile, k - k0);
    const int kpl = (kt + kWave - 1) / kWave;
    st = for_each_pass(d, TOC_OP_RIGHT, cap_rows,
                       [&](int64_t b0, int64_t n, int64_t base) -> toc_status {
      TOC_DISPATCH_KPL(kpl, right_wide_kernel, dim3((unsigned)n), dim3(kBlock), 0, s, im, b0,
                       base, W + k0, ldw, kt, R + k0, ldr, (float *)ws);
      return launch_status("right_wide_kernel");
    });
    if (st != TOC_OK) return st;
  }
  return TOC_OK;
}

}  // extern "C"

namespace {

// The left product.  fit_workers: the workspace is a fixed buffer (the static
// scratch) that may be smaller than the tiled plan's one slot per worker; the
// tiled kernel then runs with as many persistent workers per XCD as it holds
// slots for (each output element is summed in the same order by whichever worker
// takes it, so the result is the same bit for bit), and shapes whose per-batch
// minimum exceeds it are TOC_EUNSUPPORTED.
toc_status left_mul_impl(const toc_dev *d, const float *G, int32_t k, int64_t ldg, float *out,
                         int64_t ldo, int32_t accumulate, void *ws, size_t ws_bytes, void *stream,
                         bool fit_workers) {
  toc_status st = check_device(d);
  if (st != TOC_OK) return st;
  if (k < 1) return fail(TOC_EINVAL, "k must be >= 1");
  if (ldg < k || ldo < k) return fail(TOC_EINVAL, "ldg and ldo must be >= k");
  if ((!G && d->info.n_rows > 0) || (!out && d->info.n_cols > 0))
    return fail(TOC_EINVAL, "G or out is NULL");
  const int64_t nb = d->info.n_batches;
  if (nb == 0) return TOC_OK;
  const int32_t m = d->info.n_cols;
  hipStream_t s = (hipStream_t)stream;
  const Img im = image_of(d);
  if (k == 1 && k1_fits(d, TOC_OP_LEFT)) {
    const size_t lds = k1_lds(d, TOC_OP_LEFT);
    const bool wide_m = m > 4 * kBlock;      // a pass of 4 columns per thread covers 4 kBlock
    if ((st = allow_lds(wide_m ? left_k1_kernel<8> : left_k1_kernel<4>, lds))) return st;
    const uint8_t *bb = (const uint8_t *)d->buf;
    const uint32_t *occ_off = (const uint32_t *)(bb + d->layout.occ_off);
    const uint32_t *tlist = (const uint32_t *)(bb + d->layout.tlist);
    const uint32_t *cols = (const uint32_t *)(bb + d->layout.cols);
    const uint32_t *tchild = (const uint32_t *)(bb + d->layout.tchild);
    for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
      const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
      if (wide_m)
        hipLaunchKernelGGL(left_k1_kernel<8>, dim3(g), dim3(kBlock), lds, s, im, occ_off, tlist, cols,
                           tchild, b0, m, d->max_rows, d->max_codes, G, ldg, out, ldo, accumulate);
      else
        hipLaunchKernelGGL(left_k1_kernel<4>, dim3(g), dim3(kBlock), lds, s, im, occ_off, tlist, cols,
                           tchild, b0, m, d->max_rows, d->max_codes, G, ldg, out, ldo, accumulate);
      if ((st = launch_status("left_k1_kernel"))) return st;
    }
    return TOC_OK;
  }
  OpPlan plan = plan_op(d, TOC_OP_LEFT, k);
  if (fit_workers && plan.path == kPathTiled && plan.ws_floats > 0) {
    const int64_t slot_bytes = (int64_t)d->max_tree * plan.tw * 4;
    const int64_t max_spx = (int64_t)ws_bytes / (slot_bytes * kXcd);
    if (max_spx < 1)
      return fail(TOC_EUNSUPPORTED,
                  "a worker slot of %lld bytes per XCD (8) exceeds the %zu bytes of static scratch",
                  (long long)slot_bytes, ws_bytes);
    if (plan.spx > max_spx) {
      plan.spx = (int)max_spx;
      plan.grid = (unsigned)(kXcd * plan.spx);
      plan.ws_floats = (int64_t)plan.grid * d->max_tree * plan.tw;
    }
  }
  if (fit_workers && plan.path == kPathWide && plan.row_floats > 0 &&
      plan.rows_max * plan.row_floats * 4 > (int64_t)ws_bytes)
    return fail(TOC_EUNSUPPORTED, "a batch needs %lld bytes of workspace, beyond the %zu of static scratch",
                (long long)(plan.rows_max * plan.row_floats * 4), ws_bytes);
  if (plan.path == kPathTiled) {
    if (plan.ws_floats > 0 && (!ws || ws_bytes < (size_t)plan.ws_floats * 4))
      return fail(TOC_ESIZE, "workspace of %zu bytes below the %lld needed", ws_bytes,
                  (long long)plan.ws_floats * 4);
    const uint8_t *bb = (const uint8_t *)d->buf;
    const uint32_t *occ_off = (const uint32_t *)(bb + d->layout.occ_off);
    const uint32_t *tlist = (const uint32_t *)(bb + d->layout.tlist);
    const uint32_t *cols = (const uint32_t *)(bb + d->layout.cols);
    const uint32_t *tchild = (const uint32_t *)(bb + d->layout.tchild);
    const int64_t slot = plan.deep_lds ? 0 : (int64_t)d->max_tree * plan.tw;
#define TOC_LT_LAUNCH(TW, TL)                                                                  \
  do {                                                                                         \
    if ((st = allow_lds(left_tiled_kernel<TW, TL>, plan.lds))) return st;                       \
    hipLaunchKernelGGL((left_tiled_kernel<TW, TL>), dim3(plan.grid), dim3(kLtBlock), plan.lds, s, \
                       im, occ_off, tlist, cols, tchild, nb, plan.n_tiles, plan.spx,              \
                       d->max_rows, (int)d->max_tree, (int)plan.lds_rows, (int)plan.toc_lds,       \
                       plan.ocr_cap, m, G,                                                          \
                       ldg, k, out, ldo,                                                            \
                       accumulate, (float *)ws, slot);                                          \
  } while (0)
    if (plan.tw == 64) {
      if (plan.deep_lds) TOC_LT_LAUNCH(64, true);
      else TOC_LT_LAUNCH(64, false);
    } else {
      if (plan.deep_lds) TOC_LT_LAUNCH(32, true);
      else TOC_LT_LAUNCH(32, false);
    }
#undef TOC_LT_LAUNCH
    return launch_status("left_tiled_kernel");
  }
  int64_t cap_rows = 0;
  if ((st = ws_capacity(plan, ws, ws_bytes, cap_rows))) return st;
  for (int64_t k0 = 0; k0 < k; k0 += kKTile) {
    const int kt = (int)std::min<int64_t>(kKTile, k - k0);
    const int kpl = (kt + kWave - 1) / kWave;
    const uint8_t *bb = (const uint8_t *)d->buf;
    const uint32_t *occ_off = (const uint32_t *)(bb + d->layout.occ_off);
    const uint32_t *tlist = (const uint32_t *)(bb + d->layout.tlist);
    const uint32_t *cols = (const uint32_t *)(bb + d->layout.cols);
    const uint32_t *tchild = (const uint32_t *)(bb + d->layout.tchild);
    st = for_each_pass(d, TOC_OP_LEFT, cap_rows,
                       [&](int64_t b0, int64_t n, int64_t base) -> toc_status {
      TOC_DISPATCH_KPL(kpl, left_wide_kernel, dim3((unsigned)n), dim3(kBlock), 0, s, im, occ_off,
                       tlist, cols, tchild, b0, base, m, G + k0, ldg, kt, out + k0, ldo,
                       accumulate, (float *)ws);
      return launch_status("left_wide_kernel");
    });
    if (st != TOC_OK) return st;
  }
  return TOC_OK;
}

}  // namespace

extern "C" {

toc_status toc_left_mul(const toc_dev *d, const float *G, int32_t k, int64_t ldg, float *out,
                        int64_t ldo, int32_t accumulate, void *ws, size_t ws_bytes,
                        void *stream) {
  return left_mul_impl(d, G, k, ldg, out, ldo, accumulate, ws, ws_bytes, stream, false);
}

toc_status toc_left_mul_noalloc(const toc_dev *d, const float *G, int32_t k, int64_t ldg,
                                float *out, int64_t ldo, int32_t accumulate, void *stream) {
  toc_status st = check_device(d);
  if (st != TOC_OK) return st;
  void *ws = nullptr;
  if ((st = scratch_address(d->device, &ws))) return st;
  return left_mul_impl(d, G, k, ldg, out, ldo, accumulate, ws, TOC_NOALLOC_SCRATCH_BYTES, stream,
                       true);
}

toc_status toc_decode_csr(const toc_dev *d, int64_t *rowptr, int32_t *col, float *val,
                          void *stream) {
  toc_status st = check_device(d);
  if (st != TOC_OK) return st;
  if (!rowptr || (d->info.nnz > 0 && (!col || !val)))
    return fail(TOC_EINVAL, "NULL output pointer");
  const int64_t nb = d->info.n_batches;
  hipStream_t s = (hipStream_t)stream;
  if (nb == 0) {
    const int64_t zero = 0;
    if (hipMemcpyAsync(rowptr, &zero, sizeof zero, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return fail(TOC_EDEVICE, "rowptr write failed");
    return TOC_OK;
  }
  const Img im = image_of(d);
  // keys and links of every batch in LDS: a workgroup per batch
  const int64_t max_slots = d->max_keylinks;        // keys plus deep links of a batch
  const size_t lds = 8 * (size_t)max_slots + 4 * ((size_t)d->max_rows + 1);
  if (lds <= kDecLdsMax) {
    if ((st = allow_lds(decode_batch_kernel, lds))) return st;
    for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
      const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
      hipLaunchKernelGGL(decode_batch_kernel, dim3(g), dim3(kDbBlock), lds, s, im, b0, rowptr, col,
                         (uint32_t *)val, max_slots);
      if ((st = launch_status("decode_batch_kernel"))) return st;
    }
    return TOC_OK;
  }
  const uint4 *dtiles = (const uint4 *)((const uint8_t *)d->buf + d->layout.dtiles);
  for (int64_t t0 = 0; t0 < d->n_dtiles; t0 += (1 << 30)) {
    const int64_t n = std::min<int64_t>(d->n_dtiles - t0, 1 << 30);
    const unsigned g = (unsigned)(((n + kXcd - 1) / kXcd) * kXcd);
    hipLaunchKernelGGL(decode_kernel, dim3(g), dim3(kDecBlock), 0, s, im, dtiles, t0, n, rowptr,
                       col, (uint32_t *)val);
    if ((st = launch_status("decode_kernel"))) return st;
  }
  return TOC_OK;
}

toc_status toc_map_values(const toc_dev *d, int32_t op, float c, void *stream) {
  toc_status st = check_device(d);
  if (st != TOC_OK) return st;
  if (op != TOC_MAP_SCALE && op != TOC_MAP_SQUARE) return fail(TOC_EINVAL, "unknown op %d", op);
  if (op == TOC_MAP_SCALE && !std::isfinite(c)) return fail(TOC_EINVAL, "c is not finite");
  const int64_t n = d->info.n_stored;
  if (n == 0) return TOC_OK;
  uint8_t *bb = (uint8_t *)d->buf;
  const int64_t blocks = std::min<int64_t>((n + kMapBlock - 1) / kMapBlock, 64 * 256);
  const int64_t n_cval = (d->layout.end - d->layout.cval) / 4;
  hipLaunchKernelGGL(map_values_kernel, dim3((unsigned)blocks), dim3(kMapBlock), 0,
                     (hipStream_t)stream, (toc_key *)(bb + d->layout.key), n,
                     (uint32_t *)(bb + d->layout.cval), n_cval, (int)op, c);
  return launch_status("map_values_kernel");
}

toc_status toc_decode_dense(const toc_dev *d, float c, float *A, int64_t lda, void *stream) {
  toc_status st = check_device(d);
  if (st != TOC_OK) return st;
  const int m = d->info.n_cols;
  if (!std::isfinite(c)) return fail(TOC_EINVAL, "c is not finite");
  if (lda < m) return fail(TOC_EINVAL, "lda %lld < n_cols %d", (long long)lda, m);
  if (!A && d->info.n_rows > 0 && m > 0) return fail(TOC_EINVAL, "A is NULL");
  const int64_t nb = d->info.n_batches;
  if (nb == 0 || d->info.n_rows == 0 || m == 0) return TOC_OK;
  const Img im = image_of(d);
  hipStream_t s = (hipStream_t)stream;
  const size_t lds = (size_t)kDnWaves * m * sizeof(float);
  const bool row_lds = lds <= kLdsMax;
  if (row_lds && (st = allow_lds(decode_dense_kernel<true>, lds))) return st;
  for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
    const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
    if (row_lds)
      hipLaunchKernelGGL(decode_dense_kernel<true>, dim3(g), dim3(kDnBlock), lds, s, im, b0, m, c,
                         A, lda);
    else
      hipLaunchKernelGGL(decode_dense_kernel<false>, dim3(g), dim3(kDnBlock), 0, s, im, b0, m, c,
                         A, lda);
    if ((st = launch_status("decode_dense_kernel"))) return st;
  }
  return TOC_OK;
}

}  // extern "C"
