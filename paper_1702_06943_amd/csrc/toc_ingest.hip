// The upload image built on the device from physical bytes.  Each batch arrives
// as section 3.2's bit-packed (I, D) (read back as in section 4.1.1); the decoding
// tree C' is built by Algorithm 2 (the tree kernel toc_cprime_build launches), and
// the arrays the operations read are derived from it by one workgroup per batch:
// the stored codes in level order (parents before children, as the forward scan
// of Algorithm 4 and the backward scan of Algorithm 5 need), their keys and links,
// D renumbered, D inverted (the index set of the sums that define G(x) in Theorem
// 2), the column index and entries of the left multiplication, the children of
// each tree code and the decode tiles.  The image is the one toc_upload builds on
// the host from the same batches, word for word, so every operation gives the same
// results on either; only the compressed bytes cross from the host.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "toc_internal.h"
#include "toc_phys_dev.h"

namespace {

using namespace tocphys;
using toc::fail;

constexpr int kIgBlock = kCpBlock;          // the scan helper's workgroup size
constexpr int kIgWaves = kCpWaves;
constexpr int kIgGrid = 512;                // persistent workgroups, one scratch slot each
constexpr uint32_t kLive = 1u, kHasChild = 2u;
constexpr int kCensus = 8;                  // int64 counts per batch from the census

inline int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Tuple holding entry p of D (st: the n_r + 1 tuple starts; empty tuples are
// skipped, as the last tuple starting at or before p is the one holding it).
__device__ inline uint32_t tuple_of(const uint32_t *st, uint32_t n_r, uint32_t p) {
  uint32_t lo = 0, hi = n_r;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (st[mid] <= p) lo = mid;
    else hi = mid;
  }
  return lo;
}

// First tuple (0..n_r) whose start is at or after entry p.
__device__ inline uint32_t first_start_from(const uint32_t *st, uint32_t n_r, uint32_t p) {
  uint32_t lo = 0, hi = n_r;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) / 2;
    if (st[mid] < p) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// One step of an exclusive scan over a sequence taken kIgBlock items at a time:
// this thread's prefix, carry included; carry advances by the chunk's total.
__device__ inline uint32_t scan_step(uint32_t x, uint32_t *wsum, uint32_t &carry) {
  uint32_t tot;
  const uint32_t ex = block_excl_scan(x, wsum, tot);
  const uint32_t r = carry + ex;
  carry += tot;
  return r;
}

// Bits needed for keys below n (0 for n <= 1).
__device__ inline int key_bits(uint32_t n) { return n <= 1u ? 0 : 32 - __clz(n - 1u); }

// Marks a batch's live codes (kLive: the codes of D and all their ancestors, the
// only nodes the operations of section 4 touch; the walk up from an entry of D
// stops at the first node already marked) and the nodes with a live child
// (kHasChild).  flags: one word per node, cleared here.
__device__ void mark_live(const uint8_t *p_d, uint32_t w_d, uint32_t n_d, uint32_t n_nodes,
                          const uint32_t *par, uint32_t *flags) {
  for (uint32_t c = threadIdx.x; c < n_nodes; c += kIgBlock) flags[c] = 0u;
  __syncthreads();
  for (uint32_t p = threadIdx.x; p < n_d; p += kIgBlock) {
    uint32_t c = rd(p_d, p, w_d);
    while (c != 0u && (atomicOr(&flags[c], kLive) & kLive) == 0u) c = par[c];
  }
  __syncthreads();
  for (uint32_t c = 1 + threadIdx.x; c < n_nodes; c += kIgBlock)
    if ((flags[c] & kLive) && par[c] != 0u) atomicOr(&flags[par[c]], kHasChild);
  __syncthreads();
}

// Stable sort of n pairs (key below 2^bits, value) by key, 8 bits a pass, one
// workgroup.  A pass counts the digits, then places the pairs chunk by chunk of
// kIgBlock, each after the earlier pairs of its digit: those of earlier chunks
// (run), of earlier waves of its chunk (wcnt) and of lower lanes of its wave
// (found with eight ballots, one per digit bit).  wcnt must be zero on entry and
// is left zero.  Returns 1 when the result is in (k1, v1), 0 when in (k0, v0).
__device__ int block_radix_sort(uint32_t *k0, uint32_t *v0, uint32_t *k1, uint32_t *v1, uint32_t n,
                                int bits, uint32_t *run, uint32_t *wcnt, uint32_t *wsum) {
  const int tid = threadIdx.x, lane = tid % kCpWave, wave = tid / kCpWave;
  int src = 0;
  for (int sh = 0; sh < bits; sh += 8) {
    const uint32_t *ki = src ? k1 : k0, *vi = src ? v1 : v0;
    uint32_t *ko = src ? k0 : k1, *vo = src ? v0 : v1;
    if (tid < 256) run[tid] = 0u;
    __syncthreads();
    for (uint32_t e = tid; e < n; e += kIgBlock) atomicAdd(&run[(ki[e] >> sh) & 255u], 1u);
    __syncthreads();
    uint32_t tot;
    const uint32_t ex = block_excl_scan(tid < 256 ? run[tid] : 0u, wsum, tot);
    if (tid < 256) run[tid] = ex;
    __syncthreads();
    for (uint32_t e0 = 0; e0 < n; e0 += kIgBlock) {
      const uint32_t e = e0 + tid;
      const bool in = e < n;
      const uint32_t key = in ? ki[e] : 0u, val = in ? vi[e] : 0u, dg = (key >> sh) & 255u;
      uint64_t peers = __ballot(in);
#pragma unroll
      for (int bit = 0; bit < 8; ++bit) {
        const bool set = (dg >> bit) & 1u;
        const uint64_t bb = __ballot(set);
        peers &= set ? bb : ~bb;
      }
      const uint32_t rank = (uint32_t)__popcll(peers & ((1ull << lane) - 1ull));
      if (in && rank == 0u) wcnt[wave * 256 + dg] = (uint32_t)__popcll(peers);
      __syncthreads();
      if (in) {
        uint32_t pos = run[dg] + rank;
        for (int w = 0; w < wave; ++w) pos += wcnt[w * 256 + dg];
        ko[pos] = key;
        vo[pos] = val;
      }
      __syncthreads();
      if (tid < 256) {
        uint32_t s = 0;
        for (int w = 0; w < kIgWaves; ++w) {
          s += wcnt[w * 256 + tid];
          wcnt[w * 256 + tid] = 0u;
        }
        run[tid] += s;
      }
      __syncthreads();
    }
    src ^= 1;
  }
  return src;
}

// Per batch, the counts the image layout depends on (written to counts[8 b ..]):
// live codes, deepest live depth, depth-1 codes with live children, live codes of
// depth >= 2, nonzeros (the sum of the depths of D's codes: each code decodes to
// that many pairs), live depth-1 codes, and distinct key columns of live codes.
__global__ __launch_bounds__(kIgBlock) void census_kernel(
    const uint8_t *__restrict__ blobs, const int64_t *__restrict__ offs, int64_t n_batches,
    uint32_t n_cols, const int32_t *__restrict__ cp_status, const uint32_t *__restrict__ parent,
    const uint32_t *__restrict__ col, const uint32_t *__restrict__ depth,
    uint32_t *__restrict__ flags_all, uint32_t *__restrict__ colbits_all,
    int64_t *__restrict__ counts, int32_t *__restrict__ status) {
  __shared__ Hdr h;
  __shared__ unsigned long long s_nnz;
  __shared__ uint32_t s_live, s_top, s_int1, s_deep, s_lvl1, s_ucols;
  const int64_t *node_off = offs + (n_batches + 1);
  const uint32_t ncw = (n_cols + 31) / 32;
  uint32_t *colbits = colbits_all + (int64_t)blockIdx.x * ncw;
  for (int64_t b = blockIdx.x; b < n_batches; b += gridDim.x) {
    const uint8_t *blob = blobs + offs[b];
    const uint64_t size = (uint64_t)(offs[b + 1] - offs[b]);
    const int64_t no = node_off[b];
    const uint32_t n_nodes = (uint32_t)(node_off[b + 1] - no);
    if (threadIdx.x == 0) {
      h.err = cp_status[b];
      if (h.err == 0) parse_headers(blob, size, 1 << 30, h);
      s_nnz = 0ull;
      s_live = s_top = s_int1 = s_deep = s_lvl1 = s_ucols = 0u;
    }
    __syncthreads();
    if (h.err) {
      if (threadIdx.x == 0) {
        status[b] = h.err;
        for (int q = 0; q < kCensus; ++q) counts[kCensus * b + q] = 0;
      }
      __syncthreads();
      continue;
    }
    const uint32_t n_d = h.cnt[3], w_d = h.w[3];
    const uint8_t *p_d = blob + h.data[3];
    const uint32_t *par = parent + no, *cl = col + no, *dep = depth + no;
    uint32_t *fl = flags_all + no;
    mark_live(p_d, w_d, n_d, n_nodes, par, fl);
    for (uint32_t x = threadIdx.x; x < ncw; x += kIgBlock) colbits[x] = 0u;
    __syncthreads();
    uint32_t live = 0, top = 0, int1 = 0, deep = 0, lvl1 = 0;
    for (uint32_t c = 1 + threadIdx.x; c < n_nodes; c += kIgBlock) {
      const uint32_t f = fl[c];
      if (!(f & kLive)) continue;
      const uint32_t d = dep[c];
      ++live;
      top = max(top, d);
      if (d == 1u) {
        ++lvl1;
        int1 += (f & kHasChild) ? 1u : 0u;
      } else {
        ++deep;
      }
      atomicOr(&colbits[cl[c] / 32], 1u << (cl[c] % 32));
    }
    unsigned long long nnz = 0;
    for (uint32_t p = threadIdx.x; p < n_d; p += kIgBlock) nnz += dep[rd(p_d, p, w_d)];
    atomicAdd(&s_live, live);
    atomicMax(&s_top, top);
    atomicAdd(&s_int1, int1);
    atomicAdd(&s_deep, deep);
    atomicAdd(&s_lvl1, lvl1);
    atomicAdd(&s_nnz, nnz);
    __syncthreads();
    uint32_t u = 0;
    for (uint32_t x = threadIdx.x; x < ncw; x += kIgBlock) u += (uint32_t)__popc(colbits[x]);
    atomicAdd(&s_ucols, u);
    __syncthreads();
    if (threadIdx.x == 0) {
      int64_t *o = counts + kCensus * b;
      o[0] = s_live;
      o[1] = s_top;
      o[2] = s_int1;
      o[3] = s_deep;
      o[4] = (int64_t)s_nnz;
      o[5] = s_lvl1;
      o[6] = s_ucols;
      o[7] = 0;
      status[b] = 0;
    }
    __syncthreads();
  }
}

struct IgParams {
  const uint8_t *blobs;
  // n + 1 entries each: blob offsets (into blobs), node offsets and D offsets (into
  // the range's scratch, from 0), first decode tile of each batch (in the image)
  const int64_t *offs;
  int64_t n;                    // batches in the range
  int64_t b0;                   // image index of the range's first batch
  int max_rows;
  uint32_t n_cols;
  const int32_t *cp_status;
  const uint32_t *parent, *col, *val, *depth;   // C', paper numbering
  // scratch, one word per node: flags, place of each code, start of each code's
  // group in the inverted D, size of that group, code at each place, code at each
  // position of the left multiplication (as a place)
  uint32_t *flags, *newidx, *gst, *gsz, *at, *atl;
  uint32_t *occ;                // the inverted D: entries of D grouped by code
  uint32_t *g;                  // live children before each entry of occ (+1 per batch)
  uint32_t *sortbuf;            // 4 sort_len words per workgroup
  int64_t sort_len;
  uint8_t *img;
  toc_layout L;
  int32_t *status;
};

#define IG_FAIL(code)                                  \
  do {                                                 \
    if (threadIdx.x == 0) P.status[i] = (code);        \
    __syncthreads();                                   \
    goto next_batch;                                   \
  } while (0)

// The image arrays of each batch of the range (see toc_dev_layout_get for their
// meaning), at the offsets of the batch table the host wrote into the image.
__global__ __launch_bounds__(kIgBlock) void image_kernel(IgParams P) {
  extern __shared__ uint32_t sm[];              // tuple starts, then nonempty tuples before each
  __shared__ Hdr h;
  __shared__ uint32_t wsum[kIgWaves];
  __shared__ uint32_t run[256], wcnt[kIgWaves * 256];
  __shared__ uint32_t s_live, s_int1, s_top, s_max;
  uint32_t *st = sm, *nes = sm + (P.max_rows + 1);
  const int64_t n = P.n;
  const int64_t *node_off = P.offs + (n + 1), *d_off = P.offs + 2 * (n + 1),
                *dt_off = P.offs + 3 * (n + 1);
  const int tid = threadIdx.x;
  uint32_t *sk0 = P.sortbuf + (int64_t)blockIdx.x * 4 * P.sort_len, *sv0 = sk0 + P.sort_len;
  uint32_t *sk1 = sv0 + P.sort_len, *sv1 = sk1 + P.sort_len;
  const uint32_t m = P.n_cols;
  const int cbits = key_bits(m);
  for (int x = tid; x < kIgWaves * 256; x += kIgBlock) wcnt[x] = 0u;
  for (int64_t i = blockIdx.x; i < n; i += gridDim.x) {
    {
      const int64_t b = P.b0 + i;
      const uint8_t *blob = P.blobs + P.offs[i];
      const uint64_t size = (uint64_t)(P.offs[i + 1] - P.offs[i]);
      const int64_t no = node_off[i], dof = d_off[i];
      const uint32_t n_nodes = (uint32_t)(node_off[i + 1] - no);
      const toc_batch bt = ((const toc_batch *)(P.img + P.L.batches))[b];
      if (tid == 0) {
        h.err = P.cp_status[i];
        if (h.err == 0) parse_headers(blob, size, P.max_rows, h);
        if (h.err == 0 && ((int64_t)h.cnt[3] != d_off[i + 1] - dof || (int64_t)h.cnt[3] != bt.n_d ||
                           (int64_t)h.cnt[4] - 1 != bt.n_rows))
          h.err = TOC_INGEST_CHANGED;
        s_live = s_int1 = s_top = s_max = 0u;
      }
      __syncthreads();
      if (h.err) IG_FAIL(h.err);
      const uint32_t nI = h.cnt[0], n_d = h.cnt[3], n_r = h.cnt[4] - 1;
      const uint8_t *p_d = blob + h.data[3], *p_st = blob + h.data[4];
      const uint32_t w_d = h.w[3], w_st = h.w[4];
      const uint32_t *par = P.parent + no, *cl = P.col + no, *vl = P.val + no, *dep = P.depth + no;
      uint32_t *fl = P.flags + no, *nx = P.newidx + no, *gs = P.gst + no, *gz = P.gsz + no;
      uint32_t *at = P.at + no, *atl = P.atl + no;
      uint32_t *occ = P.occ + dof, *g = P.g + dof + i;
      const uint32_t L = (uint32_t)bt.n_levels, nc = (uint32_t)bt.n_codes;
      const uint32_t ni = (uint32_t)bt.n_int1, n1 = (uint32_t)bt.n_lvl1;
      const uint32_t ntree = ni + (nc - n1);
      uint32_t carry;

      // tuple starts, and the nonempty tuples before each: the entry at p of tuple
      // r makes node nI + 1 + p - nes[r] of C' unless it ends its tuple
      for (uint32_t r = tid; r <= n_r; r += kIgBlock) st[r] = rd(p_st, r, w_st);
      __syncthreads();
      carry = 0;
      for (uint32_t r0 = 0; r0 < n_r; r0 += kIgBlock) {
        const uint32_t r = r0 + tid;
        const uint32_t v = scan_step(r < n_r && st[r + 1] > st[r] ? 1u : 0u, wsum, carry);
        if (r < n_r) nes[r] = v;
      }
      mark_live(p_d, w_d, n_d, n_nodes, par, fl);

      // level offsets: live codes per depth, then running sums
      uint32_t *lv = (uint32_t *)(P.img + P.L.level) + bt.lvl_base;
      {
        uint32_t live = 0, int1 = 0, top = 0;
        for (uint32_t c = 1 + tid; c < n_nodes; c += kIgBlock) {
          const uint32_t f = fl[c];
          if (!(f & kLive)) continue;
          const uint32_t d = dep[c];
          ++live;
          top = max(top, d);
          if (d == 1u && (f & kHasChild)) ++int1;
          if (d >= 1u && d <= L) atomicAdd(&lv[d], 1u);
        }
        atomicAdd(&s_live, live);
        atomicAdd(&s_int1, int1);
        atomicMax(&s_top, top);
      }
      __syncthreads();
      if (s_live != nc || s_int1 != ni || s_top != L) IG_FAIL(TOC_INGEST_CHANGED);
      carry = 0;
      for (uint32_t d0 = 1; d0 <= L; d0 += kIgBlock) {
        const uint32_t d = d0 + tid;
        const uint32_t x = d <= L ? lv[d] : 0u;
        const uint32_t v = scan_step(x, wsum, carry);
        if (d <= L) lv[d] = v + x;
      }
      __syncthreads();
      if ((L >= 1 ? lv[1] : 0u) != n1) IG_FAIL(TOC_INGEST_CHANGED);

      // D inverted by code: group sizes, their starts, then the entries tuple by
      // tuple (a code occurs at most once in a tuple, so the entries of one tuple
      // take the next place of their groups in any order, and every group lists its
      // entries in the order of D)
      for (uint32_t c = tid; c < n_nodes; c += kIgBlock) gz[c] = 0u;
      __syncthreads();
      for (uint32_t p = tid; p < n_d; p += kIgBlock) atomicAdd(&gz[rd(p_d, p, w_d)], 1u);
      __syncthreads();
      carry = 0;
      for (uint32_t c0 = 0; c0 < n_nodes; c0 += kIgBlock) {
        const uint32_t c = c0 + tid;
        const uint32_t v = scan_step(c < n_nodes ? gz[c] : 0u, wsum, carry);
        if (c < n_nodes) gs[c] = v;
      }
      for (uint32_t c = tid; c < n_nodes; c += kIgBlock) gz[c] = 0u;
      __syncthreads();
      for (uint32_t r = 0; r < n_r; ++r) {
        for (uint32_t p = st[r] + tid; p < st[r + 1]; p += kIgBlock) {
          const uint32_t c = rd(p_d, p, w_d);
          occ[gs[c] + atomicAdd(&gz[c], 1u)] = p;
        }
        __syncthreads();
      }

      // places of depth-1 codes with children: 0 .. ni-1, in node order
      carry = 0;
      for (uint32_t c0 = 1; c0 <= nI; c0 += kIgBlock) {
        const uint32_t c = c0 + tid;
        const bool x = c <= nI && (fl[c] & (kLive | kHasChild)) == (kLive | kHasChild);
        const uint32_t v = scan_step(x ? 1u : 0u, wsum, carry);
        if (x) {
          nx[c] = v;
          at[v] = c;
        }
      }
      // places of depth-1 leaves: ni .. n1-1, in the order of their first entry in D
      carry = 0;
      for (uint32_t p0 = 0; p0 < n_d; p0 += kIgBlock) {
        const uint32_t p = p0 + tid;
        const uint32_t c = p < n_d ? rd(p_d, p, w_d) : 0u;
        const bool x = p < n_d && dep[c] == 1u && !(fl[c] & kHasChild) && occ[gs[c]] == p;
        const uint32_t v = scan_step(x ? 1u : 0u, wsum, carry);
        if (x) {
          nx[c] = ni + v;
          at[ni + v] = c;
        }
      }
      if (ni + carry != n1) IG_FAIL(TOC_INGEST_CHANGED);
      // the entry at place e of the inverted D makes a child of its code (the node
      // made there) unless it ends its tuple; g[e] counts the live ones before e
      carry = 0;
      for (uint32_t e0 = 0; e0 < n_d; e0 += kIgBlock) {
        const uint32_t e = e0 + tid;
        uint32_t x = 0;
        if (e < n_d) {
          const uint32_t p = occ[e], r = tuple_of(st, n_r, p);
          if (p + 1 < st[r + 1]) x = (fl[nI + 1 + p - nes[r]] & kLive) ? 1u : 0u;
        }
        const uint32_t v = scan_step(x, wsum, carry);
        if (e < n_d) g[e] = v;
      }
      if (tid == 0) g[n_d] = carry;
      if (n1 + carry != nc) IG_FAIL(TOC_INGEST_CHANGED);
      __syncthreads();

      // levels 2 .. L: the children of the codes of each level, parent by parent in
      // place order and each parent's in node order (the order of D), from place
      // n1 on; the start of each tree code's children is its tchild entry
      uint32_t *tch = (uint32_t *)(P.img + P.L.tchild) + bt.tree_base + b;
      carry = 0;
      for (uint32_t d = 1; d < L; ++d) {
        const uint32_t q_end = lv[d];
        for (uint32_t q0 = lv[d - 1]; q0 < q_end; q0 += kIgBlock) {
          const uint32_t q = q0 + tid;
          const bool in = q < q_end;
          const uint32_t c = in ? at[q] : 0u;
          const uint32_t ga = in ? gs[c] : 0u, ge = in ? gs[c] + gz[c] : 0u;
          const uint32_t nch = in ? g[ge] - g[ga] : 0u;
          const uint32_t base = n1 + scan_step(nch, wsum, carry);
          if (in && (q < ni || q >= n1)) tch[q < ni ? q : q - n1 + ni] = base;
          if (nch) {
            for (uint32_t e = ga; e < ge; ++e) {
              if (g[e + 1] == g[e]) continue;
              const uint32_t p = occ[e], r = tuple_of(st, n_r, p);
              const uint32_t x = nI + 1 + p - nes[r], pos = base + (g[e] - g[ga]);
              nx[x] = pos;
              at[pos] = x;
            }
          }
        }
        __syncthreads();
      }
      if (L >= 2)
        for (uint32_t q = lv[L - 1] + tid; q < lv[L]; q += kIgBlock) tch[q - n1 + ni] = nc;
      if (tid == 0) tch[ntree] = nc;
      __syncthreads();

      // keys by place, links of the codes of depth >= 2 (by place - n1); tuple
      // starts; D renumbered
      {
        toc_key *key = (toc_key *)(P.img + P.L.key) + bt.code_base;
        toc_link *lk = (toc_link *)(P.img + P.L.link) + bt.deep_base;
        for (uint32_t q = tid; q < nc; q += kIgBlock) {
          const uint32_t c = at[q], d = dep[c];
          toc_key k;
          k.col = cl[c];
          k.val = __uint_as_float(vl[c]);
          key[q] = k;
          if (q >= n1) {
            toc_link l;
            l.parent = nx[par[c]];
            l.depth = d;
            lk[q - n1] = l;
          }
        }
        uint32_t *span = (uint32_t *)(P.img + P.L.span) + bt.span_base;
        for (uint32_t r = tid; r <= n_r; r += kIgBlock) span[r] = st[r];
        uint32_t *dc = (uint32_t *)(P.img + P.L.dcodes) + bt.d_base;
        for (uint32_t p = tid; p < n_d; p += kIgBlock) dc[p] = nx[rd(p_d, p, w_d)];
      }

      // positions of the left multiplication: the leaves by (key column, place)
      for (uint32_t x = tid; x < n1 - ni; x += kIgBlock) {
        sk0[x] = cl[at[ni + x]];
        sv0[x] = ni + x;
      }
      __syncthreads();
      {
        const uint32_t *srt =
            block_radix_sort(sk0, sv0, sk1, sv1, n1 - ni, cbits, run, wcnt, wsum) ? sv1 : sv0;
        for (uint32_t q = tid; q < nc; q += kIgBlock) atl[q] = (q >= ni && q < n1) ? srt[q - ni] : q;
      }
      __syncthreads();
      // the left multiplication's entries (centry, cval), first part: the tuples of
      // each leaf position's entries of D, ascending, bit 31 on the first, the
      // key value beside each; lo: where each leaf position's start
      uint32_t *ce = (uint32_t *)(P.img + P.L.centry) + bt.d_base + bt.tree_base;
      uint32_t *cv = (uint32_t *)(P.img + P.L.cval) + bt.d_base + bt.tree_base;
      uint32_t *lo = (uint32_t *)(P.img + P.L.occ_off) + bt.code_base + 2 * b;
      uint32_t *to = lo + (n1 - ni) + 1;
      carry = 0;
      for (uint32_t q0 = ni; q0 < n1; q0 += kIgBlock) {
        const uint32_t q = q0 + tid;
        const uint32_t c = q < n1 ? at[atl[q]] : 0u, cnt = q < n1 ? gz[c] : 0u;
        const uint32_t v = scan_step(cnt, wsum, carry);
        if (q < n1) {
          lo[q - ni] = v;
          const uint32_t ga = gs[c];
          for (uint32_t x = 0; x < cnt; ++x) {
            ce[v + x] = tuple_of(st, n_r, occ[ga + x]) | (x == 0 ? 0x80000000u : 0u);
            cv[v + x] = vl[c];
          }
        }
      }
      const uint32_t n_lo = carry;      // leaf occurrences; the tree codes' entries follow
      if (tid == 0) lo[n1 - ni] = n_lo;
      // tree codes (depth-1 codes with children, codes of depth >= 2) by (key
      // column, place)
      for (uint32_t t = tid; t < ntree; t += kIgBlock) {
        const uint32_t q = t < ni ? t : n1 + (t - ni);
        sk0[t] = cl[at[q]];
        sv0[t] = q;
      }
      __syncthreads();
      uint32_t *tl = (uint32_t *)(P.img + P.L.tlist) + bt.tree_base;
      {
        const uint32_t *srt =
            block_radix_sort(sk0, sv0, sk1, sv1, ntree, cbits, run, wcnt, wsum) ? sv1 : sv0;
        for (uint32_t t = tid; t < ntree; t += kIgBlock) {
          const uint32_t q = srt[t];
          tl[t] = q;
          // second part of the entries: the tree codes by (column, place)
          ce[n_lo + t] = q | toc::kTreeEntry;
          cv[n_lo + t] = vl[at[q]];
        }
      }
      // third part: the tuples of each tree code's entries of D, ascending, by tree
      // row; to: where each tree row's start
      carry = n_lo + ntree;
      for (uint32_t h0 = 0; h0 < ntree; h0 += kIgBlock) {
        const uint32_t h = h0 + tid;
        const uint32_t c = h < ntree ? at[h < ni ? h : n1 + (h - ni)] : 0u;
        const uint32_t cnt = h < ntree ? gz[c] : 0u;
        const uint32_t v = scan_step(cnt, wsum, carry);
        if (h < ntree) {
          to[h] = v;
          const uint32_t ga = gs[c];
          for (uint32_t x = 0; x < cnt; ++x) ce[v + x] = tuple_of(st, n_r, occ[ga + x]);
        }
      }
      if (tid == 0) to[ntree] = carry;
      __syncthreads();

      // column index: per key column its leaves, their occurrences and its tree
      // codes, counted then summed up to each column (entry m closes the sums)
      uint32_t *cx = (uint32_t *)(P.img + P.L.cols) + b * 4 * ((int64_t)m + 1);
      uint32_t *c_code = cx, *c_occ = cx + (m + 1), *c_tree = cx + 2 * (m + 1), *c_ord = cx + 3 * (m + 1);
      for (uint32_t q = ni + tid; q < n1; q += kIgBlock) {
        const uint32_t c = at[atl[q]];
        atomicAdd(&c_code[cl[c]], 1u);
        atomicAdd(&c_occ[cl[c]], gz[c]);
      }
      for (uint32_t t = tid; t < ntree; t += kIgBlock) atomicAdd(&c_tree[cl[at[tl[t]]]], 1u);
      __syncthreads();
      {
        uint32_t ca = 0, co = 0, ct = 0, mx = 0;
        for (uint32_t j0 = 0; j0 <= m; j0 += kIgBlock) {
          const uint32_t j = j0 + tid;
          const bool in = j <= m;
          const uint32_t a = in ? c_code[j] : 0u, o = in ? c_occ[j] : 0u, t = in ? c_tree[j] : 0u;
          const uint32_t va = scan_step(a, wsum, ca), vo = scan_step(o, wsum, co);
          const uint32_t vt = scan_step(t, wsum, ct);
          if (in) {
            c_code[j] = ni + va;
            c_occ[j] = vo;
            c_tree[j] = vt;
          }
          if (j < m) {
            sk0[j] = o + t;
            sv0[j] = j;
            mx = max(mx, o + t);
          }
        }
        atomicMax(&s_max, mx);
      }
      __syncthreads();
      // the columns by entries (leaf occurrences plus tree codes), most first, lower
      // column first among equals
      {
        const uint32_t top = s_max;
        for (uint32_t j = tid; j < m; j += kIgBlock) sk0[j] = top - sk0[j];
        __syncthreads();
        const uint32_t *srt =
            block_radix_sort(sk0, sv0, sk1, sv1, m, key_bits(top + 1u), run, wcnt, wsum) ? sv1 : sv0;
        for (uint32_t j = tid; j < m; j += kIgBlock) c_ord[j] = srt[j];
      }
      // decode tiles: per run of kDecodeTile entries of D, the batch, the first
      // entry, the pairs before it in the batch, the first tuple starting at or
      // after it
      {
        uint32_t *dt = (uint32_t *)(P.img + P.L.dtiles) + 4 * dt_off[i];
        constexpr uint32_t kTile = (uint32_t)toc::kDecodeTile;
        carry = 0;
        for (uint32_t p0 = 0; p0 < n_d; p0 += kIgBlock) {
          const uint32_t p = p0 + tid;
          const uint32_t v = scan_step(p < n_d ? dep[rd(p_d, p, w_d)] : 0u, wsum, carry);
          if (p < n_d && p % kTile == 0u) {
            uint32_t *e = dt + 4 * (p / kTile);
            e[0] = (uint32_t)b;
            e[1] = p;
            e[2] = v;
            e[3] = first_start_from(st, n_r, p);
          }
        }
        if (n_d == 0u && tid == 0) {
          dt[0] = (uint32_t)b;
          dt[1] = dt[2] = dt[3] = 0u;
        }
      }
      if (tid == 0) P.status[i] = 0;
      __syncthreads();
    }
  next_batch:;
  }
}

// ---------------------------------------------------------------------------
// Host side: batch ranges that fit the workspace, and the two entry points.
// ---------------------------------------------------------------------------
struct RangeWs {
  int64_t offs, parent, col, val, depth, s0, s1, s2, s3, s4, flags, occ, g, status, counts, slot,
      end;
};

// Workspace layout for batches b0 .. b1-1 (nodes, D entries and the sort length
// per workgroup given).
RangeWs range_ws(int64_t nb, int64_t nodes, int64_t nd, int64_t sort_len, int64_t colwords) {
  RangeWs w;
  int64_t o = 0;
  const int64_t a = align256(4 * nodes);
  w.offs = o; o = align256(o + 8 * 4 * (nb + 1));
  w.parent = o; o += a;
  w.col = o; o += a;
  w.val = o; o += a;
  w.depth = o; o += a;
  w.s0 = o; o += a;
  w.s1 = o; o += a;
  w.s2 = o; o += a;
  w.s3 = o; o += a;
  w.s4 = o; o += a;
  w.flags = o; o += a;
  w.occ = o; o = align256(o + 4 * nd);
  w.g = o; o = align256(o + 4 * (nd + nb));
  w.status = o; o = align256(o + 4 * nb);
  w.counts = o; o = align256(o + 8 * kCensus * nb);
  w.slot = o;
  const int64_t g = std::min<int64_t>(nb, kIgGrid);
  o = align256(o + g * 4 * std::max(4 * sort_len, colwords));
  w.end = o;
  return w;
}

struct Batches {
  const toc_phys_info *info;
  int64_t n;
  int32_t n_cols;
  std::vector<int64_t> node_off, d_off;   // over all batches
};

// What a range's workspace is sized for: the census (no sorts), the build (sorts
// of up to the stored codes or the columns of a batch), or either, before the
// stored codes are known (bounded by the nodes).
enum WsFor { kWsCensus, kWsBuild, kWsBound };

int64_t sort_len_of(const Batches &B, int64_t b0, int64_t b1, const toc_dev *dev, WsFor what) {
  if (what == kWsCensus) return 0;
  int64_t s = std::max<int64_t>(B.n_cols, 1);
  for (int64_t b = b0; b < b1; ++b)
    s = std::max<int64_t>(s, what == kWsBuild ? dev->batches[(size_t)b].n_codes : B.info[b].n_nodes);
  return s;
}

RangeWs ws_for(const Batches &B, int64_t b0, int64_t b1, const toc_dev *dev, WsFor what) {
  return range_ws(b1 - b0, B.node_off[(size_t)b1] - B.node_off[(size_t)b0],
                  B.d_off[(size_t)b1] - B.d_off[(size_t)b0], sort_len_of(B, b0, b1, dev, what),
                  what == kWsBuild ? 0 : ((int64_t)B.n_cols + 31) / 32);
}

toc_status check_batches(const toc_phys_info *info, int64_t n, int32_t n_cols, Batches &B) {
  if (n < 0) return fail(TOC_EINVAL, "n_batches < 0");
  if (n > 0 && !info) return fail(TOC_EINVAL, "info is NULL");
  if (n_cols < 0) return fail(TOC_EINVAL, "n_cols < 0");
  B.info = info;
  B.n = n;
  B.n_cols = n_cols;
  B.node_off.assign((size_t)n + 1, 0);
  B.d_off.assign((size_t)n + 1, 0);
  for (int64_t b = 0; b < n; ++b) {
    const toc_phys_info &f = info[b];
    if (f.n_rows < 0 || f.n_rows > kCpMaxRows)
      return fail(TOC_EUNSUPPORTED, "batch %lld: %lld tuples (at most %d)", (long long)b,
                  (long long)f.n_rows, kCpMaxRows);
    if (f.n_nodes < 1 || f.n_nodes > (int64_t)INT32_MAX || f.n_codes < 0 ||
        f.n_codes > (int64_t)INT32_MAX || f.n_first < 0 || f.n_first >= f.n_nodes)
      return fail(TOC_EINVAL, "batch %lld: counts out of range", (long long)b);
    if (f.max_col >= n_cols) return fail(TOC_EINVAL, "batch %lld: column %lld not below n_cols %d",
                                         (long long)b, (long long)f.max_col, n_cols);
    B.node_off[(size_t)b + 1] = B.node_off[(size_t)b] + f.n_nodes;
    B.d_off[(size_t)b + 1] = B.d_off[(size_t)b] + f.n_codes;
  }
  return TOC_OK;
}

toc_status check_blob_off(const int64_t *blob_off, int64_t n, const void *blobs) {
  if (n == 0) return TOC_OK;
  if (!blob_off) return fail(TOC_EINVAL, "blob_off is NULL");
  if (blob_off[0] < 0) return fail(TOC_EINVAL, "negative offset");
  for (int64_t b = 0; b < n; ++b)
    if (blob_off[b + 1] < blob_off[b] || blob_off[b + 1] - blob_off[b] > (int64_t)UINT32_MAX)
      return fail(TOC_EINVAL, "blob_off not non-decreasing or a blob of 4 GiB or more at %lld",
                  (long long)b);
  if (blob_off[n] > 0 && !blobs) return fail(TOC_EINVAL, "blobs is NULL");
  return TOC_OK;
}

// Next range from b0: as many batches as fit ws_bytes (at least one, if it fits).
toc_status next_range(const Batches &B, int64_t b0, size_t ws_bytes, const toc_dev *dev,
                      WsFor what, int64_t &b1) {
  if ((size_t)ws_for(B, b0, b0 + 1, dev, what).end > ws_bytes)
    return fail(TOC_ESIZE, "workspace of %zu bytes below the %lld batch %lld needs", ws_bytes,
                (long long)ws_for(B, b0, b0 + 1, dev, what).end, (long long)b0);
  int64_t lo = b0 + 1, hi = B.n;              // the last end that fits, by bisection
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if ((size_t)ws_for(B, b0, mid, dev, what).end <= ws_bytes) lo = mid;
    else hi = mid - 1;
  }
  b1 = lo;
  return TOC_OK;
}

// Copies a range's offsets into the workspace and builds C' of its batches.
toc_status launch_cprime(const void *blobs, const int64_t *blob_off, const Batches &B,
                         const toc_dev *dev, int64_t b0, int64_t b1, const RangeWs &w, uint8_t *ws,
                         hipStream_t s, int &max_rows) {
  const int64_t nb = b1 - b0;
  std::vector<int64_t> h((size_t)(4 * (nb + 1)));
  max_rows = 0;
  for (int64_t x = 0; x <= nb; ++x) {
    const int64_t b = b0 + x;
    h[(size_t)x] = blob_off[b];
    h[(size_t)(nb + 1 + x)] = B.node_off[(size_t)b] - B.node_off[(size_t)b0];
    h[(size_t)(2 * (nb + 1) + x)] = B.d_off[(size_t)b] - B.d_off[(size_t)b0];
    h[(size_t)(3 * (nb + 1) + x)] =
        dev && b < B.n ? dev->dtile_base[(size_t)b] : 0;
    if (x < nb) max_rows = std::max<int>(max_rows, (int)B.info[b].n_rows);
  }
  int64_t *offs = (int64_t *)(ws + w.offs);
  if (hipMemcpyAsync(offs, h.data(), 8 * h.size(), hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(TOC_EDEVICE, "copy of the offsets failed");
  const size_t lds = 8 * ((size_t)max_rows + 1);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute((const void *)cprime_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds) != hipSuccess)
    return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  const unsigned grid = (unsigned)std::min<int64_t>(nb, 1 << 20);
  hipLaunchKernelGGL(cprime_kernel, dim3(grid), dim3(kCpBlock), lds, s, (const uint8_t *)blobs,
                     offs, nb, max_rows, (uint32_t)B.n_cols, (uint32_t *)(ws + w.parent),
                     (uint32_t *)(ws + w.col), (uint32_t *)(ws + w.val), (uint32_t *)(ws + w.depth),
                     (int32_t *)(ws + w.status), (uint32_t *)(ws + w.s0), (uint32_t *)(ws + w.s1),
                     (uint32_t *)(ws + w.s2), (uint32_t *)(ws + w.s3), (uint32_t *)(ws + w.s4));
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "cprime_kernel: %s", hipGetErrorString(e));
  return TOC_OK;
}

// The first nonzero status of a range, as an error naming its batch.
toc_status range_status(const std::vector<int32_t> &st, int64_t b0) {
  for (size_t x = 0; x < st.size(); ++x) {
    if (st[x] == 0) continue;
    if (st[x] == TOC_INGEST_CHANGED)
      return fail(TOC_EINVAL, "batch %lld: bytes differ from those planned", (long long)(b0 + (int64_t)x));
    return fail(TOC_EINVAL, "batch %lld: malformed physical encoding (TOC_CPRIME status %d)",
                (long long)(b0 + (int64_t)x), st[x]);
  }
  return TOC_OK;
}

}  // namespace

extern "C" {

toc_status toc_ingest_workspace_size(const toc_phys_info *info, int64_t n_batches, int32_t n_cols,
                                     size_t *bytes, size_t *min_bytes) {
  toc::clear_error();
  if (!bytes) return fail(TOC_EINVAL, "bytes is NULL");
  Batches B;
  try {
    toc_status st = check_batches(info, n_batches, n_cols, B);
    if (st != TOC_OK) return st;
    *bytes = n_batches ? (size_t)ws_for(B, 0, n_batches, nullptr, kWsBound).end : 0;
    if (min_bytes) {
      size_t mn = 0;
      for (int64_t b = 0; b < n_batches; ++b)
        mn = std::max(mn, (size_t)ws_for(B, b, b + 1, nullptr, kWsBound).end);
      *min_bytes = mn;
    }
  } catch (const std::bad_alloc &) {
    return fail(TOC_ENOMEM, "out of host memory");
  }
  return TOC_OK;
}

toc_status toc_ingest_plan(const void *blobs, const int64_t *blob_off, const toc_phys_info *info,
                           int64_t n_batches, int32_t n_cols, void *ws, size_t ws_bytes,
                           void *stream, size_t *image_bytes, toc_dev **out) {
  toc::clear_error();
  if (!out || !image_bytes) return fail(TOC_EINVAL, "NULL output");
  *out = nullptr;
  toc_dev *dev = new (std::nothrow) toc_dev;
  if (!dev) return fail(TOC_ENOMEM, "out of host memory");
  toc_status ret = TOC_OK;
  try {
    Batches B;
    if ((ret = check_batches(info, n_batches, n_cols, B)) != TOC_OK ||
        (ret = check_blob_off(blob_off, n_batches, blobs)) != TOC_OK) {
      delete dev;
      return ret;
    }
    if (n_batches > 0 && !ws) {
      delete dev;
      return fail(TOC_EINVAL, "ws is NULL");
    }
    hipStream_t s = (hipStream_t)stream;
    std::vector<toc::BatchCounts> bc((size_t)n_batches);
    std::vector<int64_t> n1((size_t)n_batches), nu((size_t)n_batches);
    for (int64_t b0 = 0, b1 = 0; b0 < n_batches && ret == TOC_OK; b0 = b1) {
      if ((ret = next_range(B, b0, ws_bytes, nullptr, kWsCensus, b1)) != TOC_OK) break;
      const RangeWs w = ws_for(B, b0, b1, nullptr, kWsCensus);
      uint8_t *wb = (uint8_t *)ws;
      int max_rows = 0;
      if ((ret = launch_cprime(blobs, blob_off, B, nullptr, b0, b1, w, wb, s, max_rows)) != TOC_OK)
        break;
      const int64_t nb = b1 - b0;
      const unsigned grid = (unsigned)std::min<int64_t>(nb, kIgGrid);
      hipLaunchKernelGGL(census_kernel, dim3(grid), dim3(kIgBlock), 0, s, (const uint8_t *)blobs,
                         (const int64_t *)(wb + w.offs), nb, (uint32_t)n_cols,
                         (const int32_t *)(wb + w.status), (const uint32_t *)(wb + w.parent),
                         (const uint32_t *)(wb + w.col), (const uint32_t *)(wb + w.depth),
                         (uint32_t *)(wb + w.flags), (uint32_t *)(wb + w.slot),
                         (int64_t *)(wb + w.counts), (int32_t *)(wb + w.status));
      if (hipGetLastError() != hipSuccess) {
        ret = fail(TOC_EDEVICE, "census_kernel launch failed");
        break;
      }
      std::vector<int32_t> st((size_t)nb);
      std::vector<int64_t> cn((size_t)(kCensus * nb));
      if (hipMemcpyAsync(st.data(), wb + w.status, 4 * (size_t)nb, hipMemcpyDeviceToHost, s) != hipSuccess ||
          hipMemcpyAsync(cn.data(), wb + w.counts, 8 * cn.size(), hipMemcpyDeviceToHost, s) != hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess) {
        ret = fail(TOC_EDEVICE, "census failed");
        break;
      }
      if ((ret = range_status(st, b0)) != TOC_OK) break;
      for (int64_t x = 0; x < nb; ++x) {
        const int64_t b = b0 + x, *c = &cn[(size_t)(kCensus * x)];
        const toc_phys_info &f = info[b];
        toc::BatchCounts &k = bc[(size_t)b];
        k.rows = f.n_rows;
        k.codes = c[0];
        k.levels = c[1];
        k.d = f.n_codes;
        k.deep = c[3];
        k.int1 = c[2];
        k.nnz = c[4];
        k.canon = 4 * f.n_codes + 4 * (f.n_rows + 1) + 10 * c[0] + 4 * (c[1] + 1);
        n1[(size_t)b] = c[5];
        nu[(size_t)b] = c[6];
      }
    }
    if (ret == TOC_OK) ret = toc::plan_layout(bc.data(), n_batches, n_cols, 0u, dev);
    if (ret != TOC_OK) {
      delete dev;
      return ret;
    }
    for (int64_t b = 0; b < n_batches; ++b) {
      dev->batches[(size_t)b].n_lvl1 = (int32_t)n1[(size_t)b];
      dev->batches[(size_t)b].n_ucols = (int32_t)nu[(size_t)b];
    }
    toc::finish_image(dev);
    dev->phys.assign(info, info + n_batches);
    dev->pending = true;
  } catch (const std::bad_alloc &) {
    delete dev;
    return fail(TOC_ENOMEM, "out of host memory");
  }
  *image_bytes = (size_t)dev->layout.end;
  *out = dev;
  return TOC_OK;
}

toc_status toc_ingest_build(toc_dev *dev, const void *blobs, const int64_t *blob_off, void *buf,
                            size_t bytes, void *ws, size_t ws_bytes, void *stream) {
  toc::clear_error();
  if (!dev) return fail(TOC_EINVAL, "dev is NULL");
  if (!dev->pending) return fail(TOC_EINVAL, "dev is not a planned, unbuilt image");
  if (!buf) return fail(TOC_EINVAL, "buf is NULL");
  if ((int64_t)bytes < dev->layout.end)
    return fail(TOC_ESIZE, "buffer has %zu bytes, image needs %lld", bytes, (long long)dev->layout.end);
  const int64_t n = dev->info.n_batches;
  if (n > 0 && !ws) return fail(TOC_EINVAL, "ws is NULL");
  toc_status ret = check_blob_off(blob_off, n, blobs);
  if (ret != TOC_OK) return ret;
  try {
    Batches B;
    if ((ret = check_batches(dev->phys.data(), n, dev->info.n_cols, B)) != TOC_OK) return ret;
    int device = -1;
    if (hipGetDevice(&device) != hipSuccess) return fail(TOC_EDEVICE, "hipGetDevice failed");
    hipStream_t s = (hipStream_t)stream;
    uint8_t *img = (uint8_t *)buf;
    if (hipMemsetAsync(img, 0, (size_t)dev->layout.end, s) != hipSuccess ||
        (n > 0 && hipMemcpyAsync(img + dev->layout.batches, dev->batches.data(),
                                 sizeof(toc_batch) * (size_t)n, hipMemcpyHostToDevice, s) != hipSuccess))
      return fail(TOC_EDEVICE, "image clear failed");
    for (int64_t b0 = 0, b1 = 0; b0 < n; b0 = b1) {
      if ((ret = next_range(B, b0, ws_bytes, dev, kWsBuild, b1)) != TOC_OK) return ret;
      const RangeWs w = ws_for(B, b0, b1, dev, kWsBuild);
      uint8_t *wb = (uint8_t *)ws;
      int max_rows = 0;
      if ((ret = launch_cprime(blobs, blob_off, B, dev, b0, b1, w, wb, s, max_rows)) != TOC_OK)
        return ret;
      const int64_t nb = b1 - b0;
      IgParams P;
      P.blobs = (const uint8_t *)blobs;
      P.offs = (const int64_t *)(wb + w.offs);
      P.n = nb;
      P.b0 = b0;
      P.max_rows = max_rows;
      P.n_cols = (uint32_t)dev->info.n_cols;
      P.cp_status = (const int32_t *)(wb + w.status);
      P.parent = (const uint32_t *)(wb + w.parent);
      P.col = (const uint32_t *)(wb + w.col);
      P.val = (const uint32_t *)(wb + w.val);
      P.depth = (const uint32_t *)(wb + w.depth);
      P.flags = (uint32_t *)(wb + w.flags);
      P.newidx = (uint32_t *)(wb + w.s0);
      P.gst = (uint32_t *)(wb + w.s1);
      P.gsz = (uint32_t *)(wb + w.s2);
      P.at = (uint32_t *)(wb + w.s3);
      P.atl = (uint32_t *)(wb + w.s4);
      P.occ = (uint32_t *)(wb + w.occ);
      P.g = (uint32_t *)(wb + w.g);
      P.sortbuf = (uint32_t *)(wb + w.slot);
      P.sort_len = sort_len_of(B, b0, b1, dev, kWsBuild);
      P.img = img;
      P.L = dev->layout;
      P.status = (int32_t *)(wb + w.status);
      const size_t lds = 8 * ((size_t)max_rows + 1);
      if (lds > 64 * 1024 &&
          hipFuncSetAttribute((const void *)image_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds) != hipSuccess)
        return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
      const unsigned grid = (unsigned)std::min<int64_t>(nb, kIgGrid);
      hipLaunchKernelGGL(image_kernel, dim3(grid), dim3(kIgBlock), lds, s, P);
      if (hipGetLastError() != hipSuccess) return fail(TOC_EDEVICE, "image_kernel launch failed");
      std::vector<int32_t> st((size_t)nb);
      if (hipMemcpyAsync(st.data(), wb + w.status, 4 * (size_t)nb, hipMemcpyDeviceToHost, s) != hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess)
        return fail(TOC_EDEVICE, "image build failed");
      if ((ret = range_status(st, b0)) != TOC_OK) return ret;
    }
    if (hipStreamSynchronize(s) != hipSuccess) return fail(TOC_EDEVICE, "image build failed");
    dev->buf = buf;
    dev->bytes = bytes;
    dev->device = device;
    dev->host = false;
    dev->pending = false;
  } catch (const std::bad_alloc &) {
    return fail(TOC_ENOMEM, "out of host memory");
  }
  return TOC_OK;
}

}  // extern "C"
