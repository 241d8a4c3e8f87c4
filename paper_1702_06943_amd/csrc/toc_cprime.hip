// The decoding tree C' built on the device from the physical encoding: Algorithm 2
// (BuildPrefixTree, section 4.1.2) over integers read back from bit-packed bytes
// (section 4.1.1), one workgroup per batch, batches in parallel.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "toc_internal.h"
#include "toc_phys_dev.h"

namespace tocphys {

__global__ __launch_bounds__(kCpBlock) void cprime_kernel(
    const uint8_t *__restrict__ blobs, const int64_t *__restrict__ offs, int64_t n_batches,
    int max_rows, uint32_t n_cols, uint32_t *__restrict__ parent, uint32_t *__restrict__ col,
    uint32_t *__restrict__ val, uint32_t *__restrict__ depth, int32_t *__restrict__ status,
    uint32_t *__restrict__ anc0, uint32_t *__restrict__ dist0, uint32_t *__restrict__ anc1,
    uint32_t *__restrict__ dist1, uint32_t *__restrict__ nxt) {
  extern __shared__ uint32_t sm[];              // tuple starts, then nonempty tuples before each
  __shared__ Hdr h;
  __shared__ uint32_t wsum[kCpWaves];
  __shared__ int errs;
  uint32_t *st = sm, *nes = sm + (max_rows + 1);
  const int64_t *node_off = offs + (n_batches + 1);
  for (int64_t b = blockIdx.x; b < n_batches; b += gridDim.x) {
    const uint8_t *blob = blobs + offs[b];
    const uint64_t size = (uint64_t)(offs[b + 1] - offs[b]);
    const int64_t no = node_off[b];
    const uint32_t n_decl = (uint32_t)(node_off[b + 1] - no);   // nodes node_off gives the batch
    // headers, read by one thread; every later read stays inside the arrays
    if (threadIdx.x == 0) {
      parse_headers(blob, size, max_rows, h);
      errs = 0;
    }
    __syncthreads();
    if (h.err) {
      if (threadIdx.x == 0) status[b] = h.err;
      __syncthreads();
      continue;
    }
    const uint32_t nI = h.cnt[0], U = h.cnt[1], nD = h.cnt[3], nR = h.cnt[4] - 1;
    const uint8_t *p_col = blob + h.data[0], *p_uni = blob + h.data[1], *p_vix = blob + h.data[2];
    const uint8_t *p_d = blob + h.data[3], *p_st = blob + h.data[4];
    const uint32_t w_col = h.w[0], w_vix = h.w[2], w_d = h.w[3], w_st = h.w[4];
    // tuple starts, checked, and the number of nonempty tuples before each tuple:
    // the entry at position p of tuple i matches against nI + 1 + p - nes[i] nodes
    for (uint32_t r = threadIdx.x; r <= nR; r += kCpBlock) st[r] = rd(p_st, r, w_st);
    __syncthreads();
    bool bad = threadIdx.x == 0 && (st[0] != 0 || st[nR] != nD);
    uint32_t carry = 0;
    for (uint32_t r0 = 0; r0 < nR; r0 += kCpBlock) {
      const uint32_t r = r0 + threadIdx.x;
      const bool in = r < nR;
      const uint32_t s0 = in ? st[r] : 0u, s1 = in ? st[r + 1] : 0u;
      bad |= in && s1 < s0;
      uint32_t tot;
      const uint32_t ex = block_excl_scan(in && s1 > s0 ? 1u : 0u, wsum, tot);
      if (in) nes[r] = carry + ex;
      carry += tot;
    }
    if (__syncthreads_or(bad)) {
      if (threadIdx.x == 0) status[b] = TOC_CPRIME_STARTS;
      __syncthreads();
      continue;
    }
    if ((uint64_t)1 + nI + (nD - carry) != (uint64_t)n_decl) {
      if (threadIdx.x == 0) status[b] = TOC_CPRIME_NODES;
      __syncthreads();
      continue;
    }
    const uint32_t n_nodes = n_decl;
    // the root and the first layer (nodes 1..nI are I in order); pointer-jumping
    // state: a node's nearest first-layer ancestor (itself here) and its distance
    for (uint32_t c = threadIdx.x; c <= nI; c += kCpBlock) {
      const int64_t g = no + c;
      if (c == 0) {
        parent[g] = kNone;
        col[g] = kNone;
        val[g] = 0u;
        depth[g] = 0u;
      } else {
        const uint32_t q = rd(p_vix, c - 1, w_vix);
        if (q >= U) atomicOr(&errs, 1 << TOC_CPRIME_VALUE_INDEX);
        const uint32_t cc = rd(p_col, c - 1, w_col);
        if (cc >= n_cols) atomicOr(&errs, 1 << TOC_CPRIME_COLUMN);
        parent[g] = 0u;
        col[g] = cc;
        val[g] = q < U ? rd(p_uni, q, 4) : 0u;
        depth[g] = 1u;
      }
      anc0[g] = anc1[g] = c;
      dist0[g] = dist1[g] = 0u;
    }
    // the entries of D: entry p of tuple i matches one of the nI + 1 + p - nes[i]
    // nodes existing at that point; unless it ends its tuple it makes that node,
    // child of its code, keyed by the first pair of the next entry's code
    for (uint32_t p = threadIdx.x; p < nD; p += kCpBlock) {
      uint32_t lo = 0, hi = nR;                 // last tuple starting at or before p
      while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (st[mid] <= p) lo = mid;
        else hi = mid;
      }
      const uint32_t i = lo, q = nI + 1u + p - nes[i];
      const uint32_t code = rd(p_d, p, w_d);
      if (code == 0u || code >= q) {
        atomicOr(&errs, 1 << TOC_CPRIME_CODE);
      } else if (p + 1 < st[i + 1]) {
        const int64_t g = no + q;
        parent[g] = code;
        anc0[g] = code;
        dist0[g] = 1u;
        nxt[g] = rd(p_d, p + 1, w_d);
      }
    }
    __syncthreads();
    if (errs) {
      if (threadIdx.x == 0)
        status[b] = (errs & (1 << TOC_CPRIME_VALUE_INDEX)) ? TOC_CPRIME_VALUE_INDEX
                    : (errs & (1 << TOC_CPRIME_COLUMN))    ? TOC_CPRIME_COLUMN
                                                           : TOC_CPRIME_CODE;
      __syncthreads();
      continue;
    }
    // pointer jumping over the new nodes: every node's parent has a smaller index,
    // so each round halves the distance still to go to the first layer
    uint32_t *ax = anc0, *dx = dist0, *ay = anc1, *dy = dist1;
    for (int round = 0; round < kCpMaxRounds; ++round) {
      bool changed = false;
      for (uint32_t c = nI + 1 + threadIdx.x; c < n_nodes; c += kCpBlock) {
        const int64_t g = no + c;
        const uint32_t a = ax[g], d = dx[g];
        if (a > nI) {
          ay[g] = ax[no + a];
          dy[g] = d + dx[no + a];
          changed = true;
        } else {
          ay[g] = a;
          dy[g] = d;
        }
      }
      __syncthreads();                          // this round's writes, seen by the next
      const bool any = __syncthreads_or(changed);
      uint32_t *t = ax;
      ax = ay;
      ay = t;
      t = dx;
      dx = dy;
      dy = t;
      if (!any) break;
    }
    // depth = distance to the first layer + 1; key = first pair of the next
    // entry's code, the key of its first-layer ancestor
    for (uint32_t c = nI + 1 + threadIdx.x; c < n_nodes; c += kCpBlock) {
      const int64_t g = no + c;
      depth[g] = dx[g] + 1u;
      const uint32_t f = ax[no + nxt[g]];
      col[g] = col[no + f];
      val[g] = val[no + f];
    }
    if (threadIdx.x == 0) status[b] = 0;
    __syncthreads();
  }
}

}  // namespace tocphys

namespace {

using namespace tocphys;

// The live codes of each batch in level order, from the tree toc_cprime_build made
// (parent, key, depth per node) and the blob's D: codes of D and their ancestors
// are marked live (a walk up from each entry of D stops at the first node another
// walk already marked, so each node is passed once); live codes are counted per
// depth, and each gets its place in the stable (depth, index) order from a
// per-depth running count, chunk by chunk in index order with the waves of a
// chunk taking turns; parents and D are then renumbered.
constexpr int kLvBlock = 512;
constexpr int kLvWaves = kLvBlock / kCpWave;
constexpr int kLvMaxLevels = 4096;

__global__ __launch_bounds__(kLvBlock) void level_kernel(
    const uint8_t *__restrict__ blobs, const int64_t *__restrict__ offs, int64_t n_batches,
    int max_levels, const int32_t *__restrict__ cp_status, const uint32_t *__restrict__ parent,
    const uint32_t *__restrict__ col, const uint32_t *__restrict__ val,
    const uint32_t *__restrict__ depth, uint32_t *__restrict__ l_parent,
    uint32_t *__restrict__ l_col, uint32_t *__restrict__ l_val, uint32_t *__restrict__ l_depth,
    uint32_t *__restrict__ level, uint32_t *__restrict__ l_D, int64_t *__restrict__ counts,
    int32_t *__restrict__ status, uint32_t *__restrict__ newidx) {
  extern __shared__ uint32_t run[];            // per depth: live codes placed so far
  uint32_t *wcnt = run + (max_levels + 1);     // per wave and depth: a chunk's live codes
  uint32_t *live = wcnt + kLvWaves * (max_levels + 1);   // the batch's live codes, a bit each
  __shared__ Hdr h;
  __shared__ int errs;
  __shared__ uint32_t n_lv, top_d;
  const int64_t *node_off = offs + (n_batches + 1), *d_off = offs + 2 * (n_batches + 1);
  const int lane = threadIdx.x % kCpWave, wave = threadIdx.x / kCpWave;
  for (int64_t b = blockIdx.x; b < n_batches; b += gridDim.x) {
    const uint8_t *blob = blobs + offs[b];
    const uint64_t size = (uint64_t)(offs[b + 1] - offs[b]);
    const int64_t no = node_off[b], dof = d_off[b];
    const uint32_t n_nodes = (uint32_t)(node_off[b + 1] - no);
    if (threadIdx.x == 0) {
      h.err = cp_status[b];
      if (h.err == 0) parse_headers(blob, size, 1 << 30, h);
      if (h.err == 0 && (int64_t)h.cnt[3] != d_off[b + 1] - dof) h.err = TOC_LEVEL_D;
      errs = 0;
    }
    __syncthreads();
    if (h.err) {
      if (threadIdx.x == 0) {
        status[b] = h.err;
        counts[2 * b] = counts[2 * b + 1] = 0;
      }
      __syncthreads();
      continue;
    }
    const uint32_t nD = h.cnt[3], w_d = h.w[3];
    const uint8_t *p_d = blob + h.data[3];
    for (uint32_t x = threadIdx.x; x < (n_nodes + 31) / 32; x += kLvBlock) live[x] = 0u;
    for (int d = threadIdx.x; d <= max_levels; d += kLvBlock) {
      run[d] = 0u;
      for (int v = 0; v < kLvWaves; ++v) wcnt[v * (max_levels + 1) + d] = 0u;
    }
    __syncthreads();
    // live marking: a walk up from every entry of D
    for (uint32_t p = threadIdx.x; p < nD; p += kLvBlock) {
      uint32_t c = rd(p_d, p, w_d);
      if (c == 0u || c >= n_nodes) {
        atomicOr(&errs, 1);
        continue;
      }
      while (c != 0u && (atomicOr(&live[c / 32], 1u << (c % 32)) & (1u << (c % 32))) == 0u)
        c = parent[no + c];
    }
    __syncthreads();
    if (errs) {
      if (threadIdx.x == 0) {
        status[b] = TOC_CPRIME_CODE;
        counts[2 * b] = counts[2 * b + 1] = 0;
      }
      __syncthreads();
      continue;
    }
    // live codes per depth
    for (uint32_t c = 1 + threadIdx.x; c < n_nodes; c += kLvBlock) {
      if (!((live[c / 32] >> (c % 32)) & 1u)) continue;
      const uint32_t d = depth[no + c];
      if (d == 0u || d > (uint32_t)max_levels) atomicOr(&errs, 2);
      else atomicAdd(&run[d], 1u);
    }
    __syncthreads();
    if (errs) {
      if (threadIdx.x == 0) {
        status[b] = TOC_LEVEL_DEPTH;
        counts[2 * b] = counts[2 * b + 1] = 0;
      }
      __syncthreads();
      continue;
    }
    // level offsets; run[d] becomes the first place of depth d
    if (threadIdx.x == 0) {
      uint32_t *lv = level + b * (int64_t)(max_levels + 1);
      uint32_t acc = 0, top = 0;
      lv[0] = 0u;
      for (int d = 1; d <= max_levels; ++d) {
        const uint32_t n = run[d];
        run[d] = acc;
        acc += n;
        if (n) top = (uint32_t)d;
        lv[d] = acc;
      }
      n_lv = acc;
      top_d = top;
      counts[2 * b] = acc;
      counts[2 * b + 1] = top;
    }
    __syncthreads();
    // places in (depth, index) order, chunk by chunk of kLvBlock nodes in index
    // order: each wave ranks its lanes of one depth by a ballot and counts them per
    // depth; a lane's place is the depth's running count, plus the counts of the
    // waves before its own, plus its rank; then the running counts advance
    const uint32_t L = top_d;
    for (uint32_t c0 = 1; c0 < n_nodes; c0 += kLvBlock) {
      const uint32_t c = c0 + threadIdx.x;
      const bool in = c < n_nodes && ((live[c / 32] >> (c % 32)) & 1u);
      const uint32_t d = in ? depth[no + c] : 0u;
      uint32_t rank = 0;
      bool todo = in;
      uint64_t left = __ballot(todo);
      while (left) {
        const int leader = __ffsll((unsigned long long)left) - 1;
        const uint32_t dd = (uint32_t)__shfl((int)d, leader, kCpWave);
        const bool mine = todo && d == dd;
        const uint64_t m = __ballot(mine);
        if (mine) {
          rank = (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
          todo = false;
        }
        if (lane == leader) wcnt[wave * (max_levels + 1) + dd] = (uint32_t)__popcll(m);
        left = __ballot(todo);
      }
      __syncthreads();
      if (in) {
        uint32_t at = run[d] + rank;
        for (int v = 0; v < wave; ++v) at += wcnt[v * (max_levels + 1) + d];
        newidx[no + c] = at;
      }
      __syncthreads();
      for (uint32_t dd = 1 + threadIdx.x; dd <= L; dd += kLvBlock) {
        uint32_t add = 0;
        for (int v = 0; v < kLvWaves; ++v) {
          add += wcnt[v * (max_levels + 1) + dd];
          wcnt[v * (max_levels + 1) + dd] = 0u;
        }
        run[dd] += add;
      }
      __syncthreads();
    }
    __threadfence();
    __syncthreads();
    // the live codes at their places, parents renumbered; D renumbered
    for (uint32_t c = 1 + threadIdx.x; c < n_nodes; c += kLvBlock) {
      if (!((live[c / 32] >> (c % 32)) & 1u)) continue;
      const uint32_t i = newidx[no + c], d = depth[no + c];
      l_parent[no + i] = d == 1u ? kNone : newidx[no + parent[no + c]];
      l_col[no + i] = col[no + c];
      l_val[no + i] = val[no + c];
      l_depth[no + i] = d;
    }
    for (uint32_t p = threadIdx.x; p < nD; p += kLvBlock) l_D[dof + p] = newidx[no + rd(p_d, p, w_d)];
    if (threadIdx.x == 0) status[b] = 0;
    __syncthreads();
  }
}

// A.w (k = 1, Theorem 1) straight from the device-built level order: per batch,
// H over the live codes level by level in LDS (H[c] = H[parent] + val * w[col],
// parents first), then each tuple's sum of H over its renumbered codes, the tuple
// starts read back from the blob.  Completes ingest on the device: physical bytes
// -> C' -> level order -> product, with no host pass over the batch.
__global__ __launch_bounds__(kLvBlock) void level_right_k1_kernel(
    const uint8_t *__restrict__ blobs, const int64_t *__restrict__ offs, int64_t n_batches,
    int max_levels, int64_t max_live, uint32_t n_cols, const int32_t *__restrict__ lv_status,
    const int64_t *__restrict__ counts, const uint32_t *__restrict__ level,
    const uint32_t *__restrict__ l_parent,
    const uint32_t *__restrict__ l_col, const float *__restrict__ l_val,
    const uint32_t *__restrict__ l_D, const float *__restrict__ w, float *__restrict__ r,
    int32_t *__restrict__ status) {
  extern __shared__ float H[];
  __shared__ Hdr h;
  __shared__ int bad_col;
  const int64_t *node_off = offs + (n_batches + 1), *d_off = offs + 2 * (n_batches + 1);
  const int64_t *row_off = offs + 3 * (n_batches + 1);
  for (int64_t b = blockIdx.x; b < n_batches; b += gridDim.x) {
    const uint8_t *blob = blobs + offs[b];
    const uint64_t size = (uint64_t)(offs[b + 1] - offs[b]);
    const int64_t no = node_off[b], dof = d_off[b], r0 = row_off[b];
    if (threadIdx.x == 0) {
      h.err = lv_status[b];
      if (h.err == 0) parse_headers(blob, size, 1 << 30, h);
      if (h.err == 0 && ((int64_t)h.cnt[4] - 1 != row_off[b + 1] - r0 ||
                         (int64_t)h.cnt[3] != d_off[b + 1] - dof))
        h.err = TOC_LEVEL_D;
      if (h.err == 0 && counts[2 * b] > max_live) h.err = TOC_LEVEL_LIVE;
      bad_col = 0;
    }
    __syncthreads();
    if (h.err) {
      if (threadIdx.x == 0) status[b] = h.err;
      __syncthreads();
      continue;
    }
    const uint32_t *lv = level + b * (int64_t)(max_levels + 1);
    const int top = (int)counts[2 * b + 1];
    for (int d = 1; d <= top; ++d) {
      const uint32_t a = lv[d - 1], e = lv[d];
      for (uint32_t c = a + threadIdx.x; c < e; c += kLvBlock) {
        const float base = d > 1 ? H[l_parent[no + c]] : 0.0f;
        const uint32_t cc = l_col[no + c];
        // a column past w (a tree built from another matrix's bytes) is never read
        if (cc >= n_cols) bad_col = 1;
        H[c] = fmaf(l_val[no + c], cc < n_cols ? w[cc] : 0.0f, base);
      }
      __syncthreads();
    }
    if (bad_col) {
      if (threadIdx.x == 0) status[b] = TOC_CPRIME_COLUMN;
      __syncthreads();
      continue;
    }
    const uint8_t *p_st = blob + h.data[4];
    const uint32_t w_st = h.w[4], nR = h.cnt[4] - 1;
    const int lane = threadIdx.x % 8, grp = threadIdx.x / 8;
    for (uint32_t i = grp; i < nR; i += kLvBlock / 8) {
      const uint32_t s0 = rd(p_st, i, w_st), s1 = rd(p_st, i + 1, w_st);
      // blocked summation: 16 entries per partial sum, their codes loaded together
      float acc = 0.0f;
      for (uint32_t p0 = s0 + lane; p0 < s1; p0 += 16 * 8) {
        uint32_t x[16];
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u) x[u] = p0 + 8 * u < s1 ? l_D[dof + p0 + 8 * u] : 0u;
        float part = 0.0f;
#pragma unroll
        for (uint32_t u = 0; u < 16; ++u)
          if (p0 + 8 * u < s1) part += H[x[u]];
        acc += part;
      }
#pragma unroll
      for (int o = 4; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 8);
      if (lane == 0) r[r0 + i] = acc;
    }
    if (threadIdx.x == 0) status[b] = 0;
    __syncthreads();
  }
}

inline int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

int64_t ws_nodes_offset(int64_t n_batches) { return align256(16 * (n_batches + 1)); }

}  // namespace

using namespace toc;

extern "C" {

toc_status toc_cprime_workspace_size(int64_t n_batches, int64_t n_nodes, size_t *bytes) {
  clear_error();
  if (!bytes || n_batches < 0 || n_nodes < 0) return fail(TOC_EINVAL, "bad argument");
  *bytes = (size_t)(ws_nodes_offset(n_batches) + 5 * align256(4 * n_nodes));
  return TOC_OK;
}

toc_status toc_cprime_build(const void *blobs, const int64_t *blob_off, const int64_t *node_off,
                            int64_t n_batches, int32_t max_rows, int32_t n_cols, uint32_t *parent,
                            uint32_t *col,
                            float *val, uint32_t *depth, int32_t *status, void *ws,
                            size_t ws_bytes, void *stream) {
  clear_error();
  if (n_batches < 0) return fail(TOC_EINVAL, "n_batches < 0");
  if (n_batches == 0) return TOC_OK;
  if (!blob_off || !node_off || !status || !ws) return fail(TOC_EINVAL, "NULL argument");
  if (max_rows < 0 || max_rows > kCpMaxRows)
    return fail(TOC_EUNSUPPORTED, "max_rows %d outside 0..%d", max_rows, kCpMaxRows);
  if (n_cols < 0) return fail(TOC_EINVAL, "n_cols < 0");
  if (blob_off[0] < 0 || node_off[0] < 0) return fail(TOC_EINVAL, "negative offset");
  for (int64_t b = 0; b < n_batches; ++b) {
    if (blob_off[b + 1] < blob_off[b] || blob_off[b + 1] - blob_off[b] > (int64_t)UINT32_MAX)
      return fail(TOC_EINVAL, "blob_off not non-decreasing or a blob of 4 GiB or more at %lld",
                  (long long)b);
    if (node_off[b + 1] <= node_off[b] || node_off[b + 1] - node_off[b] > (int64_t)INT32_MAX)
      return fail(TOC_EINVAL, "node_off[%lld] does not give 1..2^31-1 nodes", (long long)b);
  }
  const int64_t n_nodes = node_off[n_batches];
  if (!parent || !col || !val || !depth) return fail(TOC_EINVAL, "NULL output");
  if (blob_off[n_batches] > 0 && !blobs) return fail(TOC_EINVAL, "blobs is NULL");
  size_t need = 0;
  toc_cprime_workspace_size(n_batches, n_nodes, &need);
  if (ws_bytes < need) return fail(TOC_ESIZE, "workspace of %zu bytes below the %zu needed", ws_bytes, need);
  hipStream_t s = (hipStream_t)stream;
  int64_t *offs = (int64_t *)ws;
  if (hipMemcpyAsync(offs, blob_off, 8 * (n_batches + 1), hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(offs + n_batches + 1, node_off, 8 * (n_batches + 1), hipMemcpyHostToDevice, s) !=
          hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(TOC_EDEVICE, "copy of the offsets failed");
  uint8_t *base = (uint8_t *)ws + ws_nodes_offset(n_batches);
  const int64_t arr = align256(4 * n_nodes);
  uint32_t *a0 = (uint32_t *)base, *d0 = (uint32_t *)(base + arr), *a1 = (uint32_t *)(base + 2 * arr);
  uint32_t *d1 = (uint32_t *)(base + 3 * arr), *nx = (uint32_t *)(base + 4 * arr);
  const size_t lds = 8 * ((size_t)max_rows + 1);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute((const void *)cprime_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds) != hipSuccess)
    return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  const unsigned g = (unsigned)std::min<int64_t>(n_batches, 1 << 20);
  hipLaunchKernelGGL(cprime_kernel, dim3(g), dim3(kCpBlock), lds, s, (const uint8_t *)blobs, offs,
                     n_batches, (int)max_rows, (uint32_t)n_cols, parent, col, (uint32_t *)val, depth,
                     status, a0, d0,
                     a1, d1, nx);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "cprime_kernel: %s", hipGetErrorString(e));
  return TOC_OK;
}

toc_status toc_level_workspace_size(int64_t n_batches, int64_t n_nodes, size_t *bytes) {
  clear_error();
  if (!bytes || n_batches < 0 || n_nodes < 0) return fail(TOC_EINVAL, "bad argument");
  *bytes = (size_t)(align256(24 * (n_batches + 1)) + align256(4 * n_nodes));
  return TOC_OK;
}

toc_status toc_level_build(const void *blobs, const int64_t *blob_off, const int64_t *node_off,
                           const int64_t *d_off, int64_t n_batches, int32_t max_levels,
                           const int32_t *cprime_status, const uint32_t *parent,
                           const uint32_t *col, const float *val, const uint32_t *depth,
                           uint32_t *l_parent, uint32_t *l_col, float *l_val, uint32_t *l_depth,
                           uint32_t *level, uint32_t *l_D, int64_t *counts, int32_t *status,
                           void *ws, size_t ws_bytes, void *stream) {
  clear_error();
  if (n_batches < 0) return fail(TOC_EINVAL, "n_batches < 0");
  if (n_batches == 0) return TOC_OK;
  if (!blob_off || !node_off || !d_off || !cprime_status || !status || !counts || !level || !ws)
    return fail(TOC_EINVAL, "NULL argument");
  if (max_levels < 1 || max_levels > kLvMaxLevels)
    return fail(TOC_EUNSUPPORTED, "max_levels %d outside 1..%d", max_levels, kLvMaxLevels);
  if (blob_off[0] < 0 || node_off[0] < 0 || d_off[0] < 0) return fail(TOC_EINVAL, "negative offset");
  for (int64_t b = 0; b < n_batches; ++b) {
    if (blob_off[b + 1] < blob_off[b] || blob_off[b + 1] - blob_off[b] > (int64_t)UINT32_MAX)
      return fail(TOC_EINVAL, "blob_off not non-decreasing or a blob of 4 GiB or more at %lld",
                  (long long)b);
    if (node_off[b + 1] <= node_off[b] || node_off[b + 1] - node_off[b] > (int64_t)INT32_MAX)
      return fail(TOC_EINVAL, "node_off[%lld] does not give 1..2^31-1 nodes", (long long)b);
    if (d_off[b + 1] < d_off[b]) return fail(TOC_EINVAL, "d_off not non-decreasing at %lld", (long long)b);
  }
  const int64_t n_nodes = node_off[n_batches];
  if (!parent || !col || !val || !depth || !l_parent || !l_col || !l_val || !l_depth)
    return fail(TOC_EINVAL, "NULL node array");
  if (d_off[n_batches] > 0 && !l_D) return fail(TOC_EINVAL, "l_D is NULL");
  if (blob_off[n_batches] > 0 && !blobs) return fail(TOC_EINVAL, "blobs is NULL");
  size_t need = 0;
  toc_level_workspace_size(n_batches, n_nodes, &need);
  if (ws_bytes < need) return fail(TOC_ESIZE, "workspace of %zu bytes below the %zu needed", ws_bytes, need);
  hipStream_t s = (hipStream_t)stream;
  int64_t *offs = (int64_t *)ws;
  const size_t ob = 8 * (size_t)(n_batches + 1);
  if (hipMemcpyAsync(offs, blob_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(offs + n_batches + 1, node_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(offs + 2 * (n_batches + 1), d_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(TOC_EDEVICE, "copy of the offsets failed");
  uint32_t *newidx = (uint32_t *)((uint8_t *)ws + align256(24 * (n_batches + 1)));
  int64_t max_nodes = 0;
  for (int64_t b = 0; b < n_batches; ++b) max_nodes = std::max(max_nodes, node_off[b + 1] - node_off[b]);
  // per-depth counters and a bit per node of the batch (live marks) in LDS
  const size_t lds = 4 * ((size_t)max_levels + 1) * (1 + kLvWaves) + 4 * (size_t)((max_nodes + 31) / 32);
  if (lds > 160 * 1024)
    return fail(TOC_EUNSUPPORTED, "a batch of %lld nodes: live marks beyond LDS", (long long)max_nodes);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute((const void *)level_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                          (int)lds) != hipSuccess)
    return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  const unsigned g = (unsigned)std::min<int64_t>(n_batches, 1 << 20);
  hipLaunchKernelGGL(level_kernel, dim3(g), dim3(kLvBlock), lds, s, (const uint8_t *)blobs, offs,
                     n_batches, (int)max_levels, cprime_status, parent, col, (const uint32_t *)val,
                     depth, l_parent, l_col, (uint32_t *)l_val, l_depth, level, l_D, counts,
                     status, newidx);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "level_kernel: %s", hipGetErrorString(e));
  return TOC_OK;
}

toc_status toc_level_right_mul(const void *blobs, const int64_t *blob_off, const int64_t *node_off,
                               const int64_t *d_off, const int64_t *row_off, int64_t n_batches,
                               int32_t n_cols, int32_t max_levels, int64_t max_live,
                               const int32_t *level_status,
                               const int64_t *counts, const uint32_t *level,
                               const uint32_t *l_parent, const uint32_t *l_col, const float *l_val,
                               const uint32_t *l_D, const float *w, float *r, int32_t *status,
                               void *ws, size_t ws_bytes, void *stream) {
  clear_error();
  if (n_batches < 0) return fail(TOC_EINVAL, "n_batches < 0");
  if (n_batches == 0) return TOC_OK;
  if (!blob_off || !node_off || !d_off || !row_off || !level_status || !counts || !level ||
      !status || !ws)
    return fail(TOC_EINVAL, "NULL argument");
  if (max_levels < 1 || max_levels > kLvMaxLevels)
    return fail(TOC_EUNSUPPORTED, "max_levels %d outside 1..%d", max_levels, kLvMaxLevels);
  if (max_live < 0 || max_live * 4 > 160 * 1024)
    return fail(TOC_EUNSUPPORTED, "max_live %lld: H must fit 160 KiB of LDS", (long long)max_live);
  if (n_cols < 0) return fail(TOC_EINVAL, "n_cols < 0");
  for (int64_t b = 0; b < n_batches; ++b) {
    if (blob_off[b + 1] < blob_off[b] || node_off[b + 1] <= node_off[b] ||
        d_off[b + 1] < d_off[b] || row_off[b + 1] < row_off[b])
      return fail(TOC_EINVAL, "offsets not non-decreasing at %lld", (long long)b);
  }
  if (!l_parent || !l_col || !l_val || !w || (row_off[n_batches] > 0 && !r) ||
      (d_off[n_batches] > 0 && !l_D) || (blob_off[n_batches] > 0 && !blobs))
    return fail(TOC_EINVAL, "NULL array");
  const size_t need = (size_t)(32 * (n_batches + 1));
  if (ws_bytes < need) return fail(TOC_ESIZE, "workspace of %zu bytes below the %zu needed", ws_bytes, need);
  hipStream_t s = (hipStream_t)stream;
  int64_t *offs = (int64_t *)ws;
  const size_t ob = 8 * (size_t)(n_batches + 1);
  if (hipMemcpyAsync(offs, blob_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(offs + (n_batches + 1), node_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(offs + 2 * (n_batches + 1), d_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(offs + 3 * (n_batches + 1), row_off, ob, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(TOC_EDEVICE, "copy of the offsets failed");
  const size_t lds = 4 * (size_t)std::max<int64_t>(max_live, 1);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute((const void *)level_right_k1_kernel,
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  const unsigned g = (unsigned)std::min<int64_t>(n_batches, 1 << 20);
  hipLaunchKernelGGL(level_right_k1_kernel, dim3(g), dim3(kLvBlock), lds, s, (const uint8_t *)blobs,
                     offs, n_batches, (int)max_levels, max_live, (uint32_t)n_cols, level_status, counts,
                     level, l_parent, l_col,
                     l_val, l_D, w, r, status);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "level_right_k1_kernel: %s", hipGetErrorString(e));
  return TOC_OK;
}

}  // extern "C"
