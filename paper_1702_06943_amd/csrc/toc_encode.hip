// The logical encoding of Algorithm 1 (PrefixTreeEncode, section 3.1) on the
// device, for many mini-batches at once; each batch has its own prefix tree.
//
// Phase I (every distinct column:value pair becomes a child of the root, in order
// of first appearance) is parallel inside a batch: one workgroup per batch inserts
// the batch's pairs into an open-addressing table, keeping the smallest position
// of each pair, then numbers the first appearances with a workgroup scan.  Every
// entry leaves its pair's node index (1..|I|) in the D slot of its position.
//
// Phase II (greedy longest matches, one new node after every match that does not
// end its tuple) is sequential inside a batch by nature: the tree a tuple matches
// against is the one the earlier tuples grew.  One lane runs one batch, so a wave
// walks 64 batches at once; the children of each tree node live in a per-lane
// open-addressing table keyed by (node, pair node index).  A node's extension by a
// pair is a child of the node keyed by that pair, so the pair's first-layer node
// index stands for the pair in the key.  The codes are written over the pair
// indexes in place: a code is written only after the entries it covers were read.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <vector>

#include "toc_internal.h"

namespace {

constexpr int kEpBlock = 256;               // phase I workgroup
constexpr int kEpWave = 64;
constexpr int kEpWaves = kEpBlock / kEpWave;
constexpr int kEtBlock = 64;                // phase II: one wave per workgroup
constexpr int64_t kMaxPairGroups = 1024;    // phase I workgroups (each owns a table)
constexpr int64_t kMaxLanes = 16384;        // phase II lanes (each owns a table)
constexpr int64_t kTableBudget = (int64_t)8 << 30;   // bytes for each phase's tables
constexpr uint64_t kEmptyKey = ~0ull;
constexpr uint32_t kNone = 0xFFFFFFFFu;

// Phase I slot: the pair (column << 32 | value bits), its first position in the
// batch and, once numbered, its node index.
struct PairSlot {
  uint64_t key;
  uint32_t first;
  uint32_t node;
};

// Phase II slot: (parent node << 32 | pair node index) -> child node; `tag` is the
// batch that wrote it, so a lane's table needs no clearing between its batches.
struct ChildSlot {
  uint64_t key;
  uint32_t child;
  uint32_t tag;
};

// Slots of a table for up to n keys: a power of two at least 1.5 n (and 64).
inline int64_t table_slots(int64_t n) {
  int64_t s = 64;
  while (s < n + n / 2 + 1) s <<= 1;
  return s;
}
__device__ inline uint32_t table_slots_dev(uint32_t n) {
  uint32_t s = 64;
  while (s < n + n / 2 + 1) s <<= 1;
  return s;
}

// MurmurHash3's 64-bit finaliser (fmix64).
__device__ inline uint32_t mix64(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return (uint32_t)k;
}

__device__ inline uint32_t load_agent(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline int64_t load_agent64(const int64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix sum of x over the workgroup; total gets the sum of all.
__device__ uint32_t block_excl_scan(uint32_t x, uint32_t *wsum, uint32_t &total) {
  const int lane = threadIdx.x % kEpWave, wave = threadIdx.x / kEpWave;
  uint32_t v = x;
#pragma unroll
  for (int o = 1; o < kEpWave; o <<= 1) {
    const uint32_t y = __shfl_up(v, o, kEpWave);
    if (lane >= o) v += y;
  }
  if (lane == kEpWave - 1) wsum[wave] = v;
  __syncthreads();
  uint32_t before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kEpWaves; ++w) {
    before += w < wave ? wsum[w] : 0u;
    total += wsum[w];
  }
  __syncthreads();
  return before + v - x;
}

// Phase I.  Entry e of the input sits at index e - rowptr[0] of col, val and of the
// outputs I_col, I_val, D; batch b's entries are those of its rows.
__global__ __launch_bounds__(kEpBlock) void enc_pairs_kernel(
    const int64_t *__restrict__ rowptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, int32_t n_cols, int64_t nnz, const int64_t *__restrict__ row_off,
    int64_t n_batches, int64_t max_nnz, PairSlot *__restrict__ tables, int64_t table_stride,
    int32_t *__restrict__ I_col, float *__restrict__ I_val, uint32_t *__restrict__ D,
    int64_t *__restrict__ D_rowptr, int64_t *__restrict__ counts, int32_t *__restrict__ status) {
  __shared__ uint32_t wsum[kEpWaves];
  const int lane = threadIdx.x % kEpWave, wave = threadIdx.x / kEpWave;
  const int64_t base = rowptr[0];
  PairSlot *tab = tables + blockIdx.x * table_stride;
  const uint32_t *colu = (const uint32_t *)col;
  const uint32_t *valu = (const uint32_t *)val;
  for (int64_t b = blockIdx.x; b < n_batches; b += gridDim.x) {
    const int64_t r0 = row_off[b], r1 = row_off[b + 1];
    // row pointers of the batch: non-decreasing and inside [base, base + nnz]
    int bad = 0;
    if (threadIdx.x == 0) {                     // also against the previous batch's end
      const int64_t a = rowptr[r0];
      bad = a < base || a > base + nnz || (r0 > 0 && rowptr[r0 - 1] > a);
    }
    for (int64_t r = r0 + threadIdx.x; r < r1; r += kEpBlock) {
      const int64_t a = rowptr[r], c = rowptr[r + 1];
      bad |= c < a || c > base + nnz;
    }
    int err = __syncthreads_or(bad) ? TOC_ENCDEV_ROWPTR : 0;
    const int64_t e0 = err ? 0 : rowptr[r0] - base, e1 = err ? 0 : rowptr[r1] - base;
    if (!err && e1 - e0 > max_nnz) err = TOC_ENCDEV_SIZE;
    // columns in range and strictly increasing inside each row, values finite; the
    // nonzeros of local tuple i are counted into drp[i + 1]
    int64_t *drp = D_rowptr + r0 + b;
    int bad_col = 0, bad_val = 0;
    if (!err) {
      for (int64_t r = r0 + wave; r < r1; r += kEpWaves) {
        const int64_t a = rowptr[r] - base, c = rowptr[r + 1] - base;
        uint32_t cnt = 0;
        for (int64_t e0r = a; e0r < c; e0r += kEpWave) {
          const int64_t e = e0r + lane;
          bool nz = false;
          if (e < c) {
            const int32_t cc = col[e];
            const uint32_t bits = valu[e];
            bad_col |= cc < 0 || cc >= n_cols || (e > a && col[e - 1] >= cc);
            bad_val |= (bits & 0x7F800000u) == 0x7F800000u;
            nz = (bits & 0x7FFFFFFFu) != 0u;
          }
          cnt += (uint32_t)__popcll(__ballot(nz));
        }
        if (lane == 0) drp[r - r0 + 1] = cnt;
      }
    }
    bad_col = __syncthreads_or(bad_col);
    bad_val = __syncthreads_or(bad_val);
    if (!err && bad_col) err = TOC_ENCDEV_COLUMN;
    if (!err && bad_val) err = TOC_ENCDEV_VALUE;
    if (err) {
      if (threadIdx.x == 0) {
        status[b] = err;
        counts[4 * b] = counts[4 * b + 1] = counts[4 * b + 2] = counts[4 * b + 3] = 0;
      }
      continue;
    }
    const uint32_t n_b = (uint32_t)(e1 - e0);
    const uint32_t n_rows = (uint32_t)(r1 - r0);
    const uint32_t slots = table_slots_dev(n_b), mask = slots - 1;
    for (uint32_t s = threadIdx.x; s < slots; s += kEpBlock) {
      tab[s].key = kEmptyKey;
      tab[s].first = kNone;
      tab[s].node = 0u;
    }
    __threadfence();
    __syncthreads();
    // tuple starts among the nonzeros: drp[i] = nonzeros of tuples 0..i-1
    {
      uint32_t carry = 0;
      for (uint32_t i0 = 0; i0 < n_rows; i0 += kEpBlock) {
        const uint32_t i = i0 + threadIdx.x;
        const uint32_t cnt = i < n_rows ? (uint32_t)load_agent64(&drp[i + 1]) : 0u;
        uint32_t tot;
        const uint32_t ex = block_excl_scan(cnt, wsum, tot);
        if (i < n_rows) drp[i + 1] = carry + ex + cnt;
        carry += tot;
      }
      if (threadIdx.x == 0) drp[0] = 0;
    }
    // every nonzero entry finds or claims its pair's slot and lowers its first
    // position; D receives the slot (kNone for a zero, which the sparse encoding drops)
    for (uint32_t i = threadIdx.x; i < n_b; i += kEpBlock) {
      const int64_t e = e0 + i;
      const uint32_t bits = valu[e];
      uint32_t s = kNone;
      if ((bits & 0x7FFFFFFFu) != 0u) {
        const uint64_t key = ((uint64_t)colu[e] << 32) | bits;
        s = mix64(key) & mask;
        while (true) {
          const unsigned long long old =
              atomicCAS((unsigned long long *)&tab[s].key, (unsigned long long)kEmptyKey,
                        (unsigned long long)key);
          if (old == kEmptyKey || old == key) break;
          s = (s + 1) & mask;
        }
        atomicMin(&tab[s].first, i);
      }
      D[e] = s;
    }
    __threadfence();
    __syncthreads();
    // first appearances in entry order become nodes 1..|I| and the entries of I;
    // the slots of the nonzeros move down to their place among the nonzeros (each
    // chunk reads its slots before any of its threads writes, and writes at or
    // below them)
    uint32_t carry = 0, nzc = 0;
    for (uint32_t i0 = 0; i0 < n_b; i0 += kEpBlock) {
      const uint32_t i = i0 + threadIdx.x;
      const uint32_t s = i < n_b ? D[e0 + i] : kNone;
      const bool first = s != kNone && load_agent(&tab[s].first) == i;
      uint32_t tot, nz_tot;
      const uint32_t ex = block_excl_scan(first ? 1u : 0u, wsum, tot);
      const uint32_t nz_ex = block_excl_scan(s != kNone ? 1u : 0u, wsum, nz_tot);
      if (first) {
        tab[s].node = carry + ex + 1;
        I_col[e0 + carry + ex] = col[e0 + i];
        I_val[e0 + carry + ex] = val[e0 + i];
      }
      if (s != kNone) D[e0 + nzc + nz_ex] = s;
      carry += tot;
      nzc += nz_tot;
    }
    __threadfence();
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < nzc; i += kEpBlock) D[e0 + i] = load_agent(&tab[D[e0 + i]].node);
    if (threadIdx.x == 0) {
      counts[4 * b] = carry;
      counts[4 * b + 3] = nzc;
      status[b] = 0;
    }
    __threadfence();
    __syncthreads();                            // the table is cleared for the next batch
  }
}

// Phase II: lane g runs batches g, g + n_lanes, ...
__global__ __launch_bounds__(kEtBlock) void enc_tuples_kernel(
    const int64_t *__restrict__ rowptr, const int64_t *__restrict__ row_off, int64_t n_batches,
    int64_t n_lanes, ChildSlot *__restrict__ tables, int64_t table_stride, uint32_t *D,
    int64_t *__restrict__ D_rowptr, int64_t *__restrict__ counts,
    const int32_t *__restrict__ status) {
  const int64_t g = (int64_t)blockIdx.x * kEtBlock + threadIdx.x;
  if (g >= n_lanes) return;
  const int64_t base = rowptr[0];
  uint4 *slots4 = (uint4 *)(tables + g * table_stride);   // (key lo, key hi, child, tag)
  for (int64_t b = g; b < n_batches; b += n_lanes) {
    if (status[b] != 0) continue;
    const int64_t r0 = row_off[b], r1 = row_off[b + 1];
    const int64_t e0 = rowptr[r0] - base;
    const uint32_t mask = table_slots_dev((uint32_t)(rowptr[r1] - base - e0)) - 1;
    const uint32_t tag = (uint32_t)b;
    uint32_t next = (uint32_t)counts[4 * b] + 1;     // next node index (Algorithm 1's AddNode)
    int64_t q = e0;                                    // where the next code goes
    int64_t *drp = D_rowptr + r0 + b;
    int64_t start = e0;                                // tuple starts among the nonzeros
    for (int64_t i = 0; i < r1 - r0; ++i) {
      const int64_t end = e0 + drp[i + 1];
      drp[i] = q - e0;
      int64_t p = start;
      start = end;
      if (p == end) continue;
      // longest matches from the tree; n is the match so far, pc the pair of entry p
      // (as its first-layer node), pn the pair after it, loaded ahead of the probe
      uint32_t n = D[p++];
      uint32_t pc = p < end ? D[p] : 0u;
      while (p < end) {
        // one 16-byte load per probed slot, issued ahead of the next pair's load
        const uint64_t key = ((uint64_t)n << 32) | pc;
        uint32_t s = mix64(key) & mask;
        uint4 v = slots4[s];
        const uint32_t pn = D[p + 1 < end ? p + 1 : p];   // used only when p + 1 < end
        while (true) {
          const bool own = v.w == tag, same = ((v.x ^ (uint32_t)key) | (v.y ^ n)) == 0u;
          if (!own | same) break;
          s = (s + 1) & mask;
          v = slots4[s];
        }
        if (v.w == tag) {
          n = v.z;                              // the match goes on through entry p
        } else {                                // the match ends before entry p: emit it and
          D[q++] = n;                           // grow the tree by n extended with entry p
          slots4[s] = make_uint4((uint32_t)key, n, next++, tag);
          n = pc;
        }
        ++p;
        pc = pn;
      }
      D[q++] = n;                               // the last match ends the tuple
    }
    drp[r1 - r0] = q - e0;
    counts[4 * b + 1] = q - e0;
    counts[4 * b + 2] = next;
  }
}

inline int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

struct Plan {
  int64_t groups, lanes, pair_stride, child_stride, off_pair, off_child, end;
};

Plan plan(int64_t n_batches, int64_t max_nnz) {
  Plan p{};
  const int64_t slots = table_slots(max_nnz);
  p.pair_stride = p.child_stride = slots;
  const int64_t table_bytes = slots * (int64_t)sizeof(PairSlot);
  p.groups = std::max<int64_t>(1, std::min({n_batches, kMaxPairGroups, kTableBudget / table_bytes}));
  p.lanes = std::max<int64_t>(1, std::min({n_batches, kMaxLanes, kTableBudget / table_bytes}));
  p.off_pair = align256(8 * (n_batches + 1));
  p.off_child = p.off_pair + align256(p.groups * table_bytes);
  p.end = p.off_child + align256(p.lanes * slots * (int64_t)sizeof(ChildSlot));
  return p;
}

constexpr int64_t kMaxBatchNnz = (int64_t)1 << 30;

}  // namespace

using namespace toc;

extern "C" {

toc_status toc_encode_device_workspace_size(int64_t n_batches, int64_t max_nnz, size_t *bytes) {
  clear_error();
  if (!bytes || n_batches < 0 || max_nnz < 0) return fail(TOC_EINVAL, "bad argument");
  if (max_nnz > kMaxBatchNnz) return fail(TOC_EUNSUPPORTED, "max_nnz above 2^30");
  *bytes = n_batches == 0 ? 0 : (size_t)plan(n_batches, max_nnz).end;
  return TOC_OK;
}

toc_status toc_encode_device(int64_t n_batches, const int32_t *n_rows, int32_t n_cols,
                             const int64_t *rowptr, const int32_t *col, const float *val,
                             int64_t nnz, int64_t max_nnz, int32_t *I_col, float *I_val,
                             uint32_t *D_codes, int64_t *D_rowptr, int64_t *counts,
                             int32_t *status, void *ws, size_t ws_bytes, void *stream) {
  clear_error();
  if (n_batches < 0 || nnz < 0 || max_nnz < 0 || n_cols < 0) return fail(TOC_EINVAL, "negative size");
  if (max_nnz > kMaxBatchNnz) return fail(TOC_EUNSUPPORTED, "max_nnz above 2^30");
  if (n_batches >= (int64_t)kNone) return fail(TOC_EUNSUPPORTED, "2^32-1 batches or more");
  if (n_batches == 0) return TOC_OK;
  if (!n_rows || !rowptr || !D_rowptr || !counts || !status || !ws)
    return fail(TOC_EINVAL, "NULL argument");
  if (nnz > 0 && (!col || !val || !I_col || !I_val || !D_codes))
    return fail(TOC_EINVAL, "NULL entry array");
  std::vector<int64_t> row_off(n_batches + 1, 0);
  for (int64_t b = 0; b < n_batches; ++b) {
    if (n_rows[b] < 0) return fail(TOC_EINVAL, "n_rows[%lld] < 0", (long long)b);
    row_off[b + 1] = row_off[b] + n_rows[b];
  }
  size_t need = 0;
  toc_encode_device_workspace_size(n_batches, max_nnz, &need);
  if (ws_bytes < need) return fail(TOC_ESIZE, "workspace of %zu bytes below the %zu needed", ws_bytes, need);
  const Plan p = plan(n_batches, max_nnz);
  hipStream_t s = (hipStream_t)stream;
  uint8_t *w = (uint8_t *)ws;
  int64_t *roff = (int64_t *)w;
  if (hipMemcpyAsync(roff, row_off.data(), 8 * (n_batches + 1), hipMemcpyHostToDevice, s) !=
          hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(TOC_EDEVICE, "copy of the row offsets failed");
  ChildSlot *ctab = (ChildSlot *)(w + p.off_child);
  // tags of 0xFFFFFFFF name no batch: every child table starts empty
  if (hipMemsetAsync(ctab, 0xFF, (size_t)(p.lanes * p.child_stride) * sizeof(ChildSlot), s) !=
      hipSuccess)
    return fail(TOC_EDEVICE, "clearing the child tables failed");
  hipLaunchKernelGGL(enc_pairs_kernel, dim3((unsigned)p.groups), dim3(kEpBlock), 0, s, rowptr, col,
                     val, n_cols, nnz, roff, n_batches, max_nnz, (PairSlot *)(w + p.off_pair),
                     p.pair_stride, I_col, I_val, D_codes, D_rowptr, counts, status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "enc_pairs_kernel: %s", hipGetErrorString(e));
  hipLaunchKernelGGL(enc_tuples_kernel, dim3((unsigned)((p.lanes + kEtBlock - 1) / kEtBlock)),
                     dim3(kEtBlock), 0, s, rowptr, roff, n_batches, p.lanes, ctab, p.child_stride,
                     D_codes, D_rowptr, counts, status);
  e = hipGetLastError();
  if (e != hipSuccess) return fail(TOC_EDEVICE, "enc_tuples_kernel: %s", hipGetErrorString(e));
  return TOC_OK;
}

}  // extern "C"
