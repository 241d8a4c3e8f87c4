// Mini-batch gradient descent for the feed-forward neural network of section 5.1
// on the uploaded image: two sigmoid hidden layers, a softmax output (or one
// sigmoid output), cross-entropy loss, one step per batch (section 2.1's update
// with the batch mean).  The first layer runs on the compressed batch: its
// forward product A.W1 is Table 1's A.M (Theorem 1: the dictionary table
// H[c] = H[parent] + val * W1[col] over the deep codes, summed over each tuple's
// codes) and its weight gradient A^T dZ1 is Table 1's M.A (Theorem 2: the rows of
// dZ1 summed per code, children added into parents deepest first, val * H summed
// per key column).  A step is four launches:
//   mlp_fwd1_kernel  one workgroup per 4 hidden units: Z1 = A W1 + b1, H1 = s(Z1)
//   mlp_rows_kernel  workgroups over the tuples: layers 2 and 3, the loss gradient,
//                    dZ3, dZ2 and dZ1
//   mlp_grad_kernel  the gradients and updates of W2, b2, W3, b3
//   mlp_bwd1_kernel  one workgroup per 4 hidden units: A^T dZ1, updates of W1, b1
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "toc_internal.h"

namespace {

constexpr int kNnBlock = 1024;
constexpr int kNnLanes = 16;                 // lanes per tuple in the forward product
constexpr int kNnCodes = 8;                  // a lane's codes whose loads fly together there
constexpr uint32_t kNnFirst = 0x80000000u;   // first-occurrence bit of a leaf occurrence
constexpr size_t kNnLdsMax = 160 * 1024;
constexpr int kColGroups = 8;                // workgroups sharing a slice's key columns

struct NnImg {
  const toc_batch *batches;
  const uint32_t *level;
  const toc_key *key;
  const toc_link *link;
  const uint32_t *span, *dcodes, *occ_off, *tlist, *cols, *tchild, *centry, *cval;
};

__device__ inline float sigm(float x) { return 1.0f / (1.0f + expf(-x)); }

__device__ inline float4 fma4(float a, float4 w, float4 s) {
  return make_float4(fmaf(a, w.x, s.x), fmaf(a, w.y, s.y), fmaf(a, w.z, s.z), fmaf(a, w.w, s.w));
}
__device__ inline float4 add4(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

// Barrier after a level of table rows: rows kept in global memory also need their
// stores made visible to the workgroup's other waves.
template <bool kGlobal>
__device__ inline void rows_barrier() {
  if (kGlobal) __threadfence();
  __syncthreads();
}

// Forward first layer for hidden units u0 .. u0+3 (u0 = 4 blockIdx.x): the rows of
// the deep codes' table in LDS (or, when a batch has too many, in the workspace),
// level by level (a depth-1 code's row is val * W1[col], read when needed), then
// each tuple's sum by a 16-lane group; blockIdx.y picks 64 of the tuples.
template <bool kGlobal>
__global__ __launch_bounds__(kNnBlock) void mlp_fwd1_kernel(NnImg im, int64_t b,
                                                            const float *__restrict__ W1, int h1,
                                                            const float *__restrict__ b1,
                                                            float *__restrict__ act1,
                                                            float4 *rows_g, int64_t rows_stride) {
  extern __shared__ float4 rows_l[];
  // deep code c at Hd[c - n_lvl1]; each workgroup builds its own copy
  float4 *Hd = kGlobal ? rows_g + (blockIdx.y * gridDim.x + blockIdx.x) * rows_stride : rows_l;
  const toc_batch bt = im.batches[b];
  const int u0 = 4 * blockIdx.x;
  const uint32_t n1 = (uint32_t)bt.n_lvl1;
  const uint32_t *lvl = im.level + bt.lvl_base;
  const toc_key *key = im.key + bt.code_base;
  const toc_link *link = im.link + (bt.deep_base - (int64_t)bt.n_lvl1);   // depth >= 2 only
  auto wrow = [&](uint32_t col) { return *(const float4 *)(W1 + (int64_t)col * h1 + u0); };
  for (int d = 2; d <= bt.n_levels; ++d) {
    const uint32_t a = lvl[d - 1], e = lvl[d];
    for (uint32_t c = a + threadIdx.x; c < e; c += kNnBlock) {
      const toc_key k = key[c];
      const uint32_t p = link[c].parent;
      float4 base;
      if (p < n1) {
        const toc_key kp = key[p];
        base = fma4(kp.val, wrow(kp.col), make_float4(0.f, 0.f, 0.f, 0.f));
      } else {
        base = Hd[p - n1];
      }
      Hd[c - n1] = fma4(k.val, wrow(k.col), base);
    }
    rows_barrier<kGlobal>();
  }
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % kNnLanes, grp = threadIdx.x / kNnLanes;
  const float4 bias = *(const float4 *)(b1 + u0);
  const int r = blockIdx.y * (kNnBlock / kNnLanes) + grp;
  if (r < bt.n_rows) {
    const uint32_t s = span[r], e = span[r + 1];
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    // kNnCodes of the lane's codes at a time: their codes, then their keys, then
    // their rows are loaded together, and summed in order
    for (uint32_t j0 = s + lane; j0 < e; j0 += kNnLanes * kNnCodes) {
      uint32_t c[kNnCodes];
      toc_key k[kNnCodes];
      float4 w[kNnCodes];
#pragma unroll
      for (int q = 0; q < kNnCodes; ++q) {
        const uint32_t j = j0 + (uint32_t)(q * kNnLanes);
        c[q] = j < e ? dc[j] : 0xFFFFFFFFu;
      }
#pragma unroll
      for (int q = 0; q < kNnCodes; ++q) k[q] = c[q] < n1 ? key[c[q]] : toc_key{0u, 0.0f};
#pragma unroll
      for (int q = 0; q < kNnCodes; ++q) {
        w[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (c[q] < n1) w[q] = wrow(k[q].col);
        else if (c[q] != 0xFFFFFFFFu) w[q] = Hd[c[q] - n1];
      }
#pragma unroll
      for (int q = 0; q < kNnCodes; ++q) {
        if (c[q] < n1) acc = fma4(k[q].val, w[q], acc);
        else if (c[q] != 0xFFFFFFFFu) acc = add4(acc, w[q]);
      }
    }
#pragma unroll
    for (int o = kNnLanes / 2; o > 0; o >>= 1) {
      acc.x += __shfl_xor(acc.x, o, kNnLanes);
      acc.y += __shfl_xor(acc.y, o, kNnLanes);
      acc.z += __shfl_xor(acc.z, o, kNnLanes);
      acc.w += __shfl_xor(acc.w, o, kNnLanes);
    }
    if (lane == 0) {
      float4 z = add4(acc, bias);
      *(float4 *)(act1 + (int64_t)r * h1 + u0) = make_float4(sigm(z.x), sigm(z.y), sigm(z.z), sigm(z.w));
    }
  }
}

// Layers 2 and 3 for R tuples of a batch of n (rows R blockIdx.x onwards), and the
// gradient of the mean loss back to dZ1: every quantity here belongs to one tuple,
// so workgroups split the tuples.  H2, dZ2 and dZ3 go to the workspace for the
// weight gradients, dZ1 for the first layer's left product.
// n floats src(x) into LDS dst[x] by a workgroup of NT threads, each with kStagePer
// loads in flight before its stores (one load latency per pass, not per element)
constexpr int kStagePer = 8;
template <int NT, typename F>
__device__ inline void stage(float *dst, int n, F src) {
  for (int x0 = threadIdx.x; x0 < n; x0 += kStagePer * NT) {
    float t[kStagePer];
#pragma unroll
    for (int k = 0; k < kStagePer; ++k) {
      const int x = x0 + k * NT;
      t[k] = x < n ? src(x) : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < kStagePer; ++k) {
      const int x = x0 + k * NT;
      if (x < n) dst[x] = t[k];
    }
  }
}

template <bool kWlds>
__global__ __launch_bounds__(kNnBlock) void mlp_rows_kernel(
    int n, int R, int64_t row_base, const float *__restrict__ act1, int h1, int h2, int C,
    const float *__restrict__ W2g, const float *__restrict__ b2, const float *__restrict__ W3g,
    const float *__restrict__ b3, const int32_t *__restrict__ labels, float *__restrict__ H2g,
    float *__restrict__ dZ2g, float *__restrict__ dZ3g, float *__restrict__ dz1) {
  extern __shared__ float sm[];
  float *A = sm;                       // R x h1: the tuples' first-layer activations
  float *H = A + R * h1;               // R x h2
  float *G = H + R * h2;               // R x h2: dZ2
  float *Z = G + R * h2;               // R x C: Z3, then dZ3
  // W2 and W3 staged in LDS when they fit (kWlds), else read from global memory
  float *W2s = Z + R * C, *W3s = W2s + h1 * h2;
  const float *W2 = kWlds ? W2s : W2g, *W3 = kWlds ? W3s : W3g;
  const int i0 = R * blockIdx.x, nr = min(R, n - i0);
  stage<kNnBlock>(A, nr * h1, [&](int x) { return act1[(int64_t)i0 * h1 + x]; });
  if (kWlds) {
    stage<kNnBlock>(W2s, h1 * h2, [&](int x) { return W2g[x]; });
    stage<kNnBlock>(W3s, h2 * C, [&](int x) { return W3g[x]; });
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nr * h2; idx += kNnBlock) {
    const int i = idx / h2, u = idx - i * h2;
    const float *a = A + i * h1;
    float z = b2[u];
    for (int v = 0; v < h1; ++v) z = fmaf(a[v], W2[v * h2 + u], z);
    const float hv = sigm(z);
    H[idx] = hv;
    H2g[(int64_t)i0 * h2 + idx] = hv;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nr * C; idx += kNnBlock) {
    const int i = idx / C, c = idx - i * C;
    float z = b3[c];
    for (int u = 0; u < h2; ++u) z = fmaf(H[i * h2 + u], W3[u * C + c], z);
    Z[idx] = z;
  }
  __syncthreads();
  const float inv_n = 1.0f / (float)n;
  for (int i = threadIdx.x; i < nr; i += kNnBlock) {
    float *z = Z + i * C;
    const int y = labels[row_base + i0 + i];
    if (C == 1) {
      z[0] = (sigm(z[0]) - (y == 1 ? 1.0f : 0.0f)) * inv_n;
    } else {
      float mx = z[0];
      for (int c = 1; c < C; ++c) mx = fmaxf(mx, z[c]);
      float sum = 0.0f;
      for (int c = 0; c < C; ++c) {
        z[c] = expf(z[c] - mx);
        sum += z[c];
      }
      const float inv = 1.0f / sum;
      for (int c = 0; c < C; ++c) z[c] = (z[c] * inv - (c == y ? 1.0f : 0.0f)) * inv_n;
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nr * C; idx += kNnBlock) dZ3g[(int64_t)i0 * C + idx] = Z[idx];
  for (int idx = threadIdx.x; idx < nr * h2; idx += kNnBlock) {
    const int i = idx / h2, u = idx - i * h2;
    float g = 0.0f;
    for (int c = 0; c < C; ++c) g = fmaf(Z[i * C + c], W3[u * C + c], g);
    const float hv = H[idx];
    g = g * hv * (1.0f - hv);
    G[idx] = g;
    dZ2g[(int64_t)i0 * h2 + idx] = g;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < nr * h1; idx += kNnBlock) {
    const int i = idx / h1, v = idx - i * h1;
    const float *w = W2 + (int64_t)v * h2;
    const float *g2 = G + i * h2;
    float g = 0.0f;
    for (int u = 0; u < h2; ++u) g = fmaf(g2[u], w[u], g);
    const float a = A[idx];
    dz1[(int64_t)i0 * h1 + idx] = g * a * (1.0f - a);
  }
}

// Weight gradients of layers 2 and 3 (sums over the batch's n tuples) and their
// updates.  Workgroups below n_w2 each take a V x U block of W2 (U = min(h2, 256),
// V = 256 / U), summing over the tuples ch2 at a time with the block's columns of
// H1 and dZ2 staged in LDS (the blocks of W2's first rows also sum b2's gradient);
// the workgroups after them take 256 entries each of W3 and b3, the tuples ch3 at
// a time.  The host makes a chunk the whole batch when its rows fit 96 KiB, so a
// step stages its inputs with one load latency.  Runs after every tuple's dZ1 was
// computed from the old W2.

__global__ __launch_bounds__(256) void mlp_grad_kernel(
    int n, int n_w2, const float *__restrict__ act1, int h1, int h2, int C,
    const float *__restrict__ H2g, const float *__restrict__ dZ2g, const float *__restrict__ dZ3g,
    float lr, float *__restrict__ W2, float *__restrict__ b2, float *__restrict__ W3,
    float *__restrict__ b3, int ch2, int ch3) {
  extern __shared__ float gs[];
  if ((int)blockIdx.x < n_w2) {
    const int U = min(h2, 256), V = 256 / U, nub = (h2 + U - 1) / U;
    const int v0 = (blockIdx.x / nub) * V, u0 = (blockIdx.x % nub) * U;
    float *As = gs, *Gs = gs + ch2 * V;
    const int lv = threadIdx.x / U, lu = threadIdx.x - lv * U;
    const int v = v0 + lv, u = u0 + lu;
    float g = 0.0f, gb = 0.0f;                  // gb: b2's gradient, by the first row of blocks
    for (int i0 = 0; i0 < n; i0 += ch2) {
      const int ni = min(ch2, n - i0);
      stage<256>(As, ni * V, [&](int x) {
        const int ii = x / V, vv = v0 + (x - ii * V);
        return vv < h1 ? act1[(int64_t)(i0 + ii) * h1 + vv] : 0.0f;
      });
      stage<256>(Gs, ni * U, [&](int x) {
        const int ii = x / U, uu = u0 + (x - ii * U);
        return uu < h2 ? dZ2g[(int64_t)(i0 + ii) * h2 + uu] : 0.0f;
      });
      __syncthreads();
      if (lv < V)
        for (int ii = 0; ii < ni; ++ii) g = fmaf(As[ii * V + lv], Gs[ii * U + lu], g);
      if (v0 == 0 && lv == 0)
        for (int ii = 0; ii < ni; ++ii) gb += Gs[ii * U + lu];
      __syncthreads();
    }
    if (lv < V && v < h1 && u < h2) W2[v * h2 + u] = fmaf(-lr, g, W2[v * h2 + u]);
    if (v0 == 0 && lv == 0 && u < h2) b2[u] = fmaf(-lr, gb, b2[u]);
    return;
  }
  // W3 and b3 (b3 as a row of W3 whose H2 column is 1), tuples staged TI at a time
  const int TI = ch3;
  float *Hs = gs, *Zs = gs + TI * h2;
  const int n_out3 = (h2 + 1) * C;
  {
    const int idx = ((int)blockIdx.x - n_w2) * 256 + threadIdx.x, u = idx / C, c = idx - u * C;
    float g = 0.0f;
    for (int i0 = 0; i0 < n; i0 += TI) {
      const int ni = min(TI, n - i0);
      stage<256>(Hs, ni * h2, [&](int x) { return H2g[(int64_t)i0 * h2 + x]; });
      stage<256>(Zs, ni * C, [&](int x) { return dZ3g[(int64_t)i0 * C + x]; });
      __syncthreads();
      if (idx < n_out3)
        for (int ii = 0; ii < ni; ++ii) g = fmaf(u < h2 ? Hs[ii * h2 + u] : 1.0f, Zs[ii * C + c], g);
      __syncthreads();
    }
    if (idx < h2 * C) W3[idx] = fmaf(-lr, g, W3[idx]);
    else if (idx < n_out3) b3[c] = fmaf(-lr, g, b3[c]);
  }
}

// Weight gradient of the first layer for hidden units u0 .. u0+3, by pulling:
// each tree code's row is the sum of dZ1 over the tuples holding it, then
// children are added into parents deepest first; each key column's gradient sums
// val * (dZ1 row) over its leaf occurrences and val * (tree row) over its tree
// codes.  16-lane groups take one tree code, then one column, at a time (columns
// with the most entries first, dealt round-robin to the kColGroups workgroups of
// the slice), so a code or column with many occurrences is summed by 16 lanes;
// sums are reduced in a fixed order.
// Reads the arrays of batch b that the next step's kernels read (one word of every
// 128-byte line), so that they find them in L2: the step's kernels gather from
// them with little else to overlap.  One workgroup per XCD runs it, each reading
// the whole batch into its XCD's L2.
__device__ void nn_read_ahead(const NnImg &im, int64_t b, int32_t m, const int32_t *labels) {
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
      {im.cols + b * 4 * (int64_t)(m + 1), 4 * 4 * (int64_t)(m + 1)},
      {im.tchild + bt.tree_base + b, 4 * (nt + 1)},
      {im.level + bt.lvl_base, 4 * ((int64_t)bt.n_levels + 1)},
      {labels + bt.row_base, 4 * nr},
  };
  uint32_t acc = 0;
  for (const Range &x : r)
    for (int64_t o = (int64_t)threadIdx.x * 128; o < x.bytes; o += (int64_t)kNnBlock * 128)
      acc += *(const uint32_t *)((const char *)x.p + o);
  asm volatile("" : : "v"(acc));    // the loads are the point: keep them
}

template <bool kGlobal>
__global__ __launch_bounds__(kNnBlock) void mlp_bwd1_kernel(NnImg im, int64_t b, int32_t m,
                                                            const float *__restrict__ dz1, int h1,
                                                            float lr, float *__restrict__ W1,
                                                            float *__restrict__ b1, float4 *rows_g,
                                                            int64_t rows_stride, int64_t next,
                                                            const int32_t *__restrict__ labels) {
  // the grid's last row: the first 8 workgroups (one per XCD) read the next
  // step's batch ahead, the others have nothing to do
  if (blockIdx.y == kColGroups) {
    if (next >= 0 && blockIdx.x < 8) nn_read_ahead(im, next, m, labels);
    return;
  }
  extern __shared__ float4 rows_l[];
  // tree code c at Ht[c < ni ? c : c - n1 + ni]; each workgroup builds its own copy
  float4 *Ht = kGlobal ? rows_g + (blockIdx.y * gridDim.x + blockIdx.x) * rows_stride : rows_l;
  const toc_batch bt = im.batches[b];
  const int u0 = 4 * blockIdx.x;
  const uint32_t n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1, nc = (uint32_t)bt.n_codes;
  const uint32_t n_tree = ni + (nc - n1);
  const uint32_t *lvl = im.level + bt.lvl_base;
  // tree row t's tuples: entries to[t] .. to[t+1]-1 of the batch's entry array
  const uint32_t *to = im.occ_off + bt.code_base + 2 * b + (n1 - ni) + 1;
  const uint32_t *ce = im.centry + bt.d_base + bt.tree_base;
  const uint32_t *cv = im.cval + bt.d_base + bt.tree_base;
  const int lane = threadIdx.x % kNnLanes, grp = threadIdx.x / kNnLanes;
  constexpr int kGroups = kNnBlock / kNnLanes;
  auto grow = [&](uint32_t row) { return *(const float4 *)(dz1 + (int64_t)row * h1 + u0); };
  auto group_sum = [&](float4 v) {
#pragma unroll
    for (int o = kNnLanes / 2; o > 0; o >>= 1) {
      v.x += __shfl_xor(v.x, o, kNnLanes);
      v.y += __shfl_xor(v.y, o, kNnLanes);
      v.z += __shfl_xor(v.z, o, kNnLanes);
      v.w += __shfl_xor(v.w, o, kNnLanes);
    }
    return v;
  };
  for (uint32_t t0 = 0; t0 < n_tree; t0 += kGroups) {
    const uint32_t t = t0 + grp;
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t < n_tree) {
      const uint32_t o1 = to[t + 1];
      for (uint32_t o = to[t] + lane; o < o1; o += kNnLanes) s = add4(s, grow(ce[o]));
    }
    s = group_sum(s);
    if (t < n_tree && lane == 0) Ht[t] = s;
  }
  rows_barrier<kGlobal>();
  const uint32_t *tch = im.tchild + bt.tree_base + b;
  for (int d = bt.n_levels - 1; d >= 1; --d) {
    const uint32_t a = d == 1 ? 0u : lvl[d - 1], e = d == 1 ? ni : lvl[d];
    for (uint32_t c = a + threadIdx.x; c < e; c += kNnBlock) {
      const uint32_t t = c < ni ? c : c - n1 + ni;
      float4 s = Ht[t];
      const uint32_t c1 = tch[t + 1];
      for (uint32_t ch = tch[t]; ch < c1; ++ch) s = add4(s, Ht[ch - n1 + ni]);
      Ht[t] = s;
    }
    rows_barrier<kGlobal>();
  }
  const uint32_t *cx = im.cols + b * 4 * (int64_t)(m + 1);
  const uint32_t *Ost = cx + (m + 1), *Toff = cx + 2 * (m + 1), *Ord = cx + 3 * (m + 1);
  const uint32_t n_lo = Ost[m];   // leaf occurrences; the tree codes' entries follow
  for (int k = blockIdx.y * kGroups + grp; k < m; k += kGroups * kColGroups) {
    const uint32_t j = Ord[k];
    const uint32_t lst = Ost[j], tst = n_lo + Toff[j];
    const uint32_t nl = Ost[j + 1] - Ost[j], nt = Toff[j + 1] - Toff[j];
    if (nl + nt == 0) continue;                // no entry: the column's gradient is 0
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    // the column's leaf occurrences (val * dZ1 row of the tuple), then its tree
    // codes (val * tree row), the multiplier beside each entry
    for (uint32_t q = lane; q < nl + nt; q += kNnLanes) {
      const uint32_t at = q < nl ? lst + q : tst + (q - nl);
      const uint32_t w = ce[at];
      const float v = __uint_as_float(cv[at]);
      if (q < nl) {
        s = fma4(v, grow(w & ~kNnFirst), s);
      } else {
        const uint32_t c = w & ~toc::kTreeEntry;
        s = fma4(v, Ht[c < ni ? c : c - n1 + ni], s);
      }
    }
    s = group_sum(s);
    if (lane == 0) {
      float4 *wp = (float4 *)(W1 + (int64_t)j * h1 + u0);
      const float4 old = *wp;
      *wp = make_float4(fmaf(-lr, s.x, old.x), fmaf(-lr, s.y, old.y), fmaf(-lr, s.z, old.z),
                        fmaf(-lr, s.w, old.w));
    }
  }
  // the bias: dZ1 summed over the tuples, by the first wave of column group 0
  if (blockIdx.y == 0 && threadIdx.x < 64) {
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i = threadIdx.x; i < bt.n_rows; i += 64) s = add4(s, grow((uint32_t)i));
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      s.x += __shfl_xor(s.x, o, 64);
      s.y += __shfl_xor(s.y, o, 64);
      s.z += __shfl_xor(s.z, o, 64);
      s.w += __shfl_xor(s.w, o, 64);
    }
    if (threadIdx.x == 0) {
      float4 *bb = (float4 *)(b1 + u0);
      const float4 old = *bb;
      *bb = make_float4(fmaf(-lr, s.x, old.x), fmaf(-lr, s.y, old.y), fmaf(-lr, s.z, old.z),
                        fmaf(-lr, s.w, old.w));
    }
  }
}

toc_status allow(const void *kernel, size_t lds) {
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return toc::fail(TOC_EDEVICE, "cannot raise dynamic LDS to %zu bytes", lds);
  return TOC_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int64_t align4(int64_t x) { return (x + 3) & ~(int64_t)3; }

// Workgroups of 64 tuples the forward kernel uses for the batch with the most rows.
int64_t row_groups_max(const toc_dev *d) {
  return std::max<int64_t>(1, (d->max_rows + kNnBlock / kNnLanes - 1) / (kNnBlock / kNnLanes));
}

// Tuples per workgroup of mlp_rows_kernel: up to 8, as many as fit 40 KiB of LDS.
int rows_per_group(int h1, int h2, int C) {
  const int per = h1 + 2 * h2 + C;
  return std::max(1, std::min(8, (40 * 1024 / 4) / per));
}

// Most deep codes and most tree codes (depth-1 codes with children plus deep
// codes) of a batch in b0 .. b1-1; the table rows of a slice of 4 hidden units
// stay in LDS when they fit, else they go to the workspace.
struct Rows {
  int64_t max_deep, max_tree;
  bool deep_global, tree_global;
};

Rows table_rows(const toc_dev *d, int64_t b0, int64_t b1) {
  Rows r{0, 0, false, false};
  for (int64_t b = b0; b < b1; ++b) {
    const toc_batch &bt = d->batches[b];
    r.max_deep = std::max<int64_t>(r.max_deep, bt.n_codes - bt.n_lvl1);
    r.max_tree = std::max<int64_t>(r.max_tree, bt.n_int1 + bt.n_codes - bt.n_lvl1);
  }
  r.deep_global = r.max_deep * 16 > (int64_t)kNnLdsMax;
  r.tree_global = r.max_tree * 16 > (int64_t)kNnLdsMax;
  return r;
}

}  // namespace

using namespace toc;

extern "C" {

toc_status toc_mlp_workspace_size(const toc_dev *d, int32_t h1, int32_t h2, int32_t n_out,
                                  size_t *bytes) {
  clear_error();
  if (!d || !bytes || h1 < 1 || h2 < 1 || n_out < 1) return fail(TOC_EINVAL, "bad argument");
  const Rows r = table_rows(d, 0, d->info.n_batches);
  const int64_t nr = d->max_rows;
  const int64_t rows = align4(nr * h1) * 2 + align4(nr * h2) * 2 + align4(nr * n_out);
  *bytes = (size_t)(rows + (r.deep_global ? r.max_deep * h1 * row_groups_max(d) : 0) +
                    (r.tree_global ? r.max_tree * h1 * kColGroups : 0)) * 4;
  return TOC_OK;
}

toc_status toc_mlp_epoch(const toc_dev *d, int64_t b0, int64_t n_batches, int32_t h1, int32_t h2,
                         int32_t n_out, float *W1, float *b1, float *W2, float *b2, float *W3,
                         float *b3, const int32_t *labels, float lr, void *ws, size_t ws_bytes,
                         void *stream) {
  clear_error();
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
  if (h1 < 4 || h1 % 4 != 0 || h1 > 4096) return fail(TOC_EUNSUPPORTED, "h1 must be a multiple of 4 in 4..4096");
  if (h2 < 1 || n_out < 1 || h2 > 4096 || n_out > 4096) return fail(TOC_EINVAL, "h2 and n_out must be in 1..4096");
  if (!std::isfinite(lr)) return fail(TOC_EINVAL, "learning rate not finite");
  if (n_batches == 0) return TOC_OK;
  if (!W1 || !b1 || !W2 || !b2 || !W3 || !b3 || !labels || !ws) return fail(TOC_EINVAL, "NULL pointer");
  if (!aligned16(W1) || !aligned16(b1) || !aligned16(ws))
    return fail(TOC_EINVAL, "W1, b1 and ws must be 16-byte aligned");
  size_t need = 0;
  toc_mlp_workspace_size(d, h1, h2, n_out, &need);
  if (ws_bytes < need) return fail(TOC_ESIZE, "workspace of %zu bytes below the %zu needed", ws_bytes, need);
  // table rows sized for the whole image, so that the workspace layout does not
  // depend on the batch range
  const Rows rw = table_rows(d, 0, nb);
  const size_t lds_f = rw.deep_global ? 0 : (size_t)std::max<int64_t>(rw.max_deep, 1) * 16;
  const size_t lds_b = rw.tree_global ? 0 : (size_t)std::max<int64_t>(rw.max_tree, 1) * 16;
  const int R = rows_per_group(h1, h2, n_out);
  const size_t lds_r0 = (size_t)R * (h1 + 2 * h2 + n_out) * 4;
  const size_t lds_w = ((size_t)h1 * h2 + (size_t)h2 * n_out) * 4;
  const bool w_lds = lds_r0 + lds_w <= 96 * 1024;
  const size_t lds_r = lds_r0 + (w_lds ? lds_w : 0);
  const int gU = std::min(h2, 256), gV = 256 / gU;
  const int n_w2 = ((h1 + gV - 1) / gV) * ((h2 + gU - 1) / gU);
  const int n_w3 = ((h2 + 1) * n_out + 255) / 256;
  // W2 blocks stage ch2 (U + V) floats, the W3 workgroups ch3 (h2 + n_out): as
  // many tuples as 96 KiB holds, at most a batch
  const int ch_max = std::max<int32_t>(d->max_rows, 1);
  const int ch2 = std::max(1, std::min(ch_max, 24576 / (gU + gV)));
  const int ch3 = std::max(1, std::min(ch_max, 24576 / (h2 + n_out)));
  const size_t lds_g = (size_t)std::max(ch2 * (gU + gV), ch3 * (h2 + n_out)) * 4;
  toc_status st;
  if ((st = allow((const void *)mlp_fwd1_kernel<false>, lds_f)) ||
      (st = allow((const void *)mlp_bwd1_kernel<false>, lds_b)) ||
      (st = allow(w_lds ? (const void *)mlp_rows_kernel<true> : (const void *)mlp_rows_kernel<false>,
                  lds_r)) ||
      (st = allow((const void *)mlp_grad_kernel, lds_g)))
    return st;
  const uint8_t *base = (const uint8_t *)d->buf;
  const toc_layout &L = d->layout;
  const NnImg im{(const toc_batch *)(base + L.batches), (const uint32_t *)(base + L.level),
                 (const toc_key *)(base + L.key), (const toc_link *)(base + L.link),
                 (const uint32_t *)(base + L.span), (const uint32_t *)(base + L.dcodes),
                 (const uint32_t *)(base + L.occ_off), (const uint32_t *)(base + L.tlist),
                 (const uint32_t *)(base + L.cols), (const uint32_t *)(base + L.tchild),
                 (const uint32_t *)(base + L.centry), (const uint32_t *)(base + L.cval)};
  const int64_t nr = d->max_rows;
  float *act1 = (float *)ws;
  float *dz1 = act1 + align4(nr * h1);
  float *H2g = dz1 + align4(nr * h1);
  float *dZ2g = H2g + align4(nr * h2);
  float *dZ3g = dZ2g + align4(nr * h2);
  float4 *deep_rows = (float4 *)(dZ3g + align4(nr * n_out));
  float4 *tree_rows = deep_rows + (rw.deep_global ? rw.max_deep * (h1 / 4) * row_groups_max(d) : 0);
  hipStream_t s = (hipStream_t)stream;
  const int m = d->info.n_cols;
  const unsigned slices = (unsigned)(h1 / 4);

  for (int64_t b = b0; b < b0 + n_batches; ++b) {
    const toc_batch &bt = d->batches[b];
    if (bt.n_rows == 0) continue;               // no tuple: the step changes nothing
    const unsigned row_groups = (unsigned)((bt.n_rows + kNnBlock / kNnLanes - 1) / (kNnBlock / kNnLanes));
    if (rw.deep_global)
      hipLaunchKernelGGL(mlp_fwd1_kernel<true>, dim3(slices, row_groups), dim3(kNnBlock), 0, s, im, b, W1, h1,
                         b1, act1, deep_rows, rw.max_deep);
    else
      hipLaunchKernelGGL(mlp_fwd1_kernel<false>, dim3(slices, row_groups), dim3(kNnBlock), lds_f, s, im, b, W1,
                         h1, b1, act1, nullptr, 0);
    if (w_lds)
      hipLaunchKernelGGL(mlp_rows_kernel<true>, dim3((unsigned)((bt.n_rows + R - 1) / R)),
                         dim3(kNnBlock), lds_r, s, bt.n_rows, R, bt.row_base, act1, h1, h2, n_out,
                         W2, b2, W3, b3, labels, H2g, dZ2g, dZ3g, dz1);
    else
      hipLaunchKernelGGL(mlp_rows_kernel<false>, dim3((unsigned)((bt.n_rows + R - 1) / R)),
                         dim3(kNnBlock), lds_r, s, bt.n_rows, R, bt.row_base, act1, h1, h2, n_out,
                         W2, b2, W3, b3, labels, H2g, dZ2g, dZ3g, dz1);
    hipLaunchKernelGGL(mlp_grad_kernel, dim3((unsigned)(n_w2 + n_w3)), dim3(256), lds_g, s, bt.n_rows, n_w2,
                       act1, h1, h2, n_out, H2g, dZ2g, dZ3g, lr, W2, b2, W3, b3, ch2, ch3);
    // the next step's batch with rows (its arrays are read ahead by the last
    // kernel of this step)
    int64_t next = b + 1;
    while (next < b0 + n_batches && d->batches[next].n_rows == 0) ++next;
    if (next >= b0 + n_batches) next = -1;
    if (rw.tree_global)
      hipLaunchKernelGGL(mlp_bwd1_kernel<true>, dim3(slices, kColGroups + 1), dim3(kNnBlock), 0, s, im,
                         b, m, dz1, h1, lr, W1, b1, tree_rows, rw.max_tree, next, labels);
    else
      hipLaunchKernelGGL(mlp_bwd1_kernel<false>, dim3(slices, kColGroups + 1), dim3(kNnBlock), lds_b, s,
                         im, b, m, dz1, h1, lr, W1, b1, nullptr, 0, next, labels);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(TOC_EDEVICE, "mlp step kernels: %s", hipGetErrorString(e));
  }
  return TOC_OK;
}

}  // extern "C"
