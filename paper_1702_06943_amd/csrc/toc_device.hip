// Device side of libtoc for gfx950: upload copy, the right/left products run on
// the compressed image, and decode to CSR.
//
// Image (built on the host by Algorithm 2 + level order): per batch, codes are
// numbered 0..n_codes-1 by depth; depth-1 codes with children come first.  H, the
// dictionary table of Theorems 1 and 2, exists only inside these kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "toc_internal.h"

using toc::fail;

namespace {

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWaves = kBlock / kWave;
constexpr int kMaxKpl = 8;                    // wide kernels: up to 8 columns per lane
constexpr int kKTile = kWave * kMaxKpl;       // 512 columns per pass
constexpr int kRowsTile = 1024;               // decode: rows scanned per LDS pass
constexpr size_t kLdsMax = 160 * 1024;        // gfx950 LDS per workgroup
constexpr int kOutLdsMax = 8192;              // k = 1 left: out block kept in LDS up to m

struct Img {
  const toc_batch *batches;
  const uint32_t *level;
  const uint32_t *parent;
  const uint32_t *col;
  const float *val;
  const uint32_t *depth;
  const uint32_t *span;
  const uint32_t *dcodes;
};

Img image_of(const toc_dev *d) {
  const uint8_t *b = (const uint8_t *)d->buf;
  const toc_layout &L = d->layout;
  return Img{(const toc_batch *)(b + L.batches), (const uint32_t *)(b + L.level),
             (const uint32_t *)(b + L.parent),   (const uint32_t *)(b + L.col),
             (const float *)(b + L.val),         (const uint32_t *)(b + L.depth),
             (const uint32_t *)(b + L.span),     (const uint32_t *)(b + L.dcodes)};
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

// Load that bypasses the per-CU L1, for values other waves updated with atomics.
__device__ inline float coherent_load(const float *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ===========================================================================
// k = 1, H resident in LDS, one workgroup per batch.
// ===========================================================================

// Right multiplication (Theorem 1, Algorithm 4): H level by level, then one
// group of LPR lanes per tuple sums H over the tuple's codes.
template <int LPR>
__global__ __launch_bounds__(kBlock) void right_k1_kernel(Img im, int64_t b0,
                                                          const float *__restrict__ W,
                                                          int64_t ldw, float *__restrict__ R,
                                                          int64_t ldr) {
  extern __shared__ float H[];
  const toc_batch bt = im.batches[b0 + blockIdx.x];
  const uint32_t *lvl = im.level + bt.lvl_base;
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const float *val = im.val + bt.code_base;
  for (int d = 1; d <= bt.n_levels; ++d) {
    const uint32_t a = lvl[d - 1], e = lvl[d];
    for (uint32_t c = a + threadIdx.x; c < e; c += kBlock) {
      const float base = d > 1 ? H[par[c]] : 0.0f;
      H[c] = fmaf(val[c], W[(int64_t)col[c] * ldw], base);
    }
    __syncthreads();
  }
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % LPR, grp = threadIdx.x / LPR;
  for (int r = grp; r < bt.n_rows; r += kBlock / LPR) {
    const uint32_t s = span[r], e = span[r + 1];
    float acc = 0.0f;
    for (uint32_t j = s + lane; j < e; j += LPR) acc += H[dc[j]];
    acc = group_sum<LPR>(acc);
    if (lane == 0) R[(bt.row_base + r) * ldr] = acc;
  }
}

// Left multiplication (Theorem 2, Algorithm 5): scatter G onto codes, propagate
// child to parent deepest level first, accumulate val * H into out[col].
template <int LPR, bool OUT_LDS>
__global__ __launch_bounds__(kBlock) void left_k1_kernel(Img im, int64_t b0, int32_t m,
                                                         int32_t h_words,
                                                         const float *__restrict__ G,
                                                         int64_t ldg, float *__restrict__ out,
                                                         int64_t ldo, int accumulate) {
  extern __shared__ float sm[];
  float *H = sm;
  float *O = sm + h_words;
  const int64_t b = b0 + blockIdx.x;
  const toc_batch bt = im.batches[b];
  const uint32_t *lvl = im.level + bt.lvl_base;
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const float *val = im.val + bt.code_base;
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  float *ob = out + b * (int64_t)m * ldo;
  for (int c = threadIdx.x; c < bt.n_codes; c += kBlock) H[c] = 0.0f;
  if (OUT_LDS) {
    for (int j = threadIdx.x; j < m; j += kBlock) O[j] = 0.0f;
  } else if (!accumulate) {
    for (int j = threadIdx.x; j < m; j += kBlock) ob[(int64_t)j * ldo] = 0.0f;
    __threadfence();
  }
  __syncthreads();
  const int lane = threadIdx.x % LPR, grp = threadIdx.x / LPR;
  for (int r = grp; r < bt.n_rows; r += kBlock / LPR) {
    const float g = G[(bt.row_base + r) * ldg];
    const uint32_t s = span[r], e = span[r + 1];
    for (uint32_t j = s + lane; j < e; j += LPR) atomicAdd(&H[dc[j]], g);
  }
  __syncthreads();
  for (int d = bt.n_levels; d >= 2; --d) {
    const uint32_t a = lvl[d - 1], e = lvl[d];
    for (uint32_t c = a + threadIdx.x; c < e; c += kBlock) atomicAdd(&H[par[c]], H[c]);
    __syncthreads();
  }
  for (int c = threadIdx.x; c < bt.n_codes; c += kBlock) {
    const float x = val[c] * H[c];
    if (OUT_LDS) atomicAdd(&O[col[c]], x);
    else unsafeAtomicAdd(&ob[(int64_t)col[c] * ldo], x);
  }
  if (OUT_LDS) {
    __syncthreads();
    for (int j = threadIdx.x; j < m; j += kBlock) {
      float *p = &ob[(int64_t)j * ldo];
      *p = accumulate ? *p + O[j] : O[j];
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
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const float *val = im.val + bt.code_base;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
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
    float acc[KPL];
#pragma unroll
    for (int i = 0; i < KPL; ++i) acc[i] = 0.0f;
    const uint32_t s = span[r], e = span[r + 1];
    for (uint32_t j = s; j < e; ++j) {
      const uint32_t c = dc[j];
      if (c < n1) {
        const float v = val[c];
        const float *w = W + (int64_t)col[c] * ldw;
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          const int q = lane + kWave * i;
          if (q < kt) acc[i] = fmaf(v, w[q], acc[i]);
        }
      } else {
        const float *h = Hd + (int64_t)(c - n1) * kt;
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          const int q = lane + kWave * i;
          if (q < kt) acc[i] += h[q];
        }
      }
    }
    float *rr = R + (bt.row_base + r) * ldr;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int q = lane + kWave * i;
      if (q < kt) rr[q] = acc[i];
    }
  }
}

// Left: H rows for codes with children or depth >= 2 (a depth-1 leaf code sends
// val * G[row] straight to out[col]); scatter, then propagate and accumulate one
// level at a time from the deepest.  Algorithm 8 with the column loop innermost.
template <int KPL>
__global__ __launch_bounds__(kBlock) void left_wide_kernel(
    Img im, int64_t b0, int64_t ws_base, int32_t m, const float *__restrict__ G, int64_t ldg,
    int kt, float *__restrict__ out, int64_t ldo, int accumulate, float *__restrict__ ws) {
  const int64_t b = b0 + blockIdx.x;
  const toc_batch bt = im.batches[b];
  const uint32_t *lvl = im.level + bt.lvl_base;
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const float *val = im.val + bt.code_base;
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const uint32_t n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1;
  const int64_t n_tree = (int64_t)ni + (bt.n_codes - bt.n_lvl1);
  float *Ht = ws + (bt.tree_base - ws_base) * kt;
  float *ob = out + b * (int64_t)m * ldo;
  auto hrow = [&](uint32_t c) -> int64_t { return c < ni ? c : (int64_t)c - n1 + ni; };
  for (int64_t x = threadIdx.x; x < n_tree * kt; x += kBlock) Ht[x] = 0.0f;
  if (!accumulate)
    for (int64_t x = threadIdx.x; x < (int64_t)m * kt; x += kBlock)
      ob[(x / kt) * ldo + x % kt] = 0.0f;
  __threadfence();
  __syncthreads();
  for (int r = wave; r < bt.n_rows; r += kWaves) {
    float g[KPL];
    const float *gr = G + (bt.row_base + r) * ldg;
#pragma unroll
    for (int i = 0; i < KPL; ++i) {
      const int q = lane + kWave * i;
      g[i] = q < kt ? gr[q] : 0.0f;
    }
    const uint32_t s = span[r], e = span[r + 1];
    for (uint32_t j = s; j < e; ++j) {
      const uint32_t c = dc[j];
      if (c < ni || c >= n1) {
        float *h = Ht + hrow(c) * kt;
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          const int q = lane + kWave * i;
          if (q < kt) unsafeAtomicAdd(&h[q], g[i]);
        }
      } else {
        const float v = val[c];
        float *o = ob + (int64_t)col[c] * ldo;
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
          const int q = lane + kWave * i;
          if (q < kt) unsafeAtomicAdd(&o[q], v * g[i]);
        }
      }
    }
  }
  __threadfence();
  __syncthreads();
  for (int d = bt.n_levels; d >= 1; --d) {
    const uint32_t a = lvl[d - 1], e = d == 1 ? ni : lvl[d];
    for (uint32_t c = a + wave; c < e; c += kWaves) {
      const float *h = Ht + hrow(c) * kt;
      float *hp = d >= 2 ? Ht + hrow(par[c]) * kt : nullptr;
      const float v = val[c];
      float *o = ob + (int64_t)col[c] * ldo;
#pragma unroll
      for (int i = 0; i < KPL; ++i) {
        const int q = lane + kWave * i;
        if (q < kt) {
          const float x = coherent_load(&h[q]);
          unsafeAtomicAdd(&o[q], v * x);
          if (d >= 2) unsafeAtomicAdd(&hp[q], x);
        }
      }
    }
    __threadfence();
    __syncthreads();
  }
}

// ===========================================================================
// Decode to CSR (Algorithm 6's backtracking): per tuple, row length = sum of the
// depths of its codes; an exclusive scan gives row starts; each code writes its
// sequence backwards while walking to the root.
// ===========================================================================
__device__ void block_exclusive_scan(uint32_t *a, int n, uint32_t *wave_tot, uint32_t &total) {
  // n <= 4 * kBlock; each thread owns 4 consecutive entries
  const int t = threadIdx.x, lane = t % kWave, w = t / kWave;
  uint32_t v[4], s = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int x = 4 * t + i;
    v[i] = x < n ? a[x] : 0u;
    s += v[i];
  }
  const uint32_t incl = wave_incl_scan(s, lane);
  if (lane == kWave - 1) wave_tot[w] = incl;
  __syncthreads();
  uint32_t off = 0, tot = 0;
  for (int i = 0; i < kWaves; ++i) {
    if (i < w) off += wave_tot[i];
    tot += wave_tot[i];
  }
  uint32_t run = off + incl - s;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int x = 4 * t + i;
    if (x < n) a[x] = run;
    run += v[i];
  }
  total = tot;
  __syncthreads();
}

__global__ __launch_bounds__(kBlock) void decode_kernel(Img im, int64_t b0,
                                                        int64_t *__restrict__ rowptr,
                                                        int32_t *__restrict__ ocol,
                                                        uint32_t *__restrict__ oval) {
  __shared__ uint32_t rlen[kRowsTile];
  __shared__ uint32_t wave_tot[kWaves];
  const toc_batch bt = im.batches[b0 + blockIdx.x];
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const uint32_t *val = (const uint32_t *)im.val + bt.code_base;
  const uint32_t *dep = im.depth + bt.code_base;
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  int64_t base = bt.nnz_base;
  for (int t0 = 0; t0 < bt.n_rows; t0 += kRowsTile) {
    const int nr = min(kRowsTile, bt.n_rows - t0);
    for (int r = wave; r < nr; r += kWaves) {
      const uint32_t s = span[t0 + r], e = span[t0 + r + 1];
      uint32_t len = 0;
      for (uint32_t j = s + lane; j < e; j += kWave) len += dep[dc[j]];
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) len += __shfl_xor(len, o, kWave);
      if (lane == 0) rlen[r] = len;
    }
    __syncthreads();
    uint32_t total;
    block_exclusive_scan(rlen, nr, wave_tot, total);
    for (int r = threadIdx.x; r < nr; r += kBlock) rowptr[bt.row_base + t0 + r] = base + rlen[r];
    for (int r = wave; r < nr; r += kWaves) {
      int64_t pos = base + rlen[r];
      const uint32_t s = span[t0 + r], e = span[t0 + r + 1];
      for (uint32_t j0 = s; j0 < e; j0 += kWave) {
        const uint32_t j = j0 + lane;
        uint32_t c = 0, d = 0;
        if (j < e) {
          c = dc[j];
          d = dep[c];
        }
        const uint32_t incl = wave_incl_scan(d, lane);
        const uint32_t tot = __shfl(incl, kWave - 1, kWave);
        if (j < e) {
          int64_t p = pos + (incl - d) + d - 1;
          uint32_t x = c;
          for (uint32_t t = 0; t < d; ++t, --p) {
            ocol[p] = (int32_t)col[x];
            oval[p] = val[x];
            x = par[x];
          }
        }
        pos += tot;
      }
    }
    base += total;
    __syncthreads();
  }
  if (threadIdx.x == 0) rowptr[bt.row_base + bt.n_rows] = base;
}

// ===========================================================================
// Host helpers
// ===========================================================================
toc_status check_device(const toc_dev *d) {
  if (!d) return fail(TOC_EINVAL, "dev is NULL");
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

int lanes_per_row(const toc_dev *d) {
  const double avg = d->info.n_rows ? (double)d->info.n_codes / (double)d->info.n_rows : 0.0;
  if (avg <= 12) return 8;
  if (avg <= 24) return 16;
  if (avg <= 48) return 32;
  return 64;
}

// Whether the k = 1 kernels can keep a batch's H in LDS.
bool k1_fits(const toc_dev *d, int op) {
  size_t h = (size_t)d->max_codes * 4;
  if (op == TOC_OP_LEFT && d->info.n_cols <= kOutLdsMax) h += (size_t)d->info.n_cols * 4;
  return h + 16 <= kLdsMax;
}

int64_t rows_per_batch_need(const toc_dev *d, int op) {
  return op == TOC_OP_RIGHT ? d->max_deep : d->max_tree;
}

int64_t rows_total_need(const toc_dev *d, int op) {
  return op == TOC_OP_RIGHT ? d->total_deep : d->total_tree;
}

// Splits batches into passes whose workspace rows fit `cap_rows`; calls fn(b0, nb, base).
template <typename F>
toc_status for_each_pass(const toc_dev *d, int op, int64_t cap_rows, F fn) {
  const int64_t nb = (int64_t)d->batches.size();
  int64_t b0 = 0;
  const int64_t max_grid = 1 << 30;
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
      std::vector<uint8_t> staging((size_t)d->layout.end);
      st = toc::build_image(encs, n_batches, flags, d, staging.data());
      if (st != TOC_OK) {
        delete d;
        return st;
      }
      hipStream_t s = (hipStream_t)stream;
      if (hipMemcpyAsync(buf, staging.data(), staging.size(), hipMemcpyHostToDevice, s) !=
              hipSuccess ||
          hipStreamSynchronize(s) != hipSuccess) {
        delete d;
        return fail(TOC_EDEVICE, "upload copy failed");
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
  if (op != TOC_OP_DECODE && !(k == 1 && k1_fits(d, op))) {
    const int64_t kt = std::min<int64_t>(k, kKTile);
    minimum = (size_t)(rows_per_batch_need(d, op) * kt * 4);
    need = std::max(minimum, (size_t)(rows_total_need(d, op) * kt * 4));
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
    const size_t lds = std::max<size_t>(16, (size_t)d->max_codes * 4);
    const int lpr = lanes_per_row(d);
    for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
      const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
      switch (lpr) {
        case 8: if ((st = allow_lds(right_k1_kernel<8>, lds))) return st;
          hipLaunchKernelGGL(right_k1_kernel<8>, dim3(g), dim3(kBlock), lds, s, im, b0, W, ldw, R, ldr); break;
        case 16: if ((st = allow_lds(right_k1_kernel<16>, lds))) return st;
          hipLaunchKernelGGL(right_k1_kernel<16>, dim3(g), dim3(kBlock), lds, s, im, b0, W, ldw, R, ldr); break;
        case 32: if ((st = allow_lds(right_k1_kernel<32>, lds))) return st;
          hipLaunchKernelGGL(right_k1_kernel<32>, dim3(g), dim3(kBlock), lds, s, im, b0, W, ldw, R, ldr); break;
        default: if ((st = allow_lds(right_k1_kernel<64>, lds))) return st;
          hipLaunchKernelGGL(right_k1_kernel<64>, dim3(g), dim3(kBlock), lds, s, im, b0, W, ldw, R, ldr); break;
      }
      if ((st = launch_status("right_k1_kernel"))) return st;
    }
    return TOC_OK;
  }
  for (int64_t k0 = 0; k0 < k; k0 += kKTile) {
    const int kt = (int)std::min<int64_t>(kKTile, k - k0);
    const int kpl = (kt + kWave - 1) / kWave;
    const int64_t cap_rows = (int64_t)(ws_bytes / 4) / kt;
    if (d->max_deep > 0 && (!ws || cap_rows < d->max_deep))
      return fail(TOC_ESIZE, "workspace too small (%zu bytes)", ws_bytes);
    st = for_each_pass(d, TOC_OP_RIGHT, d->max_deep > 0 ? cap_rows : INT64_MAX / 2,
                       [&](int64_t b0, int64_t n, int64_t base) -> toc_status {
      TOC_DISPATCH_KPL(kpl, right_wide_kernel, dim3((unsigned)n), dim3(kBlock), 0, s, im, b0,
                       base, W + k0, ldw, kt, R + k0, ldr, (float *)ws);
      return launch_status("right_wide_kernel");
    });
    if (st != TOC_OK) return st;
  }
  return TOC_OK;
}

toc_status toc_left_mul(const toc_dev *d, const float *G, int32_t k, int64_t ldg, float *out,
                        int64_t ldo, int32_t accumulate, void *ws, size_t ws_bytes,
                        void *stream) {
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
    const bool out_lds = m <= kOutLdsMax;
    const int32_t hw = d->max_codes;
    const size_t lds = std::max<size_t>(16, ((size_t)hw + (out_lds ? m : 0)) * 4);
    const int lpr = lanes_per_row(d);
    for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
      const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
#define TOC_LEFT_K1(L, O)                                                                  \
  if ((st = allow_lds(left_k1_kernel<L, O>, lds))) return st;                               \
  hipLaunchKernelGGL((left_k1_kernel<L, O>), dim3(g), dim3(kBlock), lds, s, im, b0, m, hw, G, \
                     ldg, out, ldo, accumulate);
      if (out_lds) {
        switch (lpr) {
          case 8: TOC_LEFT_K1(8, true) break;
          case 16: TOC_LEFT_K1(16, true) break;
          case 32: TOC_LEFT_K1(32, true) break;
          default: TOC_LEFT_K1(64, true) break;
        }
      } else {
        switch (lpr) {
          case 8: TOC_LEFT_K1(8, false) break;
          case 16: TOC_LEFT_K1(16, false) break;
          case 32: TOC_LEFT_K1(32, false) break;
          default: TOC_LEFT_K1(64, false) break;
        }
      }
#undef TOC_LEFT_K1
      if ((st = launch_status("left_k1_kernel"))) return st;
    }
    return TOC_OK;
  }
  for (int64_t k0 = 0; k0 < k; k0 += kKTile) {
    const int kt = (int)std::min<int64_t>(kKTile, k - k0);
    const int kpl = (kt + kWave - 1) / kWave;
    const int64_t cap_rows = (int64_t)(ws_bytes / 4) / kt;
    if (d->max_tree > 0 && (!ws || cap_rows < d->max_tree))
      return fail(TOC_ESIZE, "workspace too small (%zu bytes)", ws_bytes);
    st = for_each_pass(d, TOC_OP_LEFT, d->max_tree > 0 ? cap_rows : INT64_MAX / 2,
                       [&](int64_t b0, int64_t n, int64_t base) -> toc_status {
      TOC_DISPATCH_KPL(kpl, left_wide_kernel, dim3((unsigned)n), dim3(kBlock), 0, s, im, b0,
                       base, m, G + k0, ldg, kt, out + k0, ldo, accumulate, (float *)ws);
      return launch_status("left_wide_kernel");
    });
    if (st != TOC_OK) return st;
  }
  return TOC_OK;
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
  for (int64_t b0 = 0; b0 < nb; b0 += (1 << 30)) {
    const unsigned g = (unsigned)std::min<int64_t>(nb - b0, 1 << 30);
    hipLaunchKernelGGL(decode_kernel, dim3(g), dim3(kBlock), 0, s, im, b0, rowptr, col,
                       (uint32_t *)val);
    if ((st = launch_status("decode_kernel"))) return st;
  }
  return TOC_OK;
}

}  // extern "C"
