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
// Tiled kernels for wide k.  One workgroup per (batch, column tile); the tiles of
// a batch are consecutive blocks of one XCD (the dispatcher deals blocks to the
// 8 XCDs round-robin), so they share the batch's image through that XCD's L2.
// ===========================================================================
constexpr int kXcd = 8;
constexpr int kTileBlock = 512;
constexpr int kTileWaves = kTileBlock / kWave;

__device__ inline void xcd_tile_map(int64_t blk, int n_tiles, int64_t &b, int &tile) {
  const int64_t x = blk % kXcd, j = blk / kXcd;
  tile = (int)(j % n_tiles);
  b = (j / n_tiles) * kXcd + x;
}

__device__ inline float4 f4fma(float s, float4 x, float4 a) {
  return make_float4(fmaf(s, x.x, a.x), fmaf(s, x.y, a.y), fmaf(s, x.z, a.z), fmaf(s, x.w, a.w));
}

// Right multiplication with a KT-column tile of W resident in LDS.  Lanes form 8
// groups of 8; a lane holds 4 consecutive columns, so a group covers the tile
// for one code and a wave takes 8 codes of a tuple per step.  H rows of depth >= 2
// codes are built level by level first (in LDS when they fit, else in `ws`).
constexpr int kRtKT = 32;
constexpr uint32_t kRtGlobal = 0x80000000u;   // staged address refers to ws

template <bool DEEP_LDS>
__global__ __launch_bounds__(kTileBlock) void right_tiled_kernel(
    Img im, int64_t b0, int64_t nb, int n_tiles, int m, const float *__restrict__ W,
    int64_t ldw, int k, float *__restrict__ R, int64_t ldr, float *__restrict__ ws,
    int64_t ws_base) {
  extern __shared__ float4 smem4[];
  float *lds = (float *)smem4;
  int64_t bl;
  int tile;
  xcd_tile_map(blockIdx.x, n_tiles, bl, tile);
  if (bl >= nb) return;
  const int64_t b = b0 + bl;
  const toc_batch bt = im.batches[b];
  const int k0 = tile * kRtKT;
  const int kt = min(kRtKT, k - k0);
  const uint32_t *lvl = im.level + bt.lvl_base;
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const float *val = im.val + bt.code_base;
  const uint32_t n1 = (uint32_t)bt.n_lvl1;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int grp = lane / 8, q = 4 * (lane % 8);
  float *Wt = lds;                                   // m rows of kRtKT floats
  float *Hl = lds + (size_t)m * kRtKT;               // deep rows (DEEP_LDS)
  const int64_t kpad = (int64_t)n_tiles * kRtKT;
  float *Hg = ws + (bt.deep_base - ws_base) * kpad + k0;
  // stage W[:, k0:k0+kt]
  for (int e = threadIdx.x; e < m * (kRtKT / 4); e += kTileBlock) {
    const int c = e / (kRtKT / 4), q4 = 4 * (e % (kRtKT / 4));
    const float *src = W + (int64_t)c * ldw + k0 + q4;
    float4 v;
    v.x = q4 + 0 < kt ? src[0] : 0.0f;
    v.y = q4 + 1 < kt ? src[1] : 0.0f;
    v.z = q4 + 2 < kt ? src[2] : 0.0f;
    v.w = q4 + 3 < kt ? src[3] : 0.0f;
    *(float4 *)&Wt[c * kRtKT + q4] = v;
  }
  __syncthreads();
  // H of depth >= 2 codes, level by level
  for (int d = 2; d <= bt.n_levels; ++d) {
    const uint32_t a = lvl[d - 1], e = lvl[d];
    for (uint32_t c = a + wave * 8 + grp; c < e; c += kTileWaves * 8) {
      const uint32_t p = par[c];
      float4 base;
      if (p < n1) {
        base = *(const float4 *)&Wt[col[p] * kRtKT + q];
        const float vp = val[p];
        base = make_float4(vp * base.x, vp * base.y, vp * base.z, vp * base.w);
      } else if (DEEP_LDS) {
        base = *(const float4 *)&Hl[(p - n1) * kRtKT + q];
      } else {
        base = *(const float4 *)&Hg[(int64_t)(p - n1) * kpad + q];
      }
      const float4 h = f4fma(val[c], *(const float4 *)&Wt[col[c] * kRtKT + q], base);
      if (DEEP_LDS) *(float4 *)&Hl[(c - n1) * kRtKT + q] = h;
      else *(float4 *)&Hg[(int64_t)(c - n1) * kpad + q] = h;
    }
    __syncthreads();
  }
  // per-tuple sums
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  for (int r = wave; r < bt.n_rows; r += kTileWaves) {
    const uint32_t s = span[r], e = span[r + 1];
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (uint32_t j0 = s; j0 < e; j0 += kWave) {
      const uint32_t n = min((uint32_t)kWave, e - j0);
      // lane i fetches code j0+i: LDS row offset and multiplier
      uint32_t my_addr = 0;
      float my_mult = 0.0f;
      if ((uint32_t)lane < n) {
        const uint32_t c = dc[j0 + lane];
        if (c < n1) {
          my_addr = col[c] * kRtKT;
          my_mult = val[c];
        } else {
          my_addr = DEEP_LDS ? (uint32_t)m * kRtKT + (c - n1) * kRtKT : (kRtGlobal | (c - n1));
          my_mult = 1.0f;
        }
      }
      // every lane takes part in the shuffles; lanes past n carry multiplier 0
      for (uint32_t t0 = 0; t0 < n; t0 += 8) {
        const int t = (int)t0 + grp;
        const uint32_t addr = (uint32_t)__shfl((int)my_addr, t, kWave);
        const float mult = __shfl(my_mult, t, kWave);
        float4 x;
        if (!DEEP_LDS && (addr & kRtGlobal))
          x = *(const float4 *)&Hg[(int64_t)(addr & ~kRtGlobal) * kpad + q];
        else
          x = *(const float4 *)&lds[addr + q];
        acc = f4fma(mult, x, acc);
      }
    }
#pragma unroll
    for (int o = 8; o < kWave; o <<= 1) {
      acc.x += __shfl_xor(acc.x, o, kWave);
      acc.y += __shfl_xor(acc.y, o, kWave);
      acc.z += __shfl_xor(acc.z, o, kWave);
      acc.w += __shfl_xor(acc.w, o, kWave);
    }
    if (grp == 0) {
      float *rr = R + (bt.row_base + r) * ldr + k0 + q;
      if (q + 0 < kt) rr[0] = acc.x;
      if (q + 1 < kt) rr[1] = acc.y;
      if (q + 2 < kt) rr[2] = acc.z;
      if (q + 3 < kt) rr[3] = acc.w;
    }
  }
}

// Left multiplication by pulling (Theorem 2 read as a definition): for each code,
// G(x) = sum of G rows over the entries of D equal to x (the inverted index
// occ_off/occ_row), plus the G values of its children; out[col] = sum over the
// codes with that key column of val * G(x).  No atomics: each output row and each
// H row has one writer.  A KT-column tile of G lives in LDS; lane = column.
constexpr int kLpKT = 64;
constexpr int kLpColsPerGrab = 4;

__device__ inline uint32_t rdlane(uint32_t v, uint32_t i) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)i);
}

template <int DUMMY>
__global__ __launch_bounds__(kTileBlock) void left_pull_kernel(
    Img im, const uint32_t *__restrict__ occ_off_all, const uint32_t *__restrict__ occ_row_all,
    const uint32_t *__restrict__ tlist_all, int64_t b0, int64_t nb, int n_tiles, int m,
    const float *__restrict__ G, int64_t ldg, int k, float *__restrict__ out, int64_t ldo,
    int accumulate, float *__restrict__ ws, int64_t ws_base) {
  extern __shared__ float4 smem4[];
  __shared__ uint32_t ctr;
  int64_t bl;
  int tile;
  xcd_tile_map(blockIdx.x, n_tiles, bl, tile);
  if (bl >= nb) return;
  const int64_t b = b0 + bl;
  const toc_batch bt = im.batches[b];
  const int k0 = tile * kLpKT;
  const int kt = min(kLpKT, k - k0);
  const uint32_t *lvl = im.level + bt.lvl_base;
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const float *val = im.val + bt.code_base;
  const uint32_t *oo = occ_off_all + bt.code_base + b;
  const uint32_t *orow = occ_row_all + bt.d_base;
  const uint32_t *tl = tlist_all + bt.tree_base;
  const uint32_t nc = (uint32_t)bt.n_codes, n1 = (uint32_t)bt.n_lvl1, ni = (uint32_t)bt.n_int1;
  const uint32_t n_tree = ni + (nc - n1);
  const int nrows = bt.n_rows;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  float *Gt = (float *)smem4;                          // nrows x kLpKT
  uint32_t *Loff = (uint32_t *)(Gt + (size_t)nrows * kLpKT);  // m + 1
  uint32_t *Toff = Loff + m + 1;                       // m + 1
  uint32_t *Coff = Toff + m + 1;                       // n_tree + 1
  const int64_t kpad = (int64_t)n_tiles * kLpKT;
  float *Ht = ws + (bt.tree_base - ws_base) * kpad + k0;
  auto hrow = [&](uint32_t c) -> uint32_t { return c < ni ? c : c - n1 + ni; };
  for (int e = threadIdx.x; e < nrows * kLpKT; e += kTileBlock) {
    const int r = e / kLpKT, qq = e % kLpKT;
    Gt[e] = qq < kt ? G[(bt.row_base + r) * ldg + k0 + qq] : 0.0f;
  }
  // column boundaries of the depth-1 leaves [ni, n1) (sorted by column)
  for (uint32_t i = ni + threadIdx.x; i < n1; i += kTileBlock) {
    const int64_t cc = col[i], cp = i > ni ? (int64_t)col[i - 1] : -1;
    for (int64_t j = cp + 1; j <= cc; ++j) Loff[j] = i;
  }
  {
    const int64_t last = n1 > ni ? (int64_t)col[n1 - 1] : -1;
    for (int64_t j = last + 1 + threadIdx.x; j <= m; j += kTileBlock) Loff[j] = n1;
  }
  // column boundaries of the tree-code list
  for (uint32_t t = threadIdx.x; t < n_tree; t += kTileBlock) {
    const int64_t cc = col[tl[t]], cp = t > 0 ? (int64_t)col[tl[t - 1]] : -1;
    for (int64_t j = cp + 1; j <= cc; ++j) Toff[j] = t;
  }
  {
    const int64_t last = n_tree > 0 ? (int64_t)col[tl[n_tree - 1]] : -1;
    for (int64_t j = last + 1 + threadIdx.x; j <= m; j += kTileBlock) Toff[j] = n_tree;
  }
  // children ranges: codes of depth >= 2 are sorted by (level, parent), so the
  // children of the tree code with H row h are [Coff[h], Coff[h+1])
  for (uint32_t c = n1 + threadIdx.x; c < nc; c += kTileBlock) {
    const int64_t ph = hrow(par[c]), pp = c > n1 ? (int64_t)hrow(par[c - 1]) : -1;
    for (int64_t h = pp + 1; h <= ph; ++h) Coff[h] = c;
  }
  {
    const int64_t last = nc > n1 ? (int64_t)hrow(par[nc - 1]) : -1;
    for (int64_t h = last + 1 + threadIdx.x; h <= n_tree; h += kTileBlock) Coff[h] = nc;
  }
  if (threadIdx.x == 0) ctr = 0;
  __syncthreads();
  // tree codes, deepest level first; one wave per code
  for (int d = bt.n_levels; d >= 1; --d) {
    const uint32_t a = d == 1 ? 0 : lvl[d - 1], e = d == 1 ? ni : lvl[d];
    for (uint32_t c = a + wave; c < e; c += kTileWaves) {
      const uint32_t h = hrow(c);
      float s = 0.0f;
      for (uint32_t o = oo[c]; o < oo[c + 1]; ++o) s += Gt[orow[o] * kLpKT + lane];
      for (uint32_t ch = Coff[h]; ch < Coff[h + 1]; ++ch) s += Ht[(int64_t)hrow(ch) * kpad + lane];
      Ht[(int64_t)h * kpad + lane] = s;
    }
    __syncthreads();
  }
  // columns, a few at a time per wave; code and occurrence info is fetched 64
  // entries at a time into registers and broadcast with readlane
  for (;;) {
    uint32_t base = 0;
    if (lane == 0) base = atomicAdd(&ctr, (uint32_t)kLpColsPerGrab);
    base = rdlane(base, 0);
    if (base >= (uint32_t)m) break;
    const uint32_t jend = min(base + kLpColsPerGrab, (uint32_t)m);
    bool have_c = false, have_o = false;
    uint32_t cwin = 0, owin = 0, v_oo = 0, v_val = 0, v_row = 0;
    for (uint32_t j = base; j < jend; ++j) {
      float acc = 0.0f;
      const uint32_t c_lo = Loff[j], c_hi = Loff[j + 1];
      for (uint32_t c = c_lo; c < c_hi; ++c) {
        if (!have_c || c - cwin >= 63u) {  // codes cwin..cwin+62 with both bounds
          have_c = true;
          cwin = c;
          v_oo = c + lane <= nc ? oo[c + lane] : 0u;
          v_val = c + lane < nc ? __float_as_uint(val[c + lane]) : 0u;
        }
        const uint32_t o_lo = rdlane(v_oo, c - cwin), o_hi = rdlane(v_oo, c - cwin + 1);
        const float vc = __uint_as_float(rdlane(v_val, c - cwin));
        float s = 0.0f;
        for (uint32_t o = o_lo; o < o_hi; ++o) {
          if (!have_o || o - owin >= 64u) {
            have_o = true;
            owin = o;
            v_row = o + lane < (uint32_t)bt.n_d ? orow[o + lane] : 0u;
          }
          s += Gt[rdlane(v_row, o - owin) * kLpKT + lane];
        }
        acc = fmaf(vc, s, acc);
      }
      for (uint32_t t = Toff[j]; t < Toff[j + 1]; ++t) {
        const uint32_t c = tl[t];
        acc = fmaf(val[c], Ht[(int64_t)hrow(c) * kpad + lane], acc);
      }
      if (lane < kt) {
        float *p = out + (b * m + j) * ldo + k0 + lane;
        *p = accumulate ? *p + acc : acc;
      }
    }
  }
}

// ===========================================================================
// Decode to CSR (the backtracking of Algorithm 6).  Rows are concatenated in D
// and in the CSR alike, so the output position of entry j of D is the sum of the
// depths of entries 0..j-1: one flat exclusive scan over D gives every position
// and, at the row boundaries, rowptr.  Each entry then writes its sequence
// backwards while walking to the root.
// ===========================================================================
constexpr int kDecBlock = 1024;
constexpr int kDecWaves = kDecBlock / kWave;
constexpr int kDecPer = 4;                       // entries of D per thread per tile
constexpr int kDecTile = kDecBlock * kDecPer;

__global__ __launch_bounds__(kDecBlock) void decode_kernel(Img im, int64_t b0,
                                                           int64_t *__restrict__ rowptr,
                                                           int32_t *__restrict__ ocol,
                                                           uint32_t *__restrict__ oval) {
  __shared__ uint32_t pre[kDecTile];
  __shared__ uint32_t wave_tot[kDecWaves];
  __shared__ uint32_t row_range[2];
  const toc_batch bt = im.batches[b0 + blockIdx.x];
  const uint32_t *par = im.parent + bt.code_base;
  const uint32_t *col = im.col + bt.code_base;
  const uint32_t *val = (const uint32_t *)im.val + bt.code_base;
  const uint32_t *dep = im.depth + bt.code_base;
  const uint32_t *span = im.span + bt.span_base;
  const uint32_t *dc = im.dcodes + bt.d_base;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const uint32_t nd = (uint32_t)bt.n_d;
  const int nrows = bt.n_rows;
  // first row whose span starts at or after x (spans are non-decreasing)
  auto lower_row = [&](uint32_t x) -> uint32_t {
    uint32_t lo = 0, hi = (uint32_t)nrows + 1;
    while (lo < hi) {
      const uint32_t mid = (lo + hi) / 2;
      if (span[mid] < x) lo = mid + 1;
      else hi = mid;
    }
    return lo;
  };
  int64_t base = bt.nnz_base;
  for (uint32_t t0 = 0; t0 < nd; t0 += kDecTile) {
    uint32_t c[kDecPer], d[kDecPer], s = 0;
#pragma unroll
    for (int i = 0; i < kDecPer; ++i) {
      const uint32_t j = t0 + threadIdx.x * kDecPer + i;
      c[i] = j < nd ? dc[j] : 0u;
      d[i] = j < nd ? dep[c[i]] : 0u;
      s += d[i];
    }
    const uint32_t incl = wave_incl_scan(s, lane);
    if (lane == kWave - 1) wave_tot[wave] = incl;
    if (threadIdx.x == 0) row_range[0] = lower_row(t0);
    if (threadIdx.x == 1) row_range[1] = lower_row(t0 + kDecTile);
    __syncthreads();
    uint32_t off = 0, total = 0;
    for (int w = 0; w < kDecWaves; ++w) {
      off += w < wave ? wave_tot[w] : 0u;
      total += wave_tot[w];
    }
    uint32_t run = off + incl - s;
#pragma unroll
    for (int i = 0; i < kDecPer; ++i) {
      pre[threadIdx.x * kDecPer + i] = run;
      const uint32_t j = t0 + threadIdx.x * kDecPer + i;
      if (j < nd) {
        int64_t p = base + run + d[i] - 1;
        uint32_t x = c[i];
        for (uint32_t t = 0; t < d[i]; ++t, --p) {
          ocol[p] = (int32_t)col[x];
          oval[p] = val[x];
          x = par[x];
        }
      }
      run += d[i];
    }
    __syncthreads();
    for (uint32_t r = row_range[0] + threadIdx.x; r < row_range[1]; r += kDecBlock)
      if ((int)r <= nrows && span[r] < nd) rowptr[bt.row_base + r] = base + pre[span[r] - t0];
    base += total;
    __syncthreads();
  }
  // rows whose span starts at the end of D (trailing empty rows and the end mark)
  for (uint32_t r = lower_row(nd) + threadIdx.x; r <= (uint32_t)nrows; r += kDecBlock)
    rowptr[bt.row_base + r] = base;
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

// Execution plan of an op: which kernel family, its LDS bytes, and the workspace
// it needs (rows of row_floats floats per code that needs an H row in memory).
enum { kPathK1 = 0, kPathTiled = 1, kPathWide = 2 };

struct OpPlan {
  int path = kPathWide;
  int n_tiles = 1;
  bool deep_lds = false;
  size_t lds = 0;
  int64_t row_floats = 0;     // workspace floats per H row (0: no workspace)
  int64_t rows_max = 0, rows_total = 0;
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
  if (right) {
    const size_t wt = (size_t)m * kRtKT * 4;
    if (k >= 4 && wt <= kLdsMax) {
      p.path = kPathTiled;
      p.n_tiles = (k + kRtKT - 1) / kRtKT;
      p.deep_lds = wt + (size_t)d->max_deep * kRtKT * 4 <= kLdsMax;
      p.lds = std::max<size_t>(16, p.deep_lds ? wt + (size_t)d->max_deep * kRtKT * 4 : wt);
      p.row_floats = p.deep_lds ? 0 : (int64_t)p.n_tiles * kRtKT;
      return p;
    }
  } else {
    const size_t lds = ((size_t)d->max_rows * kLpKT + 2 * ((size_t)m + 1) +
                        (size_t)d->max_tree + 1) * 4;
    if (k >= 2 && lds <= kLdsMax) {
      p.path = kPathTiled;
      p.n_tiles = (k + kLpKT - 1) / kLpKT;
      p.lds = lds;
      p.row_floats = (int64_t)p.n_tiles * kLpKT;
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
  if (op != TOC_OP_DECODE) {
    const OpPlan p = plan_op(d, op, k);
    if (p.row_floats > 0 && p.rows_max > 0) {
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
  const OpPlan plan = plan_op(d, TOC_OP_RIGHT, k);
  int64_t cap_rows = 0;
  if ((st = ws_capacity(plan, ws, ws_bytes, cap_rows))) return st;
  if (plan.path == kPathTiled) {
    const int m = d->info.n_cols;
    if ((st = plan.deep_lds ? allow_lds(right_tiled_kernel<true>, plan.lds)
                            : allow_lds(right_tiled_kernel<false>, plan.lds)))
      return st;
    return for_each_pass(d, TOC_OP_RIGHT, cap_rows,
                         [&](int64_t b0, int64_t n, int64_t base) -> toc_status {
      const unsigned grid = (unsigned)(((n + kXcd - 1) / kXcd) * kXcd * plan.n_tiles);
      if (plan.deep_lds)
        hipLaunchKernelGGL(right_tiled_kernel<true>, dim3(grid), dim3(kTileBlock), plan.lds, s,
                           im, b0, n, plan.n_tiles, m, W, ldw, k, R, ldr, (float *)ws, base);
      else
        hipLaunchKernelGGL(right_tiled_kernel<false>, dim3(grid), dim3(kTileBlock), plan.lds, s,
                           im, b0, n, plan.n_tiles, m, W, ldw, k, R, ldr, (float *)ws, base);
      return launch_status("right_tiled_kernel");
    });
  }
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
  const OpPlan plan = plan_op(d, TOC_OP_LEFT, k);
  int64_t cap_rows = 0;
  if ((st = ws_capacity(plan, ws, ws_bytes, cap_rows))) return st;
  if (plan.path == kPathTiled) {
    if ((st = allow_lds(left_pull_kernel<0>, plan.lds))) return st;
    const uint8_t *bb = (const uint8_t *)d->buf;
    const uint32_t *occ_off = (const uint32_t *)(bb + d->layout.occ_off);
    const uint32_t *occ_row = (const uint32_t *)(bb + d->layout.occ_row);
    const uint32_t *tlist = (const uint32_t *)(bb + d->layout.tlist);
    return for_each_pass(d, TOC_OP_LEFT, cap_rows,
                         [&](int64_t b0, int64_t n, int64_t base) -> toc_status {
      const unsigned grid = (unsigned)(((n + kXcd - 1) / kXcd) * kXcd * plan.n_tiles);
      hipLaunchKernelGGL(left_pull_kernel<0>, dim3(grid), dim3(kTileBlock), plan.lds, s, im,
                         occ_off, occ_row, tlist, b0, n, plan.n_tiles, m, G, ldg, k, out, ldo,
                         accumulate, (float *)ws, base);
      return launch_status("left_pull_kernel");
    });
  }
  for (int64_t k0 = 0; k0 < k; k0 += kKTile) {
    const int kt = (int)std::min<int64_t>(kKTile, k - k0);
    const int kpl = (kt + kWave - 1) / kWave;
    st = for_each_pass(d, TOC_OP_LEFT, cap_rows,
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
    hipLaunchKernelGGL(decode_kernel, dim3(g), dim3(kDecBlock), 0, s, im, b0, rowptr, col,
                       (uint32_t *)val);
    if ((st = launch_status("decode_kernel"))) return st;
  }
  return TOC_OK;
}

}  // extern "C"
