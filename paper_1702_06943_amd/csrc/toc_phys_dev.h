// Device readers of the physical encoding (section 3.2 stores (I, D) as bit-packed
// integers; section 4.1.1 reads them back) and the kernel that builds the decoding
// tree C' from them (Algorithm 2), shared by the tree builder and the image builder.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "toc_internal.h"

namespace tocphys {


constexpr int kCpBlock = 512;
constexpr int kCpWave = 64;
constexpr int kCpWaves = kCpBlock / kCpWave;
constexpr int kCpMaxRows = 16384;
constexpr int kCpMaxRounds = 48;            // pointer jumping: ceil(log2(nodes)) + 1 suffice
constexpr uint32_t kNone = 0xFFFFFFFFu;

// Integer i of a packed array of w-byte little-endian integers (w = 1..4): its
// bytes copied into a 32-bit integer, the upper bytes zero (section 4.1.1).
__device__ inline uint32_t rd(const uint8_t *p, uint64_t i, uint32_t w) {
  const uint8_t *q = p + i * w;
  uint32_t v = q[0];
  if (w > 1) v |= (uint32_t)q[1] << 8;
  if (w > 2) v |= (uint32_t)q[2] << 16;
  if (w > 3) v |= (uint32_t)q[3] << 24;
  return v;
}

// Exclusive prefix sum of x over the workgroup; total gets the sum of all.
__device__ inline uint32_t block_excl_scan(uint32_t x, uint32_t *wsum, uint32_t &total) {
  const int lane = threadIdx.x % kCpWave, wave = threadIdx.x / kCpWave;
  uint32_t v = x;
#pragma unroll
  for (int o = 1; o < kCpWave; o <<= 1) {
    const uint32_t y = __shfl_up(v, o, kCpWave);
    if (lane >= o) v += y;
  }
  if (lane == kCpWave - 1) wsum[wave] = v;
  __syncthreads();
  uint32_t before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kCpWaves; ++w) {
    before += w < wave ? wsum[w] : 0u;
    total += wsum[w];
  }
  __syncthreads();
  return before + v - x;
}

// Header of array a of a blob: count, bytes per integer, byte offset of its data.
struct Hdr {
  uint32_t cnt[5], w[5], data[5];
  int err;
};

// Reads the five array headers of a blob of `size` bytes and checks that the
// arrays fill it exactly (widths 1..4, unique values 4 bytes wide, as many value
// indexes as columns, at least one tuple start, at most max_rows tuples); h.err
// gets TOC_CPRIME_LAYOUT or TOC_CPRIME_ROWS, else 0.  Every later read of an array
// stays inside the blob.
__device__ inline void parse_headers(const uint8_t *blob, uint64_t size, int max_rows, Hdr &h) {
  int err = 0;
  uint64_t pos = 0;
  for (int a = 0; a < 5 && !err; ++a) {
    if (size < pos + 5) {
      err = TOC_CPRIME_LAYOUT;
      break;
    }
    const uint32_t cnt = rd(blob + pos, 0, 4), w = blob[pos + 4];
    if (w < 1 || w > 4 || (a == 1 && w != 4) || (size - pos - 5) / w < cnt) {
      err = TOC_CPRIME_LAYOUT;
      break;
    }
    h.cnt[a] = cnt;
    h.w[a] = w;
    h.data[a] = (uint32_t)(pos + 5);
    pos += 5 + (uint64_t)cnt * w;
  }
  if (!err && (pos != size || h.cnt[2] != h.cnt[0] || h.cnt[4] < 1)) err = TOC_CPRIME_LAYOUT;
  if (!err && h.cnt[4] - 1 > (uint32_t)max_rows) err = TOC_CPRIME_ROWS;
  h.err = err;
}

// Algorithm 2 on the device, one workgroup of kCpBlock threads per batch: the
// parent, key pair and depth of every node of each batch's C', in paper
// numbering, from the batch's blob (offs: blob offsets, then node offsets, n_batches
// + 1 each); status gets 0 or a TOC_CPRIME_* code per batch.  anc0 .. nxt are
// scratch of one word per node.  Dynamic LDS: 8 (max_rows + 1) bytes.
__global__ __launch_bounds__(kCpBlock) void cprime_kernel(
    const uint8_t *__restrict__ blobs, const int64_t *__restrict__ offs, int64_t n_batches,
    int max_rows, uint32_t n_cols, uint32_t *__restrict__ parent, uint32_t *__restrict__ col,
    uint32_t *__restrict__ val, uint32_t *__restrict__ depth, int32_t *__restrict__ status,
    uint32_t *__restrict__ anc0, uint32_t *__restrict__ dist0, uint32_t *__restrict__ anc1,
    uint32_t *__restrict__ dist1, uint32_t *__restrict__ nxt);

}  // namespace tocphys
