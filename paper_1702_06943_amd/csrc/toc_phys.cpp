// Physical encoding of an encoded batch (section 3.2): bit packing and value
// indexing, as bytes.  The byte layout is described with the declarations.
#include <algorithm>
#include <cstring>
#include <vector>

#include "toc_internal.h"

namespace toc {
namespace {

// bytes per integer of an array whose largest value is mx: ceil(log2(mx+1)/8),
// at least one
int width_of(uint64_t mx) {
  int bits = 0;
  while (bits < 64 && (mx >> bits) != 0) ++bits;
  return std::max(1, (bits + 7) / 8);
}

// Widths and unique values of one batch's arrays, computed once per call.
struct PackPlan {
  std::vector<uint32_t> u;   // unique values of I (ascending bit patterns)
  int w_col = 1, w_vix = 1, w_d = 1, w_st = 1;
  size_t bytes = 0;
};

toc_status plan(const toc_enc *e, PackPlan &pl) {
  const size_t nI = e->I_col.size(), nD = e->D_codes.size();
  if (nI > 0xFFFFFFFFu || nD > 0xFFFFFFFFu || (uint64_t)e->n_rows + 1 > 0xFFFFFFFFu)
    return fail(TOC_EUNSUPPORTED, "array longer than a u32 count");
  pl.u.assign(e->I_bits.begin(), e->I_bits.end());
  std::sort(pl.u.begin(), pl.u.end());
  pl.u.erase(std::unique(pl.u.begin(), pl.u.end()), pl.u.end());
  uint64_t mc = 0, md = 0;
  for (int32_t c : e->I_col) mc = std::max<uint64_t>(mc, (uint64_t)c);
  for (uint32_t c : e->D_codes) md = std::max<uint64_t>(md, c);
  pl.w_col = width_of(mc);
  pl.w_vix = width_of(pl.u.empty() ? 0 : pl.u.size() - 1);
  pl.w_d = width_of(md);
  pl.w_st = width_of((uint64_t)nD);
  pl.bytes = 25 + nI * (size_t)(pl.w_col + pl.w_vix) + 4 * pl.u.size() + nD * (size_t)pl.w_d +
             ((size_t)e->n_rows + 1) * (size_t)pl.w_st;
  return TOC_OK;
}

// v as w little-endian bytes at p; returns the byte after them
inline uint8_t *put(uint8_t *p, uint64_t v, int w) {
  for (int q = 0; q < w; ++q) p[q] = (uint8_t)(v >> (8 * q));
  return p + w;
}

inline uint8_t *header(uint8_t *p, uint64_t count, int w) {
  p = put(p, count, 4);
  return put(p, (uint64_t)w, 1);
}

void write(const toc_enc *e, const PackPlan &pl, uint8_t *p) {
  const size_t nI = e->I_col.size();
  p = header(p, nI, pl.w_col);
  for (int32_t c : e->I_col) p = put(p, (uint64_t)c, pl.w_col);
  p = header(p, pl.u.size(), 4);
  for (uint32_t b : pl.u) p = put(p, b, 4);
  p = header(p, nI, pl.w_vix);
  for (uint32_t b : e->I_bits)
    p = put(p, (uint64_t)(std::lower_bound(pl.u.begin(), pl.u.end(), b) - pl.u.begin()), pl.w_vix);
  p = header(p, e->D_codes.size(), pl.w_d);
  for (uint32_t c : e->D_codes) p = put(p, c, pl.w_d);
  p = header(p, (uint64_t)e->n_rows + 1, pl.w_st);
  for (int64_t s : e->D_rowptr) p = put(p, (uint64_t)s, pl.w_st);
}

uint64_t get(const uint8_t *p, int w) {
  uint64_t v = 0;
  for (int q = 0; q < w; ++q) v |= (uint64_t)p[q] << (8 * q);
  return v;
}

}  // namespace
}  // namespace toc

using namespace toc;

extern "C" {

toc_status toc_enc_pack_size(const toc_enc *enc, size_t *bytes) {
  clear_error();
  if (!enc || !bytes) return fail(TOC_EINVAL, "NULL argument");
  PackPlan pl;
  const toc_status st = plan(enc, pl);
  if (st == TOC_OK) *bytes = pl.bytes;
  return st;
}

toc_status toc_enc_pack(const toc_enc *enc, void *dst, size_t bytes) {
  clear_error();
  if (!enc || !dst) return fail(TOC_EINVAL, "NULL argument");
  PackPlan pl;
  toc_status st = plan(enc, pl);
  if (st != TOC_OK) return st;
  if (bytes < pl.bytes) return fail(TOC_ESIZE, "%zu bytes given, %zu needed", bytes, pl.bytes);
  write(enc, pl, (uint8_t *)dst);
  return TOC_OK;
}

toc_status toc_phys_info_get(const void *blob, size_t bytes, toc_phys_info *info) {
  clear_error();
  if (!info || (!blob && bytes > 0)) return fail(TOC_EINVAL, "NULL argument");
  const uint8_t *b = (const uint8_t *)blob;
  uint64_t cnt[5];
  int wid[5];
  size_t data[5], pos = 0;
  for (int a = 0; a < 5; ++a) {
    if (pos > bytes || bytes - pos < 5) return fail(TOC_EINVAL, "truncated header of array %d", a);
    cnt[a] = get(b + pos, 4);
    wid[a] = (int)b[pos + 4];
    if (wid[a] < 1 || wid[a] > 4 || (a == 1 && wid[a] != 4))
      return fail(TOC_EINVAL, "bad bytes per integer %d in array %d", wid[a], a);
    data[a] = pos + 5;
    if ((bytes - data[a]) / (uint64_t)wid[a] < cnt[a]) return fail(TOC_EINVAL, "truncated array %d", a);
    pos = data[a] + (size_t)cnt[a] * (size_t)wid[a];
  }
  if (pos != bytes) return fail(TOC_EINVAL, "%zu trailing bytes", bytes - pos);
  if (cnt[2] != cnt[0]) return fail(TOC_EINVAL, "value indexes and columns differ in count");
  if (cnt[4] < 1) return fail(TOC_EINVAL, "no tuple starts");
  uint64_t prev = 0;
  int64_t nonempty = 0;
  for (uint64_t r = 0; r < cnt[4]; ++r) {
    const uint64_t s = get(b + data[4] + r * wid[4], wid[4]);
    if ((r == 0 && s != 0) || s < prev || s > cnt[3]) return fail(TOC_EINVAL, "bad tuple start %llu", (unsigned long long)r);
    if (r > 0 && s > prev) ++nonempty;
    prev = s;
  }
  if (prev != cnt[3]) return fail(TOC_EINVAL, "tuple starts end at %llu, not |D|", (unsigned long long)prev);
  info->n_rows = (int64_t)cnt[4] - 1;
  info->n_first = (int64_t)cnt[0];
  info->n_codes = (int64_t)cnt[3];
  info->n_unique = (int64_t)cnt[1];
  info->n_nodes = 1 + (int64_t)cnt[0] + (int64_t)cnt[3] - nonempty;
  int64_t max_col = -1;
  for (uint64_t i = 0; i < cnt[0]; ++i)
    max_col = std::max<int64_t>(max_col, (int64_t)get(b + data[0] + i * wid[0], wid[0]));
  info->max_col = max_col;
  return TOC_OK;
}

}  // extern "C"
