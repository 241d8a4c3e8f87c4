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

struct Packer {
  uint8_t *out;   // null: count bytes only
  size_t n = 0;
  void put(uint64_t v, int w) {
    for (int q = 0; q < w; ++q, ++n)
      if (out) out[n] = (uint8_t)(v >> (8 * q));
  }
  void header(uint64_t count, int w) {
    put(count, 4);
    put((uint64_t)w, 1);
  }
};

// unique values of I (ascending bit patterns)
std::vector<uint32_t> uniques(const toc_enc *e) {
  std::vector<uint32_t> u(e->I_bits);
  std::sort(u.begin(), u.end());
  u.erase(std::unique(u.begin(), u.end()), u.end());
  return u;
}

toc_status pack(const toc_enc *e, Packer &pk) {
  const size_t nI = e->I_col.size(), nD = e->D_codes.size();
  if (nI > 0xFFFFFFFFu || nD > 0xFFFFFFFFu || (uint64_t)e->n_rows + 1 > 0xFFFFFFFFu)
    return fail(TOC_EUNSUPPORTED, "array longer than a u32 count");
  const std::vector<uint32_t> u = uniques(e);
  uint64_t mc = 0, md = 0;
  for (int32_t c : e->I_col) mc = std::max<uint64_t>(mc, (uint64_t)c);
  for (uint32_t c : e->D_codes) md = std::max<uint64_t>(md, c);
  int w = width_of(mc);
  pk.header(nI, w);
  for (int32_t c : e->I_col) pk.put((uint64_t)c, w);
  pk.header(u.size(), 4);
  for (uint32_t b : u) pk.put(b, 4);
  w = width_of(u.empty() ? 0 : u.size() - 1);
  pk.header(nI, w);
  for (uint32_t b : e->I_bits)
    pk.put((uint64_t)(std::lower_bound(u.begin(), u.end(), b) - u.begin()), w);
  w = width_of(md);
  pk.header(nD, w);
  for (uint32_t c : e->D_codes) pk.put(c, w);
  w = width_of((uint64_t)nD);
  pk.header((uint64_t)e->n_rows + 1, w);
  for (int64_t s : e->D_rowptr) pk.put((uint64_t)s, w);
  return TOC_OK;
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
  Packer pk{nullptr};
  const toc_status st = pack(enc, pk);
  if (st == TOC_OK) *bytes = pk.n;
  return st;
}

toc_status toc_enc_pack(const toc_enc *enc, void *dst, size_t bytes) {
  clear_error();
  if (!enc || !dst) return fail(TOC_EINVAL, "NULL argument");
  Packer cnt{nullptr};
  toc_status st = pack(enc, cnt);
  if (st != TOC_OK) return st;
  if (bytes < cnt.n) return fail(TOC_ESIZE, "%zu bytes given, %zu needed", bytes, cnt.n);
  Packer pk{(uint8_t *)dst};
  return pack(enc, pk);
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
