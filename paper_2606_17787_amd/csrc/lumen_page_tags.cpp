// Page tags and the longest checkpointed prefix: the host side of KV-reuse
// recovery.  The operations are specified in include/lumen_page_tags.h.

#include <stdint.h>
#include <string.h>

#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

#include "lumen_kv_ckpt.h"
#include "lumen_page_tags.h"

namespace {

// BLAKE2b (RFC 7693), unkeyed, 8-byte digest: initial state, message
// schedule, mixing function and compression as the RFC defines them.
constexpr uint64_t kIV[8] = {
    0x6a09e667f3bcc908ull, 0xbb67ae8584caa73bull, 0x3c6ef372fe94f82bull,
    0xa54ff53a5f1d36f1ull, 0x510e527fade682d1ull, 0x9b05688c2b3e6c1full,
    0x1f83d9abfb41bd6bull, 0x5be0cd19137e2179ull};

constexpr uint8_t kSigma[10][16] = {
    {0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15},
    {14, 10, 4, 8, 9, 15, 13, 6, 1, 12, 0, 2, 11, 7, 5, 3},
    {11, 8, 12, 0, 5, 2, 15, 13, 10, 14, 3, 6, 7, 1, 9, 4},
    {7, 9, 3, 1, 13, 12, 11, 14, 2, 6, 5, 10, 4, 0, 15, 8},
    {9, 0, 5, 7, 2, 4, 10, 15, 14, 1, 11, 12, 6, 8, 3, 13},
    {2, 12, 6, 10, 0, 11, 8, 3, 4, 13, 7, 5, 15, 14, 1, 9},
    {12, 5, 1, 15, 14, 13, 4, 10, 0, 7, 6, 3, 9, 2, 8, 11},
    {13, 11, 7, 14, 12, 1, 3, 9, 5, 0, 15, 4, 8, 6, 2, 10},
    {6, 15, 14, 9, 11, 3, 0, 8, 12, 2, 13, 7, 1, 4, 10, 5},
    {10, 2, 8, 4, 7, 6, 1, 5, 15, 11, 9, 14, 3, 12, 13, 0}};

inline uint64_t rotr(uint64_t x, int n) { return (x >> n) | (x << (64 - n)); }

inline void mix(uint64_t *v, int a, int b, int c, int d, uint64_t x,
                uint64_t y) {
  v[a] = v[a] + v[b] + x;
  v[d] = rotr(v[d] ^ v[a], 32);
  v[c] = v[c] + v[d];
  v[b] = rotr(v[b] ^ v[c], 24);
  v[a] = v[a] + v[b] + y;
  v[d] = rotr(v[d] ^ v[a], 16);
  v[c] = v[c] + v[d];
  v[b] = rotr(v[b] ^ v[c], 63);
}

inline uint64_t load_le64(const uint8_t *p) {
  uint64_t x = 0;
  for (int i = 7; i >= 0; --i) x = (x << 8) | p[i];
  return x;
}

void compress(uint64_t h[8], const uint8_t block[128], uint64_t bytes,
              bool last) {
  uint64_t m[16], v[16];
  for (int i = 0; i < 16; ++i) m[i] = load_le64(block + 8 * i);
  for (int i = 0; i < 8; ++i) {
    v[i] = h[i];
    v[i + 8] = kIV[i];
  }
  v[12] ^= bytes;  // low word of the byte counter (inputs stay below 2^64)
  if (last) v[14] = ~v[14];
  for (int r = 0; r < 12; ++r) {
    const uint8_t *s = kSigma[r % 10];
    mix(v, 0, 4, 8, 12, m[s[0]], m[s[1]]);
    mix(v, 1, 5, 9, 13, m[s[2]], m[s[3]]);
    mix(v, 2, 6, 10, 14, m[s[4]], m[s[5]]);
    mix(v, 3, 7, 11, 15, m[s[6]], m[s[7]]);
    mix(v, 0, 5, 10, 15, m[s[8]], m[s[9]]);
    mix(v, 1, 6, 11, 12, m[s[10]], m[s[11]]);
    mix(v, 2, 7, 8, 13, m[s[12]], m[s[13]]);
    mix(v, 3, 4, 9, 14, m[s[14]], m[s[15]]);
  }
  for (int i = 0; i < 8; ++i) h[i] ^= v[i] ^ v[i + 8];
}

// BLAKE2b-64 of n int32 token IDs, serialised little-endian.
uint64_t hash_tokens(const int32_t *tok, int64_t n) {
  uint64_t h[8];
  memcpy(h, kIV, sizeof(h));
  h[0] ^= 0x01010000ull ^ 8;  // depth 1, fanout 1, no key, 8-byte digest
  const uint64_t len = uint64_t(n) * 4;
  uint8_t block[128];
  uint64_t done = 0;
  int64_t t = 0;
  // Whole blocks, except that the last block (full or partial, or the
  // empty block of an empty input) is compressed with the final flag.
  while (true) {
    const uint64_t left = len - done;
    const uint64_t take = left > 128 ? 128 : left;
    memset(block, 0, sizeof(block));
    for (uint64_t i = 0; i < take; i += 4, ++t) {
      const uint32_t x = uint32_t(tok[t]);
      block[i] = uint8_t(x);
      block[i + 1] = uint8_t(x >> 8);
      block[i + 2] = uint8_t(x >> 16);
      block[i + 3] = uint8_t(x >> 24);
    }
    done += take;
    const bool last = done == len;
    compress(h, block, done, last);
    if (last) break;
  }
  return h[0];  // the first 8 output bytes, little-endian
}

int check_pages(const int32_t *tokens, int64_t num_tokens, int32_t bs,
                int64_t page_begin, int64_t page_end) {
  if (bs < 1 || num_tokens < 0 || page_begin < 0 || page_end < page_begin)
    return LUMEN_ERR_INVALID_ARG;
  if (page_end > num_tokens / bs) return LUMEN_ERR_INVALID_ARG;
  if (page_end > page_begin && !tokens) return LUMEN_ERR_INVALID_ARG;
  return LUMEN_OK;
}

// Largest page index a store accepts (so (page + 1) * block_size and the
// per-request page vector stay far from any overflow).
constexpr int64_t kMaxPage = INT32_MAX;

struct PageEntry {
  uint64_t hash = 0;
  int64_t end = 0;
  bool visible = false;
};

}  // namespace

struct lumen_tag_store {
  int32_t block_size;
  std::mutex mu;
  std::unordered_map<int64_t, std::vector<PageEntry>> pages;
  std::unordered_map<int64_t, int64_t> visible;  // count per request
};

extern "C" {

int lumen_page_tags(const int32_t *tokens, int64_t num_tokens,
                    int32_t block_size, int64_t page_begin, int64_t page_end,
                    lumen_page_tag *tags) {
  int st = check_pages(tokens, num_tokens, block_size, page_begin, page_end);
  if (st != LUMEN_OK) return st;
  if (page_end > page_begin && !tags) return LUMEN_ERR_INVALID_ARG;
  for (int64_t p = page_begin; p < page_end; ++p) {
    tags[p - page_begin].hash = hash_tokens(tokens + p * block_size, block_size);
    tags[p - page_begin].end = (p + 1) * block_size;
  }
  return LUMEN_OK;
}

lumen_tag_store *lumen_tag_store_create(int32_t block_size) {
  if (block_size < 1) return nullptr;
  lumen_tag_store *s = new (std::nothrow) lumen_tag_store;
  if (s) s->block_size = block_size;
  return s;
}

void lumen_tag_store_destroy(lumen_tag_store *store) { delete store; }

int lumen_tag_store_publish(lumen_tag_store *store, int64_t request,
                            int64_t page, lumen_page_tag tag) {
  if (!store || page < 0 || page > kMaxPage ||
      tag.end != (page + 1) * store->block_size)
    return LUMEN_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(store->mu);
  try {
    // Everything that allocates happens before the page is changed, so a
    // failed allocation leaves the store as it was.
    std::vector<PageEntry> &v = store->pages[request];
    if (v.size() <= size_t(page)) v.resize(size_t(page) + 1);
    int64_t &count = store->visible[request];
    if (!v[page].visible) ++count;
    v[page].hash = tag.hash;
    v[page].end = tag.end;
    v[page].visible = true;
  } catch (const std::bad_alloc &) {
    return LUMEN_ERR_CAPACITY;
  }
  return LUMEN_OK;
}

int lumen_tag_store_publish_pages(lumen_tag_store *store, int64_t request,
                                  const int32_t *tokens, int64_t num_tokens,
                                  int64_t page_begin, int64_t page_end) {
  if (!store) return LUMEN_ERR_INVALID_ARG;
  int st = check_pages(tokens, num_tokens, store->block_size, page_begin,
                       page_end);
  if (st != LUMEN_OK) return st;
  for (int64_t p = page_begin; p < page_end; ++p) {
    lumen_page_tag tag;
    tag.hash = hash_tokens(tokens + p * store->block_size, store->block_size);
    tag.end = (p + 1) * store->block_size;
    st = lumen_tag_store_publish(store, request, p, tag);
    if (st != LUMEN_OK) return st;
  }
  return LUMEN_OK;
}

int lumen_tag_store_release(lumen_tag_store *store, int64_t request) {
  if (!store) return LUMEN_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(store->mu);
  store->pages.erase(request);
  store->visible.erase(request);
  return LUMEN_OK;
}

int64_t lumen_tag_store_longest_prefix(lumen_tag_store *store,
                                       int64_t request, const int32_t *tokens,
                                       int64_t num_tokens) {
  if (!store || num_tokens < 0 || (num_tokens > 0 && !tokens))
    return LUMEN_ERR_INVALID_ARG;
  const int32_t bs = store->block_size;
  const int64_t complete = num_tokens / bs;
  std::lock_guard<std::mutex> lock(store->mu);
  auto it = store->pages.find(request);
  if (it == store->pages.end()) return 0;
  const std::vector<PageEntry> &v = it->second;
  int64_t n = 0;
  while (n < complete && size_t(n) < v.size() && v[n].visible &&
         v[n].end == (n + 1) * bs &&
         v[n].hash == hash_tokens(tokens + n * bs, bs))
    ++n;
  return n * bs;
}

int64_t lumen_tag_store_pages(lumen_tag_store *store, int64_t request) {
  if (!store) return LUMEN_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(store->mu);
  auto it = store->visible.find(request);
  return it == store->visible.end() ? 0 : it->second;
}

}  // extern "C"
