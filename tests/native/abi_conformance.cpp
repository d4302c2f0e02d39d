// C ABI conformance: a plain HIP host program (no Python, no torch) that
// drives liblumen_kv_ckpt through include/lumen_kv_ckpt.h with its own
// hipMalloc'd buffers and stream, and checks every result against the C
// oracle (oracle/lumen_oracle.h) on the same inputs, byte for byte.
//
// Cases: a token-major cache of 2-byte elements and a head-major cache of
// 4-byte elements; packed and per-request row plans; restore into a second
// pool under another block table; a poisoned block-table entry; the direct
// copy into pinned host memory; both staging pipelines on streams of the
// program's own; validate mode with and without a duplicate target.  Built
// by tests/native/build.py, run by tests/test_gpu_abi_c.py.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <thread>
#include <vector>

#include "lumen_kv_ckpt.h"
#include "../../oracle/lumen_oracle.h"

#define HIP_OK(x)                                                       \
  do {                                                                  \
    hipError_t e_ = (x);                                                \
    if (e_ != hipSuccess) {                                             \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x,         \
              hipGetErrorString(e_));                                   \
      exit(2);                                                          \
    }                                                                   \
  } while (0)
#define CHECK(c)                                                        \
  do {                                                                  \
    if (!(c)) {                                                         \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c);   \
      exit(1);                                                          \
    }                                                                   \
  } while (0)

// Seeded test inputs (splitmix64); holds none of the method's arithmetic.
struct Rng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
  }
  int64_t below(int64_t n) { return int64_t(next() % uint64_t(n)); }
};

template <class T>
T *dev_copy(const std::vector<T> &h) {
  T *d = nullptr;
  HIP_OK(hipMalloc(&d, std::max<size_t>(h.size(), 1) * sizeof(T)));
  if (!h.empty())
    HIP_OK(hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
  return d;
}

template <class T>
std::vector<T> host_copy(const T *d, size_t n) {
  std::vector<T> h(n);
  if (n) HIP_OK(hipMemcpy(h.data(), d, n * sizeof(T), hipMemcpyDeviceToHost));
  return h;
}

struct Case {
  int32_t L, H, D, bs, NB, R, cols, elem, head_major;
};

static void run_case(const Case &c, uint64_t seed, hipStream_t stream) {
  Rng rng{seed};
  lumen_kv_layout lay;
  lay.num_layers = c.L;
  lay.num_kv_heads = c.H;
  lay.head_dim = c.D;
  lay.block_size = c.bs;
  lay.num_blocks = c.NB;
  lay.elem_bytes = c.elem;
  lay.cache_order = c.head_major ? LUMEN_CACHE_HND : LUMEN_CACHE_NHD;
  oracle_cache_shape osh;
  osh.num_layers = c.L;
  osh.num_kv_heads = c.H;
  osh.head_dim = c.D;
  osh.block_size = c.bs;
  osh.num_blocks = c.NB;
  osh.head_major = c.head_major;
  osh.elem_bytes = c.elem;

  const size_t pool_bytes =
      size_t(c.L) * 2 * c.NB * c.bs * c.H * c.D * size_t(c.elem);
  const size_t row_bytes = size_t(c.L) * 2 * c.H * c.D * c.elem;
  std::vector<uint8_t> src(pool_bytes), dst(pool_bytes);
  for (auto &x : src) x = uint8_t(rng.next());
  for (auto &x : dst) x = uint8_t(rng.next());

  // Two block tables naming distinct blocks, and token ranges inside them
  // (one empty range, one starting mid-page).
  CHECK(c.R * c.cols <= c.NB);
  std::vector<int32_t> perm(c.NB), perm2(c.NB);
  for (int32_t i = 0; i < c.NB; ++i) perm[i] = perm2[i] = i;
  for (int32_t i = c.NB - 1; i > 0; --i) {
    std::swap(perm[i], perm[rng.below(i + 1)]);
    std::swap(perm2[i], perm2[rng.below(i + 1)]);
  }
  std::vector<int32_t> bt(perm.begin(), perm.begin() + c.R * c.cols);
  std::vector<int32_t> bt2(perm2.begin(), perm2.begin() + c.R * c.cols);
  std::vector<int32_t> s(c.R), e(c.R);
  const int32_t cap = c.cols * c.bs;
  for (int32_t r = 0; r < c.R; ++r) {
    s[r] = int32_t(rng.below(cap));
    e[r] = s[r] + int32_t(rng.below(cap - s[r] + 1));
  }
  e[0] = s[0];  // an empty range
  int64_t total = 0;
  for (int32_t r = 0; r < c.R; ++r) total += e[r] - s[r];
  CHECK(total > 0);

  // Oracle on the host.
  std::vector<uint8_t> want(size_t(total) * row_bytes);
  CHECK(oracle_pack(&osh, src.data(), bt.data(), c.cols, s.data(), e.data(),
                    c.R, 0, nullptr, want.data(), total) == ORACLE_OK);
  std::vector<uint8_t> want_dst = dst;
  CHECK(oracle_unpack(&osh, want_dst.data(), bt2.data(), c.cols, s.data(),
                      e.data(), c.R, 0, nullptr, want.data(),
                      total) == ORACLE_OK);

  // The library on the device.
  uint8_t *d_src = dev_copy(src), *d_dst = dev_copy(dst);
  int32_t *d_bt = dev_copy(bt), *d_bt2 = dev_copy(bt2);
  int32_t *d_s = dev_copy(s), *d_e = dev_copy(e);
  void *ws = nullptr;
  HIP_OK(hipMalloc(&ws, lumen_kv_ckpt_plan_workspace_bytes(c.R)));
  uint8_t *d_ck = nullptr;
  HIP_OK(hipMalloc(&d_ck, size_t(total) * row_bytes));
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_pack(&lay, d_src, d_bt, c.cols, c.R, ws, d_ck, total,
                           stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_status(ws, stream) == LUMEN_OK);
  CHECK(host_copy(d_ck, want.size()) == want);
  CHECK(lumen_kv_ckpt_unpack(&lay, d_dst, d_bt2, c.cols, c.R, ws, d_ck, total,
                             stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_status(ws, stream) == LUMEN_OK);
  CHECK(host_copy(d_dst, pool_bytes) == want_dst);

  // Per-request row mode: request r's token t at row base[r] + t.
  std::vector<int64_t> base(c.R);
  int64_t next = 3;
  for (int32_t r = 0; r < c.R; ++r) {
    base[r] = next - s[r];
    next += (e[r] - s[r]) + 1;  // a gap row after each request
  }
  const int64_t rows2 = next;
  std::vector<uint8_t> want2(size_t(rows2) * row_bytes, 0xA5);
  CHECK(oracle_pack(&osh, src.data(), bt.data(), c.cols, s.data(), e.data(),
                    c.R, 0, base.data(), want2.data(), rows2) == ORACLE_OK);
  int64_t *d_base = dev_copy(base);
  uint8_t *d_ck2 = dev_copy(std::vector<uint8_t>(want2.size(), 0xA5));
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, d_base, ws, stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_pack(&lay, d_src, d_bt, c.cols, c.R, ws, d_ck2, rows2,
                           stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_status(ws, stream) == LUMEN_OK);
  CHECK(host_copy(d_ck2, want2.size()) == want2);

  // A block-table entry outside the pool: the oracle's status.
  std::vector<int32_t> bad = bt;
  int32_t rb = 1;
  while (e[rb] == s[rb]) ++rb;  // a request with tokens (rb < R: total > 0)
  bad[size_t(rb) * c.cols + s[rb] / c.bs] = c.NB + 7;
  const int want_st = oracle_pack(&osh, src.data(), bad.data(), c.cols,
                                  s.data(), e.data(), c.R, 0, nullptr,
                                  want.data(), total);
  CHECK(want_st == ORACLE_ERR_BLOCK_ID);
  int32_t *d_bad = dev_copy(bad);
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_pack(&lay, d_src, d_bad, c.cols, c.R, ws, d_ck, total,
                           stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_status(ws, stream) == want_st);

  // The one-launch copies that plan from the ranges themselves: the same
  // rows and restored pool in both row modes, and the oracle's status for
  // the bad block id, in a status word the caller clears.
  int32_t *d_status = dev_copy(std::vector<int32_t>{LUMEN_OK});
  uint8_t *d_ck3 = nullptr;
  HIP_OK(hipMalloc(&d_ck3, size_t(total) * row_bytes));
  uint8_t *d_dst2 = dev_copy(dst);
  CHECK(lumen_kv_ckpt_pack_ranges(&lay, d_src, d_bt, c.cols, d_s, d_e, c.R, 0,
                                  nullptr, d_ck3, total, d_status,
                                  stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_unpack_ranges(&lay, d_dst2, d_bt2, c.cols, d_s, d_e,
                                    c.R, 0, nullptr, d_ck3, total, d_status,
                                    stream) == LUMEN_OK);
  HIP_OK(hipStreamSynchronize(stream));
  CHECK(host_copy(d_status, 1)[0] == LUMEN_OK);
  CHECK(host_copy(d_ck3, want.size()) == want);
  CHECK(host_copy(d_dst2, pool_bytes) == want_dst);
  uint8_t *d_ck4 = dev_copy(std::vector<uint8_t>(want2.size(), 0xA5));
  CHECK(lumen_kv_ckpt_pack_ranges(&lay, d_src, d_bt, c.cols, d_s, d_e, c.R, 0,
                                  d_base, d_ck4, rows2, d_status,
                                  stream) == LUMEN_OK);
  HIP_OK(hipStreamSynchronize(stream));
  CHECK(host_copy(d_status, 1)[0] == LUMEN_OK);
  CHECK(host_copy(d_ck4, want2.size()) == want2);
  CHECK(lumen_kv_ckpt_pack_ranges(&lay, d_src, d_bad, c.cols, d_s, d_e, c.R,
                                  0, nullptr, d_ck3, total, d_status,
                                  stream) == LUMEN_OK);
  HIP_OK(hipStreamSynchronize(stream));
  CHECK(host_copy(d_status, 1)[0] == want_st);
  CHECK(lumen_kv_ckpt_pack_ranges(&lay, d_src, d_bt, c.cols, d_s, d_e,
                                  LUMEN_KV_CKPT_RANGES_MAX_REQS + 1, 0,
                                  nullptr, d_ck3, total, d_status,
                                  stream) == LUMEN_ERR_TOO_MANY);
  HIP_OK(hipFree(d_status));
  HIP_OK(hipFree(d_ck3));
  HIP_OK(hipFree(d_ck4));
  HIP_OK(hipFree(d_dst2));

  // The direct copy into pinned host memory.
  uint8_t *h_ck = nullptr;
  HIP_OK(hipHostMalloc((void **)&h_ck, size_t(total) * row_bytes,
                       hipHostMallocDefault));
  memset(h_ck, 0, size_t(total) * row_bytes);
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_pack_to_host_direct(&lay, d_src, d_bt, c.cols, c.R, ws,
                                          0, INT64_MAX, h_ck, 0, total, 0,
                                          stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_status(ws, stream) == LUMEN_OK);
  CHECK(memcmp(h_ck, want.data(), want.size()) == 0);

  // The staging pipelines: to pinned host memory through a 2-slot ring,
  // and back into a third pool, on streams of the program's own.
  hipStream_t ps = nullptr, cs = nullptr, us = nullptr;
  HIP_OK(hipStreamCreate(&ps));
  HIP_OK(hipStreamCreate(&cs));
  HIP_OK(hipStreamCreate(&us));
  const int64_t slot_rows = 3;
  uint8_t *d_ring = nullptr;
  HIP_OK(hipMalloc(&d_ring, 2 * slot_rows * row_bytes));
  memset(h_ck, 0, size_t(total) * row_bytes);
  HIP_OK(hipStreamSynchronize(stream));
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, ps) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_pack_to_host(&lay, d_src, d_bt, c.cols, c.R, ws, total,
                                   d_ring, slot_rows, 2, h_ck, ps,
                                   cs) == LUMEN_OK);
  HIP_OK(hipStreamSynchronize(cs));
  CHECK(lumen_kv_ckpt_status(ws, ps) == LUMEN_OK);
  CHECK(memcmp(h_ck, want.data(), want.size()) == 0);
  uint8_t *d_dst3 = dev_copy(dst);
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, us) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_unpack_from_host(&lay, d_dst3, d_bt2, c.cols, c.R, ws,
                                       total, h_ck, d_ring, slot_rows, 2, cs,
                                       us) == LUMEN_OK);
  HIP_OK(hipStreamSynchronize(us));
  CHECK(lumen_kv_ckpt_status(ws, us) == LUMEN_OK);
  CHECK(host_copy(d_dst3, pool_bytes) == want_dst);

  // Validate mode: the restore table passes; a second page naming an
  // already written block is DUP_BLOCK, as the oracle says.
  const size_t mb = lumen_kv_ckpt_marks_bytes(c.NB);
  void *d_marks = nullptr;
  HIP_OK(hipMalloc(&d_marks, mb));
  CHECK(oracle_validate_targets(&osh, bt2.data(), c.cols, s.data(), e.data(),
                                c.R) == ORACLE_OK);
  CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_validate_targets(&lay, d_bt2, c.cols, c.R, ws, d_marks,
                                       mb, stream) == LUMEN_OK);
  CHECK(lumen_kv_ckpt_status(ws, stream) == LUMEN_OK);
  std::vector<int32_t> dup = bt2;
  int32_t ra = -1, rb2 = -1;  // two requests whose ranges write pages
  for (int32_t r = 0; r < c.R; ++r)
    if (e[r] > s[r]) {
      if (ra < 0) ra = r; else if (rb2 < 0) rb2 = r;
    }
  if (ra >= 0 && rb2 >= 0) {
    dup[size_t(rb2) * c.cols + s[rb2] / c.bs] =
        dup[size_t(ra) * c.cols + s[ra] / c.bs];
    const int want_v = oracle_validate_targets(&osh, dup.data(), c.cols,
                                               s.data(), e.data(), c.R);
    CHECK(want_v == ORACLE_ERR_DUP_BLOCK);
    int32_t *d_dup = dev_copy(dup);
    CHECK(lumen_kv_ckpt_plan(d_s, d_e, c.R, 0, nullptr, ws, stream) ==
          LUMEN_OK);
    CHECK(lumen_kv_ckpt_validate_targets(&lay, d_dup, c.cols, c.R, ws,
                                         d_marks, mb, stream) == LUMEN_OK);
    CHECK(lumen_kv_ckpt_status(ws, stream) == want_v);
    HIP_OK(hipFree(d_dup));
  }
  CHECK(strcmp(lumen_kv_ckpt_strerror(LUMEN_ERR_DUP_BLOCK), "unknown status"));
  CHECK(!strcmp(lumen_kv_ckpt_strerror(12345), "unknown status"));

  HIP_OK(hipFree(d_marks));
  HIP_OK(hipFree(d_dst3));
  HIP_OK(hipFree(d_ring));
  for (hipStream_t q : {ps, cs, us}) HIP_OK(hipStreamDestroy(q));
  HIP_OK(hipHostFree(h_ck));
  for (void *p : {(void *)d_src, (void *)d_dst, (void *)d_bt, (void *)d_bt2,
                  (void *)d_s, (void *)d_e, ws, (void *)d_ck, (void *)d_base,
                  (void *)d_ck2, (void *)d_bad})
    HIP_OK(hipFree(p));
}

int main() {
  hipStream_t stream = nullptr;
  HIP_OK(hipStreamCreate(&stream));  // default priority
  const Case cases[] = {
      {3, 2, 64, 16, 64, 5, 4, 2, 0},  // token-major, 2-byte elements
      {2, 3, 8, 5, 40, 4, 6, 4, 1},    // head-major, 4-byte elements
  };
  uint64_t seed = 20261202;
  for (const Case &c : cases)
    for (int rep = 0; rep < 3; ++rep) run_case(c, seed++, stream);
  HIP_OK(hipStreamDestroy(stream));
  // The same calls from four host threads at once, each on streams and
  // buffers of its own: the library's per-device state (device properties,
  // the pipelines' event pool and ring table) is shared between them.
  constexpr int kThreads = 4;
  std::vector<std::thread> threads;
  for (int t = 0; t < kThreads; ++t)
    threads.emplace_back([&cases, t] {
      HIP_OK(hipSetDevice(0));
      hipStream_t q = nullptr;
      HIP_OK(hipStreamCreate(&q));
      for (int rep = 0; rep < 2; ++rep)
        for (const Case &c : cases)
          run_case(c, 7000 + uint64_t(t) * 16 + uint64_t(rep), q);
      HIP_OK(hipStreamDestroy(q));
    });
  for (std::thread &th : threads) th.join();
  printf("abi conformance ok: %zu layouts x 3 seeds, then %d threads at once\n",
         sizeof(cases) / sizeof(cases[0]), kThreads);
  return 0;
}
