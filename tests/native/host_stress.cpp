// Randomised stress of the host libraries (page tags, scheduler, progress
// tracker) through their C ABI, built with AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py.  Besides
// being sanitizer-clean, every step checks invariants that hold for any
// sequence of calls:
//   - scheduler: the bytes reserved on a worker equal the footprints of the
//     requests it holds, never exceed its budget, and a holder is never the
//     request's serving worker; recovery reports every interrupted request
//     exactly once;
//   - progress: start <= end, start equals what was sent before;
//   - tags: the longest prefix is a whole number of pages, never longer
//     than the history, and equals the published run of matching pages.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <map>
#include <random>
#include <set>
#include <vector>

#include "lumen_kv_ckpt.h"
#include "lumen_page_tags.h"
#include "lumen_progress.h"
#include "lumen_sched.h"

#define CHECK(c)                                                      \
  do {                                                                \
    if (!(c)) {                                                       \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      exit(1);                                                        \
    }                                                                 \
  } while (0)

static void stress_sched(std::mt19937_64 &rng) {
  const int32_t W = 2 + int32_t(rng() % 7);
  std::vector<int64_t> budget(W);
  for (auto &b : budget) b = int64_t(rng() % 1000);
  lumen_sched *s = lumen_sched_create(W, budget.data(), 1e9, 0.5);
  CHECK(s);
  std::map<int64_t, std::pair<int32_t, int64_t>> live;  // id -> serving, bytes
  std::set<int32_t> dead;
  int64_t next = 0;
  for (int step = 0; step < 400; ++step) {
    const int op = int(rng() % 10);
    if (op < 5) {
      int32_t serving = int32_t(rng() % W);
      if (dead.count(serving)) continue;
      const int64_t bytes = int64_t(rng() % 300);
      int32_t holder = -2;
      CHECK(lumen_sched_place(s, next, serving, bytes, &holder) == LUMEN_OK);
      CHECK(holder >= -1 && holder < W && holder != serving);
      CHECK(holder < 0 || !dead.count(holder));
      live[next++] = {serving, bytes};
    } else if (op < 7 && !live.empty()) {
      auto it = live.begin();
      std::advance(it, rng() % live.size());
      CHECK(lumen_sched_set_persisted(s, it->first, int64_t(rng() % 400)) ==
            LUMEN_OK);
      if (rng() % 2) {
        CHECK(lumen_sched_release(s, it->first) == LUMEN_OK);
        live.erase(it);
      }
    } else if (op < 8) {
      for (int32_t w = 0; w < W; ++w)
        CHECK(lumen_sched_set_worker(s, w, double(rng() % 100) / 10.0,
                                     int64_t(rng() % 20),
                                     int64_t(rng() % 20)) == LUMEN_OK);
    } else if (op == 8) {
      const int32_t f = int32_t(rng() % W);
      std::vector<int64_t> req(live.size() + 1);
      std::vector<int32_t> wk(live.size() + 1);
      std::vector<int8_t> reuse(live.size() + 1);
      int64_t n = -1;
      CHECK(lumen_sched_recover(s, &f, 1, req.data(), wk.data(), reuse.data(),
                                int64_t(req.size()), &n) == LUMEN_OK);
      dead.insert(f);
      std::set<int64_t> seen;
      for (int64_t k = 0; k < n; ++k) {
        CHECK(live.count(req[k]) && seen.insert(req[k]).second);
        CHECK(dead.count(live[req[k]].first));
        CHECK(wk[k] == -1 || !dead.count(wk[k]));
        if (wk[k] >= 0) live[req[k]].first = wk[k];
      }
      int64_t expect = 0;
      for (auto &kv : live)
        if (dead.count(kv.second.first)) ++expect;
      // requests that found no survivor stay on a dead worker
      CHECK(n >= expect);
    }
    // reservations equal the held footprints and stay within budget
    std::vector<int64_t> held(W, 0);
    for (auto &kv : live) {
      int32_t h = -2;
      CHECK(lumen_sched_holder(s, kv.first, &h) == LUMEN_OK);
      CHECK(h >= -1 && h < W);
      if (h >= 0) {
        CHECK(h != kv.second.first || dead.count(h));
        held[h] += kv.second.second;
      }
    }
    for (int32_t w = 0; w < W; ++w) {
      const int64_t r = lumen_sched_reserved(s, w);
      CHECK(r == held[w] && r <= budget[w]);
      CHECK(!dead.count(w) || r == 0);
    }
  }
  int32_t h = 0;
  CHECK(lumen_sched_holder(s, next + 5, &h) == LUMEN_ERR_INVALID_ARG);
  CHECK(lumen_sched_place(s, 0, W, 1, &h) == LUMEN_ERR_INVALID_ARG);
  lumen_sched_destroy(s);
}

static void stress_progress(std::mt19937_64 &rng) {
  lumen_progress *p = lumen_progress_create();
  CHECK(p);
  std::map<int64_t, int32_t> sent;
  for (int step = 0; step < 300; ++step) {
    const int32_t n = int32_t(rng() % 12);
    std::set<int64_t> ids;
    while (int32_t(ids.size()) < n) ids.insert(int64_t(rng() % 40));
    std::vector<int64_t> id(ids.begin(), ids.end());
    std::vector<int32_t> len(n), st(n), en(n);
    for (int32_t i = 0; i < n; ++i) {
      const int32_t prev = sent.count(id[i]) ? sent[id[i]] : 0;
      // mostly growing histories, sometimes a rewritten (shorter) tail
      len[i] = rng() % 8 ? prev + int32_t(rng() % 20)
                         : int32_t(rng() % (prev + 1));
    }
    CHECK(lumen_progress_ranges(p, id.data(), len.data(), n, st.data(),
                                en.data()) == LUMEN_OK);
    for (int32_t i = 0; i < n; ++i) {
      const int32_t prev = sent.count(id[i]) ? sent[id[i]] : 0;
      CHECK(st[i] == (prev < len[i] ? prev : len[i]) && en[i] == len[i]);
      sent[id[i]] = len[i];
      CHECK(lumen_progress_sent(p, id[i]) == len[i]);
    }
    if (rng() % 5 == 0 && !sent.empty()) {
      auto it = sent.begin();
      std::advance(it, rng() % sent.size());
      CHECK(lumen_progress_release(p, it->first) == LUMEN_OK);
      CHECK(lumen_progress_sent(p, it->first) == 0);
      sent.erase(it);
    }
  }
  // a repeated id changes nothing
  int64_t dup[2] = {1, 1};
  int32_t len[2] = {5, 6}, st[2], en[2];
  const int64_t before = lumen_progress_sent(p, 1);
  CHECK(lumen_progress_ranges(p, dup, len, 2, st, en) == LUMEN_ERR_INVALID_ARG);
  CHECK(lumen_progress_sent(p, 1) == before);
  lumen_progress_destroy(p);
}

static void stress_tags(std::mt19937_64 &rng) {
  const int32_t bs = 1 + int32_t(rng() % 16);
  lumen_tag_store *st = lumen_tag_store_create(bs);
  CHECK(st);
  std::vector<std::vector<int32_t>> hist(6);
  for (auto &h : hist) {
    h.resize(rng() % 200);
    for (auto &x : h) x = int32_t(rng());
  }
  std::vector<std::set<int64_t>> pub(6);
  for (int step = 0; step < 300; ++step) {
    const int64_t r = int64_t(rng() % 6);
    auto &h = hist[r];
    const int64_t pages = int64_t(h.size()) / bs;
    const int op = int(rng() % 6);
    if (op < 3 && pages > 0) {
      const int64_t a = int64_t(rng() % pages);
      const int64_t b = a + int64_t(rng() % (pages - a + 1));
      CHECK(lumen_tag_store_publish_pages(st, r, h.data(), int64_t(h.size()),
                                         a, b) == LUMEN_OK);
      for (int64_t q = a; q < b; ++q) pub[r].insert(q);
    } else if (op == 3 && !h.empty()) {
      // the history's tail is rewritten: published pages there go stale
      const size_t at = rng() % h.size();
      h[at] = int32_t(rng());
    } else if (op == 4) {
      CHECK(lumen_tag_store_release(st, r) == LUMEN_OK);
      pub[r].clear();
    }
    const int64_t got =
        lumen_tag_store_longest_prefix(st, r, h.data(), int64_t(h.size()));
    CHECK(got >= 0 && got % bs == 0 && got <= int64_t(h.size()));
    CHECK(got / bs <= int64_t(pub[r].size()));
    for (int64_t q = 0; q < got / bs; ++q) CHECK(pub[r].count(q));
    CHECK(lumen_tag_store_pages(st, r) == int64_t(pub[r].size()));
  }
  lumen_page_tag t{0, 0};
  CHECK(lumen_tag_store_publish(st, 0, int64_t(1) << 40, t) ==
        LUMEN_ERR_INVALID_ARG);
  lumen_tag_store_destroy(st);
}

int main(int argc, char **argv) {
  const int rounds = argc > 1 ? atoi(argv[1]) : 50;
  std::mt19937_64 rng(20261202);
  for (int i = 0; i < rounds; ++i) {
    stress_sched(rng);
    stress_progress(rng);
    stress_tags(rng);
  }
  printf("host stress ok: %d rounds\n", rounds);
  return 0;
}
