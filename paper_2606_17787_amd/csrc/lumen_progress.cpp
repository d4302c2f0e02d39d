// Checkpoint progress of a serving worker; specified in
// include/lumen_progress.h.

#include <stdint.h>

#include <new>
#include <unordered_map>
#include <unordered_set>

#include "lumen_kv_ckpt.h"
#include "lumen_progress.h"

struct lumen_progress {
  std::unordered_map<int64_t, int32_t> sent;
};

extern "C" {

lumen_progress *lumen_progress_create(void) {
  return new (std::nothrow) lumen_progress;
}

void lumen_progress_destroy(lumen_progress *p) { delete p; }

int lumen_progress_ranges(lumen_progress *p, const int64_t *ids,
                          const int32_t *lengths, int32_t n, int32_t *start,
                          int32_t *end) {
  if (!p || n < 0) return LUMEN_ERR_INVALID_ARG;
  if (n > 0 && (!ids || !lengths || !start || !end))
    return LUMEN_ERR_INVALID_ARG;
  try {
    std::unordered_set<int64_t> seen;
    for (int32_t i = 0; i < n; ++i) {
      if (lengths[i] < 0 || !seen.insert(ids[i]).second)
        return LUMEN_ERR_INVALID_ARG;
    }
    // Allocation first: a request not seen before gets an entry of 0 sent
    // tokens, which is what an absent entry means, so a failure here
    // changes nothing a caller can observe.
    for (int32_t i = 0; i < n; ++i) p->sent.emplace(ids[i], 0);
  } catch (const std::bad_alloc &) {
    return LUMEN_ERR_CAPACITY;
  }
  for (int32_t i = 0; i < n; ++i) {
    int32_t &done = p->sent.find(ids[i])->second;
    start[i] = done < lengths[i] ? done : lengths[i];
    end[i] = lengths[i];
    done = lengths[i];
  }
  return LUMEN_OK;
}

int64_t lumen_progress_sent(lumen_progress *p, int64_t request) {
  if (!p) return LUMEN_ERR_INVALID_ARG;
  auto it = p->sent.find(request);
  return it == p->sent.end() ? 0 : it->second;
}

int lumen_progress_release(lumen_progress *p, int64_t request) {
  if (!p) return LUMEN_ERR_INVALID_ARG;
  p->sent.erase(request);
  return LUMEN_OK;
}

}  // extern "C"
