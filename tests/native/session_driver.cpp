// Drives the host session-management code of libikv (ikv_session.cpp) through its C ABI
// with a random sequence of calls, for a build under AddressSanitizer and
// UndefinedBehaviorSanitizer (g++, host code only). Exit status 0 when every call
// behaved as documented; the sanitizers abort on any memory or UB error.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <random>
#include <string>
#include <vector>

#include "ikv.h"
#include "ikv_error.hpp"

static std::string g_last;

namespace ikv {
ikv_status set_error(ikv_status code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last = buf;
  return code;
}
}  // namespace ikv

#define CHECK(c)                                                     \
  do {                                                               \
    if (!(c)) {                                                      \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                      \
    }                                                                \
  } while (0)

int main() {
  std::mt19937 rng(7);
  for (int cap : {1, 3, 64, 1024}) {
    ikv_memstore *st = nullptr;
    CHECK(ikv_memstore_create(cap, &st) == IKV_OK && st);
    std::vector<int> held;
    for (int it = 0; it < 20000; ++it) {
      ikv_key_source src{};
      std::vector<int32_t> toks(size_t(rng() % 400));
      for (auto &t : toks) t = int32_t(rng() % 7);
      std::string id = "s" + std::to_string(rng() % 50);
      switch (rng() % 4) {
        case 0: src.session_id = id.c_str(); src.session_id_len = int32_t(id.size()); break;
        case 1: src.tokens = toks.data(); src.n_tokens = int32_t(toks.size());
                src.span_start = 0; src.span_end = int32_t(toks.size() / 3); break;
        case 2: src.tokens = toks.data(); src.n_tokens = int32_t(toks.size()); break;
        default: break;
      }
      int32_t slot = -1, fresh = -1, kind = -1;
      const ikv_status r = ikv_memstore_acquire(st, &src, &slot, &fresh, &kind);
      if (r == IKV_OK) {
        CHECK(slot >= 0 && slot < cap && (fresh == 0 || fresh == 1) && kind >= 1 && kind <= 4);
        held.push_back(slot);
        int32_t fire = -1;
        CHECK(ikv_memstore_trigger(st, slot, int32_t(rng() % 20000), 8192, 512, &fire) == IKV_OK);
      } else {
        CHECK(r == IKV_EUNSUPPORTED && int(held.size()) >= cap);
      }
      while (!held.empty() && (held.size() > size_t(cap) || rng() % 3)) {
        const size_t k = rng() % held.size();
        CHECK(ikv_memstore_release(st, held[k]) == IKV_OK);
        held.erase(held.begin() + long(k));
      }
    }
    CHECK(ikv_memstore_release(st, cap + 5) == IKV_ESHAPE);
    int32_t n = -1;
    CHECK(ikv_memstore_size(st, &n) == IKV_OK && n >= 1 && n <= cap);
    ikv_memstore_destroy(st);
  }
  int32_t qs, qe;
  const int32_t a[3] = {0, 10, 50}, b[3] = {10, 50, 60};
  const uint8_t act[3] = {0, 1, 0};
  CHECK(ikv_resolve_span(60, a, b, act, 3, 32, &qs, &qe) == IKV_OK && qs == 10 && qe == 50);
  CHECK(ikv_resolve_span(60, a, b, act, 0, 32, &qs, &qe) == IKV_OK && qs == 28 && qe == 60);
  CHECK(ikv_memstore_create(0, nullptr) == IKV_EINVAL);
  puts("session driver: ok");
  return 0;
}
