// Host-side session management of the retention path (no device code):
//   session key derivation, Appendix A (session identification) and Appendix H
//   (session id derivation): an explicit session id, else the token tuple of a
//   designated session span, else the first P = 256 input tokens, else a key local
//   to the request that never matches another;
//   the QueryMemory store: an LRU of `capacity` (1,024 in the paper) memories per
//   compressor, handing out rows of a caller-owned device arena;
//   the compression trigger: N > C (Appendix H), then every `trigger` (512) new
//   tokens (Appendix A, training setup);
//   the actionable query span (Sec. 3.1) with the bounded tail fallback of W = 32
//   positions (Appendix A, compression settings).
#include <stdint.h>
#include <string.h>

#include <list>
#include <new>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "ikv_error.hpp"

using ikv::set_error;

namespace {

struct Entry {
  std::string key;          // kind byte + the key's bytes
  int32_t slot;
  int32_t refs;             // acquired and not yet released: not evictable
  int32_t last_n;           // N at the last compression event fired for this memory (0: none)
};

}  // namespace

struct ikv_memstore {
  std::mutex mu;
  int32_t capacity;
  uint64_t next_local = 1;                   // request-local keys, never reused
  std::list<Entry> lru;                      // front = most recently used
  std::unordered_map<std::string, std::list<Entry>::iterator> index;
  std::vector<int32_t> free_slots;           // arena rows never handed out or released by eviction
  std::vector<std::list<Entry>::iterator> by_slot;
  std::vector<bool> used;
};

namespace {

// The key's bytes, prefixed by its kind so that keys of different kinds never match.
ikv_status derive_key(const ikv_key_source *src, uint64_t *local_counter, std::string *key, int32_t *kind) {
  if (!src) return set_error(IKV_EINVAL, "key source is NULL");
  if (src->session_id && src->session_id_len > 0) {
    *kind = IKV_KEY_EXPLICIT;
    key->assign(1, char(IKV_KEY_EXPLICIT));
    key->append(src->session_id, size_t(src->session_id_len));
    return IKV_OK;
  }
  if (src->session_id_len < 0 || src->n_tokens < 0) return set_error(IKV_EINVAL, "negative length");
  const bool have_tokens = src->tokens != nullptr && src->n_tokens > 0;
  if (have_tokens && src->span_end > src->span_start) {
    if (src->span_start < 0 || src->span_end > src->n_tokens)
      return set_error(IKV_ESHAPE, "session span outside the request's tokens");
    *kind = IKV_KEY_SPAN;
    key->assign(1, char(IKV_KEY_SPAN));
    key->append(reinterpret_cast<const char *>(src->tokens + src->span_start),
                size_t(src->span_end - src->span_start) * sizeof(int32_t));
    return IKV_OK;
  }
  if (have_tokens) {
    const int32_t n = src->n_tokens < IKV_PREFIX_TOKENS ? src->n_tokens : IKV_PREFIX_TOKENS;
    *kind = IKV_KEY_PREFIX;
    key->assign(1, char(IKV_KEY_PREFIX));
    key->append(reinterpret_cast<const char *>(src->tokens), size_t(n) * sizeof(int32_t));
    return IKV_OK;
  }
  *kind = IKV_KEY_LOCAL;
  const uint64_t id = (*local_counter)++;
  key->assign(1, char(IKV_KEY_LOCAL));
  key->append(reinterpret_cast<const char *>(&id), sizeof id);
  return IKV_OK;
}

}  // namespace

extern "C" {

ikv_status ikv_memstore_create(int32_t capacity, ikv_memstore **out) {
  if (!out) return set_error(IKV_EINVAL, "out is NULL");
  *out = nullptr;
  if (capacity < 1) return set_error(IKV_ESHAPE, "capacity must be >= 1");
  ikv_memstore *s = new (std::nothrow) ikv_memstore;
  if (!s) return set_error(IKV_EINVAL, "out of host memory");
  s->capacity = capacity;
  s->free_slots.reserve(size_t(capacity));
  for (int32_t i = capacity - 1; i >= 0; --i) s->free_slots.push_back(i);   // slot 0 handed out first
  s->by_slot.resize(size_t(capacity));
  s->used.assign(size_t(capacity), false);
  *out = s;
  return set_error(IKV_OK, "");
}

void ikv_memstore_destroy(ikv_memstore *store) { delete store; }

ikv_status ikv_memstore_acquire(ikv_memstore *s, const ikv_key_source *src, int32_t *slot, int32_t *fresh,
                                int32_t *kind) {
  if (!s || !slot || !fresh) return set_error(IKV_EINVAL, "store / slot / fresh is NULL");
  std::lock_guard<std::mutex> lk(s->mu);
  std::string key;
  int32_t k = 0;
  ikv_status r = derive_key(src, &s->next_local, &key, &k);
  if (r) return r;
  if (kind) *kind = k;
  auto it = s->index.find(key);
  if (it != s->index.end()) {                  // a known session: most recently used now
    s->lru.splice(s->lru.begin(), s->lru, it->second);
    Entry &e = s->lru.front();
    ++e.refs;
    *slot = e.slot;
    *fresh = 0;
    return set_error(IKV_OK, "");
  }
  int32_t sl;
  if (!s->free_slots.empty()) {
    sl = s->free_slots.back();
    s->free_slots.pop_back();
  } else {                                     // evict the least recently used memory not in use
    auto victim = s->lru.end();
    for (auto v = s->lru.end(); v != s->lru.begin();) {
      --v;
      if (v->refs == 0) {
        victim = v;
        break;
      }
    }
    if (victim == s->lru.end())
      return set_error(IKV_EUNSUPPORTED, "every memory of the store is in use; none can be evicted");
    sl = victim->slot;
    s->index.erase(victim->key);
    s->lru.erase(victim);
  }
  s->lru.push_front(Entry{key, sl, 1, 0});
  s->index[key] = s->lru.begin();
  s->by_slot[size_t(sl)] = s->lru.begin();
  s->used[size_t(sl)] = true;
  *slot = sl;
  *fresh = 1;
  return set_error(IKV_OK, "");
}

ikv_status ikv_memstore_release(ikv_memstore *s, int32_t slot) {
  if (!s) return set_error(IKV_EINVAL, "store is NULL");
  std::lock_guard<std::mutex> lk(s->mu);
  if (slot < 0 || slot >= s->capacity || !s->used[size_t(slot)] || s->by_slot[size_t(slot)]->refs <= 0)
    return set_error(IKV_ESHAPE, "slot %d is not acquired", slot);
  --s->by_slot[size_t(slot)]->refs;
  return set_error(IKV_OK, "");
}

ikv_status ikv_memstore_trigger(ikv_memstore *s, int32_t slot, int32_t N, int32_t C, int32_t trigger,
                                int32_t *fire) {
  if (!s || !fire) return set_error(IKV_EINVAL, "store / fire is NULL");
  if (N < 0 || C < 0 || trigger < 0) return set_error(IKV_ESHAPE, "N, C and trigger must be >= 0");
  std::lock_guard<std::mutex> lk(s->mu);
  if (slot < 0 || slot >= s->capacity || !s->used[size_t(slot)])
    return set_error(IKV_ESHAPE, "slot is not held by a memory");
  Entry &e = *s->by_slot[size_t(slot)];
  *fire = N > C && int64_t(N) - e.last_n >= trigger;
  if (*fire) e.last_n = N;
  return set_error(IKV_OK, "");
}

ikv_status ikv_memstore_size(ikv_memstore *s, int32_t *n) {
  if (!s || !n) return set_error(IKV_EINVAL, "store / n is NULL");
  std::lock_guard<std::mutex> lk(s->mu);
  *n = int32_t(s->lru.size());
  return set_error(IKV_OK, "");
}

ikv_status ikv_resolve_span(int32_t N, const int32_t *msg_start, const int32_t *msg_end, const uint8_t *actionable,
                            int32_t n_msgs, int32_t tail_w, int32_t *qs, int32_t *qe) {
  if (!qs || !qe) return set_error(IKV_EINVAL, "qs / qe is NULL");
  if (N < 0 || n_msgs < 0 || tail_w < 0) return set_error(IKV_ESHAPE, "N, n_msgs and tail_w must be >= 0");
  if (n_msgs > 0 && (!msg_start || !msg_end || !actionable))
    return set_error(IKV_EINVAL, "message arrays are NULL");
  for (int32_t m = n_msgs - 1; m >= 0; --m) {      // the latest actionable message
    if (!actionable[m]) continue;
    if (msg_start[m] < 0 || msg_start[m] > msg_end[m] || msg_end[m] > N)
      return set_error(IKV_ESHAPE, "message outside [0, N)");
    if (msg_end[m] == msg_start[m]) continue;        // an empty message resolves nothing
    *qs = msg_start[m];
    *qe = msg_end[m];
    return set_error(IKV_OK, "");
  }
  *qe = N;                                           // the bounded query-tail fallback
  *qs = N > tail_w ? N - tail_w : 0;
  return set_error(IKV_OK, "");
}

}  // extern "C"
