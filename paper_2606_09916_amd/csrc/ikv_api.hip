// Host side of the C ABI declared in include/ikv.h: argument validation, workspace
// sizing and kernel launches. Nothing here allocates device memory.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "ikv_internal.hpp"

namespace {

// ---- per-kernel timing (ikv_timing)
struct TimingRec {
  const char *name;
  hipEvent_t a, b;
};
constexpr size_t kMaxTimingRecs = 65536;
std::mutex g_tmu;
bool g_timing = false;
std::vector<TimingRec> g_recs;      // recorded since the last read
std::vector<hipEvent_t> g_events;   // idle events, reused

hipEvent_t take_event() {
  if (!g_events.empty()) {
    hipEvent_t e = g_events.back();
    g_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}

thread_local std::string g_err;

ikv_status fail(ikv_status code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

ikv_status ok() {
  g_err.clear();
  return IKV_OK;
}

// A fault a kernel of an earlier call reported through the host fault word.
ikv_status pending_fault();

ikv_status hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return ok();
  return fail(IKV_EHIP, "%s: %s", what, hipGetErrorString(e));
}

ikv_status check_pool(const ikv_pool *p) {
  if (!p) return fail(IKV_EINVAL, "pool is NULL");
  if (p->L < 1 || p->Hq < 1 || p->Hkv < 1) return fail(IKV_ESHAPE, "pool: L, Hq, Hkv must be >= 1");
  if (p->Hq % p->Hkv) return fail(IKV_ESHAPE, "pool: Hq (%d) is not a multiple of Hkv (%d)", p->Hq, p->Hkv);
  if (p->Hq / p->Hkv > 8) return fail(IKV_EUNSUPPORTED, "pool: Hq/Hkv = %d > 8", p->Hq / p->Hkv);
  if (p->D != 64 && p->D != 128) return fail(IKV_EUNSUPPORTED, "pool: D = %d (supported: 64, 128)", p->D);
  if (p->num_slots < 1 || p->num_slots > INT32_MAX) return fail(IKV_ESHAPE, "pool: num_slots out of range");
  if (p->dead_slot < 0 || p->dead_slot >= p->num_slots) return fail(IKV_ESHAPE, "pool: dead_slot out of range");
  if (p->kv_dtype != IKV_BF16 && p->kv_dtype != IKV_F32) return fail(IKV_EINVAL, "pool: unknown kv_dtype");
  if (!p->k_pool || !p->v_pool) return fail(IKV_EINVAL, "pool: k_pool / v_pool is NULL");
  return IKV_OK;
}

ikv_status check_sessions(const ikv_session *s, const ikv_session *sd, int32_t B) {
  if (B < 0) return fail(IKV_EINVAL, "B < 0");
  if (B > 0 && (!s || !sd)) return fail(IKV_EINVAL, "sess / sess_dev is NULL");
  for (int b = 0; b < B; ++b) {
    const ikv_session &x = s[b];
    if (x.N < 0) return fail(IKV_ESHAPE, "session %d: N < 0", b);
    if (x.pi < 0 || x.pi > x.N) return fail(IKV_ESHAPE, "session %d: pi outside [0, N]", b);
    if (x.qs < 0 || x.qs > x.qe || x.qe > x.N) return fail(IKV_ESHAPE, "session %d: need 0 <= qs <= qe <= N", b);
    if (x.C < 0) return fail(IKV_ESHAPE, "session %d: C < 0", b);
    if (x.radix_prefix < 0) return fail(IKV_ESHAPE, "session %d: radix_prefix < 0", b);
    if (x.R < 1 || x.R > ikv::MAX_R) return fail(IKV_ESHAPE, "session %d: R = %d outside [1, %d]", b, x.R, ikv::MAX_R);
    if (x.nq < 0 || x.nq > ikv::MAX_NQ) return fail(IKV_ESHAPE, "session %d: nq outside [0, %d]", b, ikv::MAX_NQ);
    if (x.slot_off < 0 || x.mem_off < 0 || x.qspan_off < 0 || x.qpos_off < 0)
      return fail(IKV_ESHAPE, "session %d: negative offset", b);
  }
  return IKV_OK;
}

ikv_status check_ws(void *ws, size_t have, size_t need) {
  if (need == 0) return IKV_OK;
  if (!ws) return fail(IKV_EWORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (have < need) return fail(IKV_EWORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  if (reinterpret_cast<uintptr_t>(ws) & 255) return fail(IKV_EWORKSPACE, "workspace is not 256-byte aligned");
  return IKV_OK;
}

int max_n(const ikv_session *s, int B) {
  int m = 0;
  for (int b = 0; b < B; ++b) m = s[b].N > m ? s[b].N : m;
  return m;
}

// The MFMA score passes need D = 128 and a bf16 pool; any R (each session's memory
// rows run in 16-row slices, the last one padded).
bool use_mfma(const ikv_pool *p, const ikv_session *, int) {
  return p->D == 128 && p->kv_dtype == IKV_BF16;
}

int64_t total_positions(const ikv_session *sess, int B) {
  int64_t total = 0;
  for (int b = 0; b < B; ++b) total = std::max<int64_t>(total, sess[b].slot_off + sess[b].N);
  return total;
}

size_t score_bytes(const ikv_pool *p, const ikv_session *s, int B, uint32_t flags) {
  const bool resid = (flags & IKV_RESIDUAL) != 0;
  const int units = p->L * p->Hkv;
  int64_t f = ikv::score_offset(s, B, p->L, units, p->D, resid, use_mfma(p, s, B));
  if (resid) f += ikv::score_shared_floats(p->D);
  if (flags & IKV_POOL7) f += int64_t(units) * total_positions(s, B);    // per-unit attention masses
  f = ikv::align64f(f) + ikv::fused_exchange_floats(*p, s, B, flags);   // the one-key-pass form's exchange
  return size_t(f) * sizeof(float);
}

size_t select_bytes(const ikv_session *sess, int B) {
  return B > 0 ? ikv::select_workspace_bytes(sess, B, total_positions(sess, B)) : 0;
}

size_t redirect_bytes(int64_t num_slots, int B) {
  return size_t(B) * 2 * size_t(ikv::bitset_words(num_slots)) * sizeof(uint32_t);
}

// An upper bound on the live positions a session holds after a retention event:
// the forced set (at most pi + qe - qs positions) plus the budget, and never more
// than N. A slot map that was never pruned may hold more; the decode is then still
// exact, only with longer splits.
int live_bound(const ikv_session *s, int B) {
  int64_t m = 1;
  for (int b = 0; b < B; ++b) {
    const int64_t forced = int64_t(std::max(0, s[b].pi)) + std::max(0, s[b].qe - s[b].qs);
    m = std::max<int64_t>(m, std::min<int64_t>(s[b].N, std::max<int64_t>(s[b].C, forced)));
  }
  return int(m);
}

size_t decode_bytes(const ikv_pool *p, const ikv_session *s, int B) {
  const int splits = ikv::decode_splits(live_bound(s, B), ikv::decode_units(*p, B));
  return size_t(B) * p->L * p->Hq * splits * size_t(ikv::decode_part_floats(p->D)) * sizeof(float);
}

int prefill_splits(const ikv_pool *p, const ikv_session *s, int B) {
  int64_t keys = 1;
  for (int b = 0; b < B; ++b) keys = std::max<int64_t>(keys, int64_t(s[b].N) + std::max(0, s[b].qe - s[b].qs));
  return ikv::prefill_splits(p->L, p->Hkv, B, keys);
}

int64_t prefill_kq_floats(const ikv_pool *p, const ikv_session *s, int B) {
  int64_t n = 0;
  for (int b = 0; b < B; ++b) n += std::max(0, s[b].qe - s[b].qs);
  return ikv::align64f(n * p->L * p->D);
}

size_t prefill_bytes(const ikv_pool *p, const ikv_session *s, int B) {
  return size_t(prefill_kq_floats(p, s, B) +
                ikv::prefill_part_floats(p->L, p->Hkv, B, prefill_splits(p, s, B), p->D)) * sizeof(float);
}

ikv_status pending_fault() {
  if (ikv::take_host_fault())
    return fail(IKV_EHIP, "a wait between workgroups of an earlier call (ikv_select_budget's grid barrier or "
                          "ikv_score_history's normaliser exchange) gave up; that call's results are not valid");
  return IKV_OK;
}

// ---- IKV_DEBUG=1 in the environment (read on every call): before anything is
// enqueued, the slot ids a call reads are copied to the host, after the stream's
// earlier work, and checked. The kernels never check them; an id outside the pool
// would read or write outside it. Synchronises the stream; for debugging only.
bool debug_mode() {
  const char *e = getenv("IKV_DEBUG");
  return e != nullptr && e[0] != '\0' && e[0] != '0';
}

template <typename T>
ikv_status debug_fetch(std::vector<T> &h, const T *dev, int64_t n, hipStream_t st, const char *what, int b) {
  h.resize(size_t(n > 0 ? n : 0));
  if (n <= 0) return IKV_OK;
  hipError_t e = hipMemcpyAsync(h.data(), dev, size_t(n) * sizeof(T), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(IKV_EHIP, "IKV_DEBUG: reading %s of session %d: %s", what, b, hipGetErrorString(e));
  return IKV_OK;
}

// Entries [off, off + n) of the device array `ids` must lie in [lo, hi).
ikv_status debug_ids(const int32_t *ids, int64_t off, int64_t n, int64_t lo, int64_t hi, hipStream_t st,
                     const char *what, int b) {
  std::vector<int32_t> h;
  if (ikv_status r = debug_fetch(h, ids + off, n, st, what, b)) return r;
  for (int64_t i = 0; i < n; ++i)
    if (h[size_t(i)] < lo || h[size_t(i)] >= hi)
      return fail(IKV_EINVAL, "IKV_DEBUG: session %d: %s[%lld] = %d outside [%lld, %lld)", b, what, (long long)i,
                  h[size_t(i)], (long long)lo, (long long)hi);
  return IKV_OK;
}

// The count a device array holds for session b, clamped to [0, cap].
ikv_status debug_count(const int32_t *counts, int b, int64_t cap, hipStream_t st, const char *what, int64_t *n) {
  std::vector<int32_t> h;
  if (ikv_status r = debug_fetch(h, counts + b, 1, st, what, b)) return r;
  *n = std::min<int64_t>(std::max<int64_t>(h[0], 0), cap);
  return IKV_OK;
}

ikv_status debug_slot_maps(const ikv_session *sess, int B, const int32_t *slot_maps, int64_t num_slots,
                           hipStream_t st) {
  for (int b = 0; b < B; ++b)
    if (ikv_status r = debug_ids(slot_maps, sess[b].slot_off, sess[b].N, 0, num_slots, st, "slot map", b)) return r;
  return IKV_OK;
}

}  // namespace

namespace ikv {

ikv_status set_error(ikv_status code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

namespace {
std::mutex g_fault_mu;
std::atomic<uint32_t *> g_fault_host{nullptr};   // pinned, mapped; never freed
uint32_t *g_fault_dev = nullptr;                 // the same word as kernels address it
}  // namespace

uint32_t *host_fault_word() {
  std::lock_guard<std::mutex> lk(g_fault_mu);
  if (!g_fault_host) {
    void *h = nullptr, *d = nullptr;
    if (hipHostMalloc(&h, 64, hipHostMallocMapped | hipHostMallocPortable | hipHostMallocCoherent) != hipSuccess)
      return nullptr;
    *static_cast<volatile uint32_t *>(h) = 0u;
    if (hipHostGetDevicePointer(&d, h, 0) != hipSuccess) d = h;
    g_fault_dev = static_cast<uint32_t *>(d);
    g_fault_host.store(static_cast<uint32_t *>(h), std::memory_order_release);
  }
  return g_fault_dev;
}

uint32_t *host_fault_word_if_any() {
  std::lock_guard<std::mutex> lk(g_fault_mu);
  return g_fault_host.load(std::memory_order_acquire) ? g_fault_dev : nullptr;
}

bool take_host_fault() {
  uint32_t *h = g_fault_host.load(std::memory_order_acquire);
  return h != nullptr && __atomic_exchange_n(h, 0u, __ATOMIC_ACQ_REL) != 0u;
}

}  // namespace ikv

extern "C" {

const char *ikv_last_error(void) { return g_err.c_str(); }

namespace ikv {


KTimer::KTimer(const char *name, hipStream_t stream) : idx(-1), st(stream) {
  if (!g_timing) return;
  std::lock_guard<std::mutex> lk(g_tmu);
  if (!g_timing || g_recs.size() >= kMaxTimingRecs) return;
  TimingRec r{name, take_event(), take_event()};
  if (!r.a || !r.b || hipEventRecord(r.a, st) != hipSuccess) {
    if (r.a) g_events.push_back(r.a);
    if (r.b) g_events.push_back(r.b);
    return;
  }
  g_recs.push_back(r);
  idx = int(g_recs.size()) - 1;
}

KTimer::~KTimer() {
  if (idx < 0) return;
  std::lock_guard<std::mutex> lk(g_tmu);
  if (size_t(idx) < g_recs.size()) (void)hipEventRecord(g_recs[size_t(idx)].b, st);
}

}  // namespace ikv

ikv_status ikv_timing(int32_t enable) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = enable != 0;
  return ok();
}

int32_t ikv_timing_read(const char **names, float *ms, int32_t cap) {
  std::lock_guard<std::mutex> lk(g_tmu);
  if (cap > 0 && (!names || !ms)) return fail(IKV_EINVAL, "names / ms is NULL with cap > 0");
  const int32_t n = int32_t(g_recs.size());
  hipError_t err = hipSuccess;
  for (int32_t i = 0; i < n; ++i) {
    TimingRec &r = g_recs[size_t(i)];
    float t = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess && err == hipSuccess) err = e;
    if (i < cap) {
      names[i] = r.name;
      ms[i] = t;
    }
    g_events.push_back(r.a);
    g_events.push_back(r.b);
  }
  g_recs.clear();
  if (err != hipSuccess) return hip_status(err, "ikv_timing_read");
  ok();
  return n;
}

ikv_status ikv_workspace_bytes(const ikv_pool *pool, const ikv_session *sess, int32_t B, int32_t call,
                               uint32_t flags, size_t *bytes) {
  if (!bytes) return fail(IKV_EINVAL, "bytes is NULL");
  *bytes = 0;
  if (B < 0) return fail(IKV_EINVAL, "B < 0");
  if (B > 0 && !sess) return fail(IKV_EINVAL, "sess is NULL");
  ikv_status r;
  switch (call) {
    case IKV_CALL_SCORE:
      if ((r = check_pool(pool))) return r;
      if ((r = check_sessions(sess, sess, B))) return r;
      *bytes = score_bytes(pool, sess, B, flags);
      return ok();
    case IKV_CALL_SELECT:
      if ((r = check_sessions(sess, sess, B))) return r;
      *bytes = select_bytes(sess, B);
      return ok();
    case IKV_CALL_REDIRECT:
      if (!pool) return fail(IKV_EINVAL, "pool is NULL");
      if (pool->num_slots < 1) return fail(IKV_ESHAPE, "num_slots < 1");
      *bytes = redirect_bytes(pool->num_slots, B);
      return ok();
    case IKV_CALL_DECODE:
      if ((r = check_pool(pool))) return r;
      if ((r = check_sessions(sess, sess, B))) return r;
      *bytes = decode_bytes(pool, sess, B);
      return ok();
    case IKV_CALL_PREFILL:
      if ((r = check_pool(pool))) return r;
      if ((r = check_sessions(sess, sess, B))) return r;
      *bytes = prefill_bytes(pool, sess, B);
      return ok();
    case IKV_CALL_COMPACT:
      if ((r = check_sessions(sess, sess, B))) return r;
      *bytes = size_t(total_positions(sess, B)) * sizeof(int32_t);
      return ok();
    default:
      return fail(IKV_EINVAL, "unknown call id %d", call);
  }
}

ikv_status ikv_init_dead_slot(const ikv_pool *pool, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_pool(pool);
  if (r) return r;
  return hip_status(ikv::launch_init_dead_slot(*pool, (hipStream_t)stream), "ikv_init_dead_slot");
}

ikv_status ikv_qm_update(const ikv_pool *pool, const ikv_session *sess, const ikv_session *sess_dev, int32_t B,
                         float *M, const void *q_span, float lambda, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_pool(pool);
  if (r) return r;
  if ((r = check_sessions(sess, sess_dev, B))) return r;
  if (B == 0) return ok();
  if (!M || !q_span) return fail(IKV_EINVAL, "M / q_span is NULL");
  if (!(lambda >= 0.0f)) return fail(IKV_EINVAL, "lambda must be >= 0 (got %g)", double(lambda));
  int max_rows = 0;
  const size_t esize = pool->kv_dtype == IKV_BF16 ? 2 : 4;
  for (int b = 0; b < B; ++b) {
    const int rows = pool->L * pool->Hkv * sess[b].R;
    max_rows = rows > max_rows ? rows : max_rows;
    if ((reinterpret_cast<uintptr_t>(M) + size_t(sess[b].mem_off) * 4) % 16 ||
        (reinterpret_cast<uintptr_t>(q_span) + size_t(sess[b].qspan_off) * esize) % 16)
      return fail(IKV_EINVAL, "session %d: M + mem_off and q_span + qspan_off must be 16-byte aligned", b);
  }
  const float decay = isinf(lambda) ? 0.0f : float(exp(-double(lambda)));
  return hip_status(ikv::launch_qm_update(*pool, sess_dev, B, max_rows, M, q_span, decay, (hipStream_t)stream),
                    "ikv_qm_update");
}

ikv_status ikv_score_history(const ikv_pool *pool, const ikv_session *sess, const ikv_session *sess_dev, int32_t B,
                             const int32_t *slot_maps, const float *M, const int32_t *qpos, const float *residual,
                             uint32_t flags, float *scores, void *workspace, size_t workspace_bytes,
                             void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_pool(pool);
  if (r) return r;
  if ((r = check_sessions(sess, sess_dev, B))) return r;
  if (flags & ~(IKV_RESIDUAL | IKV_NO_XATTN | IKV_POOL7 | IKV_TWO_PASS))
    return fail(IKV_EINVAL, "unknown flag bits 0x%x", flags);
  if ((flags & IKV_POOL7) && (flags & IKV_RESIDUAL)) return fail(IKV_EINVAL, "IKV_POOL7 excludes IKV_RESIDUAL");
  if (B == 0) return ok();
  if (!slot_maps || !M || !scores) return fail(IKV_EINVAL, "slot_maps / M / scores is NULL");
  const bool resid = (flags & IKV_RESIDUAL) != 0;
  if (resid && !residual) return fail(IKV_EINVAL, "IKV_RESIDUAL set but residual is NULL");
  int maxR = 0, minR = INT32_MAX, maxNq = 0, anyq = 0;
  for (int b = 0; b < B; ++b) {
    minR = sess[b].R < minR ? sess[b].R : minR;
    if ((reinterpret_cast<uintptr_t>(M) + size_t(sess[b].mem_off) * 4) % 16)
      return fail(IKV_EINVAL, "session %d: M + mem_off must be 16-byte aligned", b);
    maxR = sess[b].R > maxR ? sess[b].R : maxR;
    maxNq = sess[b].nq > maxNq ? sess[b].nq : maxNq;
    anyq |= sess[b].nq > 0;
  }
  if (resid && anyq && !qpos) return fail(IKV_EINVAL, "qpos is NULL but a session has nq > 0");
  const size_t need = score_bytes(pool, sess, B, flags);
  if ((r = check_ws(workspace, workspace_bytes, need))) return r;
  ikv::ScoreArgs a;
  a.pool = *pool;
  a.sess_host = sess;
  a.sess_dev = sess_dev;
  a.B = B;
  a.slot_maps = slot_maps;
  a.M = M;
  a.qpos = qpos;
  a.residual = residual;
  a.flags = flags;
  a.scores = scores;
  a.ws = static_cast<float *>(workspace);
  a.mfma = use_mfma(pool, sess, B);
  a.mfma_resid = a.mfma && resid && maxNq <= 64;
  a.stats = a.mfma && maxR <= 128 && pool->Hkv % 2 == 0 &&
            int64_t(pool->num_slots) * pool->Hkv * pool->D * 2 <= int64_t(UINT32_MAX);
  // the one-key-pass form: every session at most 16 memory rows (one slice), not the
  // SnapKV-style score (which needs the unit-major pass), not turned off by the caller
  a.stash = a.mfma && maxR <= ikv::STASH_MAX_R && !(flags & (IKV_POOL7 | IKV_TWO_PASS));
  if (a.stash) a.stats = false;
  a.fused_tiles = a.mfma && !a.stash ? ikv::fused_tiles(*pool, sess, B, flags) : 0;
  if (a.fused_tiles > 0) a.stats = false;
  {
    int64_t xo = ikv::score_offset(sess, B, pool->L, pool->L * pool->Hkv, pool->D, resid, a.mfma);
    if (resid) xo += ikv::score_shared_floats(pool->D);
    if (flags & IKV_POOL7) xo += int64_t(pool->L) * pool->Hkv * total_positions(sess, B);
    a.xch = reinterpret_cast<uint64_t *>(a.ws + ikv::align64f(xo));
  }
  a.ws_shared = a.ws + ikv::score_offset(sess, B, pool->L, pool->L * pool->Hkv, pool->D, resid, a.mfma);
  a.maxN = max_n(sess, B);
  a.total_positions = total_positions(sess, B);
  if ((flags & IKV_POOL7) && !a.stats)
    return fail(IKV_EUNSUPPORTED, "IKV_POOL7 needs D = 128, a bf16 pool, an even Hkv and R <= 128");
  a.maxR = maxR;
  a.minR = minR;
  a.maxNq = maxNq;
  if (a.maxN == 0) return ok();
  if (debug_mode()) {
    if ((r = debug_slot_maps(sess, B, slot_maps, pool->num_slots, (hipStream_t)stream))) return r;
    if (resid)
      for (int b = 0; b < B; ++b)
        if ((r = debug_ids(qpos, sess[b].qpos_off, sess[b].nq, 0, sess[b].N, (hipStream_t)stream, "qpos", b))) return r;
  }
  return hip_status(ikv::launch_score(a, (hipStream_t)stream), "ikv_score_history");
}

ikv_status ikv_select_budget(const ikv_session *sess, const ikv_session *sess_dev, int32_t B,
                             const int32_t *slot_maps, int32_t dead_slot, const float *scores, uint8_t *keep,
                             int32_t *n_keep, float *tau, void *workspace, size_t workspace_bytes, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_sessions(sess, sess_dev, B);
  if (r) return r;
  if (B == 0) return ok();
  if (!slot_maps || !scores || !keep || !n_keep || !tau)
    return fail(IKV_EINVAL, "slot_maps / scores / keep / n_keep / tau is NULL");
  if (dead_slot < 0) return fail(IKV_ESHAPE, "dead_slot < 0");
  if ((r = check_ws(workspace, workspace_bytes, select_bytes(sess, B)))) return r;
  return hip_status(ikv::launch_select(sess, sess_dev, B, max_n(sess, B), slot_maps, dead_slot, scores, keep, n_keep,
                                       tau, static_cast<uint32_t *>(workspace), total_positions(sess, B),
                                       (hipStream_t)stream, true),
                    "ikv_select_budget");
}

ikv_status ikv_select_budget_static(const ikv_session *sess, const ikv_session *sess_dev, int32_t B,
                                    const int32_t *slot_maps, int32_t dead_slot, const float *scores,
                                    uint8_t *keep, int32_t *n_keep, float *tau, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_sessions(sess, sess_dev, B);
  if (r) return r;
  if (B == 0) return ok();
  if (!slot_maps || !scores || !keep || !n_keep || !tau)
    return fail(IKV_EINVAL, "slot_maps / scores / keep / n_keep / tau is NULL");
  if (dead_slot < 0) return fail(IKV_ESHAPE, "dead_slot < 0");
  const size_t need = select_bytes(sess, B);
  if (need > size_t(IKV_SELECT_STATIC_MAX_BYTES))
    return fail(IKV_EWORKSPACE, "these sessions need %zu bytes of selection scratch; the static scratch holds %zu",
                need, size_t(IKV_SELECT_STATIC_MAX_BYTES));
  uint32_t *scr = nullptr;
  if ((r = hip_status(ikv::select_static_scratch(&scr), "ikv_select_budget_static: scratch address"))) return r;
  return hip_status(ikv::launch_select(sess, sess_dev, B, max_n(sess, B), slot_maps, dead_slot, scores, keep, n_keep,
                                       tau, scr, total_positions(sess, B), (hipStream_t)stream, false),
                    "ikv_select_budget_static");
}

ikv_status ikv_redirect_slots(const ikv_session *sess, const ikv_session *sess_dev, int32_t B, int64_t num_slots,
                              int32_t *slot_maps, int32_t dead_slot, const uint8_t *keep, int32_t *freed,
                              int32_t *n_freed, int32_t *live, int32_t *n_live, void *workspace,
                              size_t workspace_bytes, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_sessions(sess, sess_dev, B);
  if (r) return r;
  if (B == 0) return ok();
  if (num_slots < 1 || num_slots > INT32_MAX) return fail(IKV_ESHAPE, "num_slots out of range");
  if (dead_slot < 0 || dead_slot >= num_slots) return fail(IKV_ESHAPE, "dead_slot out of range");
  if (!slot_maps || !keep || !freed || !n_freed || !live || !n_live)
    return fail(IKV_EINVAL, "slot_maps / keep / freed / n_freed / live / n_live is NULL");
  if ((r = check_ws(workspace, workspace_bytes, redirect_bytes(num_slots, B)))) return r;
  if (debug_mode() && (r = debug_slot_maps(sess, B, slot_maps, num_slots, (hipStream_t)stream))) return r;
  return hip_status(ikv::launch_redirect(sess_dev, B, num_slots, slot_maps, dead_slot, keep, freed, n_freed, live,
                                         n_live, static_cast<uint32_t *>(workspace), (hipStream_t)stream),
                    "ikv_redirect_slots");
}

ikv_status ikv_compact_apply(const ikv_pool *pool, const ikv_session *sess, const ikv_session *sess_dev, int32_t B,
                             const int32_t *slot_maps, const uint8_t *keep, const int32_t *dst_slots, double rope_base,
                             int32_t *n_keep, void *workspace, size_t workspace_bytes, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_pool(pool);
  if (r) return r;
  if ((r = check_sessions(sess, sess_dev, B))) return r;
  if (B == 0) return ok();
  if (!slot_maps || !keep || !dst_slots || !n_keep) return fail(IKV_EINVAL, "slot_maps / keep / dst_slots / n_keep is NULL");
  if (!(rope_base > 1.0)) return fail(IKV_EINVAL, "rope_base must be > 1");
  const size_t need = size_t(total_positions(sess, B)) * sizeof(int32_t);
  if ((r = check_ws(workspace, workspace_bytes, need))) return r;
  if (debug_mode()) {
    const hipStream_t st = (hipStream_t)stream;
    if ((r = debug_slot_maps(sess, B, slot_maps, pool->num_slots, st))) return r;
    for (int b = 0; b < B; ++b) {           // one destination slot per kept live position
      std::vector<int32_t> S;
      std::vector<uint8_t> kp;
      if ((r = debug_fetch(S, slot_maps + sess[b].slot_off, sess[b].N, st, "slot map", b))) return r;
      if ((r = debug_fetch(kp, keep + sess[b].slot_off, sess[b].N, st, "keep", b))) return r;
      int64_t nk = 0;
      for (int j = 0; j < sess[b].N; ++j) nk += kp[size_t(j)] && S[size_t(j)] != pool->dead_slot;
      if ((r = debug_ids(dst_slots, sess[b].slot_off, nk, 0, pool->num_slots, st, "dst_slots", b))) return r;
    }
  }
  return hip_status(ikv::launch_compact(*pool, sess_dev, B, max_n(sess, B), slot_maps, keep, dst_slots, rope_base,
                                        n_keep, static_cast<int32_t *>(workspace), (hipStream_t)stream),
                    "ikv_compact_apply");
}

ikv_status ikv_prefill_span(const ikv_pool *pool, const ikv_session *sess, const ikv_session *sess_dev, int32_t B,
                            const int32_t *slot_maps, const void *q_raw, const void *k_raw, const void *v_raw,
                            const int32_t *hist, const int32_t *n_hist, double rope_base, float lambda, float *M,
                            void *q_out, void *out, float *kq, void *workspace, size_t workspace_bytes, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_pool(pool);
  if (r) return r;
  if ((r = check_sessions(sess, sess_dev, B))) return r;
  if (B == 0) return ok();
  if (!slot_maps || !q_raw || !k_raw || !v_raw || !hist || !n_hist || !q_out || !out || !kq)
    return fail(IKV_EINVAL, "an input or output pointer is NULL");
  if (pool->D != 128 || pool->kv_dtype != IKV_BF16)
    return fail(IKV_EUNSUPPORTED, "ikv_prefill_span needs D = 128 and a bf16 pool");
  if (pool->Hq * pool->D > 8192 || pool->Hkv * pool->D > 2048)
    return fail(IKV_EUNSUPPORTED, "ikv_prefill_span: Hq * D must be <= 8192 and Hkv * D <= 2048");
  if (!(rope_base > 1.0)) return fail(IKV_EINVAL, "rope_base must be > 1");
  if (M && !(lambda >= 0.0f)) return fail(IKV_EINVAL, "lambda must be >= 0 (got %g)", double(lambda));
  const int G = pool->Hq / pool->Hkv;
  int max_n = 0;
  for (int b = 0; b < B; ++b) {
    const int n = sess[b].qe - sess[b].qs;
    if (n * G > 256) return fail(IKV_EUNSUPPORTED, "session %d: span of %d tokens x %d heads per KV head > 256", b, n, G);
    if (M && sess[b].R != G) return fail(IKV_ESHAPE, "session %d: the memory update needs R = Hq / Hkv = %d", b, G);
    max_n = std::max(max_n, n);
  }
  if ((r = check_ws(workspace, workspace_bytes, prefill_bytes(pool, sess, B)))) return r;
  if (max_n == 0) return ok();
  if (debug_mode()) {
    const hipStream_t st = (hipStream_t)stream;
    if ((r = debug_slot_maps(sess, B, slot_maps, pool->num_slots, st))) return r;
    for (int b = 0; b < B; ++b) {
      int64_t nh = 0;
      if ((r = debug_count(n_hist, b, sess[b].N, st, "n_hist", &nh))) return r;
      if ((r = debug_ids(hist, sess[b].slot_off, nh, 0, pool->num_slots, st, "hist", b))) return r;
    }
  }
  const float decay = isinf(lambda) ? 0.0f : float(exp(-double(lambda)));
  return hip_status(ikv::launch_prefill(*pool, sess_dev, B, max_n, prefill_splits(pool, sess, B), slot_maps, q_raw,
                                        k_raw, v_raw, hist, n_hist, rope_base, decay, M, q_out, out, kq,
                                        static_cast<float *>(workspace), prefill_kq_floats(pool, sess, B),
                                        (hipStream_t)stream),
                    "ikv_prefill_span");
}

ikv_status ikv_decode_attend_slotmap(const ikv_pool *pool, const ikv_session *sess, const ikv_session *sess_dev,
                                     int32_t B, const void *q, const int32_t *live, const int32_t *n_live, void *out,
                                     void *workspace, size_t workspace_bytes, void *stream) {
  if (ikv_status f = pending_fault()) return f;
  ikv_status r = check_pool(pool);
  if (r) return r;
  if ((r = check_sessions(sess, sess_dev, B))) return r;
  if (B == 0) return ok();
  if (!q || !live || !n_live || !out) return fail(IKV_EINVAL, "q / live / n_live / out is NULL");
  if ((r = check_ws(workspace, workspace_bytes, decode_bytes(pool, sess, B)))) return r;
  const int splits = ikv::decode_splits(live_bound(sess, B), ikv::decode_units(*pool, B));
  if (debug_mode())
    for (int b = 0; b < B; ++b) {
      int64_t nl = 0;
      if ((r = debug_count(n_live, b, sess[b].N, (hipStream_t)stream, "n_live", &nl))) return r;
      if ((r = debug_ids(live, sess[b].slot_off, nl, 0, pool->num_slots, (hipStream_t)stream, "live", b))) return r;
    }
  return hip_status(ikv::launch_decode(*pool, sess_dev, B, splits, q, live, n_live, out,
                                       static_cast<float *>(workspace), (hipStream_t)stream),
                    "ikv_decode_attend_slotmap");
}

}  // extern "C"
