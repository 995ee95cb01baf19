/*
 * ikv.h -- C ABI of the IntentKV per-step retention path on MI355X (gfx950).
 *
 * One retention step of a request (Sec. 3 of the paper; Appendix H, compression
 * event) is five calls, in order:
 *
 *   ikv_qm_update            QueryMemory recurrence, Eq. 2
 *   ikv_score_history        rule score, Eq. 3, plus the residual head, Eqs. 4-6
 *   ikv_select_budget        budgeted top-k of Eq. 1
 *   ikv_redirect_slots       slot-map eviction, Eq. 7, with the alias-aware free of Sec. 3.4
 *   ikv_decode_attend_slotmap  GQA decode attention over the live slots only
 *
 * plus ikv_init_dead_slot, run once per pool (the sentinel of Sec. 3.4).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every pointer named *_dev, every pool, map, score, mask and list is DEVICE
 *    memory; ikv_pool / ikv_session structs passed as `pool` / `sess` are HOST
 *    memory. Sessions are passed twice: `sess` (host copy, validated and used
 *    for launch geometry) and `sess_dev` (a byte-identical device copy read by
 *    the kernels). The caller owns every buffer; the library keeps no pointer
 *    to them after a call returns and allocates no device memory (the one
 *    allocation it makes is a word of pinned host memory, see ikv_select_budget).
 *  - `stream` is a hipStream_t (NULL = the default stream). Validation runs
 *    synchronously on the host; all device work is enqueued on `stream` and the
 *    call returns without synchronising.
 *  - Calls are batched over B >= 1 sessions that share one pool. Per-position
 *    arrays (slot maps, scores, keep masks, live and freed lists) of all sessions
 *    are concatenated; session b's part starts at sess[b].slot_off.
 *  - Calls that need scratch take a caller-provided `workspace` of at least
 *    ikv_workspace_bytes(...) bytes (256-byte aligned). Its contents on entry do
 *    not matter.
 *  - Results are deterministic: no result-bearing reduction uses floating-point
 *    atomics, so two runs on the same inputs give identical bytes.
 *  - Return value: IKV_OK, or a negative ikv_status; ikv_last_error() then gives
 *    a message (thread-local, valid until the next call on the same thread).
 *    On an error return nothing has been enqueued, except for IKV_EHIP, which
 *    reports a failed launch, or a fault that a kernel of an earlier call reported
 *    (see ikv_select_budget); a call that returns such a fault enqueues nothing.
 *  - Slot ids in slot maps, live lists, history and destination slot lists must
 *    lie in [0, num_slots), and cross-attention query positions in [0, N); the
 *    kernels do not check them (an id outside the pool reads or writes outside
 *    it). With IKV_DEBUG=1 in the environment (read on every call), the calls
 *    that read such ids (score_history, redirect_slots, decode_attend_slotmap,
 *    compact_apply, prefill_span) first copy them to the host, after the
 *    stream's earlier work, and return IKV_EINVAL naming the session, the array
 *    and the index of the first bad entry, with no kernel launched. This
 *    synchronises the stream on every call; it is meant for debugging.
 */
#ifndef IKV_H
#define IKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ikv_status;
#define IKV_OK            0
#define IKV_EINVAL       -1   /* null pointer, bad flag, negative size               */
#define IKV_ESHAPE       -2   /* inconsistent dimensions or ranges                   */
#define IKV_EWORKSPACE   -3   /* workspace missing, too small or misaligned          */
#define IKV_EUNSUPPORTED -4   /* valid but not implemented (e.g. D not in {64,128})  */
#define IKV_EHIP         -5   /* a HIP runtime call or kernel launch failed          */

/* K/V storage types of the pool. */
#define IKV_BF16 0
#define IKV_F32  1

/* ikv_score_history flags. */
#define IKV_RESIDUAL  1u   /* add alpha * MLP(phi ++ c), Eq. 4 (needs `residual`)           */
#define IKV_NO_XATTN  2u   /* the "- x-attn" ablation: c_j = 0 in Eq. 4 (Sec. 3.3)          */
#define IKV_POOL7     4u   /* SnapKV-style score (Sec. 4.1 baselines): see ikv_score_history  */
#define IKV_TWO_PASS  8u   /* score with two passes over the keys even where every R <= 16   */

/* ikv_workspace_bytes call ids. */
#define IKV_CALL_SCORE    1
#define IKV_CALL_SELECT   2
#define IKV_CALL_REDIRECT 3
#define IKV_CALL_DECODE   4
#define IKV_CALL_COMPACT  5
#define IKV_CALL_PREFILL  6

/*
 * The paged KV pool (Sec. 3.1: post-RoPE K, V in R^{L x Hkv x N x D}, stored by
 * physical slot as in a paged serving stack).
 *   k_pool, v_pool: device, [L][num_slots][Hkv][D] of kv_dtype, row-major.
 *   dead_slot: the sentinel slot s_dead (Sec. 3.4); never freed.
 *   Hq must be a multiple of Hkv (query head h reads KV head h / (Hq/Hkv)).
 *   Supported: D in {64, 128}; Hq / Hkv <= 8.
 */
typedef struct ikv_pool {
  int32_t L, Hq, Hkv, D;
  int64_t num_slots;
  int32_t dead_slot;
  int32_t kv_dtype;
  void *k_pool;
  void *v_pool;
} ikv_pool;

/*
 * One request r (Sec. 3.1 problem formulation; Appendix H).
 *   slot_off   first entry of this session in every per-position array
 *   mem_off    QueryMemory M_t at M + mem_off: [L][Hkv*R][D] float32. Row
 *              h*R + r of layer l pairs with KV head h (R rows per KV head; the
 *              paper's one row per query head is R = Hq/Hkv).
 *   qspan_off  query-span rows at q_span + qspan_off: [L][Hkv*R][qe-qs][D] in
 *              the pool's kv_dtype (ikv_qm_update only)
 *   qpos_off   cross-attention query positions at qpos + qpos_off: nq int32
 *              positions in [0, N) (Eq. 6; dead ones are skipped)
 *   N          positions of the request, dead ones included
 *   pi         protected prefix [0, pi); qs, qe the actionable span [qs, qe);
 *              F = ([0,pi) u [qs,qe)) restricted to live positions (Eq. 1)
 *   C          retention budget, F included: C* = max(0, C - |F|)
 *   radix_prefix  positions below it are never freed (Sec. 3.4, condition (a))
 *   R          memory rows per KV head, 1 <= R <= 256
 *   nq         number of cross-attention query positions, 0 <= nq <= 256
 */
typedef struct ikv_session {
  int64_t slot_off;
  int64_t mem_off;
  int64_t qspan_off;
  int64_t qpos_off;
  int32_t N;
  int32_t pi, qs, qe;
  int32_t C;
  int32_t radix_prefix;
  int32_t R;
  int32_t nq;
} ikv_session;

/*
 * Sentinel dead slot (Sec. 3.4, sentinel paragraph): K[l][dead_slot][h][:] = -1e4
 * (stored as bf16 -9984, the nearest bf16 value, or exactly in float32) and
 * V[l][dead_slot][h][:] = 0 on every layer and head. Run once per pool.
 */
ikv_status ikv_init_dead_slot(const ikv_pool *pool, void *stream);

/*
 * QueryMemory update, Eq. 2 with Sec. 3.2: for every session, layer and memory
 * row, Enc = mean of the qe-qs span rows; M <- exp(-lambda) * M + Enc; then the
 * row is divided by max(||row||_2, 1e-12). lambda = INFINITY drops the history
 * (the "query" scorer mode and the "- memory" ablation). In place on M.
 *   q_span: device, per session [L][Hkv*R][qe-qs][D] of the pool's kv_dtype.
 *   M + mem_off and q_span + qspan_off must be 16-byte aligned for every session
 *   (IKV_EINVAL otherwise): rows are read and written 16 bytes per lane.
 * Sessions with qe == qs leave M unchanged apart from the decay and projection.
 */
ikv_status ikv_qm_update(const ikv_pool *pool, const ikv_session *sess,
                         const ikv_session *sess_dev, int32_t B, float *M,
                         const void *q_span, float lambda, void *stream);

/*
 * Score every candidate position, Eq. 3 (and Eq. 4 with IKV_RESIDUAL).
 *   Candidates A = live positions (slot != dead_slot) outside F.
 *   rule_j = sum over layers l, KV heads h and the R memory rows r of head h of
 *            softmax_{i in A}(M[l][h*R+r] . K[l][S[i]][h] / sqrt(D)) at i = j.
 *   With IKV_RESIDUAL: s_j = rule_j + clip(alpha, -5, 5) * MLP(phi_j ++ c_j) with
 *     phi_j = [kbar_j, mbar, kbar_j * mbar, rule_j] (Eq. 5; kbar_j the mean of the
 *     key rows over layers and KV heads, mbar the mean of all memory rows),
 *     c_j the 4-head cross-attention of Eq. 6 over kbar at the live query
 *     positions (c_j = 0 with IKV_NO_XATTN or when none is live) and
 *     MLP = w_2 . GELU(W_1 x + b_1) + b_2 (exact erf GELU).
 *   residual: device float32 blob, row-major [out][in] blocks in this order:
 *     W_Q[128][3D+1] b_Q[128] W_K[128][D] b_K[128] W_V[128][D] b_V[128]
 *     W_1[256][3D+1+128] b_1[256] w_2[256] b_2[1] alpha[1]
 *     (214,274 floats at D = 128; 124,162 at D = 64). Ignored without IKV_RESIDUAL.
 *   scores: device float32, per session [N]: s_j on A, -INFINITY elsewhere.
 *   Sessions with N <= C are skipped (Appendix H): all their scores are -INFINITY.
 *   slot_maps, M, qpos: read only. M + mem_off must be 16-byte aligned for every
 *   session (IKV_EINVAL otherwise).
 */
/*
 * The same call scores for the baseline compressors of Sec. 4.1 on the same substrate
 * (Appendix: every scorer feeds the same selection, redirect and decode), with M
 * holding query rows instead of memory rows: a KV head's R rows are the n query rows
 * of each of its G query heads, so q[L][Hq][n][D] is M as it stands, with R = G * n.
 *   H2O-style (heavy hitters): flags 0, M the observed query rows: s_j is the
 *     attention j receives from them, summed over layers and query heads. The recent
 *     window of ratio mode is the forced span [qs, qe) the caller sets.
 *   SnapKV-style: flags IKV_POOL7, M the W = 32 window query rows: per (layer, KV
 *     head) the attention mass of the window's rows at each position (zero off A),
 *     max-pooled over the 7 positions j-3 .. j+3 (within [0, N)), then summed.
 *     IKV_POOL7 runs on the matrix-core path only (D = 128, bf16 pool, even Hkv,
 *     R <= 128; IKV_EUNSUPPORTED otherwise) and excludes IKV_RESIDUAL (IKV_EINVAL).
 *     Its workspace adds L * Hkv floats per position of the batch.
 * On the matrix-core path (D = 128, bf16 pool) with every session at R <= 16 the keys
 * are read once: the logits go to a float32 stash in the workspace (L * Hkv * R floats
 * per position, rounded up to 128 positions, for every session with R <= 16) and the
 * normalised sum is taken from it. IKV_TWO_PASS keeps the two passes over the keys
 * (the same scores up to float32 rounding order).
 */
ikv_status ikv_score_history(const ikv_pool *pool, const ikv_session *sess,
                             const ikv_session *sess_dev, int32_t B,
                             const int32_t *slot_maps, const float *M,
                             const int32_t *qpos, const float *residual,
                             uint32_t flags, float *scores, void *workspace,
                             size_t workspace_bytes, void *stream);

/*
 * Budgeted selection, Eq. 1 (Appendix H: K = F u topk(A, max(0, C - |F|))).
 *   Candidates are ranked by score descending, ties by lower position; NaN counts
 *   as -INFINITY and -0.0 as +0.0.
 *   keep: device uint8 per session [N]: 1 on F and on the min(C*, |A|) best
 *         candidates, 0 elsewhere (the persisted valid mask of Appendix H).
 *   n_keep: device int32 [B], |F| + min(C*, |A|).
 *   tau:    device float32 [B], score of the last candidate taken (+INFINITY if
 *           none is taken).
 *   Sessions with N <= C keep every live position (n_keep = live count,
 *   tau = -INFINITY).
 *   workspace: ikv_workspace_bytes(IKV_CALL_SELECT) bytes (per-session histograms
 *   and one 4-byte key per position, and per session the barrier flags, partial
 *   counts and histograms of the multi-workgroup path). Its contents on entry do not
 *   matter: nothing in it has to be cleared between calls. The call may be a
 *   cooperative launch (every workgroup resident at once); concurrent calls must not
 *   share a workspace. With the
 *   environment variable IKV_NO_COOP=1 the call never launches cooperatively (for
 *   tools that cannot follow such a launch); the result is the same.
 *   The workgroups of a cooperative launch meet at grid barriers whose waits are
 *   bounded (2^24 polls, or IKV_SELECT_SPINS from the environment, read on every
 *   call). Every workgroup is resident, so a wait ends well before the bound; if one
 *   ever gives up, the kernel still exits, the call's keep / n_keep / tau are not
 *   valid, and the library's next call returns IKV_EHIP (the fault travels through
 *   a word of pinned host memory that the first cooperative call allocates and the
 *   process keeps).
 */
ikv_status ikv_select_budget(const ikv_session *sess, const ikv_session *sess_dev,
                             int32_t B, const int32_t *slot_maps, int32_t dead_slot,
                             const float *scores, uint8_t *keep, int32_t *n_keep,
                             float *tau, void *workspace, size_t workspace_bytes,
                             void *stream);

/*
 * ikv_select_budget without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation). Same arguments, semantics and results as ikv_select_budget; the
 * scratch is a static device array of IKV_SELECT_STATIC_MAX_BYTES per GPU, resolved
 * on the first call on each device and held until the process ends. The call
 * allocates nothing: no hipMalloc, hipFree or allocating library routine (it reports
 * a timed-out grid barrier only if an earlier ikv_select_budget call has created the
 * host fault word).
 *   Sessions whose selection scratch (ikv_workspace_bytes with IKV_CALL_SELECT)
 *   exceeds IKV_SELECT_STATIC_MAX_BYTES are rejected with IKV_EWORKSPACE before
 *   anything is enqueued; that is about 6 bytes per position plus 44 KB per session.
 *   Every call on one GPU shares that GPU's scratch, whatever its stream: calls that
 *   overlap on one GPU race and give undefined results. Consecutive calls need
 *   nothing cleared in between.
 */
#define IKV_SELECT_STATIC_MAX_BYTES (32u << 20)
ikv_status ikv_select_budget_static(const ikv_session *sess, const ikv_session *sess_dev,
                                    int32_t B, const int32_t *slot_maps, int32_t dead_slot,
                                    const float *scores, uint8_t *keep, int32_t *n_keep,
                                    float *tau, void *stream);

/*
 * Slot-map eviction, Eq. 7, and the prefix-safe free of Sec. 3.4 / Appendix H.
 *   For every live position j with keep[j] == 0: slot_maps[j] <- dead_slot. Kept
 *   positions keep their slot; K/V rows are never touched.
 *   The old slot u of such a j is freed iff j >= radix_prefix, u != dead_slot and
 *   u is not the slot of any kept position of the same session.
 *   freed:  device int32 per session [N] (first n_freed used): the freed slots in
 *           ascending slot order, each once.
 *   live:   device int32 per session [N] (first n_live used): the slots of the
 *           positions still live afterwards, in position order.
 *   n_freed, n_live: device int32 [B].
 *   num_slots: the pool's slot count (sizes the slot sets in the workspace).
 */
ikv_status ikv_redirect_slots(const ikv_session *sess, const ikv_session *sess_dev,
                              int32_t B, int64_t num_slots, int32_t *slot_maps,
                              int32_t dead_slot, const uint8_t *keep, int32_t *freed,
                              int32_t *n_freed, int32_t *live, int32_t *n_live,
                              void *workspace, size_t workspace_bytes, void *stream);

/*
 * GQA decode attention over live slots (Sec. 3.4; Appendix C.2: the attention
 * backend strips the sentinel and reads only kept entries).
 *   For session b, layer l, query head h (KV head g = h / (Hq/Hkv)):
 *   out[b][l][h] = softmax_k(q[b][l][h] . K[l][u_k][g] / sqrt(D)) . V[l][u_k][g]
 *   over u_k = live[slot_off + k], k < n_live[b]. n_live[b] == 0 gives zeros.
 *   q, out: device [B][L][Hq][D] of the pool's kv_dtype (out rounded to nearest
 *   even). live, n_live: device, as written by ikv_redirect_slots;
 *   n_live[b] must not exceed sess[b].N.
 *   The live lists are split across workgroups by a bound known on the host,
 *   min(N, max(C, pi + qe - qs)) over the sessions (what a retention event leaves
 *   live), and by the number of (session, layer, KV head group) units, so that the
 *   workgroups fill about one resident round; a longer list is still attended
 *   exactly, with longer splits.
 */
ikv_status ikv_decode_attend_slotmap(const ikv_pool *pool, const ikv_session *sess,
                                     const ikv_session *sess_dev, int32_t B,
                                     const void *q, const int32_t *live,
                                     const int32_t *n_live, void *out, void *workspace,
                                     size_t workspace_bytes, void *stream);

/*
 * Session management on the host (no device work; every call below is synchronous,
 * thread-safe per store, and touches host memory only).
 *
 * Session key (Appendix A, session identification; Appendix H, session id
 * derivation), from the first source available, in this order:
 *   IKV_KEY_EXPLICIT  an explicit session id (session_id, session_id_len > 0 bytes);
 *   IKV_KEY_SPAN      the token tuple of a designated session span
 *                     tokens[span_start, span_end) (span_end > span_start);
 *   IKV_KEY_PREFIX    the first min(n_tokens, IKV_PREFIX_TOKENS = 256) input tokens;
 *   IKV_KEY_LOCAL     a key local to the request (no token ids), never equal to any
 *                     other key, so unrelated requests never share a memory.
 * Keys of different kinds never match, and keys match only when their bytes are
 * equal (a hash only speeds the lookup).
 */
#define IKV_KEY_EXPLICIT 1
#define IKV_KEY_SPAN     2
#define IKV_KEY_PREFIX   3
#define IKV_KEY_LOCAL    4
#define IKV_PREFIX_TOKENS 256

typedef struct ikv_key_source {
  const char *session_id;     /* host bytes of an explicit id, or NULL */
  int32_t session_id_len;     /* bytes of session_id; 0: none */
  int32_t n_tokens;           /* input token ids of the request (0: none) */
  const int32_t *tokens;      /* host, n_tokens entries, or NULL */
  int32_t span_start, span_end; /* designated session span within tokens; equal: none */
} ikv_key_source;

/*
 * The QueryMemory store of one compressor (Appendix A: an LRU of 1,024 memories per
 * compressor; concurrent requests update disjoint keys). The store maps session keys
 * to rows of a caller-owned device arena of `capacity` memories, each
 * [L][Hkv*R][D] float32; a session's memory is at arena + slot * L * Hkv * R * D
 * (its ikv_session.mem_off). The store holds no device memory.
 *   ikv_memstore_create: a store of `capacity` >= 1 memories (host allocation).
 *   ikv_memstore_acquire: the memory of src's session. A known key becomes the most
 *     recently used and *fresh = 0. A new key takes an unused row, or else the row of
 *     the least recently used memory that is not acquired (IKV_EUNSUPPORTED if every
 *     memory is acquired), and *fresh = 1: the caller zeroes that row before its
 *     first ikv_qm_update (a new session starts from M = 0). *kind (may be NULL)
 *     gets the IKV_KEY_* that was used. Every acquire pins the memory against
 *     eviction until the matching ikv_memstore_release.
 *   ikv_memstore_trigger: whether a compression event runs now for the memory at
 *     `slot` of a request of N positions and budget C: N > C (Appendix H), and at
 *     least `trigger` positions (512 in the paper, Appendix A) since the last event
 *     that fired for this memory (none yet counts as position 0). *fire = 1 records N.
 *   ikv_memstore_size: memories held.
 */
typedef struct ikv_memstore ikv_memstore;
ikv_status ikv_memstore_create(int32_t capacity, ikv_memstore **out);
void ikv_memstore_destroy(ikv_memstore *store);
ikv_status ikv_memstore_acquire(ikv_memstore *store, const ikv_key_source *src, int32_t *slot,
                                int32_t *fresh, int32_t *kind);
ikv_status ikv_memstore_release(ikv_memstore *store, int32_t slot);
ikv_status ikv_memstore_trigger(ikv_memstore *store, int32_t slot, int32_t N, int32_t C,
                                int32_t trigger, int32_t *fire);
ikv_status ikv_memstore_size(ikv_memstore *store, int32_t *n);

/*
 * The actionable query span [qs, qe) (Sec. 3.1: the latest user, tool or function
 * message that can affect the next decision, after template rendering). The caller
 * passes the rendered request's messages as position ranges [msg_start, msg_end)
 * in order, with actionable[m] != 0 for user, tool and function messages. The span
 * is the latest non-empty actionable message; with none, the bounded query-tail
 * fallback [max(0, N - tail_w), N) (W = 32 in the paper, Appendix A). Host arrays.
 */
ikv_status ikv_resolve_span(int32_t N, const int32_t *msg_start, const int32_t *msg_end,
                            const uint8_t *actionable, int32_t n_msgs, int32_t tail_w,
                            int32_t *qs, int32_t *qe);

/*
 * The compact apply path that the standard compactors use (Sec. 3.4; the Appendix
 * layout ablation, Table 7, compares it with ikv_redirect_slots): the kept positions
 * of each session are left-packed. The t-th kept live position j (position order)
 * moves to position t and slot dst_slots[slot_off + t]: on every layer and KV head
 *   K[l][dst][h] = RoPE_{t - j}(K[l][S[j]][h])   (Neox rotate-half: channel pair
 *                  (i, i + D/2) turns by (t - j) * rope_base^(-2i/D); angles in float64,
 *                  rotation in float32, one rounding to the pool's type),
 *   V[l][dst][h] = V[l][S[j]][h].
 * The session's new slot map is dst_slots[slot_off .. slot_off + n_keep[b]) and its new
 * length n_keep[b]; every old slot can go back to the allocator, and the radix prefix
 * cache no longer matches (the compact layout forces it off). No source slot may be a
 * destination slot (results undefined otherwise).
 *   keep: device uint8 per session [N] (ikv_select_budget's mask); dead positions are
 *   never kept. dst_slots: device int32 per session [N] (first n_keep used).
 *   n_keep: device int32 [B]. workspace: ikv_workspace_bytes(IKV_CALL_COMPACT).
 */
ikv_status ikv_compact_apply(const ikv_pool *pool, const ikv_session *sess,
                             const ikv_session *sess_dev, int32_t B, const int32_t *slot_maps,
                             const uint8_t *keep, const int32_t *dst_slots, double rope_base,
                             int32_t *n_keep, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Prefill of each session's actionable query span [qs, qe), n = qe - qs tokens, with the
 * retention step's inputs produced on the way (Sec. 3.5: the post-RoPE Q and K that the
 * step uses are the ones the model's attention computes; Sec. 3.2: Enc(q_t); Eq. 2;
 * Eq. 6's keys). For every layer, token t of the span (position qs + t) and head:
 *   q' = RoPE_{qs+t}(q_raw), k' = RoPE_{qs+t}(k_raw) (Neox rotate-half, base rope_base;
 *        float64 angles, float32 rotation, one rounding to the pool's type);
 *   k', v_raw are written into the pool at slot_maps[slot_off + qs + t] (the caller has
 *        assigned the span's slots);
 *   q_out = q'; out = causal attention of q' over the history slots
 *        hist[slot_off .. slot_off + n_hist[b]) (positions before qs; every span query
 *        sees all of them) and the span's slots of tokens 0 .. t;
 *   with M (not NULL): Eq. 2 with Enc = the mean of the n rows q' of each query head,
 *        in place (the memory's R must equal Hq / Hkv: one row per query head, the
 *        paper's M_t in R^{L x Hq x D});
 *   kq[t] = the mean of k' over layers and KV heads (Eq. 5's key mean at the span's
 *        positions, the cross-attention keys of Eq. 6), float32.
 * Packing: sessions in order; session b's rows start after those of the sessions before
 * it: q_raw, q_out, out [L][Hq][n][D] and k_raw, v_raw [L][Hkv][n][D] (pool's type), kq
 * [n][D]. Supported: D = 128, a bf16 pool, n * (Hq / Hkv) <= 256, Hq * D <= 8192 and
 * Hkv * D <= 2048 (IKV_EUNSUPPORTED otherwise). lambda as in ikv_qm_update.
 * workspace: ikv_workspace_bytes(IKV_CALL_PREFILL).
 */
ikv_status ikv_prefill_span(const ikv_pool *pool, const ikv_session *sess,
                            const ikv_session *sess_dev, int32_t B, const int32_t *slot_maps,
                            const void *q_raw, const void *k_raw, const void *v_raw,
                            const int32_t *hist, const int32_t *n_hist, double rope_base,
                            float lambda, float *M, void *q_out, void *out, float *kq,
                            void *workspace, size_t workspace_bytes, void *stream);

/*
 * Workspace size of one call (IKV_CALL_*) for these sessions, in bytes (0 when
 * the call needs none). `pool` may be NULL for SELECT; REDIRECT reads only
 * pool->num_slots. `flags` matter for SCORE only and are the score call's flags.
 */
ikv_status ikv_workspace_bytes(const ikv_pool *pool, const ikv_session *sess, int32_t B,
                               int32_t call, uint32_t flags, size_t *bytes);

/* Message of the last error on this thread ("" if none). */
const char *ikv_last_error(void);

/*
 * Per-kernel timing, a tracing aid for profiling the calls above.
 * ikv_timing(1) makes every following call record a pair of HIP events around
 * each kernel it launches, on that call's stream; ikv_timing(0) stops recording
 * (records already taken stay until read). ikv_timing returns IKV_OK.
 * ikv_timing_read waits for the recorded events, writes up to `cap` entries in
 * launch order (kernel name: a static string; elapsed milliseconds), drops every
 * record and returns how many records it held (a count above cap means the rest
 * were not written), or IKV_EHIP if an event call failed. At most 65536 records
 * are kept between reads; later launches are not recorded. names and ms are host
 * memory and may be NULL when cap is 0. The record list is process-wide: switch
 * timing on, launch and read from one thread. Event pairs add a little time
 * between kernels; time whole calls with timing off.
 */
ikv_status ikv_timing(int32_t enable);
int32_t ikv_timing_read(const char **names, float *ms, int32_t cap);

#ifdef __cplusplus
}
#endif

#endif /* IKV_H */
