"""Plain float64 CPU oracle of the IntentKV per-step retention path.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's CPU
baseline may import this module. The product path (the HIP library and its Python
binding) never calls it, and it shares no code with that path: it reads the same
seeded input bytes and nothing else.

Every function computes the paper's plain definition, step by step, in float64
(bf16 / fp32 inputs are widened exactly). A library primitive (matrix product, erf,
stable sort) may serve as one step; there is no blocking, fusion or reordering.

Notation (Sec. 3.1): S slot map, K/V post-RoPE keys/values in a paged pool indexed
by physical slot, s_dead the sentinel slot, [0, pi) the protected prefix, [qs, qe)
the actionable query span, F the forced set, A the candidate set, C the budget,
C* = max(0, C - |F|), M the QueryMemory.

Parity status: every function here is pinned by tests/test_oracle_pins.py against
closed forms, textbook special cases, hand-worked examples or brute force. No
function is "parity unpinned". What no pin can settle is how the authors' code read
the passages the paper leaves open; those readings are listed in the design notes.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

LAMBDA = 0.5            # memory decay (Appendix A, session identification paragraph)
NORM_EPS = 1e-12        # floor of the row norm in the unit-norm projection
H_C, D_C, HIDDEN = 4, 128, 256   # cross-attention heads / width, MLP hidden width (Sec. 3.3)
ALPHA_CLIP = 5.0        # alpha in [-5, 5], clipped at inference (Eq. 4)
SENTINEL_K = -1.0e4     # sentinel key value on every layer; sentinel value is 0 (Sec. 3.4)

FLAG_RESIDUAL = 1       # add the residual head of Eq. 4
FLAG_NO_XATTN = 2       # the "- x-attn" ablation: c_j = 0 (Sec. 3.3, ablation knobs)


def widen(a) -> np.ndarray:
    """bf16 bit patterns (uint16) or float32 to float64, exactly."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ----------------------------------------------------------------------------- sets

def sets(S, pi, qs, qe, C, dead):
    """Live, forced and candidate positions and the residual budget.

    Appendix H (compression event): skip when N <= C; live set L = {j : S[j] != s_dead};
    L splits into forced F and candidates A. Sec. 3.1 / Eq. 1: F = [0, pi) u [qs, qe),
    C* = max(0, C - |F|). Forced positions that are already dead are not live and are
    not counted in |F|.
    """
    S = np.asarray(S)
    N = len(S)
    j = np.arange(N)
    live = S != dead
    forced = ((j < pi) | ((j >= qs) & (j < qe))) & live
    cand = live & ~forced
    return {
        "N": N, "live": live, "forced": forced, "cand": cand,
        "Cstar": max(0, C - int(forced.sum())), "skip": N <= C,
    }


# ----------------------------------------------------------------------------- Eq. 2

def qm_update(M_prev, q_span, lam=LAMBDA):
    """One QueryMemory step, Eq. 2 and Sec. 3.2.

    Enc(q_t) is the mean of the span's post-RoPE query rows; M_t = exp(-lam) M_{t-1}
    + Enc(q_t); then every row is projected to unit norm along the head dimension.
    ``M_prev`` [rows][D], ``q_span`` [rows][n][D]. A new session starts from M = 0.
    """
    M_prev = widen(M_prev)
    q = widen(q_span)
    enc = q.mean(axis=-2)
    decay = 0.0 if math.isinf(lam) else math.exp(-lam)
    M = decay * M_prev + enc
    norm = np.sqrt((M * M).sum(axis=-1, keepdims=True))
    return M / np.maximum(norm, NORM_EPS)


# ----------------------------------------------------------------------------- Eq. 3

def rule_scores(k_pool, S, cand, M, Hkv, R):
    """Rule score of every candidate, Eq. 3.

    For every layer l, KV head h and memory row r paired with h (rows h*R .. h*R+R-1
    of M[l]), a_{r,j} = softmax over the candidate set A of M[l, r] . K[l, S[j], h] / sqrt(D);
    rule_j = sum of a_{r,j} over all (l, h, r). Returns float64 [N], -inf off A.
    """
    S = np.asarray(S)
    idx = np.nonzero(cand)[0]
    N = len(S)
    out = np.full(N, -np.inf)
    if len(idx) == 0:
        return out
    L = k_pool.shape[0]
    D = k_pool.shape[-1]
    M = widen(M).reshape(L, Hkv * R, D)
    rule = np.zeros(len(idx))
    slots = S[idx]
    for l in range(L):
        Kl = widen(k_pool[l][slots])                 # [|A|][Hkv][D]
        for h in range(Hkv):
            X = M[l, h * R:(h + 1) * R] @ Kl[:, h, :].T / math.sqrt(D)   # [R][|A|]
            X = X - X.max(axis=1, keepdims=True)
            P = np.exp(X)
            P = P / P.sum(axis=1, keepdims=True)
            rule += P.sum(axis=0)
    out[idx] = rule
    return out


def row_lse(k_pool, S, cand, M, Hkv, R):
    """log sum_{j in A} exp(M[l,r] . K[l,S[j],h] / sqrt(D)) for every memory row: the
    normaliser of Eq. 3, float64 [L][Hkv*R]."""
    S = np.asarray(S)
    idx = np.nonzero(cand)[0]
    L, D = k_pool.shape[0], k_pool.shape[-1]
    M = widen(M).reshape(L, Hkv * R, D)
    out = np.full((L, Hkv * R), -np.inf)
    if len(idx) == 0:
        return out
    for l in range(L):
        Kl = widen(k_pool[l][S[idx]])
        for h in range(Hkv):
            X = M[l, h * R:(h + 1) * R] @ Kl[:, h, :].T / math.sqrt(D)
            m = X.max(axis=1)
            out[l, h * R:(h + 1) * R] = m + np.log(np.exp(X - m[:, None]).sum(axis=1))
    return out


# ----------------------------------------------------------------------------- Eq. 5

def kbar(k_pool, S, positions):
    """k-bar_j: mean of K[l, S[j], h] over layers and KV heads, Eq. 5 (the mean over
    GQA-expanded heads equals the mean over KV heads). float64 [len(positions)][D]."""
    S = np.asarray(S)
    positions = np.asarray(positions, dtype=np.int64)
    L, _, Hkv, D = k_pool.shape
    acc = np.zeros((len(positions), D))
    slots = S[positions]
    for l in range(L):
        acc += widen(k_pool[l][slots]).sum(axis=1)
    return acc / (L * Hkv)


def mbar(M):
    """m-bar: mean of all QueryMemory rows (Eq. 5), float64 [D]."""
    M = widen(M)
    return M.reshape(-1, M.shape[-1]).mean(axis=0)


# ----------------------------------------------------------------------------- Eqs. 4-6

def residual_layout(D):
    """Parameter blocks of the residual head in packing order, (name, shape).

    Sec. 3.3: phi_j in R^{3D+1}; cross-attention with H_c = 4 heads of width
    d_c = 128 (W_Q, W_K, W_V with biases, no output projection); a two-layer GELU
    MLP of hidden width 256 over [phi_j ; c_j]; the scalar alpha. Matrices are
    row-major [out][in].
    """
    f = 3 * D + 1
    return [("W_Q", (D_C, f)), ("b_Q", (D_C,)), ("W_K", (D_C, D)), ("b_K", (D_C,)),
            ("W_V", (D_C, D)), ("b_V", (D_C,)), ("W_1", (HIDDEN, f + D_C)), ("b_1", (HIDDEN,)),
            ("w_2", (HIDDEN,)), ("b_2", (1,)), ("alpha", (1,))]


def residual_param_count(D):
    return sum(int(np.prod(shape)) for _, shape in residual_layout(D))


def residual_unpack(blob, D):
    blob = np.asarray(blob, dtype=np.float64)
    out, o = {}, 0
    for name, shape in residual_layout(D):
        n = int(np.prod(shape))
        out[name] = blob[o:o + n].reshape(shape)
        o += n
    if o != len(blob):
        raise ValueError(f"residual blob has {len(blob)} floats, layout needs {o}")
    return out


def gelu(x):
    """GELU in its exact erf form: x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def cross_attention(Qc, kq, W):
    """c_j = CrossAttn(W_Q phi_j, W_K Kq, W_V Kq), Eq. 6.

    ``Qc`` [n][128] are the projected candidate queries W_Q phi_j + b_Q; ``kq``
    [n_q][D] the k-bar rows at the live query positions. Each of the 4 heads takes
    32 consecutive channels, scores with scale 1/sqrt(32) and a softmax over the
    n_q query keys, and reads the matching 32 channels of the values.
    """
    n = Qc.shape[0]
    c = np.zeros((n, D_C))
    if kq.shape[0] == 0:
        return c
    Kp = kq @ W["W_K"].T + W["b_K"]
    Vp = kq @ W["W_V"].T + W["b_V"]
    dh = D_C // H_C
    for h in range(H_C):
        sl = slice(h * dh, (h + 1) * dh)
        X = Qc[:, sl] @ Kp[:, sl].T / math.sqrt(dh)
        X = X - X.max(axis=1, keepdims=True)
        P = np.exp(X)
        P = P / P.sum(axis=1, keepdims=True)
        c[:, sl] = P @ Vp[:, sl]
    return c


def residual_scores(rule, kb, mb, kq, blob, D, xattn=True):
    """s_j = rule_j + clip(alpha, -5, 5) * MLP(phi_j ++ c_j), Eq. 4 with Eqs. 5-6.

    ``rule`` [n] and ``kb`` [n][D] for the candidates, ``mb`` [D] the memory mean,
    ``kq`` [n_q][D] the k-bar rows of the live query positions.
    phi_j = [k-bar_j, m-bar, k-bar_j * m-bar, rule_j]; MLP = w_2 . GELU(W_1 x + b_1) + b_2.
    """
    W = residual_unpack(blob, D)
    n = len(rule)
    phi = np.concatenate([kb, np.broadcast_to(mb, (n, D)), kb * mb[None, :], rule[:, None]], axis=1)
    Qc = phi @ W["W_Q"].T + W["b_Q"]
    c = cross_attention(Qc, kq, W) if xattn else np.zeros((n, D_C))
    hidden = gelu(np.concatenate([phi, c], axis=1) @ W["W_1"].T + W["b_1"])
    y = hidden @ W["w_2"] + W["b_2"][0]
    alpha = min(max(W["alpha"][0], -ALPHA_CLIP), ALPHA_CLIP)
    return rule + alpha * y


def scores(k_pool, S, st, M, Hkv, R, blob=None, flags=0, qpos=None, dead=0):
    """Score vector of one session: Eq. 3, plus Eq. 4 when FLAG_RESIDUAL is set.

    Returns float64 [N]: s_j on the candidate set, -inf elsewhere; all -inf when
    the compression gate skips the session (N <= C).
    """
    N = len(S)
    if st["skip"]:
        return np.full(N, -np.inf)
    rule = rule_scores(k_pool, S, st["cand"], M, Hkv, R)
    if not (flags & FLAG_RESIDUAL) or blob is None:
        return rule
    D = k_pool.shape[-1]
    idx = np.nonzero(st["cand"])[0]
    out = np.full(N, -np.inf)
    if len(idx) == 0:
        return out
    qpos = np.asarray(qpos if qpos is not None else [], dtype=np.int64)
    qlive = qpos[np.asarray(S)[qpos] != dead] if len(qpos) else qpos
    kq = kbar(k_pool, S, qlive)
    out[idx] = residual_scores(rule[idx], kbar(k_pool, S, idx), mbar(M), kq, blob, D,
                               xattn=not (flags & FLAG_NO_XATTN))
    return out


# ----------------------------------------------------------------------------- Eq. 1

def select_budget(s, st):
    """Kept set of Eq. 1: F together with the C* best candidates.

    Candidates are ordered by score descending, ties by lower position (a NaN score
    counts as -inf). Returns (keep bool [N], n_keep, tau) with tau the score of the
    last candidate taken, +inf when none is taken. When the gate skips the session
    (N <= C) every live position is kept and tau = -inf.
    """
    live, forced, cand = st["live"], st["forced"], st["cand"]
    if st["skip"]:
        return live.copy(), int(live.sum()), -math.inf
    idx = np.nonzero(cand)[0]
    key = np.asarray(s, dtype=np.float64)[idx]
    key = np.where(np.isnan(key), -np.inf, key)
    order = np.lexsort((idx, -key))            # last key is primary: score desc, then position asc
    take = min(st["Cstar"], len(idx))
    keep = forced.copy()
    keep[idx[order[:take]]] = True
    tau = float(key[order[take - 1]]) if take > 0 else math.inf
    return keep, int(keep.sum()), tau


# ----------------------------------------------------------------------------- Eq. 7 + Sec. 3.4

def redirect(S, keep, dead, radix_prefix):
    """Slot-map eviction, Eq. 7, with the alias-aware free of Sec. 3.4 / Appendix H.

    Every live position outside the kept set is rerouted to the sentinel; kept
    positions keep their slot. The old slot u = S[j] of a newly dropped position j
    is freed only if j is outside the radix-protected prefix, u is not the sentinel
    and u is not a slot of any kept position.

    Returns (S_new, freed, live_list): freed as ascending unique slot ids, live_list
    the slot ids of the positions still live after the redirect, in position order.
    """
    S = np.asarray(S).astype(np.int64)
    keep = np.asarray(keep, dtype=bool)
    live = S != dead
    drop = live & ~keep
    kept_slots = set(S[keep & live].tolist())
    S_new = S.copy()
    S_new[drop] = dead
    freed = set()
    for j in np.nonzero(drop)[0]:
        u = int(S[j])
        if j >= radix_prefix and u != dead and u not in kept_slots:
            freed.add(u)
    live_list = S_new[S_new != dead]
    return S_new.astype(np.int32), np.array(sorted(freed), dtype=np.int32), live_list.astype(np.int32)


# ----------------------------------------------------------------------------- decode

def decode(q, k_pool, v_pool, live_slots):
    """GQA decode attention of one query row per head over the live slots.

    The attention backend reads the kept entries through the slot map with the
    sentinel stripped (Sec. 3.4; Appendix C.2): for layer l and query head h with
    KV head g = h // G, o = softmax_k(q . K[l, u_k, g] / sqrt(D)) V[l, u_k, g] over the
    live list u_0 .. u_{n-1}. An empty list gives o = 0. float64 [L][Hq][D].
    """
    q = widen(q)
    L, Hq, D = q.shape
    Hkv = k_pool.shape[2]
    G = Hq // Hkv
    live_slots = np.asarray(live_slots, dtype=np.int64)
    o = np.zeros((L, Hq, D))
    if len(live_slots) == 0:
        return o
    for l in range(L):
        Kl = widen(k_pool[l][live_slots])
        Vl = widen(v_pool[l][live_slots])
        for h in range(Hq):
            g = h // G
            x = Kl[:, g, :] @ q[l, h] / math.sqrt(D)
            x = x - x.max()
            p = np.exp(x)
            p = p / p.sum()
            o[l, h] = p @ Vl[:, g, :]
    return o


# ----------------------------------------------------------------------------- one step

def step(k_pool, v_pool, S, M, q_dec, Hkv, R, pi, qs, qe, C, radix_prefix, dead=0,
         blob=None, flags=0, qpos=None):
    """One retention step of one session: score, select, redirect, decode."""
    st = sets(S, pi, qs, qe, C, dead)
    s = scores(k_pool, S, st, M, Hkv, R, blob, flags, qpos, dead)
    keep, n_keep, tau = select_budget(s, st)
    S_new, freed, live = redirect(S, keep, dead, radix_prefix)
    o = decode(q_dec, k_pool, v_pool, live)
    return {"sets": st, "scores": s, "keep": keep, "n_keep": n_keep, "tau": tau,
            "S": S_new, "freed": freed, "live": live, "out": o}


# ----------------------------------------------------------------------------- baseline scorers on the substrate
# Sec. 4.1 (baselines) and Appendix A (compression settings): SnapKV with an observation
# window of W = 32 tail query rows, kernel-7 max-pool smoothing; H2O in ratio mode with
# a recent-window floor. Appendix "substrate integration": every scorer feeds the same
# selection, dead-slot redirect and decode. Query head h reads KV head h // G.

def attention_mass(k_pool, S, cand, q_rows, Hkv):
    """Attention each candidate receives from a set of query rows, per (layer, KV head).

    ``q_rows`` [L][Hq][n][D]: n post-RoPE query rows of every query head. For layer l
    and KV head g, every row of the G query heads h with h // G = g takes a softmax
    over the candidate set A of q . K[l, S[i], g] / sqrt(D); v[l, g, j] is the sum of
    those softmax weights at j. Returns float64 [L][Hkv][N], zero off A.
    """
    S = np.asarray(S)
    q = widen(q_rows)
    L, Hq, n, D = q.shape
    G = Hq // Hkv
    N = len(S)
    v = np.zeros((L, Hkv, N))
    idx = np.nonzero(cand)[0]
    if len(idx) == 0 or n == 0:
        return v
    for l in range(L):
        Kl = widen(k_pool[l][S[idx]])              # [|A|][Hkv][D]
        for h in range(Hq):
            g = h // G
            X = q[l, h] @ Kl[:, g, :].T / math.sqrt(D)   # [n][|A|]
            X = X - X.max(axis=1, keepdims=True)
            P = np.exp(X)
            P = P / P.sum(axis=1, keepdims=True)
            v[l, g, idx] += P.sum(axis=0)
    return v


def h2o_scores(k_pool, S, st, q_obs, Hkv):
    """H2O-style heavy-hitter score: the attention a candidate has received from the
    observed query rows, summed over layers and query heads. -inf off A; all -inf when
    the compression gate skips the session."""
    N = len(S)
    if st["skip"]:
        return np.full(N, -np.inf)
    v = attention_mass(k_pool, S, st["cand"], q_obs, Hkv)
    out = v.sum(axis=(0, 1))
    out[~st["cand"]] = -np.inf
    return out


def max_pool(v, kernel):
    """1-D max pooling of v along its last axis, stride 1, window of `kernel` (odd)
    positions centred on each position, positions past either end left out."""
    r = kernel // 2
    N = v.shape[-1]
    out = np.empty_like(v)
    for j in range(N):
        out[..., j] = v[..., max(0, j - r):min(N, j + r + 1)].max(axis=-1)
    return out


def snapkv_scores(k_pool, S, st, q_win, Hkv, kernel=7):
    """SnapKV-style score: per (layer, KV head) the attention mass from the observation
    window's query rows (attention_mass), smoothed by a max pool of `kernel` positions
    along the position axis (non-candidates hold zero mass), then summed over layers
    and KV heads. -inf off A; all -inf when the compression gate skips the session."""
    N = len(S)
    if st["skip"]:
        return np.full(N, -np.inf)
    v = attention_mass(k_pool, S, st["cand"], q_win, Hkv)
    out = max_pool(v, kernel).sum(axis=(0, 1))
    out[~st["cand"]] = -np.inf
    return out


def recent_window(N, C, recent_ratio):
    """H2O's ratio mode with a recent-window floor: the last ceil(recent_ratio * C)
    positions form the forced recent window [qs, N); the rest of the budget goes to the
    heavy hitters."""
    w = min(N, int(math.ceil(recent_ratio * C)))
    return N - w, N


# ----------------------------------------------------------------------------- compact apply path
# Sec. 3.4 (standard compactors left-pack the kept rows and re-index RoPE) and the
# Appendix layout ablation (Table 7: compact vs dead-slot apply path).

def rope_rotate(x, delta, base, D):
    """Neox (rotate-half) RoPE rotation of rows x[..., D] by `delta` positions: channel
    pair (i, i + D/2) turns by delta * base^(-2i/D). Rotating a key made at position j by
    t - j gives the key the same projection would have made at position t."""
    x = np.asarray(x, dtype=np.float64)
    h = D // 2
    ang = float(delta) * base ** (-2.0 * np.arange(h) / D)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def compact_apply(k_pool, v_pool, S, keep, dst, base):
    """Left-pack the kept positions of one session. The t-th kept position j (in position
    order) moves to position t and slot dst[t]: on every layer and KV head its key is
    re-rotated by t - j and its value copied. Returns float64 (K', V') [L][n_keep][Hkv][D],
    the rows written at dst[0 .. n_keep), and the new slot map dst[0 .. n_keep)."""
    S = np.asarray(S)
    kept = np.nonzero(np.asarray(keep, dtype=bool))[0]
    D = k_pool.shape[-1]
    L, Hkv = k_pool.shape[0], k_pool.shape[2]
    Kn = np.zeros((L, len(kept), Hkv, D))
    Vn = np.zeros((L, len(kept), Hkv, D))
    for t, j in enumerate(kept):
        Kn[:, t] = rope_rotate(widen(k_pool[:, S[j]]), t - int(j), base, D)
        Vn[:, t] = widen(v_pool[:, S[j]])
    return Kn, Vn, np.asarray(dst[:len(kept)], dtype=np.int32)


# ----------------------------------------------------------------------------- prefill of the query span
# Sec. 3.5 (post-RoPE Q and K captured from the model's attention: the RoPE hook) with
# Sec. 3.2 (Enc(q_t) is the mean of the span's post-RoPE Q rows) and Eq. 6 (the
# cross-attention keys are the mean key rows at the query positions): the span's
# prefill attention produces everything the retention step needs from the span.

def prefill_attention(q, k_pool, v_pool, hist_slots, span_slots):
    """Causal attention of the span's query rows. ``q`` [L][Hq][n][D] post-RoPE query
    rows of span tokens 0 .. n-1. Query row t of head h (KV head h // G) attends over
    the history slots (every one) and the span's own slots span_slots[u] for u <= t:
    o = softmax(q . K / sqrt(D)) V. float64 [L][Hq][n][D]."""
    q = widen(q)
    L, Hq, n, D = q.shape
    Hkv = k_pool.shape[2]
    G = Hq // Hkv
    hist = np.asarray(hist_slots, dtype=np.int64)
    span = np.asarray(span_slots, dtype=np.int64)
    out = np.zeros((L, Hq, n, D))
    for l in range(L):
        for t in range(n):
            slots = np.concatenate([hist, span[:t + 1]])
            Kl = widen(k_pool[l][slots])
            Vl = widen(v_pool[l][slots])
            for h in range(Hq):
                g = h // G
                x = Kl[:, g, :] @ q[l, h, t] / math.sqrt(D)
                x = x - x.max()
                p = np.exp(x)
                p = p / p.sum()
                out[l, h, t] = p @ Vl[:, g, :]
    return out
