"""Seeded synthetic inputs for the IntentKV retention path.

This module draws what a serving stack would hand to the retention step: post-RoPE
keys and values in a paged pool, per-session slot maps, QueryMemory rows, query-span
rows, a decode query and residual-head weights. Every tensor comes from its own
counter-keyed Philox stream ``(seed, tensor id, chunk)``, so any chunk can be
regenerated alone.

It holds none of the method's arithmetic (no scoring, selection, eviction or
attention). Both the HIP path and the oracle consume the exact bytes produced here;
nothing else is shared between them.

Layout conventions (the C-ABI's):
  * pools ``[L][num_slots][Hkv][D]``, bf16 bit patterns (uint16) or float32;
  * slot 0 is the dead slot; live slots are handed out in pages of ``page`` slots
    from a seeded shuffle of the free pages;
  * QueryMemory ``[L][Hkv*R][D]`` float32 per session, concatenated;
  * query-span rows ``[L][Hkv*R][n_span][D]`` in the pool dtype, concatenated;
  * decode queries ``[B][L][Hq][D]`` in the pool dtype.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
import dataclasses
from dataclasses import dataclass, field

import numpy as np

BF16, F32 = 0, 1
DEAD_SLOT = 0
# Rotary base of the public Qwen3 / Qwen2.5 configs. Both sides consume the
# rotated bytes, so the value only shapes the inputs.
ROPE_BASE = 1.0e6

# Philox key tensor ids.
T_K, T_V, T_M, T_QDEC, T_QSPAN, T_RESID, T_PAGES, T_HEAVY, T_DEAD, T_SHUF = range(10)


def stream(seed: int, tensor: int, chunk: int = 0) -> np.random.Generator:
    """Independent Philox stream keyed by (seed, tensor id, chunk)."""
    key = np.array([seed & 0xFFFFFFFFFFFFFFFF, ((tensor & 0xFFFF) << 48) | (chunk & 0xFFFFFFFFFFFF)],
                   dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


# ----------------------------------------------------------------------------- bf16

def f64_to_bf16(x) -> np.ndarray:
    """Round float64 values to bfloat16 (round-to-nearest-even), returned as uint16 bits.

    Rounds the float64 significand directly to 8 bits, so there is no double
    rounding through float32.
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    u = x.view(np.uint64)
    lsb = (u >> np.uint64(45)) & np.uint64(1)
    r = ((u + np.uint64((1 << 44) - 1) + lsb) >> np.uint64(45)) << np.uint64(45)
    f32 = r.view(np.float64).astype(np.float32)  # exact: at most 8 significant bits
    return (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(b) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float32."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_dtype(x64: np.ndarray, kv_dtype: int) -> np.ndarray:
    """Round float64 data to the storage dtype (bf16 bits or float32, both RNE)."""
    return f64_to_bf16(x64) if kv_dtype == BF16 else x64.astype(np.float32)


def widen(a: np.ndarray) -> np.ndarray:
    """Storage array (bf16 bits or float32) to float64, exactly."""
    if a.dtype == np.uint16:
        return bf16_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------- RoPE

def rope_cos_sin(positions, D: int, base: float = ROPE_BASE):
    inv = base ** (-np.arange(0, D, 2, dtype=np.float64) / D)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope_neox(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half (Neox) RoPE of float64 rows ``x[n, ..., D]`` at the n positions."""
    h = x.shape[-1] // 2
    shape = (cos.shape[0],) + (1,) * (x.ndim - 2) + (h,)
    c, s = cos.reshape(shape), sin.reshape(shape)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ----------------------------------------------------------------------------- specs

@dataclass
class Shape:
    L: int
    Hq: int
    Hkv: int
    D: int

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


@dataclass
class SessionSpec:
    """One request: N positions, budget C, forced prefix [0,pi) and span [qs,qe)."""
    N: int
    C: int
    pi: int
    qs: int
    qe: int
    R: int
    radix_prefix: int = 0
    qpos: np.ndarray | None = None       # query positions for the cross-attention (default: span)
    dead_frac: float = 0.0               # fraction of non-forced positions already redirected
    heavy_frac: float = 0.0              # fraction of non-forced positions with K scaled
    heavy_scale: float = 4.0

    def query_positions(self) -> np.ndarray:
        if self.qpos is not None:
            return np.asarray(self.qpos, dtype=np.int32)
        return np.arange(self.qs, self.qe, dtype=np.int32)


@dataclass
class Batch:
    shape: Shape
    kv_dtype: int
    sessions: list
    num_slots: int
    k_pool: np.ndarray            # [L][num_slots][Hkv][D]
    v_pool: np.ndarray
    slot_maps: np.ndarray         # int32 [sum N]
    slot_off: np.ndarray          # int64 [B]
    M: np.ndarray                 # float32 flat
    mem_off: np.ndarray           # int64 [B]
    q_span: np.ndarray            # pool dtype, flat
    qspan_off: np.ndarray         # int64 [B]
    qpos: np.ndarray              # int32 flat
    qpos_off: np.ndarray          # int64 [B]
    q_dec: np.ndarray             # [B][L][Hq][D] pool dtype
    heavy: list = field(default_factory=list)   # per session: positions with scaled K

    def S(self, b: int) -> np.ndarray:
        o = int(self.slot_off[b])
        return self.slot_maps[o:o + self.sessions[b].N]

    def M_of(self, b: int) -> np.ndarray:
        s, sh = self.sessions[b], self.shape
        o = int(self.mem_off[b])
        return self.M[o:o + sh.L * sh.Hkv * s.R * sh.D].reshape(sh.L, sh.Hkv * s.R, sh.D)

    def q_span_of(self, b: int) -> np.ndarray:
        s, sh = self.sessions[b], self.shape
        n = s.qe - s.qs
        o = int(self.qspan_off[b])
        return self.q_span[o:o + sh.L * sh.Hkv * s.R * n * sh.D].reshape(sh.L, sh.Hkv * s.R, n, sh.D)

    def qpos_of(self, b: int) -> np.ndarray:
        o = int(self.qpos_off[b])
        return self.qpos[o:o + len(self.sessions[b].query_positions())]


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def paged_slots(Ns, seed: int, page: int = 16, spare_pages: int = 0):
    """Physical slots of sessions of lengths ``Ns`` in one paged pool: pages of ``page``
    slots dealt in order from a seeded shuffle of all pages (slot 0 stays the dead
    slot). Returns (list of int64 slot arrays, num_slots)."""
    pages_per = [(int(n) + page - 1) // page for n in Ns]
    total_pages = sum(pages_per) + spare_pages
    order = stream(seed, T_PAGES).permutation(total_pages).astype(np.int64)
    alloc, p0 = [], 0
    for n, pp in zip(Ns, pages_per):
        pages = order[p0:p0 + pp]
        p0 += pp
        j = np.arange(int(n), dtype=np.int64)
        alloc.append(1 + pages[j // page] * page + (j % page))
    return alloc, 1 + total_pages * page


def make_batch(shape: Shape, sessions: list, seed: int, kv_dtype: int = BF16,
               layout: str = "paged", page: int = 16, spare_pages: int = 0, span_rows: bool = True) -> Batch:
    """Draw a batch of sessions sharing one paged pool.

    ``span_rows``: draw the query-span rows of the memory update ([L][Hkv*R][qe-qs][D]
    per session); False leaves them empty (a step without a memory update).

    ``layout``: ``"identity"`` (single session, S[j] = j + 1), ``"shuffled"``
    (single session, S a seeded permutation of 1..N) or ``"paged"`` (pages of
    ``page`` slots handed out from a seeded shuffle of all pages).
    """
    L, Hkv, D = shape.L, shape.Hkv, shape.D
    B = len(sessions)
    Ns = [s.N for s in sessions]

    # --- physical slots ------------------------------------------------------
    alloc = []
    if layout in ("identity", "shuffled"):
        assert B == 1
        n = Ns[0]
        num_slots = 1 + n
        if layout == "identity":
            alloc.append(np.arange(1, n + 1, dtype=np.int64))
        else:
            alloc.append(1 + stream(seed, T_SHUF).permutation(n).astype(np.int64))
    else:
        alloc, num_slots = paged_slots(Ns, seed, page, spare_pages)

    # --- slot maps with already-dead positions ---------------------------------
    slot_off = np.zeros(B, dtype=np.int64)
    slot_maps = np.zeros(sum(Ns), dtype=np.int32)
    heavy = []
    o = 0
    for b, s in enumerate(sessions):
        slot_off[b] = o
        S = alloc[b].astype(np.int32).copy()
        j = np.arange(s.N)
        forced = (j < s.pi) | ((j >= s.qs) & (j < s.qe))
        free_pos = np.nonzero(~forced)[0]
        if s.dead_frac > 0:
            nd = int(round(s.dead_frac * len(free_pos)))
            dead = stream(seed, T_DEAD, b).choice(free_pos, size=nd, replace=False)
            S[dead] = DEAD_SLOT
        if s.heavy_frac > 0:
            nh = min(len(free_pos), int(round(s.heavy_frac * s.N)))
            heavy.append(np.sort(stream(seed, T_HEAVY, b).choice(free_pos, size=nh, replace=False)))
        else:
            heavy.append(np.zeros(0, dtype=np.int64))
        slot_maps[o:o + s.N] = S
        o += s.N

    # --- pools -------------------------------------------------------------------
    st = np.uint16 if kv_dtype == BF16 else np.float32
    k_pool = np.zeros((L, num_slots, Hkv, D), dtype=st)
    v_pool = np.zeros((L, num_slots, Hkv, D), dtype=st)
    rope = [rope_cos_sin(np.arange(s.N), D) for s in sessions]

    def fill(job):
        b, l = job
        s = sessions[b]
        k = stream(seed, T_K, (b << 16) | l).standard_normal((s.N, Hkv, D), dtype=np.float32)
        k = rope_neox(k.astype(np.float64), *rope[b])
        if len(heavy[b]):
            k[heavy[b]] *= s.heavy_scale
        k_pool[l, alloc[b]] = to_dtype(k, kv_dtype)
        del k
        v = stream(seed, T_V, (b << 16) | l).standard_normal((s.N, Hkv, D), dtype=np.float32)
        v_pool[l, alloc[b]] = to_dtype(v.astype(np.float64), kv_dtype)

    jobs = [(b, l) for b in range(B) for l in range(L)]
    with ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, jobs))

    return Batch(shape=shape, kv_dtype=kv_dtype, sessions=sessions, num_slots=num_slots,
                 k_pool=k_pool, v_pool=v_pool, slot_maps=slot_maps, slot_off=slot_off, heavy=heavy,
                 **_queries(shape, sessions, seed, kv_dtype, span_rows))


def _queries(shape: Shape, sessions: list, seed: int, kv_dtype: int, span_rows: bool) -> dict:
    """QueryMemory, span rows, query positions and decode queries of a batch (the fields
    of Batch that depend on the memory rows R, not on the pool)."""
    L, Hkv, D = shape.L, shape.Hkv, shape.D
    B = len(sessions)
    mem_off = np.zeros(B, dtype=np.int64)
    qspan_off = np.zeros(B, dtype=np.int64)
    qpos_off = np.zeros(B, dtype=np.int64)
    Ms, spans, qps = [], [], []
    om = osp = oq = 0
    for b, s in enumerate(sessions):
        mem_off[b], qspan_off[b], qpos_off[b] = om, osp, oq
        m = stream(seed, T_M, b).standard_normal((L, Hkv * s.R, D), dtype=np.float32)
        Ms.append(m.ravel())
        om += m.size
        n = s.qe - s.qs if span_rows else 0
        q = stream(seed, T_QSPAN, b).standard_normal((n, L, Hkv * s.R, D), dtype=np.float32)
        cs = rope_cos_sin(np.arange(s.qs, s.qs + n), D)
        q = rope_neox(q.astype(np.float64), *cs).transpose(1, 2, 0, 3)
        spans.append(to_dtype(np.ascontiguousarray(q), kv_dtype).ravel())
        osp += spans[-1].size
        qp = s.query_positions()
        qps.append(qp)
        oq += len(qp)
    q_dec = np.zeros((B, L, shape.Hq, D), dtype=np.uint16 if kv_dtype == BF16 else np.float32)
    for b, s in enumerate(sessions):
        q = stream(seed, T_QDEC, b).standard_normal((1, L, shape.Hq, D), dtype=np.float32)
        q = rope_neox(q.astype(np.float64), *rope_cos_sin(np.array([s.N]), D))
        q_dec[b] = to_dtype(q[0], kv_dtype)
    return dict(M=np.concatenate(Ms) if Ms else np.zeros(0, np.float32), mem_off=mem_off,
                q_span=np.concatenate(spans), qspan_off=qspan_off,
                qpos=np.concatenate(qps).astype(np.int32), qpos_off=qpos_off, q_dec=q_dec)


def with_memory_rows(batch: Batch, R: int, seed: int, span_rows: bool = True) -> Batch:
    """The same sessions over the same pool (keys, values and slot maps shared, not
    copied) with R memory rows per KV head: QueryMemory, span rows and queries drawn
    afresh from `seed`."""
    sessions = [dataclasses.replace(s, R=R) for s in batch.sessions]
    return dataclasses.replace(batch, sessions=sessions,
                               **_queries(batch.shape, sessions, seed, batch.kv_dtype, span_rows))


# ----------------------------------------------------------------------------- residual weights

def residual_sizes(D: int, h_c: int = 128, hidden: int = 256):
    """Packed parameter blocks of the residual head, in packing order (name, count)."""
    f = 3 * D + 1
    return [("W_Q", h_c * f), ("b_Q", h_c), ("W_K", h_c * D), ("b_K", h_c),
            ("W_V", h_c * D), ("b_V", h_c), ("W_1", hidden * (f + h_c)), ("b_1", hidden),
            ("w_2", hidden), ("b_2", 1), ("alpha", 1)]


def residual_blob(D: int, seed: int, variant: str = "random", alpha: float = 1.0,
                  std: float = 0.02, units: int = 1, out_std: float = 0.01) -> np.ndarray:
    """Residual-head parameters as one float32 blob.

    ``random``: every weight and bias ~ N(0, std^2), alpha as given.
    ``zero``: as ``random`` but the output projection (w_2, b_2) is zero, which is
    the head's initial state.
    ``scaled``: weights under which every term of the head moves the scores of a
    full-size workload. The mean key row averages ``units`` = L * Hkv rows, so its
    entries are about sqrt(units) times smaller than a key's; random weights of a
    fixed scale then leave the cross-attention logits near zero and its output near
    constant across candidates. Here every matrix entry is N(0, 1/fan_in), the
    columns that read the mean key row (and its product with the memory mean), and
    W_K, W_V, are multiplied by sqrt(units); W_Q by 2 (attention over the query
    keys well away from uniform) and W_1's cross-attention columns by 4; biases are
    N(0, 0.1^2); w_2 and b_2 are N(0, (out_std / 4)^2) and N(0, out_std^2), so the
    head's output varies across candidates by about ``out_std`` (pick it near the
    spread of the rule scores).
    """
    sizes = residual_sizes(D)
    total = sum(n for _, n in sizes)
    if variant == "scaled":
        return _residual_blob_scaled(D, seed, alpha, units, out_std)
    blob = stream(seed, T_RESID).standard_normal(total, dtype=np.float32) * np.float32(std)
    o = 0
    for name, n in sizes:
        if name in ("w_2", "b_2") and variant == "zero":
            blob[o:o + n] = 0
        if name == "alpha":
            blob[o] = alpha
        o += n
    return blob


def _residual_blob_scaled(D: int, seed: int, alpha: float, units: int, out_std: float) -> np.ndarray:
    f, hc, hid = 3 * D + 1, 128, 256
    g = stream(seed, T_RESID, 1)
    ku = np.sqrt(float(units))
    WQ = g.standard_normal((hc, f)) / np.sqrt(f)
    WQ[:, :D] *= ku
    WQ[:, 2 * D:3 * D] *= ku
    WQ *= 2.0
    WK = g.standard_normal((hc, D)) / np.sqrt(D) * ku
    WV = g.standard_normal((hc, D)) / np.sqrt(D) * ku
    W1 = g.standard_normal((hid, f + hc)) / np.sqrt(f + hc)
    W1[:, :D] *= ku
    W1[:, 2 * D:3 * D] *= ku
    W1[:, f:] *= 4.0
    parts = {"W_Q": WQ, "b_Q": 0.1 * g.standard_normal(hc), "W_K": WK, "b_K": 0.1 * g.standard_normal(hc),
             "W_V": WV, "b_V": 0.1 * g.standard_normal(hc), "W_1": W1, "b_1": 0.1 * g.standard_normal(hid),
             "w_2": out_std / 4.0 * g.standard_normal(hid), "b_2": out_std * g.standard_normal(1),
             "alpha": np.array([alpha])}
    return np.concatenate([np.asarray(parts[n], np.float64).ravel() for n, _ in residual_sizes(D)]).astype(np.float32)


# ----------------------------------------------------------------------------- named workloads

def tiny_shape() -> Shape:
    return Shape(L=1, Hq=8, Hkv=2, D=64)


def qwen3_8b_shape() -> Shape:
    return Shape(L=36, Hq=32, Hkv=8, D=128)


def qwen25_14b_shape() -> Shape:
    return Shape(L=48, Hq=40, Hkv=8, D=128)


def tiny_single_layer(R: int = 16, layout: str = "identity", seed: int = 1, dead_frac: float = 0.0) -> Batch:
    """Single layer, 8 query / 2 KV heads, D=64, fp32 K/V, N=2048, budget 512, span = last 32."""
    N = 2048
    s = SessionSpec(N=N, C=512, pi=0, qs=N - 32, qe=N, R=R, dead_frac=dead_frac)
    return make_batch(tiny_shape(), [s], seed=seed, kv_dtype=F32, layout=layout)


def qwen3_8b_32k(R: int = 64, seed: int = 2) -> Batch:
    """Qwen3-8B shape, bf16 K/V, history 32768, budget 8192, span = last 64 positions."""
    N = 32768
    s = SessionSpec(N=N, C=8192, pi=0, qs=N - 64, qe=N, R=R)
    return make_batch(qwen3_8b_shape(), [s], seed=seed, kv_dtype=BF16, layout="paged")


def qwen25_14b_92k_heavy(R: int = 64, seed: int = 3) -> Batch:
    """Qwen2.5-14B shape, history 92,300 pruned to 8192; 5% of non-forced keys scaled x4."""
    N = 92300
    s = SessionSpec(N=N, C=8192, pi=0, qs=N - 64, qe=N, R=R, heavy_frac=0.05, heavy_scale=4.0)
    return make_batch(qwen25_14b_shape(), [s], seed=seed, kv_dtype=BF16, layout="paged")


# ----------------------------------------------------------------------------- query rows of the baseline scorers

def window_queries(shape: Shape, N: int, W: int, seed: int, session: int = 0) -> np.ndarray:
    """Post-RoPE query rows of the last W positions N-W .. N-1 of every query head, as a
    model in bf16 would emit them: N(0,1), rotated at their positions, rounded to bf16,
    returned widened to float32 [L][Hq][W][D]. Viewed as [L][Hkv*G*W][D] this is the
    memory-row argument of the scorer with R = G * W (query head h pairs with KV head
    h // G, its rows contiguous)."""
    q = stream(seed, T_QWIN, session).standard_normal((W, shape.L, shape.Hq, shape.D), dtype=np.float32)
    q = rope_neox(q.astype(np.float64), *rope_cos_sin(np.arange(N - W, N), shape.D)).transpose(1, 2, 0, 3)
    return bf16_to_f32(f64_to_bf16(np.ascontiguousarray(q)))


# ----------------------------------------------------------------------------- isolated-call inputs

def score_vector(n: int, seed: int, ties: bool = True) -> np.ndarray:
    """float32 scores for selection tests: many exact ties, NaN, -0.0, +0.0 and infinities."""
    g = stream(seed, T_MISC_SCORES)
    if ties:
        s = g.integers(-20, 20, n).astype(np.float32) * np.float32(0.125)
    else:
        s = g.standard_normal(n).astype(np.float32)
    k = max(1, n // 50)
    idx = g.choice(n, size=min(n, 5 * k), replace=False)
    s[idx[:k]] = np.nan
    s[idx[k:2 * k]] = -0.0
    s[idx[2 * k:3 * k]] = 0.0
    s[idx[3 * k:4 * k]] = -np.inf
    s[idx[4 * k:5 * k]] = np.float32(1e30)
    return s


def keep_mask(S: np.ndarray, seed: int, frac: float = 0.3, dead: int = DEAD_SLOT) -> np.ndarray:
    """uint8 keep mask over live positions (about `frac` of them), for isolated redirect tests."""
    g = stream(seed, T_MISC_KEEP)
    return ((g.random(len(S)) < frac) & (S != dead)).astype(np.uint8)


def alias_slots(S: np.ndarray, seed: int, pairs: int) -> np.ndarray:
    """Copy of S where `pairs` live positions reuse the slot of another live position."""
    g = stream(seed, T_MISC_ALIAS)
    S = S.copy()
    live = np.nonzero(S != DEAD_SLOT)[0]
    pick = g.choice(live, size=2 * pairs, replace=False)
    S[pick[:pairs]] = S[pick[pairs:]]
    return S


def slot_map(n: int, num_slots: int, seed: int, dead_frac: float = 0.1, dead: int = DEAD_SLOT) -> np.ndarray:
    """int32 slot map of n positions: distinct slots drawn from [0, num_slots) minus the
    dead slot, about `dead_frac` of the positions pointing at the dead slot."""
    g = stream(seed, T_MISC_SLOTS)
    pool = np.delete(np.arange(num_slots, dtype=np.int64), dead)
    S = g.choice(pool, size=n, replace=False).astype(np.int32)
    S[g.random(n) < dead_frac] = dead
    return S


T_MISC_SCORES, T_MISC_KEEP, T_MISC_ALIAS, T_MISC_SLOTS = 20, 21, 22, 23
T_TURNS = 24
T_TABLE_K, T_TABLE_V = 25, 26
T_QWIN = 27


# ----------------------------------------------------------------------------- multi-turn session

def multi_turn_plan(seed: int, turns: int = 8, first: int = 4096, final: int = 49152) -> list:
    """Token counts of a multi-turn agent session: [(appended tool tokens, query tokens)].

    Turn 1 holds `first` positions, the last 32-64 of them the query. Each later turn
    appends a tool output of ~U[2048, 8192] tokens (rescaled so that the last turn
    ends at `final` positions) and then a 32-64 token query.
    """
    g = stream(seed, T_TURNS)
    nq = g.integers(32, 65, turns)
    tool = g.integers(2048, 8193, turns - 1).astype(np.float64)
    target = final - first - int(nq[1:].sum())
    tool = np.floor(tool * target / tool.sum()).astype(np.int64)
    tool[-1] += target - int(tool.sum())
    return [(first - int(nq[0]), int(nq[0]))] + [(int(a), int(q)) for a, q in zip(tool, nq[1:])]


def turn_kv_rows(seed: int, turn: int, start: int, n: int, shape: Shape, kv_dtype: int = BF16):
    """K (post-RoPE at positions start .. start+n-1) and V rows appended in one turn,
    each [L][n][Hkv][D] in the storage type (bf16 bits or float32)."""
    L, Hkv, D = shape.L, shape.Hkv, shape.D
    cs = rope_cos_sin(np.arange(start, start + n), D)
    st = np.uint16 if kv_dtype == BF16 else np.float32
    k = np.empty((L, n, Hkv, D), st)
    v = np.empty((L, n, Hkv, D), st)

    def fill(l):
        x = stream(seed, T_K, (turn << 16) | l).standard_normal((n, Hkv, D), dtype=np.float32)
        k[l] = to_dtype(rope_neox(x.astype(np.float64), *cs), kv_dtype)
        y = stream(seed, T_V, (turn << 16) | l).standard_normal((n, Hkv, D), dtype=np.float32)
        v[l] = to_dtype(y.astype(np.float64), kv_dtype)

    with ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, range(L)))
    return k, v


def turn_span_rows(seed: int, turn: int, positions: np.ndarray, shape: Shape, R: int, kv_dtype: int = BF16):
    """Query rows of a turn's span for the QueryMemory update: [L][Hkv*R][n][D], post-RoPE."""
    n = len(positions)
    q = stream(seed, T_QSPAN, turn).standard_normal((n, shape.L, shape.Hkv * R, shape.D), dtype=np.float32)
    q = rope_neox(q.astype(np.float64), *rope_cos_sin(positions, shape.D)).transpose(1, 2, 0, 3)
    return to_dtype(np.ascontiguousarray(q), kv_dtype)


def turn_decode_query(seed: int, turn: int, position: int, shape: Shape, kv_dtype: int = BF16):
    """The decode query of a turn, [L][Hq][D], post-RoPE at `position`."""
    q = stream(seed, T_QDEC, turn).standard_normal((1, shape.L, shape.Hq, shape.D), dtype=np.float32)
    q = rope_neox(q.astype(np.float64), *rope_cos_sin(np.array([position]), shape.D))
    return to_dtype(q[0], kv_dtype)


# ----------------------------------------------------------------------------- table rows
# Pools too large to draw on the host (the batched one-GPU share: about 219 GB of keys
# and values) are filled on the GPU from a table: row (l, slot, h) is the window
# table[o : o + D] of T + D N(0,1) values in bf16, at o = splitmix64(key + (r + 1) *
# GAMMA) >> (64 - log2 T), r = (l * num_slots + slot) * Hkv + h (SplitMix64's output
# function: Steele, Lea and Flood, OOPSLA 2014). The device kernel (table_rows.hip)
# and table_rows() below produce the same bytes, so the oracle regenerates any row on
# the host. Every row holds D N(0,1) values; rows whose windows overlap share values,
# shifted. No RoPE is applied: a rotation of i.i.d. N(0,1) pairs is again i.i.d. N(0,1).

TABLE_LOG2 = 24
_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_SYNTH_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth.so")


def f32_to_bf16(x) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest even), as uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def table(seed: int, tensor: int, D: int, log2_T: int = TABLE_LOG2) -> np.ndarray:
    """2^log2_T + D N(0,1) values rounded to bf16 (nearest even), as uint16 bits."""
    return f32_to_bf16(stream(seed, tensor).standard_normal((1 << log2_T) + D, dtype=np.float32))


def table_key(seed: int, tensor: int) -> int:
    return (int(seed) << 32) | int(tensor)


def _splitmix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def table_offsets(l: int, num_slots: int, Hkv: int, slots, key: int, log2_T: int = TABLE_LOG2) -> np.ndarray:
    """Window offsets of rows (l, slots[k], h): int64 [len(slots)][Hkv]."""
    slots = np.asarray(slots, dtype=np.uint64)
    r = (np.uint64(l) * np.uint64(num_slots) + slots)[:, None] * np.uint64(Hkv) + np.arange(Hkv, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key) + (r + np.uint64(1)) * _GAMMA
        return (_splitmix64(z) >> np.uint64(64 - log2_T)).astype(np.int64)


def table_rows(tab: np.ndarray, L: int, num_slots: int, Hkv: int, D: int, slots, key: int,
               log2_T: int = TABLE_LOG2) -> np.ndarray:
    """Host copy of pool rows [L][len(slots)][Hkv][D] (uint16 bf16 bits), the same bytes
    as the device fill."""
    slots = np.asarray(slots)
    out = np.empty((L, len(slots), Hkv, D), dtype=np.uint16)
    d = np.arange(D, dtype=np.int64)
    for l in range(L):
        o = table_offsets(l, num_slots, Hkv, slots, key, log2_T)
        out[l] = tab[o[:, :, None] + d]
    return out


def device_table_rows(pool, L: int, num_slots: int, Hkv: int, D: int, slots, tab_dev, key: int,
                      log2_T: int = TABLE_LOG2, stream_=None) -> None:
    """Fill rows of a device bf16 pool tensor [L][num_slots][Hkv][D] from a device table:
    every slot (slots=None) or the slots of a device int32 tensor."""
    import ctypes
    import torch
    if not os.path.exists(_SYNTH_LIB):
        raise RuntimeError(f"{_SYNTH_LIB} is missing: run __graft_entry__.build()")
    lib = ctypes.CDLL(_SYNTH_LIB)
    fn = lib.synth_table_rows
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                   ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_uint64, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    st = (stream_ or torch.cuda.current_stream()).cuda_stream
    n = num_slots if slots is None else int(slots.numel())
    err = fn(pool.data_ptr(), L, num_slots, Hkv, D, None if slots is None else slots.data_ptr(), n,
             tab_dev.data_ptr(), log2_T, key, st)
    if err != 0:
        raise RuntimeError(f"synth_table_rows failed with HIP error {err}")


def read_ceiling(k_pool, v_pool, live, n: int, hpw: int, splits: int, stream_=None):
    """Plain read of the key and value rows of the first n slots of the device int32
    tensor `live`, every layer, in pieces of hpw adjacent heads (read_ceiling.hip): the
    bench's reference rate for decode attention. Returns the device tensor of per-
    workgroup words (asynchronous)."""
    import ctypes
    import torch
    if not os.path.exists(_SYNTH_LIB):
        raise RuntimeError(f"{_SYNTH_LIB} is missing: run __graft_entry__.build()")
    lib = ctypes.CDLL(_SYNTH_LIB)
    fn = lib.synth_read_ceiling
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                   ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    L, num_slots, Hkv, D = k_pool.shape
    out = torch.empty(splits * L * (Hkv // hpw), dtype=torch.int32, device=k_pool.device)
    st = (stream_ or torch.cuda.current_stream()).cuda_stream
    err = fn(k_pool.data_ptr(), v_pool.data_ptr(), L, num_slots, Hkv, D, hpw, live.data_ptr(), int(n), splits,
             out.data_ptr(), st)
    if err != 0:
        raise RuntimeError(f"synth_read_ceiling failed with HIP error {err}")
    return out


_probe_stamp = [1]


def exchange_probe(G: int, U: int, lag: int, mode: int, work_ns: int, device, spins: int = 1 << 16) -> dict:
    """Time the per-unit normaliser exchange probe (exchange_probe.hip) on a resident grid
    of G workgroups: U steps of `work_ns` spin each, with (mode 1) or without (mode 0) the
    exchange, normalisers awaited `lag` steps after their partials. Returns microseconds
    per step (the median of 5 launches) and the failure bits (1: a reader's wait ran out,
    2: an owner's)."""
    import ctypes
    import torch
    if not os.path.exists(_SYNTH_LIB):
        raise RuntimeError(f"{_SYNTH_LIB} is missing: run __graft_entry__.build()")
    lib = ctypes.CDLL(_SYNTH_LIB)
    fn = lib.synth_exchange_probe
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                   ctypes.c_int, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    part = torch.zeros(U * 64 * G, dtype=torch.int64, device=device)
    nrm = torch.zeros(U * 64, dtype=torch.int64, device=device)
    fail = torch.zeros(1, dtype=torch.int32, device=device)
    st = torch.cuda.current_stream()
    times = []
    for _ in range(6):
        stamp = _probe_stamp[0]
        _probe_stamp[0] += U + 1
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        err = fn(part.data_ptr(), nrm.data_ptr(), G, U, lag, mode, work_ns, spins, stamp, fail.data_ptr(),
                 st.cuda_stream)
        b.record()
        if err != 0:
            raise RuntimeError(f"synth_exchange_probe failed with HIP error {err}")
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b) * 1e3 / U)
    return {"us_per_step": round(float(np.median(times[1:])), 3), "fail": int(fail.item())}


def build_native(verbose: bool = False) -> str:
    """Compile table_rows.hip, read_ceiling.hip and exchange_probe.hip into
    synth/libsynth.so (gfx950)."""
    import shutil
    import subprocess
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    here = os.path.dirname(_SYNTH_LIB)
    srcs = [os.path.join(here, f) for f in ("table_rows.hip", "read_ceiling.hip", "exchange_probe.hip")]
    cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", *srcs, "-o", _SYNTH_LIB + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on synth's sources:\n{r.stdout}\n{r.stderr}")
    os.replace(_SYNTH_LIB + ".tmp", _SYNTH_LIB)
    if verbose:
        print(f"built {_SYNTH_LIB}")
    return _SYNTH_LIB


# ----------------------------------------------------------------------------- the batched share
def batched_share_full(seed: int = 5, B: int = 64) -> Batch:
    """The batched one-GPU share at full size: B sessions in the shape of one GPU's half of
    a Qwen2.5-14B tensor-parallel pair (48 layers, 20 query / 4 KV heads, D = 128), N ~
    U{4096..65536}, R ~ U{32..128}, budget 8192, the last 64 positions the query span and
    the cross-attention queries, one shared paged pool. Keys and values are not drawn
    here (k_pool = v_pool = None): fill_share_pools() writes them on the GPU, and
    share_rows() regenerates any rows on the host. No span rows (no memory update)."""
    g = stream(seed, T_TURNS, 2)
    Ns = [int(n) for n in g.integers(4096, 65537, B)]
    Rs = [int(r) for r in g.integers(32, 129, B)]
    shape = Shape(L=48, Hq=20, Hkv=4, D=128)
    alloc, num_slots = paged_slots(Ns, seed, 16, spare_pages=64)
    sessions = [SessionSpec(N=n, C=8192, pi=0, qs=n - 64, qe=n, R=r) for n, r in zip(Ns, Rs)]
    slot_maps = np.concatenate(alloc).astype(np.int32)
    slot_off = np.concatenate([[0], np.cumsum(Ns)[:-1]]).astype(np.int64)
    Ms, mem_off, om = [], np.zeros(B, np.int64), 0
    for b in range(B):
        mem_off[b] = om
        Ms.append(stream(seed, T_M, b).standard_normal((shape.L, shape.Hkv * Rs[b], shape.D), dtype=np.float32).ravel())
        om += Ms[-1].size
    qpos = np.concatenate([np.arange(n - 64, n) for n in Ns]).astype(np.int32)
    q_dec = np.stack([f32_to_bf16(stream(seed, T_QDEC, b).standard_normal((shape.L, shape.Hq, shape.D),
                                                                          dtype=np.float32)) for b in range(B)])
    batch = Batch(shape=shape, kv_dtype=BF16, sessions=sessions, num_slots=num_slots, k_pool=None, v_pool=None,
                  slot_maps=slot_maps, slot_off=slot_off, M=np.concatenate(Ms), mem_off=mem_off,
                  q_span=np.zeros(0, np.uint16), qspan_off=np.zeros(B, np.int64), qpos=qpos,
                  qpos_off=64 * np.arange(B, dtype=np.int64), q_dec=q_dec)
    batch.table_seed = seed                        # the seed of the tables its rows come from
    return batch


def fill_share_pools(k, v, batch: Batch) -> None:
    """Write every key and value row of the batched share's pool on the GPU (device bf16
    tensors [L][num_slots][Hkv][D]) from the seeded tables."""
    import torch
    sh = batch.shape
    for pool, tensor in ((k, T_TABLE_K), (v, T_TABLE_V)):
        tab = table(batch.table_seed, tensor, sh.D)
        tab_dev = torch.from_numpy(tab.view(np.int16)).to(pool.device)
        device_table_rows(pool, sh.L, batch.num_slots, sh.Hkv, sh.D, None, tab_dev,
                          table_key(batch.table_seed, tensor))


def share_rows(batch: Batch, slots, values: bool = False, layers: int | None = None) -> np.ndarray:
    """Host copy of the batched share's key (or value) rows at `slots`: [layers][len][Hkv][D]
    (the first `layers` layers, every layer by default)."""
    sh = batch.shape
    tensor = T_TABLE_V if values else T_TABLE_K
    return table_rows(table(batch.table_seed, tensor, sh.D), sh.L if layers is None else layers, batch.num_slots,
                      sh.Hkv, sh.D, slots, table_key(batch.table_seed, tensor))
