"""Pins of the float64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: hand-worked
numbers, closed forms, textbook special cases, invariants the paper states, or brute
force on tiny inputs. They run on the CPU only.
"""
import itertools
import math
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def pool_from_logical(K, slots, num_slots):
    """Scatter logical rows K[L][N][Hkv][D] into a pool [L][num_slots][Hkv][D]."""
    L, N, Hkv, D = K.shape
    pool = np.zeros((L, num_slots, Hkv, D), dtype=np.float32)
    pool[:, slots] = K
    return pool


def rand_pool(rng, L, N, Hkv, D, scale=1.0):
    K = (rng.standard_normal((L, N, Hkv, D)) * scale).astype(np.float32)
    S = (1 + rng.permutation(N)).astype(np.int32)
    return pool_from_logical(K, S, N + 1), S


# ============================================================================ sets

def test_sets_hand_example():
    S = np.array([5, 0, 3, 7, 2, 0, 9, 4, 6, 8], dtype=np.int32)
    st = oracle.sets(S, pi=2, qs=7, qe=9, C=5, dead=0)
    assert np.nonzero(st["live"])[0].tolist() == [0, 2, 3, 4, 6, 7, 8, 9]
    assert np.nonzero(st["forced"])[0].tolist() == [0, 7, 8]        # position 1 is dead
    assert np.nonzero(st["cand"])[0].tolist() == [2, 3, 4, 6, 9]
    assert st["Cstar"] == 2 and st["skip"] is False
    assert oracle.sets(S, 2, 7, 9, C=10, dead=0)["skip"] is True    # N <= C
    assert oracle.sets(S, 2, 7, 9, C=1, dead=0)["Cstar"] == 0       # |F| > C


# ============================================================================ Eq. 2

def test_qm_update_from_zero_hand():
    q = np.array([[[1.0, 2.0], [3.0, 4.0]]], dtype=np.float32)      # one row, span of 2
    M1 = oracle.qm_update(np.zeros((1, 2)), q)
    np.testing.assert_allclose(M1[0], [0.5547001962252291, 0.8320502943378437], rtol=0, atol=1e-15)


def test_qm_update_two_steps_hand():
    M1 = oracle.qm_update(np.zeros((1, 2)), np.array([[[1.0, 2.0], [3.0, 4.0]]], np.float32))
    M2 = oracle.qm_update(M1, np.array([[[0.0, 0.0], [0.0, 2.0]]], np.float32))   # Enc = [0, 1]
    np.testing.assert_allclose(M2[0], [0.2182114501672475, 0.9759015129693708], rtol=0, atol=1e-15)


def test_qm_update_unit_norm_zero_and_query_mode():
    rng = np.random.default_rng(0)
    Mp = rng.standard_normal((6, 16))
    q = rng.standard_normal((6, 5, 16)).astype(np.float32)
    M = oracle.qm_update(Mp, q)
    np.testing.assert_allclose(np.linalg.norm(M, axis=1), 1.0, atol=1e-12)
    assert np.all(oracle.qm_update(np.zeros((2, 4)), np.zeros((2, 3, 4), np.float32)) == 0)
    # lambda -> infinity forgets the past: the 'query' scorer mode / '- memory' ablation
    Mq = oracle.qm_update(Mp, q, lam=math.inf)
    Mz = oracle.qm_update(np.zeros_like(Mp), q)
    np.testing.assert_array_equal(Mq, Mz)
    # the projection makes the result invariant to a positive (exact, power-of-two) scale
    np.testing.assert_allclose(oracle.qm_update(np.zeros_like(Mp), 4 * q), Mz, atol=1e-15)


# ============================================================================ Eq. 3

def test_rule_single_row_is_textbook_softmax():
    # One layer, one KV head, one memory row, D = 4: logits are M.K/2 = v_j by construction.
    v = [0.5, -1.0, 2.0, 0.0, 1.5]
    K = np.array([[[[x, 1.0, -1.0, 0.0]] for x in v]], dtype=np.float32)   # [1][5][1][4]
    S = np.arange(1, 6, dtype=np.int32)
    pool = pool_from_logical(K, S, 6)
    M = np.array([[[2.0, 0.0, 0.0, 0.0]]])
    st = oracle.sets(S, 0, 5, 5, 0, 0)
    rule = oracle.rule_scores(pool, S, st["cand"], M, 1, 1)
    expect = [0.11074648791419399, 0.024710881584170254, 0.4963313244633698,
              0.06717114037545327, 0.3010401656628128]
    np.testing.assert_allclose(rule, expect, rtol=1e-14)


def test_rule_sums_to_row_count():
    rng = np.random.default_rng(1)
    L, N, Hkv, D, R = 3, 200, 2, 16, 5
    pool, S = rand_pool(rng, L, N, Hkv, D)
    S[rng.choice(N, 30, replace=False)] = 0
    M = rng.standard_normal((L, Hkv * R, D))
    st = oracle.sets(S, 10, 180, 190, 50, 0)
    rule = oracle.rule_scores(pool, S, st["cand"], M, Hkv, R)
    assert np.all(np.isneginf(rule[~st["cand"]]))
    assert math.isclose(rule[st["cand"]].sum(), L * Hkv * R, rel_tol=1e-12)


def test_rule_uniform_cases():
    rng = np.random.default_rng(2)
    L, N, Hkv, D, R = 2, 50, 2, 8, 3
    same = rng.standard_normal(D).astype(np.float32)
    K = np.broadcast_to(same, (L, N, Hkv, D)).copy()
    S = np.arange(1, N + 1, dtype=np.int32)
    st = oracle.sets(S, 5, 45, 50, 10, 0)
    nA = int(st["cand"].sum())
    M = rng.standard_normal((L, Hkv * R, D))
    rule = oracle.rule_scores(pool_from_logical(K, S, N + 1), S, st["cand"], M, Hkv, R)
    np.testing.assert_allclose(rule[st["cand"]], L * Hkv * R / nA, rtol=1e-13)
    pool, S2 = rand_pool(rng, L, N, Hkv, D)
    rule0 = oracle.rule_scores(pool, S2, st["cand"], np.zeros((L, Hkv * R, D)), Hkv, R)
    np.testing.assert_allclose(rule0[st["cand"]], L * Hkv * R / nA, rtol=1e-13)


def test_rule_row_to_kv_head_and_layer_pairing():
    # KV head 1 and layer 1 carry identical keys; the memory rows paired with the
    # distinct keys (layer 0, head 0) are zero. With the pairing of Eq. 3 (memory rows
    # h*R..h*R+R-1 of layer l score K[l, :, h]) every row then sees a uniform softmax.
    rng = np.random.default_rng(3)
    L, N, Hkv, D, R = 2, 40, 2, 8, 2
    K = rng.standard_normal((L, N, Hkv, D)).astype(np.float32)
    K[:, :, 1, :] = K[0, 0, 1, :]
    K[1] = K[1, 0]
    S = np.arange(1, N + 1, dtype=np.int32)
    pool = pool_from_logical(K, S, N + 1)
    st = oracle.sets(S, 0, N, N, 0, 0)
    M = rng.standard_normal((L, Hkv * R, D)) * 3
    M[0, :R] = 0
    rule = oracle.rule_scores(pool, S, st["cand"], M, Hkv, R)
    np.testing.assert_allclose(rule, L * Hkv * R / N, rtol=1e-13)


def test_rule_excludes_dead_and_forced_from_softmax():
    rng = np.random.default_rng(4)
    L, N, Hkv, D, R = 1, 30, 1, 8, 2
    pool, S = rand_pool(rng, L, N, Hkv, D)
    M = rng.standard_normal((L, Hkv * R, D))
    pool[:, S[7]] = 50.0          # huge key at a position that will be forced
    pool[:, S[9]] = 50.0          # ... and at one that will be dead
    Sd = S.copy()
    Sd[9] = 0
    st = oracle.sets(Sd, 0, 7, 8, 5, 0)
    r1 = oracle.rule_scores(pool, Sd, st["cand"], M, Hkv, R)
    Sd2 = Sd.copy()
    Sd2[7] = 0                    # same candidate set, position 7 now dead instead of forced
    st2 = oracle.sets(Sd2, 0, 7, 8, 5, 0)
    assert np.array_equal(st["cand"], st2["cand"])
    r2 = oracle.rule_scores(pool, Sd2, st2["cand"], M, Hkv, R)
    np.testing.assert_array_equal(r1, r2)
    assert math.isclose(r1[st["cand"]].sum(), L * Hkv * R, rel_tol=1e-12)


def test_rule_brute_force_loops():
    rng = np.random.default_rng(5)
    L, N, Hkv, D, R = 2, 9, 2, 4, 2
    pool, S = rand_pool(rng, L, N, Hkv, D)
    S[3] = 0
    M = rng.standard_normal((L, Hkv * R, D))
    pi, qs, qe = 1, 7, 8
    st = oracle.sets(S, pi, qs, qe, 3, 0)
    rule = oracle.rule_scores(pool, S, st["cand"], M, Hkv, R)
    cand = [j for j in range(N) if S[j] != 0 and not (j < pi or qs <= j < qe)]
    for j in range(N):
        if j not in cand:
            assert rule[j] == -math.inf
            continue
        total = 0.0
        for l in range(L):
            for h in range(Hkv):
                for r in range(R):
                    row = M[l][h * R + r]
                    def logit(i):
                        return sum(float(row[d]) * float(pool[l][S[i]][h][d]) for d in range(D)) / math.sqrt(D)
                    den = sum(math.exp(logit(i)) for i in cand)
                    total += math.exp(logit(j)) / den
        assert math.isclose(rule[j], total, rel_tol=1e-12)


def test_rule_slot_permutation_invariance():
    rng = np.random.default_rng(6)
    L, N, Hkv, D, R = 2, 64, 2, 8, 3
    K = rng.standard_normal((L, N, Hkv, D)).astype(np.float32)
    S1 = (1 + rng.permutation(N)).astype(np.int32)
    S2 = (1 + rng.permutation(N)).astype(np.int32)
    M = rng.standard_normal((L, Hkv * R, D))
    st = oracle.sets(S1, 2, 60, 64, 10, 0)
    r1 = oracle.rule_scores(pool_from_logical(K, S1, N + 1), S1, st["cand"], M, Hkv, R)
    r2 = oracle.rule_scores(pool_from_logical(K, S2, N + 1), S2, st["cand"], M, Hkv, R)
    np.testing.assert_array_equal(r1, r2)


def test_row_lse_brute_force():
    rng = np.random.default_rng(7)
    L, N, Hkv, D, R = 1, 6, 2, 4, 2
    pool, S = rand_pool(rng, L, N, Hkv, D)
    M = rng.standard_normal((L, Hkv * R, D))
    st = oracle.sets(S, 0, 5, 6, 0, 0)
    lse = oracle.row_lse(pool, S, st["cand"], M, Hkv, R)
    for h in range(Hkv):
        for r in range(R):
            xs = [float(M[0, h * R + r] @ pool[0, S[j], h].astype(np.float64)) / 2.0 for j in range(5)]
            assert math.isclose(lse[0, h * R + r], math.log(sum(math.exp(x) for x in xs)), rel_tol=1e-13)


# ============================================================================ Eq. 5

def test_kbar_and_mbar_hand():
    K = np.zeros((2, 3, 2, 2), dtype=np.float32)        # L=2, N=3, Hkv=2, D=2
    K[0, 1] = [[1, 2], [3, 4]]
    K[1, 1] = [[5, 6], [7, 8]]
    S = np.array([3, 1, 2], dtype=np.int32)
    pool = pool_from_logical(K, S, 4)
    np.testing.assert_array_equal(oracle.kbar(pool, S, [1]), [[4.0, 5.0]])
    M = np.array([[[1.0, 0.0], [0.0, 1.0]], [[3.0, 2.0], [4.0, 1.0]]])
    np.testing.assert_array_equal(oracle.mbar(M), [2.0, 1.0])


# ============================================================================ Eqs. 4-6

def test_residual_parameter_count_golden():
    with open(os.path.join(GOLDEN, "residual_param_count.txt")) as f:
        line = [ln for ln in f if ln.startswith("D=")][0]
    D, n = [int(t.split("=")[1]) for t in line.split()]
    assert oracle.residual_param_count(D) == n == 214274
    # the same topology at D = 64 (the single-layer workload)
    assert oracle.residual_param_count(64) == 124162
    assert sum(n for _, n in synth.residual_sizes(128)) == 214274


def test_gelu_is_exact_erf_form():
    with open(os.path.join(GOLDEN, "normal_cdf.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    for x, phi in rows:
        x, phi = float(x), float(phi)
        assert math.isclose(oracle.ikv_oracle.gelu(np.array(x)), x * phi, rel_tol=1e-14, abs_tol=1e-16)


def _session(seed, D=16, L=2, Hkv=2, R=3, N=40):
    rng = np.random.default_rng(seed)
    pool, S = rand_pool(rng, L, N, Hkv, D)
    M = rng.standard_normal((L, Hkv * R, D))
    return rng, pool, S, M


def _blob(rng, D, std=0.3, alpha=1.0):
    n = oracle.residual_param_count(D)
    b = rng.standard_normal(n) * std
    b[-1] = alpha
    return b


def _set_block(blob, D, name, value):
    o = 0
    for nm, shape in oracle.ikv_oracle.residual_layout(D):
        k = int(np.prod(shape))
        if nm == name:
            blob[o:o + k] = np.asarray(value, dtype=np.float64).ravel()
            return blob
        o += k
    raise KeyError(name)


def test_zero_initialised_head_recovers_rule_exactly():
    rng, pool, S, M = _session(8)
    D = 16
    st = oracle.sets(S, 2, 36, 40, 10, 0)
    blob = _blob(rng, D)
    _set_block(blob, D, "w_2", np.zeros(256))
    _set_block(blob, D, "b_2", [0.0])
    qpos = np.arange(36, 40)
    s = oracle.scores(pool, S, st, M, 2, 3, blob, oracle.FLAG_RESIDUAL, qpos)
    rule = oracle.rule_scores(pool, S, st["cand"], M, 2, 3)
    np.testing.assert_array_equal(s, rule)
    # alpha = 0 with a live fc2: the '- residual' ablation, also exactly the rule
    blob2 = _blob(rng, D, alpha=0.0)
    np.testing.assert_array_equal(oracle.scores(pool, S, st, M, 2, 3, blob2, oracle.FLAG_RESIDUAL, qpos), rule)


@pytest.mark.parametrize("block,index", [("kbar", 3), ("mbar", 5), ("prod", 7), ("rule", 0), ("c", 2)])
def test_residual_feature_order_one_hot_probes(block, index):
    """W_1 reads exactly one input feature; the MLP output is then GELU of that feature,
    which pins the order [k-bar ; m-bar ; k-bar*m-bar ; rule ; c] and the [out][in] layout."""
    D = 8
    rng, pool, S, M = _session(9, D=D)
    st = oracle.sets(S, 0, 39, 40, 5, 0)     # single query position 39 -> c = V' exactly
    blob = np.zeros(oracle.residual_param_count(D))
    blob[-1] = 1.0
    col = {"kbar": index, "mbar": D + index, "prod": 2 * D + index, "rule": 3 * D, "c": 3 * D + 1 + index}[block]
    W1 = np.zeros((256, 3 * D + 1 + 128))
    W1[0, col] = 1.0
    _set_block(blob, D, "W_1", W1)
    w2 = np.zeros(256)
    w2[0] = 1.0
    _set_block(blob, D, "w_2", w2)
    WV = np.zeros((128, D))
    WV[index, 1] = 1.0                        # c channel `index` = k-bar_q[1] (+ b_V = 0)
    _set_block(blob, D, "W_V", WV)
    s = oracle.scores(pool, S, st, M, 2, 3, blob, oracle.FLAG_RESIDUAL, np.array([39]))
    rule = oracle.rule_scores(pool, S, st["cand"], M, 2, 3)
    idx = np.nonzero(st["cand"])[0]
    kb = oracle.kbar(pool, S, idx)
    mb = oracle.mbar(M)
    feat = {"kbar": kb[:, index], "mbar": np.full(len(idx), mb[index]), "prod": kb[:, index] * mb[index],
            "rule": rule[idx], "c": np.full(len(idx), oracle.kbar(pool, S, [39])[0, 1])}[block]
    phi = np.array([0.5 * x * (1 + math.erf(x / math.sqrt(2))) for x in feat])
    np.testing.assert_allclose(s[idx] - rule[idx], phi, rtol=1e-12, atol=1e-15)


def test_cross_attention_head_split():
    D = 4
    W = {"W_K": np.zeros((128, D)), "b_K": np.zeros(128), "W_V": np.zeros((128, D)), "b_V": np.zeros(128)}
    W["W_K"][0, 0] = 10.0          # head 0 key channel 0 = +10 * kq[:, 0]
    W["W_K"][32, 0] = -10.0        # head 1 key channel 32 = -10 * kq[:, 0]
    W["W_V"][:, 1] = 1.0           # every value channel = kq[:, 1]
    kq = np.array([[1.0, 3.0, 0, 0], [-1.0, 7.0, 0, 0]])
    Qc = np.zeros((1, 128))
    Qc[0, 0] = 10.0
    Qc[0, 32] = 10.0
    c = oracle.ikv_oracle.cross_attention(Qc, kq, W)
    np.testing.assert_allclose(c[0, 0:32], 3.0, atol=1e-12)    # head 0 picks query key 0
    np.testing.assert_allclose(c[0, 32:64], 7.0, atol=1e-12)   # head 1 picks query key 1
    np.testing.assert_allclose(c[0, 64:], 5.0, atol=1e-12)     # heads 2-3: uniform over both


def test_alpha_clip_and_xattn_switches():
    D = 16
    rng, pool, S, M = _session(10, D=D)
    st = oracle.sets(S, 2, 36, 40, 10, 0)
    qpos = np.arange(36, 40)
    base = _blob(rng, D)

    def run(blob, flags=oracle.FLAG_RESIDUAL, q=qpos):
        return oracle.scores(pool, S, st, M, 2, 3, blob, flags, q)

    b7, b5 = base.copy(), base.copy()
    b7[-1], b5[-1] = 7.0, 5.0
    np.testing.assert_array_equal(run(b7), run(b5))
    bm9, bm5 = base.copy(), base.copy()
    bm9[-1], bm5[-1] = -9.0, -5.0
    np.testing.assert_array_equal(run(bm9), run(bm5))
    no_x = run(base, oracle.FLAG_RESIDUAL | oracle.FLAG_NO_XATTN)
    vzero = _set_block(_set_block(base.copy(), D, "W_V", np.zeros((128, D))), D, "b_V", np.zeros(128))
    np.testing.assert_allclose(run(vzero), no_x, rtol=0, atol=1e-14)
    # every query position dead: the cross-attention has no live evidence, c = 0
    S2 = S.copy()
    S2[36:40] = 0
    st2 = oracle.sets(S2, 2, 36, 40, 10, 0)
    a = oracle.scores(pool, S2, st2, M, 2, 3, base, oracle.FLAG_RESIDUAL, qpos)
    b = oracle.scores(pool, S2, st2, M, 2, 3, base, oracle.FLAG_RESIDUAL | oracle.FLAG_NO_XATTN, qpos)
    np.testing.assert_array_equal(a, b)


# ============================================================================ Eq. 1

def test_select_brute_force_argtop():
    rng = np.random.default_rng(11)
    for trial in range(20):
        N = 9
        S = np.arange(1, N + 1, dtype=np.int32)
        S[rng.choice(N, 2, replace=False)] = 0
        st = oracle.sets(S, 1, 7, 8, C=int(rng.integers(2, 7)), dead=0)
        s = rng.standard_normal(N)
        keep, n_keep, tau = oracle.select_budget(s, st)
        cand = np.nonzero(st["cand"])[0].tolist()
        k = min(st["Cstar"], len(cand))
        best = max(itertools.combinations(cand, k), key=lambda c: sum(s[j] for j in c))
        expect = set(np.nonzero(st["forced"])[0].tolist()) | set(best)
        assert set(np.nonzero(keep)[0].tolist()) == expect
        assert n_keep == len(expect)
        if k:
            assert tau == min(s[j] for j in best)


def test_select_ties_nan_and_signed_zero():
    N = 8
    S = np.arange(1, N + 1, dtype=np.int32)
    st = oracle.sets(S, 0, 8, 8, C=3, dead=0)
    keep, _, _ = oracle.select_budget(np.full(N, 0.25), st)
    assert np.nonzero(keep)[0].tolist() == [0, 1, 2]            # equal scores: lowest positions
    s = np.array([np.nan, -0.0, 0.0, -1.0, np.nan, -0.0, -2.0, -3.0])
    keep, _, tau = oracle.select_budget(s, st)
    assert np.nonzero(keep)[0].tolist() == [1, 2, 5] and tau == 0.0
    st0 = oracle.sets(S, 0, 8, 8, C=7, dead=0)
    keep, _, tau = oracle.select_budget(s, st0)
    assert np.nonzero(keep)[0].tolist() == [0, 1, 2, 3, 5, 6, 7] and tau == -math.inf


def test_select_counts_gate_and_optimality():
    rng = np.random.default_rng(12)
    N = 500
    S = (1 + rng.permutation(N)).astype(np.int32)
    S[rng.choice(N, 100, replace=False)] = 0
    st = oracle.sets(S, 20, 480, 500, C=150, dead=0)
    s = rng.standard_normal(N)
    keep, n_keep, tau = oracle.select_budget(s, st)
    nF, nA = int(st["forced"].sum()), int(st["cand"].sum())
    assert n_keep == nF + min(st["Cstar"], nA)
    assert np.all(keep[st["forced"]]) and not np.any(keep[~st["live"]])
    kept_c = st["cand"] & keep
    drop_c = st["cand"] & ~keep
    assert s[kept_c].min() >= s[drop_c].max() and tau == s[kept_c].min()
    # a budget at least the live count keeps everything live
    st_all = oracle.sets(S, 20, 480, 500, C=499, dead=0)
    assert np.array_equal(oracle.select_budget(s, st_all)[0], st["live"])
    # N <= C: the compression event is skipped
    st_skip = oracle.sets(S, 20, 480, 500, C=500, dead=0)
    keep, n, tau = oracle.select_budget(s, st_skip)
    assert np.array_equal(keep, st["live"]) and tau == -math.inf


# ============================================================================ Eq. 7 / Sec. 3.4

def test_redirect_hand_example():
    S = np.array([11, 12, 0, 13, 14, 12, 15, 16], dtype=np.int32)
    keep = np.array([1, 0, 0, 1, 0, 1, 0, 1], dtype=bool)
    # position 1 aliases slot 12 with kept position 5 -> not freed; position 4 is in the
    # radix-protected prefix [0, 5) -> not freed; position 6 frees slot 15.
    S_new, freed, live = oracle.redirect(S, keep, dead=0, radix_prefix=5)
    assert S_new.tolist() == [11, 0, 0, 13, 0, 12, 0, 16]
    assert freed.tolist() == [15]
    assert live.tolist() == [11, 13, 12, 16]


def test_redirect_invariants_random():
    rng = np.random.default_rng(13)
    N = 1000
    S = (1 + rng.permutation(N)).astype(np.int32)
    S[rng.choice(N, 150, replace=False)] = 0
    dup = rng.choice(np.nonzero(S)[0], 20, replace=False)
    S[dup[:10]] = S[dup[10:]]                          # shared slots inside the request
    keep = (rng.random(N) < 0.3) & (S != 0)
    S_new, freed, live = oracle.redirect(S, keep, 0, radix_prefix=100)
    assert np.array_equal(S_new[keep], S[keep])                          # kept slots untouched
    assert np.all(S_new[~keep] == 0)                                     # dropped -> sentinel
    kept_slots = set(S[keep].tolist())
    assert not (set(freed.tolist()) & kept_slots) and 0 not in freed
    assert len(set(freed.tolist())) == len(freed) and np.all(np.diff(freed) > 0)
    pos_of = {}
    for j in range(N):
        pos_of.setdefault(int(S[j]), []).append(j)
    for u in freed:
        assert any(j >= 100 and not keep[j] for j in pos_of[int(u)])
    assert np.array_equal(live, S_new[S_new != 0])


# ============================================================================ decode

def test_decode_brute_force_loops():
    rng = np.random.default_rng(14)
    L, Hq, Hkv, D, n = 2, 4, 2, 4, 5
    pool_k = rng.standard_normal((L, 9, Hkv, D)).astype(np.float32)
    pool_v = rng.standard_normal((L, 9, Hkv, D)).astype(np.float32)
    live = np.array([3, 8, 1, 6, 2])
    q = rng.standard_normal((L, Hq, D)).astype(np.float32)
    o = oracle.decode(q, pool_k, pool_v, live)
    for l in range(L):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            xs = [sum(float(q[l, h, d]) * float(pool_k[l, u, g, d]) for d in range(D)) / 2.0 for u in live]
            ws = [math.exp(x) for x in xs]
            for d in range(D):
                ref = sum(w * float(pool_v[l, u, g, d]) for w, u in zip(ws, live)) / sum(ws)
                assert math.isclose(o[l, h, d], ref, rel_tol=1e-12, abs_tol=1e-14)


def test_decode_special_cases():
    rng = np.random.default_rng(15)
    L, Hq, Hkv, D = 1, 4, 2, 8
    pk = rng.standard_normal((L, 10, Hkv, D)).astype(np.float32)
    pv = rng.standard_normal((L, 10, Hkv, D)).astype(np.float32)
    q = rng.standard_normal((L, Hq, D)).astype(np.float32)
    o = oracle.decode(q, pk, pv, [4])
    np.testing.assert_allclose(o[0, 0], pv[0, 4, 0], rtol=0, atol=0)      # one live row: o = V
    np.testing.assert_allclose(o[0, 3], pv[0, 4, 1], rtol=0, atol=0)      # head 3 -> KV head 1
    assert np.all(oracle.decode(q, pk, pv, []) == 0)
    pk2 = pk.copy()
    pk2[0, :, :, :] = pk[0, 1]
    o = oracle.decode(q, pk2, pv, [1, 2, 3])
    np.testing.assert_allclose(o[0, 1], pv[0, [1, 2, 3], 0].astype(np.float64).mean(0), atol=1e-14)
    pv2 = pv.copy()
    pv2[0, :, 1, :] = 0.75                                                # KV head 1 values constant
    o = oracle.decode(q, pk, pv2, [1, 5, 7])
    np.testing.assert_allclose(o[0, 2:4], 0.75, atol=1e-15)


def test_decode_slot_permutation_invariance():
    rng = np.random.default_rng(16)
    L, Hq, Hkv, D, n = 2, 8, 2, 16, 30
    K = rng.standard_normal((L, n, Hkv, D)).astype(np.float32)
    V = rng.standard_normal((L, n, Hkv, D)).astype(np.float32)
    q = rng.standard_normal((L, Hq, D)).astype(np.float32)
    s1 = 1 + rng.permutation(n)
    s2 = 1 + rng.permutation(n)
    o1 = oracle.decode(q, pool_from_logical(K, s1, n + 1), pool_from_logical(V, s1, n + 1), s1)
    o2 = oracle.decode(q, pool_from_logical(K, s2, n + 1), pool_from_logical(V, s2, n + 1), s2)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-15)


def test_sentinel_is_not_a_mask_when_query_sum_is_negative():
    """The sentinel's logit is -1e4 * sum_d(q_d) / sqrt(D), not -1e4 * sqrt(D): attending
    to it only masks when sum_d q_d > 0. This is why decode strips dead slots."""
    rng = np.random.default_rng(17)
    L, Hq, Hkv, D = 1, 2, 1, 8
    pk = rng.standard_normal((L, 6, Hkv, D)).astype(np.float32)
    pv = rng.standard_normal((L, 6, Hkv, D)).astype(np.float32)
    pk[:, 0] = oracle.ikv_oracle.SENTINEL_K
    pv[:, 0] = 0.0
    q = np.ones((L, Hq, D), dtype=np.float32)
    q[0, 1] *= -1.0                                 # head 1: sum of q is negative
    masked = oracle.decode(q, pk, pv, [1, 2, 3, 4, 5])
    with_sentinel = oracle.decode(q, pk, pv, [0, 1, 2, 3, 4, 5])
    np.testing.assert_allclose(with_sentinel[0, 0], masked[0, 0], atol=1e-12)
    np.testing.assert_allclose(with_sentinel[0, 1], 0.0, atol=1e-12)
    assert np.abs(masked[0, 1]).max() > 1e-3


# ============================================================================ whole step

def test_step_tiny_single_layer_end_to_end():
    b = synth.tiny_single_layer(R=4)
    s = b.sessions[0]
    S = b.S(0)
    r = oracle.step(b.k_pool, b.v_pool, S, b.M_of(0), b.q_dec[0], 2, s.R, s.pi, s.qs, s.qe, s.C, 0)
    st = r["sets"]
    assert r["n_keep"] == s.C and r["keep"][s.qs:s.qe].all()
    assert math.isclose(r["scores"][st["cand"]].sum(), 1 * 2 * s.R, rel_tol=1e-12)
    assert len(r["live"]) == s.C and len(r["freed"]) == s.N - s.C
    kept = np.nonzero(r["keep"])[0]
    o = oracle.decode(b.q_dec[0], b.k_pool, b.v_pool, S[kept])
    np.testing.assert_array_equal(o, r["out"])


def test_cross_attention_per_head_scale():
    """Head width 32 gives the scale 1/sqrt(32): a logit gap of sqrt(32) * ln 3 puts weight
    3/4 on the first query key (hand-worked: 0.75 * 4 + 0.25 * 8 = 5)."""
    D = 4
    W = {"W_K": np.zeros((128, D)), "b_K": np.zeros(128), "W_V": np.zeros((128, D)), "b_V": np.zeros(128)}
    W["W_K"][0, 0] = 1.0
    W["W_V"][:, 1] = 1.0
    kq = np.array([[1.0, 4.0, 0, 0], [0.0, 8.0, 0, 0]])
    Qc = np.zeros((1, 128))
    Qc[0, 0] = math.sqrt(32.0) * math.log(3.0)
    c = oracle.ikv_oracle.cross_attention(Qc, kq, W)
    np.testing.assert_allclose(c[0, :32], 5.0, rtol=1e-14)
    np.testing.assert_allclose(c[0, 32:], 6.0, rtol=1e-14)


# ============================================================================ Eqs. 4-6, hand-worked

def _hand_residual(b_K=0.7, b_V=0.5, b_Q=1.0, b_1=-1.0, b_2=0.25, alpha=1.0):
    """A residual head whose every output is worked out by hand (Sec. 3.3, Eqs. 4-6).

    Two layers, one KV head, one memory row, D = 4; positions 0 and 1 are the
    candidates, 2 and 3 the query span (the live cross-attention keys), 4 a dead
    query position whose sentinel row would dominate if it were read. Layer-1 rows
    are 3x layer-0 rows, so k-bar (the mean over layers) is 2x the layer-0 row:
        k-bar_0 = e0, k-bar_1 = e1, k-bar_2 = 2 e2, k-bar_3 = 2 e3.
    M = 0, so every row's softmax over the two candidates is uniform: rule = 1.
    Weights (all else zero): W_Q[0, 0] = 1 (one-hot: query channel 0 reads
    k-bar_j[0]), b_Q[0]; W_K[0, 2] = g = sqrt(32) ln 3 / 4, b_K[0]; W_V[0, 2] = 1,
    b_V[0]; W_1[0, 3D + 1] = 1 (hidden unit 0 reads c_j[0]), b_1[0]; w_2[0] = 1, b_2.
    Head 0 (channels 0..31, scale 1/sqrt(32)): the logit gap between query keys 2 and
    3 is Q_j[0] * 2g / sqrt(32) = Q_j[0] ln 3 / 2, with Q_j[0] = k-bar_j[0] + b_Q[0].
    """
    D = 4
    kb = np.array([[1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 2, 0], [0, 0, 0, 2]], dtype=np.float64)
    K = np.zeros((2, 6, 1, D), dtype=np.float32)          # pool [L][slots][Hkv][D]; slot 0 the sentinel
    K[0, 1:5, 0] = kb / 2
    K[1, 1:5, 0] = 3 * kb / 2
    K[:, 0, 0] = [0.0, 0.0, 50.0, 0.0]                     # read only if a dead query position leaked in
    S = np.array([1, 2, 3, 4, 0], dtype=np.int32)
    M = np.zeros((2, 1, D))
    st = oracle.sets(S, pi=0, qs=2, qe=4, C=3, dead=0)
    g = math.sqrt(32.0) * math.log(3.0) / 4.0
    blob = np.zeros(oracle.residual_param_count(D))
    WQ = np.zeros((128, 3 * D + 1))
    WQ[0, 0] = 1.0
    WK = np.zeros((128, D))
    WK[0, 2] = g
    WV = np.zeros((128, D))
    WV[0, 2] = 1.0
    W1 = np.zeros((256, 3 * D + 1 + 128))
    W1[0, 3 * D + 1] = 1.0
    vec = lambda i, x, n: np.eye(n)[i] * x                 # noqa: E731
    for name, val in (("W_Q", WQ), ("b_Q", vec(0, b_Q, 128)), ("W_K", WK), ("b_K", vec(0, b_K, 128)),
                      ("W_V", WV), ("b_V", vec(0, b_V, 128)), ("W_1", W1), ("b_1", vec(0, b_1, 256)),
                      ("w_2", vec(0, 1.0, 256)), ("b_2", [b_2]), ("alpha", [alpha])):
        _set_block(blob, D, name, val)
    s = oracle.scores(K, S, st, M, 1, 1, blob, oracle.FLAG_RESIDUAL, np.array([2, 3, 4]), 0)
    return s, st


def _gelu_hand(x):
    return 0.5 * x * (1.0 + math.erf(x / math.sqrt(2.0)))


def test_residual_hand_worked_two_query_keys():
    """Candidate 0: Q = 1 + 1 = 2, gap ln 3: weights (3/4, 1/4) on V'[0] = (2.5, 0.5), so
    c_0[0] = 2 and s_0 = 1 + GELU(2 - 1) + 0.25. Candidate 1: Q = 0 + 1 = 1, gap ln 3 / 2:
    weights (sqrt3, 1) / (1 + sqrt3), c_1[0] = (2.5 sqrt3 + 0.5) / (1 + sqrt3)."""
    s, st = _hand_residual()
    assert np.nonzero(st["cand"])[0].tolist() == [0, 1]
    r3 = math.sqrt(3.0)
    c1 = (2.5 * r3 + 0.5) / (1.0 + r3)
    assert math.isclose(c1, 1.7679491924311228, rel_tol=1e-15)
    assert math.isclose(s[0], 1.0 + 0.8413447460685429 + 0.25, rel_tol=1e-14)      # GELU(1) = Phi(1)
    assert math.isclose(s[0], 2.091344746068543, rel_tol=1e-14)
    assert math.isclose(s[1], 1.0 + _gelu_hand(c1 - 1.0) + 0.25, rel_tol=1e-14)
    assert math.isclose(s[1], 1.8480337638176736, rel_tol=1e-13)
    assert np.all(np.isneginf(s[2:]))


@pytest.mark.parametrize("kw,want", [
    # b_Q = 0: both candidates see Q = k-bar_j[0]: candidate 0 the ln 3 / 2 gap, candidate 1 a uniform mix
    (dict(b_Q=0.0), (1.25 + _gelu_hand((2.5 * math.sqrt(3) + 0.5) / (1 + math.sqrt(3)) - 1), 1.25 + _gelu_hand(0.5))),
    # b_V = 0: V'[0] = (2, 0): c_0[0] = 1.5, c_1[0] = 2 sqrt3 / (1 + sqrt3)
    (dict(b_V=0.0), (1.25 + _gelu_hand(0.5), 1.25 + _gelu_hand(2 * math.sqrt(3) / (1 + math.sqrt(3)) - 1))),
    # b_1 = 0: the hidden unit sees c_j[0] itself
    (dict(b_1=0.0), (1.25 + _gelu_hand(2.0), 1.25 + _gelu_hand((2.5 * math.sqrt(3) + 0.5) / (1 + math.sqrt(3))))),
    # b_2 = -1 and alpha = -2: s = rule - 2 (GELU(c - 1) - 1)
    (dict(b_2=-1.0, alpha=-2.0), (1.0 - 2 * (_gelu_hand(1.0) - 1.0),
                                  1.0 - 2 * (_gelu_hand((2.5 * math.sqrt(3) + 0.5) / (1 + math.sqrt(3)) - 1) - 1.0))),
])
def test_residual_hand_worked_biases(kw, want):
    s, _ = _hand_residual(**kw)
    np.testing.assert_allclose(s[:2], want, rtol=1e-14)


def test_residual_key_bias_cancels_in_the_softmax():
    """b_K adds Q_j . b_K / sqrt(32) to every logit of candidate j alike, so the softmax
    over the query keys, and hence every score, does not depend on it."""
    a, _ = _hand_residual(b_K=0.7)
    b, _ = _hand_residual(b_K=-13.0)
    np.testing.assert_allclose(a, b, rtol=1e-14)


def test_gate_counts_dead_positions():
    """Appendix H skips the event when N <= C with N counting dead positions too. With
    N > C but only C live positions the event still runs: candidates are scored and
    every live one is kept, the threshold being the lowest candidate score."""
    rng = np.random.default_rng(18)
    L, N, Hkv, D, R = 1, 12, 1, 4, 2
    pool, S = rand_pool(rng, L, N, Hkv, D)
    S[[1, 4, 6]] = 0                                    # 9 live positions, N = 12
    M = rng.standard_normal((L, Hkv * R, D))
    st = oracle.sets(S, 0, 10, 12, C=9, dead=0)
    assert not st["skip"] and st["Cstar"] == 7 and int(st["cand"].sum()) == 7
    s = oracle.scores(pool, S, st, M, Hkv, R)
    assert np.all(np.isfinite(s[st["cand"]]))
    keep, n_keep, tau = oracle.select_budget(s, st)
    assert np.array_equal(keep, st["live"]) and n_keep == 9 and tau == s[st["cand"]].min()
    st12 = oracle.sets(S, 0, 10, 12, C=12, dead=0)
    assert st12["skip"] and np.all(np.isneginf(oracle.scores(pool, S, st12, M, Hkv, R)))


# ============================================================================ baseline scorers (Sec. 4.1)

def test_max_pool_hand():
    v = np.array([0, 3, 1, 0, 0, 0, 0, 0, 5, 2], dtype=np.float64)
    np.testing.assert_array_equal(oracle.ikv_oracle.max_pool(v, 7), [3, 3, 3, 3, 3, 5, 5, 5, 5, 5])
    np.testing.assert_array_equal(oracle.ikv_oracle.max_pool(v, 3), [3, 3, 3, 1, 0, 0, 0, 5, 5, 5])
    np.testing.assert_array_equal(oracle.ikv_oracle.max_pool(v, 1), v)


def _one_row_pool(x):
    """One layer, one KV head, one query head, one query row q = e0, D = 4: the logit of
    position i is x_i by construction (K_i = 2 x_i e0, scale 1/sqrt(4))."""
    N = len(x)
    K = np.zeros((1, N, 1, 4), np.float32)
    K[0, :, 0, 0] = 2 * np.asarray(x)
    S = np.arange(1, N + 1, dtype=np.int32)
    pool = pool_from_logical(K, S, N + 1)
    q = np.zeros((1, 1, 1, 4), np.float32)
    q[0, 0, 0, 0] = 1.0
    return pool, S, q


def test_snapkv_hand_worked():
    """Logits (ln 4, 0, 0, 0, 0, ln 2, 0, 0, 0, 0): softmax weights (4,1,1,1,1,2,1,1,1,1)/14,
    max-pooled over 7 positions: (4,4,4,4,2,2,2,2,2,1)/14. The keys are float32, so the
    logits carry the float32 rounding of ln 2 (relative 1e-8 in the weights)."""
    ln2 = math.log(2.0)
    x = [2 * ln2, 0, 0, 0, 0, ln2, 0, 0, 0, 0]
    pool, S, q = _one_row_pool(x)
    st = oracle.sets(S, 0, 10, 10, 0, 0)                  # no forced positions, C = 0: every position scored
    np.testing.assert_allclose(oracle.ikv_oracle.snapkv_scores(pool, S, st, q, 1),
                               np.array([4, 4, 4, 4, 2, 2, 2, 2, 2, 1]) / 14.0, rtol=1e-7)
    np.testing.assert_allclose(oracle.ikv_oracle.h2o_scores(pool, S, st, q, 1),
                               np.array([4, 1, 1, 1, 1, 2, 1, 1, 1, 1]) / 14.0, rtol=1e-7)
    # position 0 forced: out of the softmax, zero mass in the pool windows; weights
    # (1,1,1,1,2,1,1,1,1)/10 on positions 1..9, position 5's 2/10 reaching positions 2..8
    st_f = oracle.sets(S, 1, 10, 10, 0, 0)
    s = oracle.ikv_oracle.snapkv_scores(pool, S, st_f, q, 1)
    assert s[0] == -math.inf
    np.testing.assert_allclose(s[1:], np.array([1, 2, 2, 2, 2, 2, 2, 2, 1]) / 10.0, rtol=1e-7)


def _baseline_case(seed, L=2, N=40, Hkv=2, G=3, D=8, n=5):
    rng = np.random.default_rng(seed)
    pool, S = rand_pool(rng, L, N, Hkv, D)
    S[rng.choice(N, 6, replace=False)] = 0
    q = rng.standard_normal((L, Hkv * G, n, D)).astype(np.float32)
    st = oracle.sets(S, 2, N - 4, N, 10, 0)
    return pool, S, q, st


def test_attention_mass_closed_form_and_brute_force():
    pool, S, q, st = _baseline_case(21)
    L, Hq, n, D = q.shape
    Hkv = 2
    v = oracle.ikv_oracle.attention_mass(pool, S, st["cand"], q, Hkv)
    # every query row's softmax sums to one: each KV head collects G * n, the total L * Hq * n
    np.testing.assert_allclose(v.sum(axis=2), (Hq // Hkv) * n, rtol=1e-13)
    assert np.all(v[:, :, ~st["cand"]] == 0)
    cand = np.nonzero(st["cand"])[0]
    for l in range(L):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            for t in range(n):
                logit = {i: float(q[l, h, t].astype(np.float64) @ pool[l, S[i], g].astype(np.float64)) / math.sqrt(D)
                         for i in cand}
                den = sum(math.exp(x) for x in logit.values())
                for i in cand[:3]:
                    v[l, g, i] -= math.exp(logit[i]) / den
    assert np.abs(v[:, :, cand[:3]]).max() < 1e-12


def test_snapkv_pool_bounds_and_kernel_one():
    pool, S, q, st = _baseline_case(22)
    h2o = oracle.ikv_oracle.h2o_scores(pool, S, st, q, 2)
    np.testing.assert_array_equal(oracle.ikv_oracle.snapkv_scores(pool, S, st, q, 2, kernel=1), h2o)
    snap = oracle.ikv_oracle.snapkv_scores(pool, S, st, q, 2)
    c = st["cand"]
    assert np.all(snap[c] >= h2o[c]) and np.all(np.isneginf(snap[~c]))
    # the pooled sum is at most the sum of the per-unit maxima over each window
    v = oracle.ikv_oracle.attention_mass(pool, S, c, q, 2)
    j = int(np.nonzero(c)[0][5])
    lo, hi = max(0, j - 3), j + 4
    assert math.isclose(snap[j], v[:, :, lo:hi].max(axis=2).sum(), rel_tol=1e-13)


def test_recent_window_hand():
    assert oracle.ikv_oracle.recent_window(32768, 8192, 0.5) == (32768 - 4096, 32768)
    assert oracle.ikv_oracle.recent_window(100, 8192, 0.5) == (0, 100)
    assert oracle.ikv_oracle.recent_window(1000, 301, 0.5) == (849, 1000)


# ============================================================================ compact apply path (Sec. 3.4, Table 7)

def test_rope_rotate_hand():
    """D = 4, base 1e4: the pairs (0, 2) and (1, 3) turn by delta and delta / 100."""
    x = np.array([1.0, 0.0, 0.0, 2.0])
    y = oracle.ikv_oracle.rope_rotate(x, -2, 1.0e4, 4)
    np.testing.assert_allclose(y, [math.cos(2.0), -2 * math.sin(-0.02), -math.sin(2.0), 2 * math.cos(0.02)],
                               rtol=0, atol=1e-15)
    np.testing.assert_array_equal(oracle.ikv_oracle.rope_rotate(x, 0, 1.0e4, 4), x)


def test_rope_rotate_composes_with_the_generator_rope():
    """A key rotated at position j (the input generator's own RoPE) and re-rotated by
    t - j equals the key rotated at t."""
    rng = np.random.default_rng(30)
    D = 128
    x = rng.standard_normal((5, D))
    j, t = np.array([700, 91000, 33, 5000, 12]), np.array([3, 8191, 33, 77, 0])
    a = synth.rope_neox(x, *synth.rope_cos_sin(j, D))
    b = synth.rope_neox(x, *synth.rope_cos_sin(t, D))
    for k in range(5):
        np.testing.assert_allclose(oracle.ikv_oracle.rope_rotate(a[k], t[k] - j[k], synth.ROPE_BASE, D), b[k],
                                   rtol=0, atol=1e-9)


def test_compact_apply_order_values_and_norms():
    rng = np.random.default_rng(31)
    L, N, Hkv, D = 2, 30, 2, 8
    kp, S = rand_pool(rng, L, N, Hkv, D)
    vp, _ = rand_pool(rng, L, N, Hkv, D)
    vp = vp[:, :]                                            # values by the same slots
    keep = rng.random(N) < 0.4
    keep[3] = True
    dst = np.arange(100, 100 + N, dtype=np.int32)
    Kn, Vn, Sn = oracle.ikv_oracle.compact_apply(kp, vp, S, keep, dst, 1.0e4)
    kept = np.nonzero(keep)[0]
    assert len(Sn) == len(kept) and np.array_equal(Sn, dst[:len(kept)])
    np.testing.assert_array_equal(Vn, vp[:, S[kept]].astype(np.float64))          # values move unchanged
    np.testing.assert_allclose(np.linalg.norm(Kn, axis=-1),                       # rotations keep norms
                               np.linalg.norm(kp[:, S[kept]].astype(np.float64), axis=-1), rtol=1e-13)
    t0 = int(np.nonzero(kept == 3)[0][0])
    np.testing.assert_allclose(Kn[:, t0], oracle.ikv_oracle.rope_rotate(kp[:, S[3]], t0 - 3, 1.0e4, D), rtol=0,
                               atol=1e-15)
    # everything kept: no position moves, every key stays as it was
    Kall, _, _ = oracle.ikv_oracle.compact_apply(kp, vp, S, np.ones(N, bool), dst, 1.0e4)
    np.testing.assert_array_equal(Kall, kp[:, S].astype(np.float64))


# ============================================================================ span prefill (Sec. 3.5)

def test_prefill_attention_causal_brute_force():
    rng = np.random.default_rng(40)
    L, Hq, Hkv, D, n = 2, 4, 2, 4, 3
    kp = rng.standard_normal((L, 12, Hkv, D)).astype(np.float32)
    vp = rng.standard_normal((L, 12, Hkv, D)).astype(np.float32)
    q = rng.standard_normal((L, Hq, n, D)).astype(np.float32)
    hist, span = [5, 1, 9], [2, 7, 11]
    o = oracle.ikv_oracle.prefill_attention(q, kp, vp, hist, span)
    for l in range(L):
        for h in range(Hq):
            g = h // 2
            for t in range(n):
                slots = hist + span[:t + 1]
                xs = [sum(float(q[l, h, t, d]) * float(kp[l, u, g, d]) for d in range(D)) / 2.0 for u in slots]
                ws = [math.exp(x) for x in xs]
                for d in range(D):
                    ref = sum(w * float(vp[l, u, g, d]) for w, u in zip(ws, slots)) / sum(ws)
                    assert math.isclose(o[l, h, t, d], ref, rel_tol=1e-12, abs_tol=1e-14)


def test_prefill_attention_reduces_to_decode():
    """One span token attends over the history and itself: the decode of that query over
    the history slots followed by its own slot."""
    rng = np.random.default_rng(41)
    L, Hq, Hkv, D = 2, 8, 2, 16
    kp = rng.standard_normal((L, 40, Hkv, D)).astype(np.float32)
    vp = rng.standard_normal((L, 40, Hkv, D)).astype(np.float32)
    q = rng.standard_normal((L, Hq, 1, D)).astype(np.float32)
    hist = [3, 17, 8, 30, 22]
    o = oracle.ikv_oracle.prefill_attention(q, kp, vp, hist, [39])
    np.testing.assert_allclose(o[:, :, 0], oracle.decode(q[:, :, 0], kp, vp, hist + [39]), rtol=1e-13, atol=1e-15)
    # the first span token of a longer span sees only its own span key
    o2 = oracle.ikv_oracle.prefill_attention(np.repeat(q, 3, axis=2), kp, vp, hist, [39, 4, 5])
    np.testing.assert_allclose(o2[:, :, 0], o[:, :, 0], rtol=1e-13, atol=1e-15)
