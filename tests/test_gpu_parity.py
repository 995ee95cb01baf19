"""HIP path vs the float64 oracle, call by call and end to end, through the C ABI.

Inputs come from the seeded generator; expected values come from the oracle only.
Where several results are correct (kept-set members whose score lies within the
selection band of the threshold), the unique parts are compared and the rest is
checked for validity.
"""
import math

import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import (RESID_MFMA_FLOOR, SCORE_FLOOR, band_positions, check_attention, check_decode_on, check_keep,
                    check_scores, check_xattn_visible, oracle_scores_pair)

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def sess_sets(batch, b, S=None):
    s = batch.sessions[b]
    S = batch.S(b) if S is None else S
    return oracle.sets(S, s.pi, s.qs, s.qe, s.C, synth.DEAD_SLOT)


def seg(arr, batch, b):
    o = int(batch.slot_off[b])
    return arr[o:o + batch.sessions[b].N]


def oracle_scores(batch, b, blob=None, flags=0, M=None, S=None):
    s = batch.sessions[b]
    S = batch.S(b) if S is None else S
    M = batch.M_of(b) if M is None else M
    st = sess_sets(batch, b, S)
    return oracle.scores(batch.k_pool, S, st, M, batch.shape.Hkv, s.R, blob, flags,
                         batch.qpos_of(b), synth.DEAD_SLOT), st


def tiny_bf16(R=16, seed=11):
    N = 2048
    s = synth.SessionSpec(N=N, C=512, pi=0, qs=N - 32, qe=N, R=R)
    return synth.make_batch(synth.tiny_shape(), [s], seed=seed, kv_dtype=synth.BF16, layout="paged")


# ============================================================================ sentinel

@pytest.mark.parametrize("kind", ["f32", "bf16"])
def test_init_dead_slot(dev, kind):
    batch = synth.tiny_single_layer() if kind == "f32" else tiny_bf16()
    st = RetentionStep(batch, dev)
    st.init_dead_slot()
    k, v = st.host("k_pool"), st.host("v_pool")
    kw = synth.widen(k[:, 0])
    assert np.all(kw == (-1.0e4 if kind == "f32" else -9984.0))
    assert np.all(synth.widen(v[:, 0]) == 0)
    assert np.array_equal(k[:, 1:], batch.k_pool[:, 1:]) and np.array_equal(v[:, 1:], batch.v_pool[:, 1:])


# ============================================================================ Eq. 2

@pytest.mark.parametrize("kind,lam", [("f32", 0.5), ("bf16", 0.5), ("f32", math.inf)])
def test_qm_update(dev, kind, lam):
    batch = synth.tiny_single_layer() if kind == "f32" else tiny_bf16()
    st = RetentionStep(batch, dev)
    st.qm_update(lam)
    got = st.host("M").reshape(batch.M_of(0).shape)
    want = oracle.qm_update(batch.M_of(0), batch.q_span_of(0), lam)
    np.testing.assert_allclose(got, want, rtol=0, atol=2e-6)
    st.qm_update(lam)                                  # a second turn on the updated memory
    want2 = oracle.qm_update(want, batch.q_span_of(0), lam)
    np.testing.assert_allclose(st.host("M").reshape(want.shape), want2, rtol=0, atol=4e-6)


# ============================================================================ Eq. 3

@pytest.mark.parametrize("layout,R,dead_frac", [("identity", 16, 0.0), ("shuffled", 16, 0.2), ("identity", 4, 0.0),
                                                ("shuffled", 7, 0.5)])
def test_rule_scores_tiny(dev, layout, R, dead_frac):
    batch = synth.tiny_single_layer(R=R, layout=layout, dead_frac=dead_frac)
    st = RetentionStep(batch, dev)
    st.init_dead_slot()
    st.score(flags=0)
    want, sets = oracle_scores(batch, 0)
    rel = check_scores(st.host("scores"), want, sets["cand"])
    assert rel < 1e-5, rel
    assert math.isclose(float(st.host("scores")[sets["cand"]].astype(np.float64).sum()), 2 * R, rel_tol=1e-5)


def test_rule_scores_bf16_tiny(dev):
    batch = tiny_bf16(R=32)
    st = RetentionStep(batch, dev)
    st.score(flags=0)
    want, sets = oracle_scores(batch, 0)
    assert check_scores(st.host("scores"), want, sets["cand"]) < 1e-5


def small_d128(R=64, N=1000, seed=31, dead_frac=0.1, C=300, L=2, Hkv=2, G=4):
    s = synth.SessionSpec(N=N, C=min(C, N // 3), pi=4, qs=N - 16, qe=N, R=R, dead_frac=dead_frac)
    return synth.make_batch(synth.Shape(L=L, Hq=Hkv * G, Hkv=Hkv, D=128), [s], seed=seed, kv_dtype=synth.BF16,
                            layout="paged")


@pytest.mark.parametrize("R,N", [(16, 1000), (48, 777), (64, 1000), (80, 333), (96, 900), (112, 1500), (128, 1280),
                                 (64, 129), (1, 500), (4, 640), (33, 777), (47, 1000), (63, 300), (65, 700),
                                 (100, 900), (127, 1280), (150, 600), (256, 300)])
def test_rule_scores_d128_matrix_cores(dev, R, N):
    """Head dimension 128, bf16 pool: the MFMA score passes, for any R (the last 16-row
    slice of memory rows padded), including R > 128 (split rows and the four-wave passes)."""
    batch = small_d128(R=R, N=N, seed=R + N)
    st = RetentionStep(batch, dev)
    st.init_dead_slot()
    st.score(flags=0)
    want, sets = oracle_scores(batch, 0)
    rel = check_scores(st.host("scores"), want, sets["cand"])
    assert rel < 1e-5, rel
    st.select()
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, sets["cand"])


@pytest.mark.parametrize("R,N,Hkv,flags", [(64, 1000, 3, 0), (16, 700, 1, 0), (48, 1300, 3, ikv.IKV_RESIDUAL),
                                            (96, 800, 3, ikv.IKV_RESIDUAL), (37, 900, 3, ikv.IKV_RESIDUAL),
                                            (90, 700, 1, 0), (140, 500, 3, 0)])
def test_scores_d128_odd_kv_heads(dev, R, N, Hkv, flags):
    """An odd number of KV heads: the first pass runs position-major over all units
    (64-position partials), the second pass as for even Hkv."""
    batch = small_d128(R=R, N=N, seed=3 * R + N, L=3, Hkv=Hkv, G=2)
    blob = synth.residual_blob(128, seed=R) if flags else None
    st = RetentionStep(batch, dev, residual=blob, flags=flags)
    st.init_dead_slot()
    st.score(flags=flags)
    want, sets = oracle_scores(batch, 0, blob, flags)
    rel = check_scores(st.host("scores"), want, sets["cand"], floor=RESID_MFMA_FLOOR if flags else SCORE_FLOOR)
    assert rel < 1e-5, rel
    st.select()
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, sets["cand"])


@pytest.mark.parametrize("R,flags,nq", [(16, ikv.IKV_RESIDUAL, 16), (64, ikv.IKV_RESIDUAL, 16),
                                        (64, ikv.IKV_RESIDUAL | ikv.IKV_NO_XATTN, 16),
                                        (32, ikv.IKV_RESIDUAL, 64), (48, ikv.IKV_RESIDUAL, 100),
                                        (128, ikv.IKV_RESIDUAL, 16)])
def test_residual_scores_d128_matrix_cores(dev, R, flags, nq):
    """Residual head at D = 128: on the matrix cores up to 64 live query positions,
    on the vector units beyond."""
    batch = small_d128(R=R, N=1500, seed=40 + R, dead_frac=0.05)
    s = batch.sessions[0]
    s.qpos = np.arange(s.N - nq, s.N, dtype=np.int32)
    batch.qpos = s.qpos.copy()
    blob = synth.residual_blob(128, seed=R)
    st = RetentionStep(batch, dev, residual=blob, flags=flags)
    st.score()
    want, sets = oracle_scores(batch, 0, blob, flags)
    # up to 64 live query rows the head runs on the matrix cores, beyond on the vector units
    rel = check_scores(st.host("scores"), want, sets["cand"], floor=RESID_MFMA_FLOOR if nq <= 64 else SCORE_FLOOR)
    print(f"max scale-aware relative score error {rel:.2e}")
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    st.select()
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, sets["cand"])


def test_zero_initialised_head_is_bitwise_the_rule_d128(dev):
    batch = small_d128(R=64, N=1200, seed=77)
    st = RetentionStep(batch, dev, residual=synth.residual_blob(128, seed=3, variant="zero"),
                       flags=ikv.IKV_RESIDUAL)
    st.score()
    with_head = st.host("scores").copy()
    st.score(flags=0)
    assert np.array_equal(with_head, st.host("scores"))


def test_step_batched_d128_matrix_cores(dev):
    shape = synth.Shape(L=3, Hq=10, Hkv=2, D=128)
    sessions = [synth.SessionSpec(N=900, C=200, pi=8, qs=880, qe=900, R=16, dead_frac=0.1),
                synth.SessionSpec(N=2000, C=500, pi=0, qs=1950, qe=2000, R=48),
                synth.SessionSpec(N=150, C=400, pi=0, qs=140, qe=150, R=32),
                synth.SessionSpec(N=1300, C=100, pi=16, qs=1240, qe=1300, R=64, radix_prefix=16)]
    batch = synth.make_batch(shape, sessions, seed=41, kv_dtype=synth.BF16, layout="paged", spare_pages=3)
    blob = synth.residual_blob(128, seed=42)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    for b in range(len(sessions)):
        _compare_step(st, batch, b, blob, ikv.IKV_RESIDUAL, True)


def test_step_batched_d128_mixed_row_counts(dev):
    """Sessions of up to 64 and of more memory rows in one batch: each score pass runs
    one launch per kind, and each launch skips the other kind's sessions. One session is
    at its budget (skipped), others carry dead positions, a forced prefix and a
    protected radix prefix."""
    shape = synth.Shape(L=2, Hq=8, Hkv=2, D=128)
    sessions = [synth.SessionSpec(N=1100, C=300, pi=8, qs=1080, qe=1100, R=96, dead_frac=0.1),
                synth.SessionSpec(N=700, C=200, pi=0, qs=650, qe=700, R=32),
                synth.SessionSpec(N=400, C=400, pi=0, qs=380, qe=400, R=128),
                synth.SessionSpec(N=1500, C=150, pi=16, qs=1440, qe=1500, R=128, radix_prefix=16),
                synth.SessionSpec(N=900, C=500, pi=0, qs=860, qe=900, R=16, dead_frac=0.2)]
    batch = synth.make_batch(shape, sessions, seed=43, kv_dtype=synth.BF16, layout="paged", spare_pages=4)
    blob = synth.residual_blob(128, seed=44)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    for b in range(len(sessions)):
        _compare_step(st, batch, b, blob, ikv.IKV_RESIDUAL, True)


def test_step_batched_d128_residual_setup_edges(dev):
    """The residual head's set-up, fold and K', V' on the matrix-core path, at its edges:
    session 0 at its budget (its workgroups write only the weights every session shares),
    query lists holding dead positions (the live ones keep their list order), a list
    with no live position (no cross-attention), and one with exactly 64 live positions
    (every key row of the fragments)."""
    shape = synth.Shape(L=2, Hq=8, Hkv=2, D=128)
    specs = [synth.SessionSpec(N=300, C=300, pi=0, qs=280, qe=300, R=32),
             synth.SessionSpec(N=1200, C=300, pi=0, qs=1180, qe=1200, R=64, dead_frac=0.3,
                               qpos=np.zeros(48, np.int32)),
             synth.SessionSpec(N=900, C=200, pi=0, qs=890, qe=900, R=16, dead_frac=0.3,
                               qpos=np.zeros(12, np.int32)),
             synth.SessionSpec(N=1000, C=250, pi=0, qs=936, qe=1000, R=48)]
    batch = synth.make_batch(shape, specs, seed=47, kv_dtype=synth.BF16, layout="paged", spare_pages=2)
    dead = [np.flatnonzero(batch.S(b) == synth.DEAD_SLOT) for b in range(len(specs))]
    live = [np.flatnonzero(batch.S(b) != synth.DEAD_SLOT) for b in range(len(specs))]
    rng = np.random.default_rng(48)
    # session 1: 24 dead and 24 live history positions, shuffled; session 2: dead only
    q1 = np.concatenate([rng.choice(dead[1], 24, replace=False), rng.choice(live[1][:1000], 24, replace=False)])
    rng.shuffle(q1)
    q2 = rng.choice(dead[2], 12, replace=False)
    for b, q in ((1, q1), (2, q2)):
        specs[b].qpos = q.astype(np.int32)
        o = int(batch.qpos_off[b])
        batch.qpos[o:o + len(q)] = q
    blob = synth.residual_blob(128, seed=49)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=False)
    for b in range(len(specs)):
        _compare_step(st, batch, b, blob, ikv.IKV_RESIDUAL, False)


# ============================================================================ Eqs. 4-6

@pytest.mark.parametrize("variant,flags", [("random", ikv.IKV_RESIDUAL), ("random", ikv.IKV_RESIDUAL | ikv.IKV_NO_XATTN),
                                           ("alpha7", ikv.IKV_RESIDUAL)])
def test_residual_scores_tiny(dev, variant, flags):
    batch = synth.tiny_single_layer(R=16, layout="shuffled")
    blob = synth.residual_blob(64, seed=5, variant="random", alpha=7.0 if variant == "alpha7" else 1.0)
    st = RetentionStep(batch, dev, residual=blob, flags=flags)
    st.score()
    want, sets = oracle_scores(batch, 0, blob, flags)
    rel = check_scores(st.host("scores"), want, sets["cand"])
    print(f"max scale-aware relative score error {rel:.2e}")


def test_zero_initialised_head_is_bitwise_the_rule(dev):
    batch = synth.tiny_single_layer(R=16)
    blob = synth.residual_blob(64, seed=6, variant="zero")
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.score()
    with_head = st.host("scores").copy()
    st.score(flags=0)
    assert np.array_equal(with_head, st.host("scores"))
    blob0 = synth.residual_blob(64, seed=6, variant="random", alpha=0.0)
    st0 = RetentionStep(batch, dev, residual=blob0, flags=ikv.IKV_RESIDUAL)
    st0.score()
    assert np.array_equal(st0.host("scores"), with_head)


def test_residual_without_live_query_positions(dev):
    batch = synth.tiny_single_layer(R=8)
    s = batch.sessions[0]
    s.qpos = np.array([10, 20, 30], dtype=np.int32)
    batch.qpos = s.qpos.copy()
    batch.slot_maps[[10, 20, 30]] = synth.DEAD_SLOT
    blob = synth.residual_blob(64, seed=7)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.score()
    want, sets = oracle_scores(batch, 0, blob, ikv.IKV_RESIDUAL)
    check_scores(st.host("scores"), want, sets["cand"])
    st.score(flags=ikv.IKV_RESIDUAL | ikv.IKV_NO_XATTN)
    want2, _ = oracle_scores(batch, 0, blob, ikv.IKV_RESIDUAL | ikv.IKV_NO_XATTN)
    np.testing.assert_array_equal(want, want2)
    check_scores(st.host("scores"), want2, sets["cand"])


# ============================================================================ Eq. 1

@pytest.mark.parametrize("C,pi", [(512, 0), (300, 40), (60, 50), (10, 40), (2000, 0), (2048, 0), (5000, 0)])
def test_select_isolated_exact(dev, C, pi):
    torch = _torch()
    batch = synth.tiny_single_layer(R=4, layout="shuffled", dead_frac=0.1)
    s = batch.sessions[0]
    s.C, s.pi = C, pi
    st = RetentionStep(batch, dev)
    sc = synth.score_vector(s.N, seed=C + pi)
    st.scores.copy_(torch.from_numpy(sc).to(dev))
    st.select()
    sets = sess_sets(batch, 0)
    keep_o, n_o, tau_o = oracle.select_budget(sc.astype(np.float64), sets)
    assert np.array_equal(st.host("keep").astype(bool), keep_o)
    assert int(st.host("n_keep")[0]) == n_o
    tau = float(st.host("tau")[0])
    assert tau == tau_o or (math.isnan(tau) and math.isnan(tau_o))


def test_select_on_scores_tiny(dev):
    batch = synth.tiny_single_layer(R=16, layout="shuffled", dead_frac=0.1)
    blob = synth.residual_blob(64, seed=8)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.score()
    st.select()
    want, sets = oracle_scores(batch, 0, blob, ikv.IKV_RESIDUAL)
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, sets["cand"])
    assert math.isclose(float(st.host("tau")[0]), tau_o, rel_tol=1e-5)


# ============================================================================ Eq. 7

@pytest.mark.parametrize("radix,aliases", [(0, 0), (100, 0), (300, 40)])
def test_redirect_isolated_exact(dev, radix, aliases):
    torch = _torch()
    batch = synth.tiny_single_layer(R=4, layout="shuffled", dead_frac=0.15)
    s = batch.sessions[0]
    s.radix_prefix = radix
    S = batch.S(0)
    if aliases:
        S = synth.alias_slots(S, seed=radix, pairs=aliases)
        batch.slot_maps[:] = S
    keep = synth.keep_mask(S, seed=radix + 1)
    st = RetentionStep(batch, dev)
    st.keep.copy_(torch.from_numpy(keep).to(dev))
    k_before = st.host("k_pool").copy()
    st.redirect()
    S_o, freed_o, live_o = oracle.redirect(S, keep.astype(bool), synth.DEAD_SLOT, radix)
    assert np.array_equal(st.host("S"), S_o)
    nf, nl = int(st.host("n_freed")[0]), int(st.host("n_live")[0])
    assert np.array_equal(st.host("freed")[:nf], freed_o)
    assert np.array_equal(st.host("live")[:nl], live_o)
    assert np.array_equal(st.host("k_pool"), k_before)          # no K/V row moves


# ============================================================================ decode

@pytest.mark.parametrize("kind,frac", [("f32", 0.25), ("bf16", 0.25), ("f32", 0.0005), ("bf16", 1.0)])
def test_decode_isolated(dev, kind, frac):
    torch = _torch()
    batch = synth.tiny_single_layer() if kind == "f32" else tiny_bf16()
    S = batch.S(0)
    keep = synth.keep_mask(S, seed=3, frac=frac)
    live = S[keep.astype(bool)].astype(np.int32)
    st = RetentionStep(batch, dev)
    st.live[:len(live)].copy_(torch.from_numpy(live).to(dev))
    st.n_live.fill_(len(live))
    st.decode()
    want = oracle.decode(batch.q_dec[0], batch.k_pool, batch.v_pool, live)
    got = synth.widen(st.host("out")[0])
    check_attention(got, want, bf16=(kind == "bf16"))


@pytest.mark.parametrize("Hkv,G,n_live", [(1, 1, 700), (2, 2, 129), (3, 3, 64), (4, 4, 1000), (8, 5, 300),
                                          (2, 6, 513), (4, 7, 77), (8, 8, 2100), (4, 4, 3), (8, 8, 1),
                                          (4, 4, 640)])
def test_decode_heads_kernel_variants(dev, Hkv, G, n_live):
    """bf16 pool, D = 128: the head-group decode with one, two or four KV heads per
    workgroup (Hkv odd, 2 mod 4, 0 mod 4), G from 1 to 8 (halves of 32 live slots up to
    G = 4, of 16 above), against the oracle. The live bound of these sessions is 300, so
    the lists are split five ways: splits that end inside a half or on a pair boundary
    (640: two whole pairs each), splits shorter than a half, empty splits (3 and 1 live
    rows), and lists longer than the bound (513, 1000, 2100)."""
    torch = _torch()
    batch = small_d128(R=16, N=max(2400, n_live + 100), seed=7 * Hkv + G, dead_frac=0.0, L=2, Hkv=Hkv, G=G)
    S = batch.S(0)
    live = S[synth.stream(8, synth.T_MISC_KEEP, Hkv * 16 + G).permutation(len(S))[:n_live]].astype(np.int32)
    st = RetentionStep(batch, dev)
    st.init_dead_slot()
    st.live[:len(live)].copy_(torch.from_numpy(live).to(dev))
    st.n_live.fill_(len(live))
    st.decode()
    want = oracle.decode(batch.q_dec[0], batch.k_pool, batch.v_pool, live)
    check_attention(synth.widen(st.host("out")[0]), want, bf16=True)


def test_decode_empty_live_list(dev):
    batch = synth.tiny_single_layer()
    st = RetentionStep(batch, dev)
    st.n_live.fill_(0)
    st.decode()
    assert np.all(st.host("out") == 0)


# ============================================================================ whole step

def _compare_step(st, batch, b, blob, flags, update_memory, xattn_check=False):
    """One session of a step against the oracle. The kept set must match outside the
    selection band; the slot map, freed and live lists then follow from it. Decode is
    always checked against the oracle's attention over the GPU's own live list (a valid
    answer whenever the kept set is), and against the oracle's list when the kept sets
    agree. With `xattn_check` the residual head's cross-attention must also visibly
    move the scores and the kept set (Sec. 3.3, Eq. 6), so that the comparison sees it."""
    s = batch.sessions[b]
    M = oracle.qm_update(batch.M_of(b), batch.q_span_of(b)) if update_memory else batch.M_of(b)
    if update_memory:
        np.testing.assert_allclose(seg_M(st, batch, b), M, atol=4e-6, rtol=0)
    if xattn_check:
        sets = sess_sets(batch, b)
        want, nox = oracle_scores_pair(batch.k_pool, batch.S(b), sets, M, batch.shape.Hkv, s.R, blob,
                                       batch.qpos_of(b), synth.DEAD_SLOT)
        ratio, nd = check_xattn_visible(want, nox, sets)
        print(f"cross-attention: moves scores by up to {ratio:.1f}x the tolerance, {nd} kept positions")
    else:
        want, sets = oracle_scores(batch, b, blob, flags, M=M)
    if sets["skip"]:
        assert np.all(np.isneginf(seg(st.host("scores"), batch, b)))
    else:
        mfma_head = (flags & ikv.IKV_RESIDUAL) and batch.shape.D == 128 and batch.kv_dtype == synth.BF16
        check_scores(seg(st.host("scores"), batch, b), want, sets["cand"],
                     floor=RESID_MFMA_FLOOR if mfma_head else SCORE_FLOOR)
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    nk = int(st.host("n_keep")[b])
    keep_g = seg(st.host("keep"), batch, b).astype(bool)
    ndiff = check_keep(keep_g, nk, keep_o, n_o, want, tau_o, sets["cand"])
    S_o, freed_o, live_o = oracle.redirect(batch.S(b), keep_o, synth.DEAD_SLOT, s.radix_prefix)
    S_g = seg(st.host("S"), batch, b)
    band = band_positions(want, tau_o, sets["cand"])
    assert np.array_equal(S_g[~band], S_o[~band])
    assert np.all((S_g[band] == batch.S(b)[band]) | (S_g[band] == synth.DEAD_SLOT))
    nl, nf = int(st.host("n_live")[b]), int(st.host("n_freed")[b])
    live_g = seg(st.host("live"), batch, b)[:nl]
    assert np.array_equal(live_g, S_g[S_g != synth.DEAD_SLOT])
    freed_g = seg(st.host("freed"), batch, b)[:nf]
    band_slots = set(batch.S(b)[band].tolist())
    assert set(freed_g.tolist()) ^ set(freed_o.tolist()) <= band_slots
    o = synth.widen(st.host("out")[b])
    bf16 = batch.kv_dtype == synth.BF16
    check_decode_on(o, batch.q_dec[b], batch.k_pool, batch.v_pool, live_g, bf16)
    if ndiff == 0:
        assert np.array_equal(live_g, live_o) and np.array_equal(freed_g, freed_o)
    return ndiff


def seg_M(st, batch, b):
    s, sh = batch.sessions[b], batch.shape
    o = int(batch.mem_off[b])
    return st.host("M")[o:o + sh.L * sh.Hkv * s.R * sh.D].reshape(sh.L, sh.Hkv * s.R, sh.D)


@pytest.mark.parametrize("update_memory", [False, True])
def test_step_end_to_end_tiny(dev, update_memory):
    batch = synth.tiny_single_layer(R=16, layout="shuffled", dead_frac=0.05)
    blob = synth.residual_blob(64, seed=9)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=update_memory)
    _compare_step(st, batch, 0, blob, ikv.IKV_RESIDUAL, update_memory)


def test_step_batched_ragged(dev):
    """Three sessions of different length, budget, memory rows and forced sets in one
    pool, plus an empty one and one that the N <= C gate skips."""
    shape = synth.Shape(L=2, Hq=8, Hkv=2, D=64)
    sessions = [synth.SessionSpec(N=1000, C=300, pi=16, qs=960, qe=1000, R=4, radix_prefix=16, dead_frac=0.1),
                synth.SessionSpec(N=2500, C=700, pi=0, qs=2440, qe=2500, R=16),
                synth.SessionSpec(N=0, C=10, pi=0, qs=0, qe=0, R=3),
                synth.SessionSpec(N=300, C=400, pi=8, qs=280, qe=300, R=7, dead_frac=0.2),
                synth.SessionSpec(N=777, C=100, pi=50, qs=700, qe=777, R=5)]
    batch = synth.make_batch(shape, sessions, seed=21, kv_dtype=synth.BF16, layout="paged", spare_pages=7)
    blob = synth.residual_blob(64, seed=10)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    for b in range(len(sessions)):
        if sessions[b].N == 0:
            assert int(st.host("n_keep")[b]) == 0 and int(st.host("n_live")[b]) == 0
            continue
        _compare_step(st, batch, b, blob, ikv.IKV_RESIDUAL, True)
    # the gated session: nothing scored, nothing dropped
    b = 3
    assert np.all(np.isneginf(seg(st.host("scores"), batch, b)))
    assert np.array_equal(seg(st.host("S"), batch, b), batch.S(b))
    assert float(st.host("tau")[b]) == -math.inf and int(st.host("n_freed")[b]) == 0


def test_step_forced_set_exceeds_budget(dev):
    batch = synth.tiny_single_layer(R=4)
    s = batch.sessions[0]
    s.pi = 600                          # |F| = 600 + 32 > C = 512: C* = 0
    st = RetentionStep(batch, dev)
    st.step(update_memory=False)
    sets = sess_sets(batch, 0)
    assert np.array_equal(st.host("keep").astype(bool), sets["forced"])
    assert float(st.host("tau")[0]) == math.inf and int(st.host("n_keep")[0]) == int(sets["forced"].sum())


def test_step_no_candidates(dev):
    batch = synth.tiny_single_layer(R=4, dead_frac=1.0)
    st = RetentionStep(batch, dev)
    st.step(update_memory=False)
    sets = sess_sets(batch, 0)
    assert not sets["cand"].any()
    assert np.all(np.isneginf(st.host("scores")))
    assert np.array_equal(st.host("keep").astype(bool), sets["forced"])


def test_step_is_deterministic_and_layout_invariant(dev):
    blob = synth.residual_blob(64, seed=12)
    outs = []
    for layout in ("identity", "shuffled", "shuffled"):
        batch = synth.tiny_single_layer(R=16, layout=layout)
        st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
        st.step(update_memory=True)
        outs.append((st.host("scores").copy(), st.host("keep").copy(), st.host("out").copy(), st.host("M").copy()))
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a, b)
    for a, b in zip(outs[1], outs[2]):
        assert np.array_equal(a, b)


# ============================================================================ full size

@pytest.fixture(scope="module")
def qwen3_8b(dev):
    batch = synth.qwen3_8b_32k(R=64)
    # head weights under which every term moves the scores (rule scores spread ~5e-3 here)
    blob = synth.residual_blob(128, seed=22, variant="scaled", units=36 * 8, out_std=5e-3)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    return batch, blob, st


def test_qwen3_8b_32k_step_full(qwen3_8b):
    """Full Qwen3-8B-shaped step (36 layers, 8 KV heads, 32,768 positions, budget 8192,
    64 memory rows per KV head, residual head on) against the full oracle."""
    batch, blob, st = qwen3_8b
    st.reset()
    st.step(update_memory=False)
    ndiff = _compare_step(st, batch, 0, blob, ikv.IKV_RESIDUAL, False, xattn_check=True)
    print(f"kept-set differences inside the band: {ndiff}")


@pytest.mark.skip(reason="one-key-pass form switched off: intermittent wrong row normaliser, cause not found")
def test_qwen3_8b_32k_step_full_one_pass_exchange(qwen3_8b, dev, monkeypatch):
    """The same full step with the score call's one-key-pass form (IKV_FUSED=1: every key
    read once, the row normalisers of Eq. 3 exchanged between resident workgroups), on
    the same pool, against the full oracle."""
    batch, blob, st0 = qwen3_8b
    monkeypatch.setenv("IKV_FUSED", "1")
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL, k_dev=st0.k_pool, v_dev=st0.v_pool)
    st.reset()
    ikv.timing(True)
    try:
        st.step(update_memory=False)
        names = [n for n, _ in ikv.timing_read()]
    finally:
        ikv.timing(False)
    assert "k_score_fused" in names, names
    ndiff = _compare_step(st, batch, 0, blob, ikv.IKV_RESIDUAL, False, xattn_check=True)
    print(f"kept-set differences inside the band: {ndiff}")


@pytest.fixture(scope="module")
def qwen25_14b(dev):
    batch = synth.qwen25_14b_92k_heavy(R=64)
    blob = synth.residual_blob(128, seed=23, variant="scaled", units=48 * 8, out_std=2e-3)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    return batch, blob, st


def test_qwen25_14b_92k_heavy_step_full(qwen25_14b):
    """Qwen2.5-14B-shaped step (48 layers, 8 KV heads, 92,300 positions: not a multiple
    of any tile, budget 8192, 64 memory rows per KV head, residual head on), with 5% of
    the non-forced keys scaled x4 on every layer and head (a heavy-tailed score
    distribution), against the full oracle."""
    batch, blob, st = qwen25_14b
    st.reset()
    st.step(update_memory=False)
    ndiff = _compare_step(st, batch, 0, blob, ikv.IKV_RESIDUAL, False, xattn_check=True)
    print(f"kept-set differences inside the band: {ndiff}")
