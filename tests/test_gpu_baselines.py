"""The baseline compressors of Sec. 4.1 scored on the same substrate (the matrix-core
scorer, then the same selection and redirect): H2O-style heavy-hitter scores (the
attention received from observed query rows, the recent window of ratio mode forced)
and SnapKV-style scores (the W = 32 window rows' attention mass per layer and KV head,
max-pooled over 7 positions, summed), against the float64 oracle."""
import math

import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import check_keep, check_scores

pytestmark = pytest.mark.gpu
W = 32


def _batch(shape, N, C, seed, recent=None, dead_frac=0.0, qs=None):
    G = shape.Hq // shape.Hkv
    if recent is not None:                                  # ratio mode: the recent window is the forced floor
        qs, qe = oracle.ikv_oracle.recent_window(N, C, recent)
    else:
        qs, qe = (N - W if qs is None else qs), N
    # no memory update and no residual head: no span rows, no cross-attention positions
    spec = synth.SessionSpec(N=N, C=C, pi=0, qs=qs, qe=qe, R=G * W, dead_frac=dead_frac, qpos=np.zeros(0, np.int32))
    batch = synth.make_batch(shape, [spec], seed=seed, kv_dtype=synth.BF16, layout="paged", span_rows=False)
    q = synth.window_queries(shape, N, W, seed)
    batch.M = q.reshape(-1).copy()                          # [L][Hq][W][D] is M with R = G * W
    return batch, q


def _run(dev, batch, flags):
    st = RetentionStep(batch, dev, flags=flags)
    st.init_dead_slot()
    st.score(flags=flags)
    st.select()
    return st


@pytest.mark.parametrize("kind,N,Hkv,G,dead", [("snapkv", 1000, 2, 4, 0.0), ("snapkv", 777, 2, 2, 0.2),
                                               ("snapkv", 2100, 4, 1, 0.1), ("h2o", 1000, 2, 4, 0.1),
                                               ("h2o", 1500, 2, 3, 0.0)])
def test_baseline_scores_small(dev, kind, N, Hkv, G, dead):
    shape = synth.Shape(L=2, Hq=Hkv * G, Hkv=Hkv, D=128)
    C = N // 3
    batch, q = _batch(shape, N, C, seed=N + G, recent=0.5 if kind == "h2o" else None, dead_frac=dead)
    flags = ikv.IKV_POOL7 if kind == "snapkv" else 0
    st = _run(dev, batch, flags)
    S, s = batch.S(0), batch.sessions[0]
    sets = oracle.sets(S, s.pi, s.qs, s.qe, s.C, synth.DEAD_SLOT)
    fn = oracle.ikv_oracle.snapkv_scores if kind == "snapkv" else oracle.ikv_oracle.h2o_scores
    want = fn(batch.k_pool, S, sets, q, Hkv)
    rel = check_scores(st.host("scores"), want, sets["cand"])
    assert rel < 1e-5, rel
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, sets["cand"])
    if kind == "h2o":                                       # every query row's softmax sums to one
        got = st.host("scores").astype(np.float64)
        assert math.isclose(got[sets["cand"]].sum(), shape.L * shape.Hq * W, rel_tol=1e-5)


@pytest.mark.parametrize("kind", ["snapkv", "h2o"])
def test_baseline_scores_qwen3_8b_32k(dev, kind):
    """Qwen3-8B shape, 32,768 positions, budget 8192, full size, then redirect and decode
    on the kept set as for IntentKV."""
    shape = synth.qwen3_8b_shape()
    N, C = 32768, 8192
    batch, q = _batch(shape, N, C, seed=2, recent=0.5 if kind == "h2o" else None)
    flags = ikv.IKV_POOL7 if kind == "snapkv" else 0
    st = _run(dev, batch, flags)
    st.redirect()
    st.decode()
    S, s = batch.S(0), batch.sessions[0]
    sets = oracle.sets(S, s.pi, s.qs, s.qe, s.C, synth.DEAD_SLOT)
    fn = oracle.ikv_oracle.snapkv_scores if kind == "snapkv" else oracle.ikv_oracle.h2o_scores
    want = fn(batch.k_pool, S, sets, q, shape.Hkv)
    rel = check_scores(st.host("scores"), want, sets["cand"])
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    nd = check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, sets["cand"])
    nl = int(st.host("n_live")[0])
    live = st.host("live")[:nl]
    S_g = st.host("S")
    assert np.array_equal(live, S_g[S_g != synth.DEAD_SLOT]) and nl == n_o
    from parity import check_decode_on
    err = check_decode_on(synth.widen(st.host("out")[0]), batch.q_dec[0], batch.k_pool, batch.v_pool, live, True)
    print(f"{kind}: score error {rel:.1e}, band differences {nd}, attention error {err:.1e}")


def test_pool7_rejections(dev):
    shape = synth.Shape(L=2, Hq=6, Hkv=3, D=128)            # odd Hkv: not on the unit-major path
    batch, _ = _batch(shape, 600, 200, seed=9)
    with pytest.raises(ikv.IkvError) as e:
        _run(dev, batch, ikv.IKV_POOL7)
    assert e.value.status == -4
    shape = synth.Shape(L=2, Hq=4, Hkv=2, D=128)
    batch, _ = _batch(shape, 600, 200, seed=9)
    st = RetentionStep(batch, dev, residual=synth.residual_blob(128, seed=1), flags=ikv.IKV_RESIDUAL)
    with pytest.raises(ikv.IkvError) as e:
        st.score(flags=ikv.IKV_POOL7 | ikv.IKV_RESIDUAL)
    assert e.value.status == -1
