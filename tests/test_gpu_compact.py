"""The compact apply path (Sec. 3.4; the layout ablation of Table 7) against the float64
oracle: kept positions left-packed into destination slots, keys re-rotated from their
old position to their new one, values copied. Keys stored in bf16 must match the oracle
within one bf16 unit in the last place (one rounding of a float32 rotation); float32
keys within 1e-6; values, counts and untouched rows exactly."""
import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _bf16_ulp(x):
    ax = np.abs(np.asarray(x, np.float64))
    return np.exp2(np.floor(np.log2(np.where(ax > 0, ax, 1.0))) - 7)


def _check_rows(got_k, got_v, want_k, want_v, bf16):
    got_k, got_v = synth.widen(got_k), synth.widen(got_v)
    if bf16:
        tol = np.maximum(_bf16_ulp(want_k), 1e-6)
    else:
        tol = 1e-6 * np.maximum(1.0, np.abs(want_k))
    err = np.abs(got_k - want_k)
    assert np.all(err <= tol), f"key error {err.max():.3e}"
    np.testing.assert_array_equal(got_v, want_v)
    return float((err / tol).max())


def _dst_slots(batch, b, n):
    used = set(batch.slot_maps.tolist())
    free = np.array(sorted(set(range(1, batch.num_slots)) - used), np.int32)
    assert len(free) >= n
    return free[:n]


@pytest.mark.parametrize("kind,dead", [("f32", 0.0), ("f32", 0.2), ("bf16", 0.1)])
def test_compact_apply_small(dev, kind, dead):
    torch = _torch()
    N = 1500
    shape = synth.Shape(L=2, Hq=8, Hkv=2, D=64 if kind == "f32" else 128)
    spec = synth.SessionSpec(N=N, C=400, pi=0, qs=N - 32, qe=N, R=4, dead_frac=dead)
    batch = synth.make_batch(shape, [spec], seed=51, kv_dtype=synth.F32 if kind == "f32" else synth.BF16,
                             layout="paged", spare_pages=N // 16 + 2)
    S = batch.S(0)
    keep = synth.keep_mask(S, seed=52, frac=0.35)
    dst_h = np.zeros(N, np.int32)
    nk_o = int(keep.sum())
    dst_h[:nk_o] = _dst_slots(batch, 0, nk_o)
    st = RetentionStep(batch, dev)
    k_before = st.host("k_pool").copy()
    keep_d = torch.from_numpy(keep).to(dev)
    dst_d = torch.from_numpy(dst_h).to(dev)
    n_keep = torch.zeros(1, dtype=torch.int32, device=dev)
    ikv.compact_apply(st.pool, st.sess, st.S, keep_d, dst_d, n_keep, st.ws, rope_base=synth.ROPE_BASE)
    torch.cuda.synchronize()
    assert int(n_keep.item()) == nk_o
    Kn, Vn, Sn = oracle.ikv_oracle.compact_apply(batch.k_pool, batch.v_pool, S, keep, dst_h, synth.ROPE_BASE)
    k, v = st.host("k_pool"), st.host("v_pool")
    frac = _check_rows(k[:, Sn], v[:, Sn], Kn, Vn, kind == "bf16")
    other = np.setdiff1d(np.arange(batch.num_slots), Sn)
    assert np.array_equal(k[:, other], k_before[:, other])   # nothing else written
    print(f"{kind}: worst key error {frac:.2f} of the tolerance")


def test_compact_apply_qwen3_8b_32k(dev):
    """After the full Qwen3-8B 32k step's selection and redirect, the 8192 kept rows
    left-packed into freed slots (the rows a compactor reuses), checked against the oracle
    on a sample of kept indices spanning the whole range, every layer and head."""
    torch = _torch()
    batch = synth.qwen3_8b_32k(R=64)
    st = RetentionStep(batch, dev)
    st.init_dead_slot()
    st.score(flags=0)
    st.select()
    keep = st.host("keep")
    st.redirect()
    nf = int(st.host("n_freed")[0])
    dst = st.freed.clone()
    n_keep = torch.zeros(1, dtype=torch.int32, device=dev)
    assert nf >= int(keep.sum())
    S0 = batch.S(0)
    ikv.compact_apply(st.pool, st.sess, st.S0, st.keep, dst, n_keep, st.ws, rope_base=synth.ROPE_BASE)
    torch.cuda.synchronize()
    nk = int(n_keep.item())
    assert nk == int(keep.sum()) == 8192
    dst_h = dst.cpu().numpy()
    kept = np.nonzero(keep)[0]
    sample = np.unique(np.concatenate([np.arange(0, nk, 97), [0, nk - 1]]))
    kpool, vpool = st.host("k_pool"), st.host("v_pool")
    # the oracle on the sampled kept positions: their ranks among all kept ones decide the shift
    for t in sample:
        j = int(kept[t])
        want_k = oracle.ikv_oracle.rope_rotate(synth.widen(batch.k_pool[:, S0[j]]), int(t) - j, synth.ROPE_BASE, 128)
        want_v = synth.widen(batch.v_pool[:, S0[j]])
        _check_rows(kpool[:, dst_h[t]], vpool[:, dst_h[t]], want_k, want_v, True)
