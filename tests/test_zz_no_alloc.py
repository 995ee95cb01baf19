"""The allocation-free selection, ikv_select_budget_static, against ikv_select_budget on
the same inputs: two calls in a row on the library's static scratch, the second on a
smaller input than the first, each bit for bit equal to the workspace call's keep
mask, kept count and threshold; device memory stays as it was; sessions whose scratch
would exceed the static array are rejected before anything is enqueued."""
import numpy as np
import pytest

import synth
from paper_2606_09916_amd import ikv

pytestmark = pytest.mark.gpu
DEAD = synth.DEAD_SLOT


def _batch(lengths, seed):
    rows, off = [], 0
    Ss, scs = [], []
    for b, n in enumerate(lengths):
        rows.append(dict(slot_off=off, mem_off=0, qspan_off=0, qpos_off=0, N=n, pi=3, qs=max(0, n - 64), qe=n,
                         C=max(1, n // 4), radix_prefix=0, R=16, nq=0))
        off += n
        Ss.append(synth.slot_map(n, 2 * n + 1, seed=seed * 10 + b, dead_frac=0.1))
        scs.append(synth.score_vector(n, seed=seed * 10 + 5 + b, ties=b % 2 == 0))
    return rows, np.concatenate(Ss), np.concatenate(scs)


def _buffers(dev, rows, S_all, sc_all):
    import torch
    B, tot = len(rows), len(S_all)
    return dict(sess=ikv.Sessions(rows, dev), S=torch.from_numpy(S_all).to(dev),
                sc=torch.from_numpy(sc_all).to(dev), keep=torch.full((tot,), 7, dtype=torch.uint8, device=dev),
                n_keep=torch.full((B,), -9, dtype=torch.int32, device=dev),
                tau=torch.full((B,), 3.0, dtype=torch.float32, device=dev))


def _host(b):
    return b["keep"].cpu().numpy(), b["n_keep"].cpu().numpy(), b["tau"].cpu().numpy()


@pytest.mark.parametrize("no_coop", [False, True])
def test_static_select_matches_workspace_select(dev, monkeypatch, no_coop):
    import torch
    if no_coop:
        monkeypatch.setenv("IKV_NO_COOP", "1")
    # first input: one session past the cooperative path's 131,072 positions (the three-kernel
    # path) and two shorter ones; second input: smaller, the cooperative (or one-workgroup) path
    inputs = [_batch((150000, 3000, 40000), 1), _batch((40000, 777), 2)]
    want, bufs = [], []
    ws = ikv.Workspace(dev)
    for rows, S_all, sc_all in inputs:
        b = _buffers(dev, rows, S_all, sc_all)
        ikv.select_budget(b["sess"], b["S"], DEAD, b["sc"], b["keep"], b["n_keep"], b["tau"], ws)
        torch.cuda.synchronize()
        want.append(_host(b))
        bufs.append(_buffers(dev, rows, S_all, sc_all))
    free0 = torch.cuda.mem_get_info()[0]
    for b in bufs:                                   # two calls in a row, the second on the smaller input
        ikv.select_budget_static(b["sess"], b["S"], DEAD, b["sc"], b["keep"], b["n_keep"], b["tau"])
    torch.cuda.synchronize()
    assert torch.cuda.mem_get_info()[0] == free0, "device memory changed across the static calls"
    for (k0, n0, t0), b in zip(want, bufs):
        k1, n1, t1 = _host(b)
        assert np.array_equal(k0, k1)
        assert np.array_equal(n0, n1)
        assert np.array_equal(t0.view(np.uint32), t1.view(np.uint32))


def test_static_select_rejects_oversized_sessions(dev):
    import torch
    rows, S_all, sc_all = _batch((3000,), 3)
    rows[0]["N"] = 6_000_000                         # host descriptor only: rejected before any launch
    b = _buffers(dev, [rows[0]], S_all, sc_all)
    keep_before = b["keep"].clone()
    with pytest.raises(ikv.IkvError) as e:
        ikv.select_budget_static(b["sess"], b["S"], DEAD, b["sc"], b["keep"], b["n_keep"], b["tau"])
    assert e.value.status == -3 and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.equal(b["keep"], keep_before)
