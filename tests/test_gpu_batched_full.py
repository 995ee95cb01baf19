"""The batched one-GPU share at full size: 64 sessions in the shape of one GPU's half
of a Qwen2.5-14B tensor-parallel pair (48 layers, 20 query / 4 KV heads, D = 128) with
4096-65536 positions each (2.29 million in all), 32-128 memory rows (any count), budget
8192, the last 64 positions the query span and the cross-attention queries, residual head
on (weights under which its cross-attention visibly moves the checked sessions' scores);
one scoring + selection + redirect + decode pass over the whole batch, as one call
each. The pool holds 210 GiB of bf16 keys and values, too much to draw on the host:
they are filled on the GPU from seeded tables (synth.fill_share_pools). Every session's
kept count, slot map, freed list and live list are checked against their definitions,
and a second scoring call without the residual head checks every session's rule scores
against the closed form (they sum to L * Hkv * R); five sessions (the longest, the
shortest, the shortest above its budget, the ones with the most and the fewest memory
rows) against the float64 oracle on rows regenerated on the host (synth.share_rows)."""
import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import (RESID_MFMA_FLOOR, check_attention, check_keep, check_scores, check_xattn_visible,
                    oracle_scores_pair)

pytestmark = pytest.mark.gpu
SEED = 5
L, HQ, HKV, D, C, SPAN = 48, 20, 4, 128, 8192, 64


def _t(a, dev):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(a).to(dev)


def test_table_rows_device_matches_host(dev):
    import torch
    Ls, ns, Hkv, Dd = 3, 700, 4, 128
    tab = synth.table(9, synth.T_TABLE_K, Dd, log2_T=16)
    key = synth.table_key(9, synth.T_TABLE_K)
    pool = torch.zeros((Ls, ns, Hkv, Dd), dtype=torch.bfloat16, device=dev)
    synth.device_table_rows(pool, Ls, ns, Hkv, Dd, None, _t(tab, dev), key, log2_T=16)
    want = synth.table_rows(tab, Ls, ns, Hkv, Dd, np.arange(ns), key, log2_T=16)
    assert np.array_equal(pool.view(torch.int16).cpu().numpy().view(np.uint16), want)
    part = torch.zeros_like(pool)
    sl = np.array([5, 699, 0, 321], np.int32)
    synth.device_table_rows(part, Ls, ns, Hkv, Dd, _t(sl, dev), _t(tab, dev), key, log2_T=16)
    got = part.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got[:, sl], want[:, sl])
    assert not got[:, 1].any()


def test_batched_share_full_size(dev):
    import time

    import torch
    batch = synth.batched_share_full(SEED)
    B, Ns, Rs = len(batch.sessions), [x.N for x in batch.sessions], [x.R for x in batch.sessions]
    num_slots, slot_maps, slot_off = batch.num_slots, batch.slot_maps, batch.slot_off
    blob = synth.residual_blob(D, seed=26, variant="scaled", units=L * HKV, out_std=0.01)
    print(f"c5 share: {sum(Ns)} positions in {num_slots} slots, "
          f"{2 * L * num_slots * HKV * D * 2 / 2 ** 30:.1f} GiB of K and V", flush=True)
    clock = [time.perf_counter()]

    def lap(what):
        torch.cuda.synchronize()
        clock.append(time.perf_counter())
        print(f"  {what}: {clock[-1] - clock[-2]:.2f} s", flush=True)

    k = torch.empty((L, num_slots, HKV, D), dtype=torch.bfloat16, device=dev)
    v = torch.empty((L, num_slots, HKV, D), dtype=torch.bfloat16, device=dev)
    synth.fill_share_pools(k, v, batch)
    lap("fill keys and values")
    # spot check of the fill: rows of the last layer at a few slots, against the host
    probe = np.array([1, num_slots // 2, num_slots - 1])
    got = k[L - 1, torch.from_numpy(probe).to(dev)].view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, synth.share_rows(batch, probe)[L - 1])
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL, k_dev=k, v_dev=v)
    st.init_dead_slot()
    lap("inputs")
    st.score()
    lap("score")
    st.select()
    st.redirect()
    lap("select + redirect")
    st.decode()
    lap("decode")

    sc, kp = st.host("scores"), st.host("keep").astype(bool)
    S_new, fr, nf = st.host("S"), st.host("freed"), st.host("n_freed")
    live_h, nl, o_all = st.host("live"), st.host("n_live"), st.host("out")
    nk = st.host("n_keep")
    # the rule score alone over the redirected maps: each scored session's candidates are
    # now its kept ones, and their rule scores still sum to the row count L * Hkv * R
    st.score(flags=0)
    lap("rule-only score")
    rs = st.host("scores").astype(np.float64)
    for b in range(B):
        x = rs[slot_off[b]:slot_off[b] + Ns[b]]
        if Ns[b] <= C:
            assert np.all(np.isneginf(x))
            continue
        assert abs(x[np.isfinite(x)].sum() - L * HKV * Rs[b]) < 1e-4 * L * HKV * Rs[b], b
    del st, k, v
    torch.cuda.empty_cache()
    # every session: the kept count, the slot map, the freed and live lists by definition.
    # A session at or under its budget skips the event: all -inf scores, everything kept.
    kept = np.minimum(Ns, C)
    assert np.array_equal(nk, kept) and np.array_equal(nl, kept)
    for b in range(B):
        sl = slice(slot_off[b], slot_off[b] + Ns[b])
        kb = kp[sl]
        assert kb[Ns[b] - SPAN:].all() and int(kb.sum()) == kept[b]
        assert np.array_equal(S_new[sl], np.where(kb, slot_maps[sl], synth.DEAD_SLOT))
        assert np.array_equal(live_h[slot_off[b]:slot_off[b] + kept[b]], slot_maps[sl][kb])
        assert np.array_equal(fr[slot_off[b]:slot_off[b] + nf[b]], np.sort(slot_maps[sl][~kb]))
        if Ns[b] <= C:
            assert np.all(np.isneginf(sc[sl]))
            continue
        assert np.all(np.isfinite(sc[sl][:Ns[b] - SPAN])) and np.all(np.isneginf(sc[sl][Ns[b] - SPAN:]))
        # the kept set is the top of the scores: the lowest kept candidate beats the highest dropped one
        cand = np.arange(Ns[b]) < Ns[b] - SPAN
        assert sc[sl][cand & kb].min() >= sc[sl][cand & ~kb].max()
    # sessions against the oracle, on rows regenerated on the host: the longest, the
    # shortest (at or under the budget), the shortest above it, the most and fewest rows
    above = [b for b in range(B) if Ns[b] > C]
    picks = sorted({int(np.argmax(Ns)), int(np.argmin(Ns)), min(above, key=lambda b: Ns[b]), int(np.argmax(Rs)),
                    min(above, key=lambda b: Rs[b])})
    for b in picks:
        N, R = Ns[b], Rs[b]
        print(f"oracle on session {b} (N={N}, R={R})", flush=True)
        sl = slice(slot_off[b], slot_off[b] + N)
        Sb = slot_maps[sl]
        kc = np.zeros((L, N + 1, HKV, D), np.uint16)     # compact pool: position j at row j + 1
        kc[:, 1:] = synth.share_rows(batch, Sb)
        Sc = np.arange(1, N + 1, dtype=np.int32)
        sets = oracle.sets(Sc, 0, N - SPAN, N, C, 0)
        want, nox = oracle_scores_pair(kc, Sc, sets, batch.M_of(b), HKV, R, blob, np.arange(N - SPAN, N), 0)
        if N <= C:                                     # the event is skipped: nothing scored
            assert np.all(np.isneginf(want)) and np.all(np.isneginf(sc[sl]))
            rel = 0.0
        else:
            ratio, nd = check_xattn_visible(want, nox, sets)
            print(f"session {b}: cross-attention moves scores by up to {ratio:.0f}x the tolerance, {nd} kept",
                  flush=True)
            rel = check_scores(sc[sl], want, sets["cand"], floor=RESID_MFMA_FLOOR)
        keep_o, n_o, tau_o = oracle.select_budget(want, sets)
        check_keep(kp[sl], int(kept[b]), keep_o, n_o, want, tau_o, sets["cand"])
        S_o, freed_o, live_o = oracle.redirect(Sb, kp[sl], synth.DEAD_SLOT, 0)
        n = len(live_o)
        assert np.array_equal(S_new[sl], S_o) and np.array_equal(live_h[slot_off[b]:slot_off[b] + n], live_o)
        assert np.array_equal(fr[slot_off[b]:slot_off[b] + nf[b]], freed_o)
        kl = np.zeros((L, n + 1, HKV, D), np.uint16)
        vl = np.zeros((L, n + 1, HKV, D), np.uint16)
        kl[:, 1:] = synth.share_rows(batch, live_o)
        vl[:, 1:] = synth.share_rows(batch, live_o, values=True)
        o_o = oracle.decode(batch.q_dec[b], kl, vl, np.arange(1, n + 1))
        err = check_attention(synth.widen(o_all[b]), o_o, bf16=True)
        print(f"session {b}: N={N} R={R} score rel err {rel:.2e}, attention err {err:.2e}", flush=True)
