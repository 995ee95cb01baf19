"""The batched one-GPU share at full size: 64 sessions in the shape of one GPU's half
of a Qwen2.5-14B tensor-parallel pair (48 layers, 20 query / 4 KV heads, D = 128) with
4096-65536 positions each (2.29 million in all), 32-128 memory rows, budget 8192, the
last 64 positions the query span and the cross-attention queries, residual head on;
one scoring + selection + redirect + decode pass over the whole batch, as one call
each. The pool holds 210 GiB of bf16 keys and values, too much to draw on the host:
keys are filled on the GPU from a seeded table (synth.device_table_rows), values only
at the slots still live after the redirect. Every session's kept count, slot map, freed
list and live list are checked against their definitions; four sessions (the longest,
the shortest, the shortest above its budget, one with the most memory rows) against the
float64 oracle on rows regenerated on the host (synth.table_rows)."""
import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from parity import check_attention, check_keep, check_scores

pytestmark = pytest.mark.gpu
SEED = 5
L, HQ, HKV, D, C, SPAN = 48, 20, 4, 128, 8192, 64


def _bf16(x32):
    u = np.ascontiguousarray(x32, np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


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
    import torch
    g = synth.stream(SEED, synth.T_TURNS, 2)
    B = 64
    Ns = [int(n) for n in g.integers(4096, 65537, B)]
    Rs = [int(r) for r in 16 * g.integers(2, 9, B)]
    alloc, num_slots = synth.paged_slots(Ns, SEED, 16, spare_pages=64)
    slot_maps = np.concatenate(alloc).astype(np.int32)
    slot_off = np.concatenate([[0], np.cumsum(Ns)[:-1]]).astype(np.int64)
    rows, Ms, mem_off = [], [], 0
    for b in range(B):
        rows.append(dict(slot_off=int(slot_off[b]), mem_off=mem_off, qspan_off=0, qpos_off=SPAN * b, N=Ns[b],
                         pi=0, qs=Ns[b] - SPAN, qe=Ns[b], C=C, radix_prefix=0, R=Rs[b], nq=SPAN))
        Ms.append(synth.stream(SEED, synth.T_M, b).standard_normal((L, HKV * Rs[b], D), dtype=np.float32))
        mem_off += Ms[-1].size
    qpos = np.concatenate([np.arange(n - SPAN, n) for n in Ns]).astype(np.int32)
    q_dec = np.stack([_bf16(synth.stream(SEED, synth.T_QDEC, b).standard_normal((L, HQ, D), dtype=np.float32))
                      for b in range(B)])
    blob = synth.residual_blob(D, seed=26)
    tabK, tabV = synth.table(SEED, synth.T_TABLE_K, D), synth.table(SEED, synth.T_TABLE_V, D)
    keyK, keyV = synth.table_key(SEED, synth.T_TABLE_K), synth.table_key(SEED, synth.T_TABLE_V)
    print(f"c5 share: {sum(Ns)} positions in {num_slots} slots, "
          f"{2 * L * num_slots * HKV * D * 2 / 2 ** 30:.1f} GiB of K and V", flush=True)

    import time
    clock = [time.perf_counter()]

    def lap(what):
        torch.cuda.synchronize()
        clock.append(time.perf_counter())
        print(f"  {what}: {clock[-1] - clock[-2]:.2f} s", flush=True)

    k = torch.empty((L, num_slots, HKV, D), dtype=torch.bfloat16, device=dev)
    v = torch.empty((L, num_slots, HKV, D), dtype=torch.bfloat16, device=dev)
    lap("allocate")
    synth.device_table_rows(k, L, num_slots, HKV, D, None, _t(tabK, dev), keyK)
    lap("fill keys")
    # spot check of the fill: rows of the last layer at a few slots, against the host
    probe = np.array([1, num_slots // 2, num_slots - 1])
    got = k[L - 1, torch.from_numpy(probe).to(dev)].view(torch.int16).cpu().numpy().view(np.uint16)
    want = synth.table_rows(tabK, L, num_slots, HKV, D, probe, keyK)[L - 1]
    assert np.array_equal(got, want)
    pool = ikv.make_pool(k, v, L, HQ, HKV, D, num_slots, synth.DEAD_SLOT)
    ikv.init_dead_slot(pool)
    sess = ikv.Sessions(rows, dev)
    total = len(slot_maps)
    S = _t(slot_maps, dev)
    M = _t(np.concatenate([m.ravel() for m in Ms]), dev)
    scores = torch.empty(total, dtype=torch.float32, device=dev)
    keep = torch.empty(total, dtype=torch.uint8, device=dev)
    freed = torch.empty(total, dtype=torch.int32, device=dev)
    live = torch.empty(total, dtype=torch.int32, device=dev)
    n_keep, n_freed, n_live = (torch.empty(B, dtype=torch.int32, device=dev) for _ in range(3))
    tau = torch.empty(B, dtype=torch.float32, device=dev)
    out = torch.empty((B, L, HQ, D), dtype=torch.bfloat16, device=dev)
    ws = ikv.Workspace(dev)
    lap("inputs")
    ikv.score_history(pool, sess, S, M, scores, ws, qpos=_t(qpos, dev), residual=_t(blob, dev),
                      flags=ikv.IKV_RESIDUAL)
    lap("score")
    ikv.select_budget(sess, S, synth.DEAD_SLOT, scores, keep, n_keep, tau, ws)
    ikv.redirect_slots(sess, num_slots, S, synth.DEAD_SLOT, keep, freed, n_freed, live, n_live, ws)
    lap("select + redirect")
    nl = n_live.cpu().numpy()
    live_h = live.cpu().numpy()
    live_slots = np.concatenate([live_h[slot_off[b]:slot_off[b] + nl[b]] for b in range(B)])
    synth.device_table_rows(v, L, num_slots, HKV, D, _t(live_slots, dev), _t(tabV, dev), keyV)
    lap("fill live values")
    ikv.decode_attend_slotmap(pool, sess, _t(q_dec, dev), live, n_live, out, ws)
    lap("decode")

    sc, kp = scores.cpu().numpy(), keep.cpu().numpy().astype(bool)
    S_new, fr, nf = S.cpu().numpy(), freed.cpu().numpy(), n_freed.cpu().numpy()
    o_all = out.view(torch.int16).cpu().numpy().view(np.uint16)
    del k, v
    torch.cuda.empty_cache()
    # every session: the kept count, the slot map, the freed and live lists by definition.
    # A session at or under its budget skips the event: all -inf scores, everything kept.
    kept = np.minimum(Ns, C)
    assert np.array_equal(n_keep.cpu().numpy(), kept) and np.array_equal(nl, kept)
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
    # shortest (at or under the budget), the shortest above it, one with the most rows
    above = [b for b in range(B) if Ns[b] > C]
    picks = sorted({int(np.argmax(Ns)), int(np.argmin(Ns)), min(above, key=lambda b: Ns[b]), int(np.argmax(Rs))})
    for b in picks:
        N, R = Ns[b], Rs[b]
        print(f"oracle on session {b} (N={N}, R={R})", flush=True)
        sl = slice(slot_off[b], slot_off[b] + N)
        Sb = slot_maps[sl]
        kc = np.zeros((L, N + 1, HKV, D), np.uint16)     # compact pool: position j at row j + 1
        kc[:, 1:] = synth.table_rows(tabK, L, num_slots, HKV, D, Sb, keyK)
        Sc = np.arange(1, N + 1, dtype=np.int32)
        sets = oracle.sets(Sc, 0, N - SPAN, N, C, 0)
        want = oracle.scores(kc, Sc, sets, Ms[b], HKV, R, blob, oracle.FLAG_RESIDUAL,
                             np.arange(N - SPAN, N), 0)
        if N <= C:                                     # the event is skipped: nothing scored
            assert np.all(np.isneginf(want)) and np.all(np.isneginf(sc[sl]))
            rel = 0.0
        else:
            rel = check_scores(sc[sl], want, sets["cand"])
        keep_o, n_o, tau_o = oracle.select_budget(want, sets)
        check_keep(kp[sl], int(kept[b]), keep_o, n_o, want, tau_o, sets["cand"])
        S_o, freed_o, live_o = oracle.redirect(Sb, kp[sl], synth.DEAD_SLOT, 0)
        n = len(live_o)
        assert np.array_equal(S_new[sl], S_o) and np.array_equal(live_h[slot_off[b]:slot_off[b] + n], live_o)
        assert np.array_equal(fr[slot_off[b]:slot_off[b] + nf[b]], freed_o)
        kl = np.zeros((L, n + 1, HKV, D), np.uint16)
        vl = np.zeros((L, n + 1, HKV, D), np.uint16)
        kl[:, 1:] = synth.table_rows(tabK, L, num_slots, HKV, D, live_o, keyK)
        vl[:, 1:] = synth.table_rows(tabV, L, num_slots, HKV, D, live_o, keyV)
        o_o = oracle.decode(q_dec[b], kl, vl, np.arange(1, n + 1))
        err = check_attention(synth.widen(o_all[b]), o_o, bf16=True)
        print(f"session {b}: N={N} R={R} score rel err {rel:.2e}, attention err {err:.2e}", flush=True)
