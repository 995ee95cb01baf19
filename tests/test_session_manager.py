"""Host session management (no GPU): the session-key priority of Appendix A /
Appendix H, the LRU QueryMemory store, the compression trigger and the actionable
span with its tail fallback, called through the C ABI."""
from collections import OrderedDict

import numpy as np
import pytest

from paper_2606_09916_amd import ikv


def test_key_priority_order():
    st = ikv.MemStore(16)
    toks = np.arange(1000, 1600)
    # an explicit id wins over everything else
    s1, f1, k1 = st.acquire(b"sess-A", tokens=toks, span=(10, 20))
    assert (f1, k1) == (True, ikv.IKV_KEY_EXPLICIT)
    s2, f2, _ = st.acquire(b"sess-A", tokens=np.arange(5))            # same id, other tokens: same memory
    assert (s2, f2) == (s1, False)
    # no id: the designated span's tokens
    s3, f3, k3 = st.acquire(None, tokens=toks, span=(10, 20))
    assert (f3, k3) == (True, ikv.IKV_KEY_SPAN) and s3 != s1
    other = toks.copy()
    other[0] = -5                                                    # outside the span: still the same session
    assert st.acquire(None, tokens=other, span=(10, 20))[:2] == (s3, False)
    # no span: the first 256 tokens
    s4, f4, k4 = st.acquire(None, tokens=toks)
    assert (f4, k4) == (True, ikv.IKV_KEY_PREFIX)
    tail = toks.copy()
    tail[256:] = 7                                                   # differs only past the prefix
    assert st.acquire(None, tokens=tail)[:2] == (s4, False)
    head = toks.copy()
    head[255] = 7                                                    # differs inside the prefix
    assert st.acquire(None, tokens=head)[1] is True
    # no tokens at all: request-local keys never match
    a, fa, ka = st.acquire(None)
    b, fb, kb = st.acquire(None)
    assert ka == kb == ikv.IKV_KEY_LOCAL and fa and fb and a != b


def test_keys_of_different_kinds_never_match():
    st = ikv.MemStore(8)
    toks = np.array([0x41424344, 0x45464748], np.int32)
    as_bytes = toks.tobytes()                                        # an explicit id with the same bytes
    s_id = st.acquire(as_bytes)[0]
    s_span = st.acquire(None, tokens=toks, span=(0, 2))[0]
    s_pre = st.acquire(None, tokens=toks)[0]
    assert len({s_id, s_span, s_pre}) == 3


def test_short_prefix_and_empty_span():
    st = ikv.MemStore(4)
    s, f, k = st.acquire(None, tokens=[1, 2, 3], span=(2, 2))       # empty span: not a span key
    assert k == ikv.IKV_KEY_PREFIX and f
    assert st.acquire(None, tokens=[1, 2, 3])[:2] == (s, False)
    assert st.acquire(None, tokens=[1, 2])[1] is True               # a different (shorter) prefix


def test_span_outside_tokens_is_rejected():
    st = ikv.MemStore(4)
    with pytest.raises(ikv.IkvError) as e:
        st.acquire(None, tokens=[1, 2, 3], span=(1, 9))
    assert e.value.status == -2


def test_lru_eviction_and_pinning():
    st = ikv.MemStore(3)
    slots = {}
    for k in (b"a", b"b", b"c"):
        slots[k], fresh, _ = st.acquire(k)
        assert fresh
        st.release(slots[k])
    assert sorted(slots.values()) == [0, 1, 2] and len(st) == 3
    st.release(st.acquire(b"a")[0])                                  # "a" is now the most recently used
    s_d, fresh, _ = st.acquire(b"d")                                  # evicts "b", the least recently used
    assert fresh and s_d == slots[b"b"] and len(st) == 3
    s_b, fresh, _ = st.acquire(b"b")                                  # "b" comes back fresh, evicting "c"
    assert fresh and s_b == slots[b"c"]
    # "d" and "b" are still held: a new key can only take "a"'s row
    s_e, fresh, _ = st.acquire(b"e")
    assert fresh and s_e == slots[b"a"]
    with pytest.raises(ikv.IkvError) as e:                            # every memory held: nothing to evict
        st.acquire(b"f")
    assert e.value.status == -4
    st.release(s_d)
    assert st.acquire(b"f")[0] == s_d                                 # "d" released: its row goes first


def test_release_errors():
    st = ikv.MemStore(2)
    s, _, _ = st.acquire(b"x")
    st.release(s)
    with pytest.raises(ikv.IkvError):
        st.release(s)                                                # released twice
    with pytest.raises(ikv.IkvError):
        st.release(5)                                                # not a row of the store


def test_store_against_a_reference_lru():
    """A random sequence of acquires and releases on the paper's 1,024-memory store,
    against a plain model: an ordered map of key -> row, most recently used last, the
    least recently used memory that is not held evicted when every row is taken."""
    cap = 1024
    st = ikv.MemStore(cap)
    rng = np.random.default_rng(0)
    model, held, free = OrderedDict(), {}, list(range(cap))
    pinned = []
    for step in range(6000):
        key = b"k%d" % int(rng.integers(0, 1500))
        slot, fresh, _ = st.acquire(key)
        if key in model:
            assert not fresh and slot == model[key]
            model.move_to_end(key)
        else:
            assert fresh
            if free:
                want = free.pop(0)
            else:
                victim = next(k for k in model if held.get(k, 0) == 0)
                want = model.pop(victim)
            assert slot == want
            model[key] = slot
        held[key] = held.get(key, 0) + 1
        pinned.append((key, slot))
        # release most acquires at once, keep a few held for a while
        while pinned and (len(pinned) > 20 or rng.random() < 0.7):
            k, s = pinned.pop(int(rng.integers(0, len(pinned))))
            st.release(s)
            held[k] -= 1
    assert len(st) == len(model) == cap


def test_trigger_policy():
    st = ikv.MemStore(2)
    s, _, _ = st.acquire(b"t")
    C = 8192
    assert not st.trigger(s, 8192, C)                               # N <= C: never
    assert st.trigger(s, 8193, C)                                   # first event once N > C
    assert not st.trigger(s, 8193 + 511, C)                          # fewer than 512 new positions
    assert st.trigger(s, 8193 + 512, C)
    assert not st.trigger(s, 8193 + 600, C)
    assert st.trigger(s, 20000, C, trigger=0) and st.trigger(s, 20000, C, trigger=0)


def test_resolve_span():
    # system prompt, user task, assistant turn, tool output, assistant header
    msgs = [(0, 64, False), (64, 300, True), (300, 420, False), (420, 900, True), (900, 910, False)]
    assert ikv.resolve_span(910, msgs) == (420, 900)                # the latest actionable message
    assert ikv.resolve_span(910, msgs[:3]) == (64, 300)
    assert ikv.resolve_span(910, msgs + [(910, 910, True)]) == (420, 900)   # empty message skipped
    assert ikv.resolve_span(910, [(0, 64, False)]) == (878, 910)    # fallback: the last W = 32 positions
    assert ikv.resolve_span(20, []) == (0, 20)
    assert ikv.resolve_span(910, [], tail_w=64) == (846, 910)
    with pytest.raises(ikv.IkvError):
        ikv.resolve_span(100, [(50, 120, True)])                   # past N
