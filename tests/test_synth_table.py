"""The table-row input generator (synth.table_rows, and its GPU twin in
synth/table_rows.hip): SplitMix64 against its published outputs, rows as windows of
the table, and the value distribution."""
import numpy as np

import synth


def test_splitmix64_matches_published_outputs():
    # SplitMix64 started from state 0 (state += 0x9E3779B97F4A7C15, then the output
    # function): the first four outputs of the published reference generator
    gamma = np.uint64(0x9E3779B97F4A7C15)
    with np.errstate(over="ignore"):
        states = np.arange(1, 5, dtype=np.uint64) * gamma
    got = [int(x) for x in synth._splitmix64(states)]
    assert got == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]


def test_rows_are_table_windows_at_their_offsets():
    D, L, ns, Hkv = 64, 3, 500, 2
    tab = synth.table(7, synth.T_TABLE_K, D, log2_T=12)
    key = synth.table_key(7, synth.T_TABLE_K)
    slots = np.array([0, 17, 499, 17])
    rows = synth.table_rows(tab, L, ns, Hkv, D, slots, key, log2_T=12)
    assert rows.shape == (L, 4, Hkv, D)
    for l in range(L):
        o = synth.table_offsets(l, ns, Hkv, slots, key, log2_T=12)
        assert o.min() >= 0 and o.max() < 1 << 12
        for k in range(4):
            for h in range(Hkv):
                assert np.array_equal(rows[l, k, h], tab[o[k, h]:o[k, h] + D])
    assert np.array_equal(rows[:, 1], rows[:, 3])            # a row depends only on (l, slot, h)
    # offset of row (l, slot, h): the generator's definition written out for one row
    r = (2 * ns + 499) * Hkv + 1
    z = (key + (r + 1) * 0x9E3779B97F4A7C15) % (1 << 64)
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) % (1 << 64)
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) % (1 << 64)
    z ^= z >> 31
    assert synth.table_offsets(2, ns, Hkv, [499], key, log2_T=12)[0, 1] == z >> (64 - 12)


def test_table_values_are_standard_normal_in_bf16():
    tab = synth.table(5, synth.T_TABLE_K, 128, log2_T=20)
    x = synth.widen(tab)
    assert len(x) == (1 << 20) + 128
    assert abs(x.mean()) < 5e-3 and abs(x.std() - 1.0) < 5e-3
    # bf16: the low 16 bits of every float32 value are zero and rounding is to nearest
    f = np.asarray(synth.stream(5, synth.T_TABLE_K).standard_normal(1000, dtype=np.float32), np.float64)
    assert np.all(np.abs(x[:1000] - f) <= np.abs(f) * 2.0 ** -8)
