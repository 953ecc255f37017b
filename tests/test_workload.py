"""Sanity of the seeded input generators (shapes, ranges, sharing structure)."""
import numpy as np

from paper_2606_17081_amd import workload as wl


def test_deterministic_and_seed_dependent():
    a, b, c = wl.tiny_trace(0), wl.tiny_trace(0), wl.tiny_trace(1)
    assert np.array_equal(a.tokens, b.tokens) and np.array_equal(a.turn_blocks, b.turn_blocks)
    assert not np.array_equal(a.turn_blocks, c.turn_blocks)


def test_tiny_trace_shape():
    t = wl.tiny_trace(0)
    assert t.n_conv == t.n_turns == 64
    assert t.turn_blocks.min() >= 4 and t.turn_blocks.max() <= 32
    assert np.array_equal(np.diff(t.tok_off), t.turn_blocks.astype(np.int64) * 16)
    assert t.tokens.min() >= 0 and t.tokens.max() < wl.VOCAB
    P = t.turn_blocks
    assert np.all(t.shared >= (P + 3) // 4) and np.all(t.shared <= (3 * P) // 4)
    assert t.group.min() >= 0 and t.group.max() < 8
    # requests of one group share their first min(s_a, s_b) blocks of tokens
    for g in np.unique(t.group):
        idx = np.nonzero(t.group == g)[0]
        for a, b in zip(idx, idx[1:]):
            k = 16 * min(t.shared[a], t.shared[b])
            ta = t.tokens[t.tok_off[a]:t.tok_off[a] + k]
            tb = t.tokens[t.tok_off[b]:t.tok_off[b] + k]
            assert np.array_equal(ta, tb)


def test_zipf_finite_frequencies():
    rng = np.random.default_rng(0)
    x = wl.zipf_finite(rng, 8, 1.1, 200000)
    w = np.arange(1, 9, dtype=float) ** -1.1
    p = w / w.sum()
    f = np.bincount(x, minlength=8) / x.size
    assert np.allclose(f, p, atol=0.005)
    y = wl.zipf_finite(rng, 64, 1.0, 1000)        # s = 1 is allowed (finite support)
    assert y.min() >= 0 and y.max() < 64


def test_lognormal_lengths_clipped():
    t = wl.sweep70b_trace(0, n_req=4096)
    assert t.turn_blocks.min() >= 8 and t.turn_blocks.max() <= 512
    assert 80 < t.turn_blocks.mean() < 120
    s = wl.saturation_trace(0, n_req=2048)
    assert s.turn_blocks.min() >= 8 and s.turn_blocks.max() <= 1024


def test_multiturn_trace():
    t = wl.multiturn_trace(0, n_conv=64)
    assert t.n_conv == 64
    nt = np.diff(t.turn_off)
    assert nt.min() >= 1 and nt.max() <= 16
    for c in range(t.n_conv):
        tb = t.turn_blocks[t.turn_off[c]:t.turn_off[c + 1]]
        assert np.all(np.diff(tb) >= 0)
        assert tb[-1] == t.chain_blocks[c] and tb[-1] <= 2048
        if nt[c] < 2:
            assert tb[-1] == 2048        # ended early only by reaching the context limit


def test_scoring_instance_structure():
    inst = wl.scoring_instance(seed=3, B=300, W=5, log2_slots=11, len_hi=64, len_lo=4)
    half = (1 << 11) // 2
    assert np.all(np.diff(inst.key_off) == half)
    assert np.all(inst.keys != 0) and np.all(inst.chains != 0)
    assert np.unique(inst.keys[inst.key_off[0]:inst.key_off[1]]).size == half
    L = np.diff(inst.chain_off)
    assert L.min() >= 4 and L.max() <= 64
    # membership along every chain is monotone (tables hold prefix-closed sets)
    for j in range(inst.W):
        s = set(int(k) for k in inst.keys[inst.key_off[j]:inst.key_off[j + 1]])
        for i in range(inst.B):
            ch = inst.chains[inst.chain_off[i]:inst.chain_off[i + 1]]
            m = np.array([int(h) in s for h in ch])
            if m.size:
                assert not np.any(m[1:] & ~m[:-1])
