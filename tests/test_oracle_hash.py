"""Pins of the oracle's block-hash chain against published vectors and identities."""
import json
import os
import struct

import numpy as np

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hash_vectors.json")


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def test_fnv1a64_published_vectors(orc):
    for text, hexval in _gold()["fnv1a64"]:
        assert orc.fnv1a64(text.encode()) == int(hexval, 16), text


def test_splitmix64_reference_outputs(orc):
    # splitmix64.c: state += 0x9E3779B97F4A7C15, then mix; orc.splitmix64(x) mixes x + gamma.
    gamma = 0x9E3779B97F4A7C15
    state = 0
    for hexval in _gold()["splitmix64_state0_outputs"]:
        assert orc.splitmix64(state) == int(hexval, 16)
        state = (state + gamma) & 0xFFFFFFFFFFFFFFFF


def test_block_bytes_are_little_endian_int32(orc):
    rng = np.random.default_rng(1)
    for _ in range(20):
        tok = rng.integers(0, 32000, size=16).astype(np.int32)
        raw = struct.pack("<16i", *[int(t) for t in tok])
        assert orc.block_fnv(tok) == orc.fnv1a64(raw)
    # a token's high bytes matter too (ids above 65535 are hashed as four bytes)
    tok = np.zeros(16, np.int32)
    tok[3] = 1 << 20
    assert orc.block_fnv(tok) == orc.fnv1a64(struct.pack("<16i", *[int(t) for t in tok]))
    assert orc.block_fnv(tok) != orc.block_fnv(np.zeros(16, np.int32))


def test_chain_worked_value(orc):
    g = _gold()["chain_tokens_0_15"]
    f = orc.block_fnv(np.arange(16, dtype=np.int32))
    assert f == int(g["fnv"], 16)
    assert orc.chain_step(0, f) == int(g["h0"], 16)
    out = orc.hash_chains(np.arange(16, dtype=np.int32), np.array([0, 16]), np.array([1]))
    assert int(out[0]) == int(g["h0"], 16)


def test_chain_is_iterated_step_and_prefix_determined(orc):
    rng = np.random.default_rng(7)
    shared = rng.integers(0, 32000, size=5 * 16).astype(np.int32)
    a = np.concatenate([shared, rng.integers(0, 32000, size=3 * 16).astype(np.int32)])
    b = np.concatenate([shared, rng.integers(0, 32000, size=4 * 16 + 9).astype(np.int32)])
    tokens = np.concatenate([a, b])
    tok_off = np.array([0, a.size, a.size + b.size])
    ch = orc.hash_chains(tokens, tok_off, np.array([8, 9]))
    ca, cb = ch[:8], ch[8:]
    # identical first five blocks -> identical hashes; the chain separates them afterwards
    assert np.array_equal(ca[:5], cb[:5])
    assert not np.any(ca[5:8] == cb[5:8])
    # h_i = step(h_{i-1}, fnv(block_i)) with h_{-1} = 0
    h = 0
    for i in range(8):
        h = orc.chain_step(h, orc.block_fnv(a[16 * i:16 * i + 16]))
        assert int(ca[i]) == h
    # changing a token in block 2 changes every later hash, not the earlier ones
    a2 = a.copy()
    a2[2 * 16 + 5] ^= 1
    ch2 = orc.hash_chains(a2, np.array([0, a2.size]), np.array([8]))
    assert np.array_equal(ch2[:2], ca[:2])
    assert not np.any(ch2[2:] == ca[2:])


def test_trailing_partial_block_is_not_hashed(orc):
    rng = np.random.default_rng(3)
    t = rng.integers(0, 32000, size=3 * 16 + 7).astype(np.int32)
    c1 = orc.hash_chains(t, np.array([0, t.size]), np.array([3]))
    t2 = t.copy()
    t2[-3:] += 1
    c2 = orc.hash_chains(t2, np.array([0, t2.size]), np.array([3]))
    assert np.array_equal(c1, c2)


def test_zero_hash_is_remapped(orc):
    gamma = 0x9E3779B97F4A7C15
    # splitmix64 mixes x + gamma with a bijection that maps 0 to 0, so x = -gamma hashes to 0
    x = (-gamma) & 0xFFFFFFFFFFFFFFFF
    assert orc.splitmix64(x) == 0
    assert orc.chain_step(0, x) == gamma
    assert orc.chain_step(x ^ 5, 5) == gamma
