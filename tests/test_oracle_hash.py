"""Pins for the oracle's hashed front-end (appendix 'Vocabulary Compression',
section 'Model Dictionary Compression'): raw ids -> MurmurHash64A -> the 64 bits
read as two 32-bit numbers (low half B, high half C), each QR-indexing its own
pair of tables.

What fixes the oracle here, independently of its own code:
  - the hash's published verification procedure and value (SMHasher: hash the
    keys {}, {0}, {0,1}, ... {0..254} with seeds 256, 255, ... 1, then hash the
    concatenated 8-byte little-endian results with seed 0; the low 32 bits of
    that hash are 0x1F0D3804 for MurmurHash64A);
  - an inverse written here from the mixing steps (xor-shift by 47 is an
    involution on 64 bits, the multiplier is odd): unhashing recovers every id,
    so the 8-byte hash is a bijection (no two ids collide);
  - the split of a hash into B and C is the bitcast of the 64-bit value into
    two 32-bit words (numpy view);
  - gather and backward against one-hot / scatter-add formulations in numpy
    from those indices;
  - distinct ids give distinct combined embeddings (QR keeps uniqueness).
"""
import struct

import numpy as np
import pytest

import oracle

M64 = 0xc6a4a7935bd1e995
MASK = (1 << 64) - 1


def xs47(x):
    return x ^ (x >> 47)


def unhash8(h: int, seed: int) -> int:
    """Inverse of MurmurHash64A on an 8-byte key."""
    minv = pow(M64, -1, 1 << 64)
    h = xs47(h)
    h = (h * minv) & MASK
    h = xs47(h)
    h = (h * minv) & MASK            # undo the block's h *= m
    k = h ^ (seed ^ ((8 * M64) & MASK))
    k = (k * minv) & MASK
    k = xs47(k)
    k = (k * minv) & MASK
    return k


def test_published_verification_value():
    key = bytes(range(256))
    hashes = b"".join(struct.pack("<Q", oracle.murmur64a(key[:i], 256 - i)) for i in range(256))
    assert oracle.murmur64a(hashes, 0) & 0xffffffff == 0x1F0D3804


@pytest.mark.parametrize("seed", [0, 42, (1 << 63) + 12345])
def test_inverse_recovers_ids(seed):
    rng = np.random.default_rng(1)
    ids = np.concatenate([rng.integers(-(1 << 62), 1 << 62, 20000), np.arange(-100, 5000),
                          np.array([np.iinfo(np.int64).min, np.iinfo(np.int64).max])]).astype(np.int64)
    h = oracle.hash_ids(ids, seed)
    back = np.array([unhash8(int(x), seed) for x in h], dtype=np.uint64).view(np.int64)
    assert np.array_equal(back, ids)
    assert np.unique(h).size == np.unique(ids).size


def test_halves_are_the_bitcast_words():
    ids = np.arange(1000, dtype=np.int64) * 7919
    h = oracle.hash_ids(ids)
    words = h.view(np.uint32).reshape(-1, 2)  # little-endian: (low, high)
    assert np.array_equal(words[:, 0].astype(np.uint64), h & np.uint64(0xffffffff))
    assert np.array_equal(words[:, 1].astype(np.uint64), h >> np.uint64(32))


def hashed_inputs(rng, B, F, D, rows_q, m, bags=False):
    if bags:
        lens = rng.integers(0, 5, B * F)
        offsets = np.zeros(B * F + 1, np.int64)
        np.cumsum(lens, out=offsets[1:])
        ids = rng.integers(-(1 << 62), 1 << 62, int(offsets[-1]))
    else:
        offsets = None
        ids = rng.integers(-(1 << 62), 1 << 62, (B, F))
    qt = rng.standard_normal((F, 2, rows_q, D)).astype(np.float32)
    rt = rng.standard_normal((F, 2, m, D)).astype(np.float32)
    return ids.astype(np.int64), offsets, qt, rt


@pytest.mark.parametrize("combine", ["sum", "mul"])
def test_gather_vs_numpy(combine):
    rng = np.random.default_rng(2)
    B, F, D, Nd, rows_q, m = 40, 3, 8, 4, 1 << 16, 1 << 16
    ids, _, qt, rt = hashed_inputs(rng, B, F, D, rows_q, m)
    dense = rng.standard_normal((B, Nd)).astype(np.float32)
    x0 = oracle.gather_hashed(B, F, D, Nd, rows_q, m, combine, False, 9, ids, None, qt, rt, dense)
    h = oracle.hash_ids(ids, 9).reshape(B, F)
    op = (lambda a, b: a * b) if combine == "mul" else (lambda a, b: a + b)
    for f in range(F):
        e = np.zeros((B, D), np.float32)
        parts = []
        for s, half in enumerate((h[:, f] & np.uint64(0xffffffff), h[:, f] >> np.uint64(32))):
            qi, ri = (half // np.uint64(m)).astype(np.int64), (half % np.uint64(m)).astype(np.int64)
            parts.append(op(qt[f, s][qi], rt[f, s][ri]))
        e = parts[0] + parts[1]
        assert np.array_equal(x0[:, f * D:(f + 1) * D], e)
    assert np.array_equal(x0[:, F * D:], dense)


def test_rejects_tables_that_do_not_cover_32_bits():
    with pytest.raises(ValueError):
        oracle.gather_hashed(1, 1, 8, 0, 1 << 15, 1 << 16, "sum", False, 0, np.zeros((1, 1), np.int64), None,
                             np.zeros((1, 2, 1 << 15, 8), np.float32), np.zeros((1, 2, 1 << 16, 8), np.float32),
                             np.zeros((1, 0), np.float32))


@pytest.mark.parametrize("combine,bags", [("sum", False), ("mul", True)])
def test_backward_vs_scatter_add(combine, bags):
    rng = np.random.default_rng(3)
    B, F, D, Nd, rows_q, m = 30, 2, 4, 3, 1 << 16, 1 << 16
    ids, offsets, qt, rt = hashed_inputs(rng, B, F, D, rows_q, m, bags)
    d = F * D + Nd
    G = rng.standard_normal((B, d))
    gq, gr = oracle.embed_backward_hashed(B, F, D, Nd, rows_q, m, combine, 5, ids, offsets, qt, rt, G)
    eq, er = np.zeros_like(gq), np.zeros_like(gr)
    h = oracle.hash_ids(ids, 5)
    flat = ids.reshape(-1)
    for bag in range(B * F):
        b, f = divmod(bag, F)
        ps = range(offsets[bag], offsets[bag + 1]) if bags else [bag]
        for p in ps:
            for s in (0, 1):
                x = int(h[p]) >> (32 * s) & 0xffffffff
                qi, ri = divmod(x, m)
                g = G[b, f * D:(f + 1) * D]
                if combine == "mul":
                    eq[f, s, qi] += g * rt[f, s, ri]
                    er[f, s, ri] += g * qt[f, s, qi]
                else:
                    eq[f, s, qi] += g
                    er[f, s, ri] += g
    np.testing.assert_allclose(gq, eq, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(gr, er, rtol=1e-12, atol=1e-14)


def test_distinct_ids_give_distinct_embeddings():
    rng = np.random.default_rng(4)
    n, D, rows_q, m = 20000, 8, 1 << 16, 1 << 16
    ids = np.unique(rng.integers(0, 1 << 40, n)).astype(np.int64)
    qt = rng.standard_normal((1, 2, rows_q, D)).astype(np.float32)
    rt = rng.standard_normal((1, 2, m, D)).astype(np.float32)
    x0 = oracle.gather_hashed(ids.size, 1, D, 0, rows_q, m, "sum", False, 0, ids.reshape(-1, 1), None, qt, rt,
                              np.zeros((ids.size, 0), np.float32))
    assert np.unique(x0, axis=0).shape[0] == ids.size
