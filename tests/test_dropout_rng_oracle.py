"""Pins of the oracle's counter-based dropout mask (oracle/dropout_rng.py).

  * the Philox4x64-10 block against numpy's own Philox bit generator, a
    library implementation of the same published generator (numpy advances
    its 256-bit counter before each block, so its first block for counter c is
    the block at c + 1), including carries across counter words;
  * the mask: p = 0 keeps every element; for a fixed (seed, offset) the masks
    of increasing p are nested (a draw kept at a higher rate is kept at every
    lower one); the keep rate lies within the binomial bounds; the counter
    layout (bytes 2t and 2t+1 of a call are the block at counter offset + t,
    bit e of the pair the 16-bit quarter e of its output; with k a multiple of
    16, row i of a call is row 0 of the call at offset + i k/16);
  * planted mistakes in the block or the layout fail the numpy pin or the
    layout pin.
"""
import numpy as np
import pytest

from oracle import dropout_rng as rng


def _numpy_block(ctr, key):
    """numpy's Philox block for counter ctr (4 x 64-bit) and key (2 x 64-bit)."""
    c = ctr[0] | (ctr[1] << 64) | (ctr[2] << 128) | (ctr[3] << 192)
    c = (c - 1) % (1 << 256)                      # numpy increments before the block
    words = [(c >> (64 * i)) & ((1 << 64) - 1) for i in range(4)]
    g = np.random.Philox(counter=np.array(words, dtype=np.uint64), key=np.array(key, dtype=np.uint64))
    return tuple(int(x) for x in g.random_raw(4))


CASES = [((0, 0, 0, 0), (0, 0)), ((1, 0, 0, 0), (0x123456789ABCDEF0, 0x0FEDCBA987654321)),
         ((0, 1, 0, 0), (7, 0)), ((2**64 - 1, 2**64 - 1, 5, 9), (2**64 - 1, 2**64 - 1)),
         ((12345, 678, 91011, 1213), (1415, 1617))]


@pytest.mark.parametrize("ctr,key", CASES)
def test_block_matches_numpy_philox(ctr, key):
    assert rng.philox4x64_10(ctr, key) == _numpy_block(ctr, key)


def test_threshold():
    assert rng.keep_threshold(0.0) == 2**16
    assert rng.keep_threshold(0.5) == 2**15
    assert rng.keep_threshold(np.float32(0.05)) == 62259     # 0.95 * 65536 = 62259.2


def test_p_zero_keeps_all():
    assert (rng.dropout_keep_philox(3, 10, 0.0, 5, 64) == 0xFF).all()


def test_masks_nest_with_the_rate():
    a = rng.dropout_keep_philox(11, 0, 0.1, 6, 128)
    b = rng.dropout_keep_philox(11, 0, 0.3, 6, 128)
    c = rng.dropout_keep_philox(11, 0, 0.7, 6, 128)
    assert ((b & ~a) == 0).all() and ((c & ~b) == 0).all()
    assert (a != b).any() and (b != c).any()


@pytest.mark.parametrize("p", [0.05, 0.5])
def test_keep_rate_within_binomial_bounds(p):
    m, k = 64, 1024
    bits = np.unpackbits(rng.dropout_keep_philox(5, 1000, p, m, k), bitorder="little")
    n = bits.size
    q = rng.keep_threshold(p) / 2**16
    assert abs(bits.mean() - q) <= 5 * np.sqrt(q * (1 - q) / n)


def _bits(seed, ctr, thr):
    words = _numpy_block((ctr & (2**64 - 1), ctr >> 64, 0, 0), (seed, 0))
    return sum(1 << e for e in range(16) if ((words[e // 4] >> (16 * (e % 4))) & 0xFFFF) < thr)


def test_counter_layout():
    seed, p = 99, 0.25
    thr = rng.keep_threshold(p)
    # k = 24: three bytes a row, so rows start inside blocks; the counter carries into its second word
    off, m, k = 2**64 - 3, 4, 24
    full = rng.dropout_keep_philox(seed, off, p, m, k)
    flat = full.reshape(-1)
    for b in range(m * k // 8):
        assert flat[b] == (_bits(seed, off + b // 2, thr) >> (8 * (b % 2))) & 0xFF, b
    # k a multiple of 16: row i of a call is row 0 of the call at offset + i k / 16
    off, m, k = 2**64 - 9, 4, 48
    full = rng.dropout_keep_philox(seed, off, p, m, k)
    for i in range(m):
        assert (rng.dropout_keep_philox(seed, off + i * (k // 16), p, 1, k)[0] == full[i]).all()
    # rows passed explicitly give the same bytes
    assert (rng.dropout_keep_philox(seed, off, p, m, k, rows=[3, 1]) == full[[3, 1]]).all()


def test_planted_mistakes_fail_the_pins(monkeypatch):
    ctr, key = CASES[1]
    ref = _numpy_block(ctr, key)
    # round multiplier typo
    monkeypatch.setattr(rng, "_M1", rng._M1 ^ 1)
    assert rng.philox4x64_10(ctr, key) != ref
    monkeypatch.undo()
    # key bumped before the first round
    orig = rng.philox4x64_10

    def early_bump(c, k):
        return orig(c, ((k[0] + rng._W0) % 2**64, (k[1] + rng._W1) % 2**64))
    assert early_bump(ctr, key) != ref
    # byte layout: one block per byte instead of one per byte pair
    seed, off, p, m, k = 99, 7, 0.25, 3, 48
    full = rng.dropout_keep_philox(seed, off, p, m, k)
    thr = rng.keep_threshold(p)
    wrong = np.array([_bits(seed, off + b, thr) & 0xFF for b in range(k // 8)], dtype=np.uint8)
    assert not (wrong == full[0]).all()
