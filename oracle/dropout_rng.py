"""The dropout keep mask drawn from a counter-based generator -- TEST
INFRASTRUCTURE (the oracle of the device mask generator; only tests, the
package smoke check and the benchmark's CPU-baseline leg may use it).

Listing 3's configuration carries LORA_DROPOUT; the dropout of the adapter's
input needs one keep/drop draw per element of X.  The library draws them on
the device with Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC 2011); this module evaluates the same
definition with Python integers, one block at a time:

  block(counter c0..c3, key k0, k1): ten rounds; in each, the 128-bit products
  P0 = M0 * c0 and P1 = M1 * c2 give the new counter
      (hi(P1) ^ c1 ^ k0,  lo(P1),  hi(P0) ^ c3 ^ k1,  lo(P0)),
  and after each round the key is advanced by the Weyl constants (W0, W1).

  mask bytes 2t and 2t+1 (byte b = i * (k/8) + q holds elements 8q .. 8q+7 of
  row i): the block at counter (offset + t as a 128-bit integer in c0, c1;
  c2 = c3 = 0) and key (seed, 0); its words split into sixteen 16-bit values
  u_e (u_4h+j = bits 16j .. 16j+15 of word h); bit e of the byte pair (e = 0..7
  in byte 2t, 8..15 in byte 2t+1) is set (element kept) iff
  u_e < T = floor((1 - p) * 2^16 + 1/2), with p the float32 rate taken to
  float64.

Pins (tests/test_dropout_rng_oracle.py): the block against numpy's own
Philox bit generator (a library implementation of the same published
generator), the keep rate against its binomial bounds, p = 0 keeping all,
nested masks for increasing p, and the counter layout across rows and calls.
"""
import numpy as np

_MASK64 = (1 << 64) - 1
_M0, _M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157   # round multipliers
_W0, _W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B   # key increments (Weyl sequence)


def philox4x64_10(ctr, key):
    """One Philox4x64-10 block: ctr a 4-tuple and key a 2-tuple of unsigned
    64-bit integers; returns the 4 output words."""
    c0, c1, c2, c3 = (int(x) & _MASK64 for x in ctr)
    k0, k1 = (int(x) & _MASK64 for x in key)
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _W0) & _MASK64
            k1 = (k1 + _W1) & _MASK64
        p0 = _M0 * c0
        p1 = _M1 * c2
        c0, c1, c2, c3 = ((p1 >> 64) ^ c1 ^ k0, p1 & _MASK64, (p0 >> 64) ^ c3 ^ k1, p0 & _MASK64)
    return c0, c1, c2, c3


def keep_threshold(p) -> int:
    """T = floor((1 - p) 2^16 + 1/2) for the float32 rate p, in float64."""
    return int(np.floor((1.0 - float(np.float32(p))) * 65536.0 + 0.5))


def _pair(seed: int, ctr: int, thr: int) -> int:
    """The 16 keep bits of the block at the 128-bit counter ctr."""
    words = philox4x64_10((ctr & _MASK64, ctr >> 64, 0, 0), (int(seed), 0))
    bits = 0
    for e in range(16):
        if ((words[e // 4] >> (16 * (e % 4))) & 0xFFFF) < thr:
            bits |= 1 << e
    return bits


def dropout_keep_philox(seed: int, offset: int, p, m: int, k: int, rows=None) -> np.ndarray:
    """Packed keep mask [len(rows), k/8] (rows default: all m rows) of the
    call (seed, offset, p, m, k); see the module docstring."""
    assert k % 8 == 0
    kb = k // 8
    rows = range(m) if rows is None else rows
    thr = keep_threshold(p)
    out = np.zeros((len(rows), kb), dtype=np.uint8)
    for ri, i in enumerate(rows):
        for q in range(kb):
            b = int(i) * kb + q                       # byte of the call
            bits = _pair(seed, int(offset) + b // 2, thr)
            out[ri, q] = (bits >> (8 * (b % 2))) & 0xFF
    return out
