"""Counter-based dropout masks (oracle).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper draws its dropout masks with cuRAND and stores them
(Sec. "Fusion Implementation"; Table 3 counts the masks among the outputs).
This build instead regenerates masks from a counter-based generator, so the
mask is a pure function of (seed, site, layer, logical element index):

* Generator: Philox4x32 with 10 rounds, as defined by Salmon, Moraes, Dror
  and Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11), Sec. 3:
  each round multiplies counter words 0 and 2 by the two round multipliers,
  keeps both halves of the 64-bit products, and mixes the high halves with
  the other two counter words and the round key; the two key words are
  bumped by the Weyl constants between rounds.
* Counter for logical element e: (lo32(e >> 2), hi32(e >> 2), site, layer);
  key: (lo32(seed), hi32(seed)); element e uses output word e & 3.
* Keep iff that word < thr, thr = floor((1 - p) * 2^32) (computed in double).
  p = 0 means no dropout at all (identity, no draws).
* Kept elements are scaled by 1 / (1 - p) (inverted dropout).

Parity: pinned against rocRAND's independent philox4x32_10 engine
(tests/test_oracle_philox.py) and by keep-rate statistics.
"""
from __future__ import annotations

import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF

# Dropout sites (the third counter word).
SITE_ATTN = 0       # attention probabilities, logical order (h, b, j, k)
SITE_ATTN_OUT = 1   # attention-block output, logical order (b, j, i)
SITE_FFN_OUT = 2    # feed-forward output, logical order (b, j, i)
SITE_FFN_ACT = 3    # after the feed-forward activation (paper's fourth dropout), (b, j, f)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Ten Philox4x32 rounds on uint32 counter words (arrays or scalars) and
    a two-word key.  Returns the four uint32 output words."""
    x = [np.asarray(c, dtype=np.uint64) & MASK32 for c in (c0, c1, c2, c3)]
    x = np.broadcast_arrays(*x)
    x = [a.copy() for a in x]
    ka = np.uint64(int(k0) & MASK32)
    kb = np.uint64(int(k1) & MASK32)
    for rnd in range(10):
        if rnd > 0:
            ka = np.uint64((int(ka) + W0) & MASK32)
            kb = np.uint64((int(kb) + W1) & MASK32)
        p0 = x[0] * np.uint64(M0)          # < 2^64: exact in uint64
        p1 = x[2] * np.uint64(M1)
        hi0, lo0 = p0 >> np.uint64(32), p0 & np.uint64(MASK32)
        hi1, lo1 = p1 >> np.uint64(32), p1 & np.uint64(MASK32)
        x = [hi1 ^ x[1] ^ ka, lo1, hi0 ^ x[3] ^ kb, lo0]
    return [a.astype(np.uint32) for a in x]


def keep_threshold(p: float) -> int:
    """Largest excluded 32-bit word: keep iff word < thr."""
    if not (0.0 <= p < 1.0):
        raise ValueError("dropout probability must lie in [0, 1)")
    return int(np.floor((1.0 - p) * 4294967296.0))


def random_words(seed: int, site: int, layer: int, e) -> np.ndarray:
    """The 32-bit word that decides logical element(s) e."""
    e = np.asarray(e, dtype=np.uint64)
    blk = e >> np.uint64(2)
    words = philox4x32_10(blk & np.uint64(MASK32), blk >> np.uint64(32),
                          np.uint64(site), np.uint64(layer),
                          seed & MASK32, (seed >> 32) & MASK32)
    sel = (e & np.uint64(3)).astype(np.int64)
    out = np.choose(sel, words)
    return out.astype(np.uint32)


def keep_mask(seed: int, site: int, layer: int, p: float, n: int, offset: int = 0) -> np.ndarray:
    """Boolean keep mask of logical elements offset .. offset+n-1."""
    if p == 0.0:
        return np.ones(n, dtype=bool)
    thr = keep_threshold(p)
    e = np.arange(offset, offset + n, dtype=np.uint64)
    return random_words(seed, site, layer, e).astype(np.uint64) < np.uint64(thr)


def dropout_factor(seed: int, site: int, layer: int, p: float, shape) -> np.ndarray:
    """float64 factor M / (1 - p) over a tensor whose C-order flat index is the
    logical element index."""
    n = int(np.prod(shape))
    if p == 0.0:
        return np.ones(shape)
    m = keep_mask(seed, site, layer, p, n).reshape(shape)
    return m.astype(np.float64) / (1.0 - p)
