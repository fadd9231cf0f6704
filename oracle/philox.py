"""Philox4x32 counter-based random numbers (oracle; test infrastructure only).

Definition: J. Salmon, M. Moraes, R. Dror, D. Shaw, "Parallel random numbers:
as easy as 1, 2, 3", SC'11, Sec. 3 (the Philox S-box and key schedule).  The
round count is a parameter of the family: the authors found Philox4x32 to pass
their statistical test batteries from seven rounds on and recommend ten for
a safety margin.  The FQT stream uses seven (ROUNDS): the paper asks only for
independent uniforms (Sec. 3.3), and each round costs the GPU quantizer two
wide multiplies per four elements.

One bijection maps a 128-bit counter (four 32-bit words) under a 64-bit key
(two 32-bit words) to four 32-bit outputs.  A round multiplies words 0 and 2 by
two fixed odd multipliers; the high halves of the 64-bit products are XOR-ed
with the other two words and the round key, and the low halves are carried
through with the word order swapped.  Between rounds the key is advanced by
two Weyl increments (the golden ratio and sqrt(3)-1 scaled to 32 bits).

The FQT stochastic-rounding stream uses Philox4x32-7 as follows:

  key     = (lo32(seed), hi32(seed))
  counter = (lo32(e >> 2), hi32(e >> 2), stream, 0)
  draw    = output word (e & 3)

where e is the logical row-major element index.  Vectorised over numpy uint64
arrays holding 32-bit values.
"""
import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)
# Multipliers and Weyl increments of Philox4x32 (Salmon et al., SC'11).
PHILOX_M0 = np.uint64(0xD2511F53)
PHILOX_M1 = np.uint64(0xCD9E8D57)
PHILOX_W0 = np.uint64(0x9E3779B9)
PHILOX_W1 = np.uint64(0xBB67AE85)
ROUNDS = 7  # the FQT stream; philox4x32(..., rounds=10) is the authors' default


def philox4x32(c0, c1, c2, c3, k0, k1, rounds=ROUNDS):
    """Apply Philox4x32-`rounds` to counters (c0..c3) under key (k0, k1).

    All arguments are numpy arrays (or scalars) of 32-bit values held in
    uint64.  Returns a tuple of four uint64 arrays of 32-bit outputs.
    """
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & MASK32 for c in (c0, c1, c2, c3))
    k0 = np.asarray(k0, dtype=np.uint64) & MASK32
    k1 = np.asarray(k1, dtype=np.uint64) & MASK32
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + PHILOX_W0) & MASK32
            k1 = (k1 + PHILOX_W1) & MASK32
        p0 = PHILOX_M0 * c0          # < 2^64, exact in uint64
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def draws(elem_index, seed, stream):
    """32-bit Philox words for logical element indices `elem_index` (uint64 array).

    Element e takes word (e & 3) of the block at counter e >> 2.  When the
    indices come in aligned runs of four (e, e+1, e+2, e+3 with e % 4 == 0),
    each block is evaluated once and its four words are used in order; the
    result is the same as evaluating every element on its own.
    """
    e = np.asarray(elem_index, dtype=np.uint64)
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    k0, k1 = np.uint64(seed & 0xFFFFFFFF), np.uint64(seed >> 32)
    flat = e.reshape(-1)
    if flat.size and flat.size % 4 == 0:
        quads = flat.reshape(-1, 4)
        first = quads[:, 0]
        if ((first & np.uint64(3)) == 0).all() and (quads == first[:, None] + np.arange(4, dtype=np.uint64)).all():
            q = first >> np.uint64(2)
            o = philox4x32(q & MASK32, q >> np.uint64(32), np.uint64(stream), np.uint64(0), k0, k1)
            return np.stack(o, axis=1).reshape(e.shape).astype(np.uint64)
    q = e >> np.uint64(2)
    o = philox4x32(q & MASK32, q >> np.uint64(32), np.uint64(stream), np.uint64(0), k0, k1)
    w = (e & np.uint64(3)).astype(np.int64)
    out = np.where(w == 0, o[0], np.where(w == 1, o[1], np.where(w == 2, o[2], o[3])))
    return out.astype(np.uint64)
