"""Philox4x32-10 counter-based generator, uniforms and Gumbel noise (oracle side).

TEST INFRASTRUCTURE ONLY. This module belongs to the CPU oracle: only the
test suite, the smoke check and the benchmark's CPU-baseline leg may import
it. The product path (the HIP library) has its own, independent generator.

The generator is Philox4x32 with 10 rounds as defined by Salmon, Moraes, Dror
and Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11): a 128-bit
counter (four 32-bit words) and a 64-bit key (two words); each round
multiplies counter words 0 and 2 by two fixed 32-bit constants, and the new
counter is (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0));
the key is bumped by two Weyl constants between rounds.

The paper fixes no RNG; the method only needs independent uniforms per
(request, node, token) so that every random decision of replay (Section 3.2,
eq. (2)) and verification (Appendix A, recursive rejection sampling) is
addressable. Counter layout used by both sides of this project:

    word0 = draw >> 2            (element group of four draws)
    word1 = node | stream << 16  (tree node index, stream tag)
    word2 = request index
    word3 = step
    key   = (seed mod 2**32, seed >> 32);  output word = draw & 3

Streams: REPLAY (node = parent being refilled, draw = token id), ACCEPT
(node = child under test, draw = 0), BONUS (node = terminal node, draw =
token id).

All arithmetic below is on numpy uint64 arrays holding 32-bit values, so that
32x32 products are exact.
"""
import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint64(0x9E3779B9)
W1 = np.uint64(0xBB67AE85)
MASK32 = np.uint64(0xFFFFFFFF)
SH32 = np.uint64(32)

STREAM_REPLAY = 0
STREAM_ACCEPT = 1
STREAM_BONUS = 2


def philox4x32_10(ctr, key):
    """Philox4x32-10 on broadcastable uint64 arrays.

    ctr: tuple of 4 arrays (or ints) holding 32-bit counter words.
    key: tuple of 2 arrays (or ints) holding 32-bit key words.
    Returns the four 32-bit output words as uint64 arrays.
    """
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) & MASK32 for c in ctr)
    k0, k1 = (np.asarray(k, dtype=np.uint64) & MASK32 for k in key)
    for rnd in range(10):
        p0 = M0 * c0
        p1 = M1 * c2
        hi0, lo0 = p0 >> SH32, p0 & MASK32
        hi1, lo1 = p1 >> SH32, p1 & MASK32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
        if rnd != 9:
            k0 = (k0 + W0) & MASK32
            k1 = (k1 + W1) & MASK32
    return c0, c1, c2, c3


def seed_key(seed):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return (seed & 0xFFFFFFFF, seed >> 32)


def draw_words(seed, step, request, node, stream, draws):
    """32-bit words for the given draw indices of one (step, request, node, stream)."""
    draws = np.asarray(draws, dtype=np.uint64)
    ctr = (draws >> np.uint64(2),
           np.uint64((int(node) & 0xFFFF) | (int(stream) << 16)),
           np.uint64(int(request) & 0xFFFFFFFF),
           np.uint64(int(step) & 0xFFFFFFFF))
    words = philox4x32_10(ctr, seed_key(seed))
    sel = (draws & np.uint64(3)).astype(np.int64)
    out = np.choose(sel, words) if draws.ndim else words[int(sel)]
    return np.asarray(out, dtype=np.uint64)


def u24(words):
    """Uniform in (0, 1): (2*(w >> 9) + 1) * 2**-24, exact in binary32 and binary64."""
    w = np.asarray(words, dtype=np.uint64)
    k = (w >> np.uint64(9)).astype(np.float64)
    return (2.0 * k + 1.0) * (2.0 ** -24)


def gumbel(u):
    """Standard Gumbel noise -ln(-ln u), in binary64."""
    u = np.asarray(u, dtype=np.float64)
    return -np.log(-np.log(u))


def uniforms(seed, step, request, node, stream, draws):
    return u24(draw_words(seed, step, request, node, stream, draws))


def gumbels(seed, step, request, node, stream, n):
    """Gumbel noise for draws 0..n-1 of one (step, request, node, stream)."""
    return gumbel(uniforms(seed, step, request, node, stream, np.arange(n, dtype=np.uint64)))


# Largest and smallest Gumbel value the 24-bit uniform can produce.
G_MAX = float(gumbel((2.0 ** 24 - 1.0) * 2.0 ** -24))
G_MIN = float(gumbel(2.0 ** -24))
