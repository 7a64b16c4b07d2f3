"""Philox4xW-R in pure Python integers, written from its published
definition (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11).  TEST INFRASTRUCTURE ONLY.

This is an implementation independent of the C oracle's: it is generic over
the word width, so that its round function, key schedule and output order can
be checked against numpy's Philox4x64-10 bit generator, and its 32-bit
instance then pins the C oracle's Philox4x32-10 by agreement.
"""

# Round multipliers and Weyl key increments from the Philox definition.
CONSTANTS = {
    32: ((0xD2511F53, 0xCD9E8D57), (0x9E3779B9, 0xBB67AE85)),
    64: ((0xD2E7470EE14C6C93, 0xCA5A826395121157), (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)),
}


def philox4(counter, key, width=32, rounds=10):
    """One Philox4xW block: four W-bit output words for a four-word counter
    and a two-word key."""
    mult, weyl = CONSTANTS[width]
    mask = (1 << width) - 1
    c = [int(x) & mask for x in counter]
    k = [int(x) & mask for x in key]
    for r in range(rounds):
        if r:
            k = [(k[0] + weyl[0]) & mask, (k[1] + weyl[1]) & mask]
        p0 = mult[0] * c[0]
        p1 = mult[1] * c[2]
        c = [(p1 >> width) ^ c[1] ^ k[0], p1 & mask, (p0 >> width) ^ c[3] ^ k[1], p0 & mask]
    return c


def uniform(seed, i, m, t):
    """The stochastic-rounding uniform of element i, worker m, iteration t:
    counter (lo32(i>>2), m, t, hi32(i>>2)), key (lo32(seed), hi32(seed)),
    output word i & 3, u = (word >> 8) / 2**24 (exact in binary32)."""
    block = i >> 2
    words = philox4([block & 0xFFFFFFFF, m, t, block >> 32], [seed & 0xFFFFFFFF, seed >> 32], 32, 10)
    return (words[i & 3] >> 8) / float(1 << 24)
