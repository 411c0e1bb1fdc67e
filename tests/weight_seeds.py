"""Seeds whose round-0 weight of colour 0 is a chosen 64-bit word.

Algorithm 1 draws the weight of colour b in round r from a counter-based
SplitMix64 stream (Steele, Lea and Flood 2014): with the increment g and the
output function mix,

    key(seed, r) = mix(mix(seed + g) + (r + 1) g),   W = mix(key + (b + 1) g),

taken as it is in Z/2^64 and reduced mod p = 2^61 - 1 in F_p.  mix is a
composition of xor-shifts and multiplications by odd constants, each a
bijection of 64-bit words, so W for r = 0, b = 0 is inverted step by step.
The weights that come out are degenerate on purpose: 2^62 in Z/2^64 makes the
one-colour round's values d W depend on d mod 4 only, and 0 in F_p makes all
of them equal.  tests/test_oracle_degenerate_weight.py checks these seeds
against the oracle's own weight function.
"""
M = (1 << 64) - 1
G = 0x9E3779B97F4A7C15
C1 = 0xBF58476D1CE4E5B9
C2 = 0x94D049BB133111EB


def mix(z):
    z &= M
    z = ((z ^ (z >> 30)) * C1) & M
    z = ((z ^ (z >> 27)) * C2) & M
    return z ^ (z >> 31)


def _unxorshift(y, s):
    # y = x ^ (x >> s)  =>  x = y ^ (y >> s) ^ (y >> 2s) ^ ...
    x, t = y, y >> s
    while t:
        x ^= t
        t >>= s
    return x


def unmix(z):
    z = _unxorshift(z & M, 31)
    z = (z * pow(C2, -1, 1 << 64)) & M
    z = _unxorshift(z, 27)
    z = (z * pow(C1, -1, 1 << 64)) & M
    return _unxorshift(z, 30)


def seed_for_weight0(w):
    """The seed whose stream gives colour 0 the raw output w in round 0."""
    key = (unmix(w) - G) & M
    s1 = (unmix(key) - G) & M
    return (unmix(s1) - G) & M
