"""Arithmetic in GF(2)[x] / p(x) with p(x) = x^32 + x^22 + x^2 + x + 1 (test helper).

Polynomials are Python ints, bit k = coefficient of x^k.  Used to pin the LFSR
register of the comparator sequence to the algebra it is meant to implement:
a Galois right-shift step multiplies the state polynomial by x^{-1} mod p, so the
state after n steps from S_0 is S_0 * x^{-n} mod p, and the period is the order of
x, which is 2^32 - 1 exactly when p is primitive.
"""

P = (1 << 32) | (1 << 22) | (1 << 2) | (1 << 1) | 1
ORDER = (1 << 32) - 1
ORDER_PRIME_FACTORS = (3, 5, 17, 257, 65537)


def pmod(a, p=P):
    dp = p.bit_length() - 1
    while a.bit_length() - 1 >= dp:
        a ^= p << (a.bit_length() - 1 - dp)
    return a


def pmul(a, b, p=P):
    r = 0
    while b:
        if b & 1:
            r ^= a
        a <<= 1
        b >>= 1
    return pmod(r, p)


def ppow(a, e, p=P):
    r = 1
    a = pmod(a, p)
    while e:
        if e & 1:
            r = pmul(r, a, p)
        a = pmul(a, a, p)
        e >>= 1
    return r


def x_inverse():
    """x^{-1} mod p = x^{ORDER-1} (valid once x has order ORDER)."""
    return ppow(2, ORDER - 1)
