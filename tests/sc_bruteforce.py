"""Pure-Python brute force of the SC GEMM for tiny inputs (test helper).

An implementation independent of the C oracle (no shared code): its own
SplitMix64, its own LFSR, its own boundary maps, explicit lists of stream bits,
XNOR/AND per bit, and an exact rational decode with ``fractions.Fraction``.
Only for M, N, K <= a few and L <= a few hundred.

Follows the paper's Sec. 3.1 (encoding, comparator SNG, Eq. (1)), Sec. 4.2
(boundaries, per-row lengths) and Sec. A.1 (LFSR), with the same readings as the
oracle (R-LFSR, R-SEED, R-BETA, R-SHARE, R-L0, R-UNI).
"""
from fractions import Fraction

MASK64 = (1 << 64) - 1
QMAX = 127


def splitmix64(x):
    z = (x + 0x9E3779B97F4A7C15) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def seed_state(seed, op):
    s = splitmix64((2 * seed + op) & MASK64) >> 32
    return s if s != 0 else 1


def lfsr_bits(state, nbits):
    """Output bits of the Galois right-shift register with taps x^32+x^22+x^2+x+1."""
    s = state
    out = []
    for _ in range(nbits):
        b = s & 1
        out.append(b)
        s >>= 1
        if b:
            s ^= (1 << 31) | (1 << 21) | (1 << 1) | 1
    return out


def draws(seed, op, n):
    bits = lfsr_bits(seed_state(seed, op), 8 * n)
    r = []
    for l in range(n):
        v = 0
        for t in range(8):
            v = 2 * v + bits[8 * l + t]
        r.append(v)
    return r


def beta_bipolar(q):
    # round half up of 256 (q + 127) / 254
    num = 256 * (q + QMAX)
    return (2 * num + 254) // (2 * 254)


def beta_unipolar(q):
    # round half up of 256 |q| / 127 ... written as floor((256|q| + 63)/127)
    return (256 * abs(q) + 63) // 127


def stream(r, beta, length):
    return [1 if r[l] < beta else 0 for l in range(length)]


def sc_gemm(A, B, sA, sB, L, polarity, seed):
    """A: list of M lists of K ints; B: N lists of K ints.  Returns (counts, out).

    ``out`` entries are exact Fractions of the float32 scales.
    """
    M, N = len(A), len(B)
    K = len(A[0]) if M else 0
    Lmax = max(L) if L else 0
    rA = draws(seed, 0, Lmax)
    rB = draws(seed, 1, Lmax)
    counts = [[0] * N for _ in range(M)]
    out = [[Fraction(0)] * N for _ in range(M)]
    for i in range(M):
        Li = L[i]
        for j in range(N):
            c = 0
            for d in range(K):
                a, b = A[i][d], B[j][d]
                if polarity == 0:
                    za = stream(rA, beta_bipolar(a), Li)
                    zb = stream(rB, beta_bipolar(b), Li)
                    c += sum(1 - (x ^ y) for x, y in zip(za, zb))
                else:
                    za = stream(rA, beta_unipolar(a), Li)
                    zb = stream(rB, beta_unipolar(b), Li)
                    p = sum(x & y for x, y in zip(za, zb))
                    c += p if (a < 0) == (b < 0) else -p
            counts[i][j] = c
            if Li > 0:
                scale = Fraction(sA[i]) * Fraction(sB[j]) * QMAX * QMAX
                if polarity == 0:
                    out[i][j] = scale * (Fraction(2 * c, Li) - K)
                else:
                    out[i][j] = scale * Fraction(c, Li)
    return counts, out


# ---------------------------------------------------------------------------
# Sobol-8 and conditional bitstream generation, written independently
# ---------------------------------------------------------------------------

def sobol8_points(dim, shift, n=256):
    """Natural-order Sobol points of dimension 1 or 2 as 8-bit integers.

    Dimension 1 is the base-2 radical inverse; dimension 2 uses direction numbers of
    the polynomial x + 1, computed here as bit-reversed binomial coefficients mod 2.
    """
    pts = []
    for k in range(n):
        if dim == 1:
            x = int("{:08b}".format(k)[::-1], 2)
        else:
            x = 0
            for j in range(8):
                if (k >> j) & 1:
                    # m_{j+1} of x + 1 is the odd number whose bits are row j of Pascal's
                    # triangle mod 2
                    m = sum(((1 if (j & i) == i else 0) << i) for i in range(j + 1))
                    x ^= m << (8 - (j + 1))
        pts.append(x ^ shift)
    return pts


def cbsg_gemm(A, B, sA, sB, L, polarity, seed):
    M, N = len(A), len(B)
    K = len(A[0]) if M else 0
    sh_a = splitmix64((2 * seed) & MASK64) >> 56
    sh_b = splitmix64((2 * seed + 1) & MASK64) >> 56
    rA = sobol8_points(1, sh_a)
    rB = sobol8_points(2, sh_b)
    counts = [[0] * N for _ in range(M)]
    out = [[Fraction(0)] * N for _ in range(M)]
    bfun = beta_bipolar if polarity == 0 else beta_unipolar
    for i in range(M):
        Li = L[i]
        for j in range(N):
            c = 0
            for d in range(K):
                ba, bb = bfun(A[i][d]), bfun(B[j][d])
                ones = zeros = 0
                s = 0
                for l in range(Li):
                    a = 1 if rA[l] < ba else 0
                    if a:
                        bbit = 1 if rB[ones] < bb else 0
                        ones += 1
                    else:
                        bbit = 1 if rB[zeros] < bb else 0
                        zeros += 1
                    if polarity == 0:
                        s += 1 if a == bbit else 0
                    else:
                        s += a & bbit
                if polarity == 1 and (A[i][d] < 0) != (B[j][d] < 0):
                    s = -s
                c += s
            counts[i][j] = c
            if Li > 0:
                scale = Fraction(sA[i]) * Fraction(sB[j]) * QMAX * QMAX
                out[i][j] = scale * (Fraction(2 * c, Li) - K) if polarity == 0 else scale * Fraction(c, Li)
    return counts, out
