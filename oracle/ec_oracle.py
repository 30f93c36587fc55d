"""Pedersen vector commitments over secp256k1, plain and slow.

TEST INFRASTRUCTURE ONLY: nothing in the product library imports, loads or
calls this file, and it shares no code with the GPU path.

The paper commits to a vector a by the group element g^a = prod g_i^{a_i}
(Sec. II-C; multiplicative notation), with public generators g of a group in
which discrete logarithms are hard, instantiated on secp256k1 or BLS12-381
(Sec. IV, security parameters).  Here, additively, P = sum_i a_i G_i on
secp256k1: y^2 = x^3 + 7 over F_q, q = 2^256 - 2^32 - 977, with the group
order and base point of the SEC 2 standard.

Generators (a reading: the paper only asks for public generators): G_i is
found by try-and-increment from SHA-256: for c = 0, 1, ...,
x = SHA-256("range-arithmetic generators v1" || domain || LE64(i) || LE32(c))
read big-endian, mod q; the first x for which x^3 + 7 is a square mod q gives
G_i = (x, y) with y its even square root.  Nobody knows a relation between
them.

Encoding of a point: 64 bytes, x then y, big-endian; the identity is 64 zero
bytes.  Every operation is Python integer arithmetic on affine points (the
chord-and-tangent law), scalar multiplication by double-and-add.
"""
import hashlib

Q = 2 ** 256 - 2 ** 32 - 977
N = 0xFFFFFFFFFFFFFFFFFFFFFFFFFFFFFFFEBAAEDCE6AF48A03BBFD25E8CD0364141
G = (0x79BE667EF9DCBBAC55A06295CE870B07029BFCDB2DCE28D959F2815B16F81798,
     0x483ADA7726A3C4655DA4FBFC0E1108A8FD17B448A68554199C47D08FFB10D4B8)
GEN_TAG = b"range-arithmetic generators v1"


def on_curve(pt) -> bool:
    if pt is None:
        return True
    x, y = pt
    return 0 <= x < Q and 0 <= y < Q and (y * y - x * x * x - 7) % Q == 0


def neg(pt):
    return None if pt is None else (pt[0], (-pt[1]) % Q)


def add(p1, p2):
    """The group law on affine points (None is the identity)."""
    if p1 is None:
        return p2
    if p2 is None:
        return p1
    (x1, y1), (x2, y2) = p1, p2
    if x1 == x2:
        if (y1 + y2) % Q == 0:
            return None
        lam = 3 * x1 * x1 * pow(2 * y1, -1, Q) % Q          # tangent
    else:
        lam = (y2 - y1) * pow(x2 - x1, -1, Q) % Q            # chord
    x3 = (lam * lam - x1 - x2) % Q
    return x3, (lam * (x1 - x3) - y1) % Q


def mul(k: int, pt):
    """k pt for any integer k (double-and-add over |k|)."""
    if k < 0:
        return mul(-k, neg(pt))
    acc, base = None, pt
    while k:
        if k & 1:
            acc = add(acc, base)
        base = add(base, base)
        k >>= 1
    return acc


def generator_with_counter(domain: bytes, i: int):
    """(G_i, the counter c that gave it)."""
    assert len(domain) == 32
    c = 0
    while True:
        h = hashlib.sha256(GEN_TAG + domain + i.to_bytes(8, "little") + c.to_bytes(4, "little")).digest()
        x = int.from_bytes(h, "big") % Q
        rhs = (x * x * x + 7) % Q
        if pow(rhs, (Q - 1) // 2, Q) == 1:                    # Euler's criterion
            y = pow(rhs, (Q + 1) // 4, Q)                     # q = 3 mod 4
            if y & 1:
                y = Q - y
            return (x, y), c
        c += 1


def generator(domain: bytes, i: int):
    return generator_with_counter(domain, i)[0]


def generators(domain: bytes, count: int):
    return [generator(domain, i) for i in range(count)]


def commit(values, gens):
    """sum_i values[i] gens[i] (values: integers, any sign)."""
    acc = None
    for v, g in zip(values, gens):
        if int(v):
            acc = add(acc, mul(int(v), g))
    return acc


def encode(pt) -> bytes:
    if pt is None:
        return bytes(64)
    return pt[0].to_bytes(32, "big") + pt[1].to_bytes(32, "big")


def decode(b: bytes):
    if b == bytes(64):
        return None
    return int.from_bytes(b[:32], "big"), int.from_bytes(b[32:], "big")
