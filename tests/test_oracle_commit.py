"""Pins of the commitment oracle (oracle/ec_oracle.py), each against
something other than the oracle: the published group order of secp256k1
(n G is the identity, a property a wrong constant, a wrong curve equation or a
wrong group law would break), group-law identities, the defining properties
of the generator rule (the hash, Euler's criterion on every counter tried,
the even root), and the homomorphism of the commitment."""
import hashlib
import random

from oracle import ec_oracle as ec


def test_base_point_and_order():
    assert ec.on_curve(ec.G)
    assert ec.mul(ec.N, ec.G) is None
    assert ec.mul(ec.N - 1, ec.G) == ec.neg(ec.G)
    assert ec.mul(ec.N + 5, ec.G) == ec.mul(5, ec.G)
    assert ec.Q % 4 == 3


def test_group_law_identities():
    rng = random.Random(7)
    pts = [ec.mul(rng.randrange(1, ec.N), ec.G) for _ in range(6)]
    for p in pts:
        assert ec.on_curve(p)
        assert ec.add(p, ec.neg(p)) is None
        assert ec.add(p, None) == p
        assert ec.add(p, p) == ec.mul(2, p)
    a, b, c = pts[:3]
    assert ec.add(a, b) == ec.add(b, a)
    assert ec.add(ec.add(a, b), c) == ec.add(a, ec.add(b, c))
    for _ in range(5):
        k1, k2 = rng.randrange(-2 ** 40, 2 ** 40), rng.randrange(-2 ** 40, 2 ** 40)
        assert ec.add(ec.mul(k1, a), ec.mul(k2, a)) == ec.mul(k1 + k2, a)
        assert ec.mul(k1, ec.mul(k2, b)) == ec.mul(k1 * k2, b)


def test_generator_rule():
    domain = hashlib.sha256(b"generator pins").digest()
    for i in (0, 1, 2, 17, 2 ** 20):
        (x, y), c = ec.generator_with_counter(domain, i)
        assert ec.on_curve((x, y)) and y % 2 == 0
        for cc in range(c + 1):
            h = hashlib.sha256(ec.GEN_TAG + domain + i.to_bytes(8, "little") + cc.to_bytes(4, "little")).digest()
            xx = int.from_bytes(h, "big") % ec.Q
            square = pow((xx ** 3 + 7) % ec.Q, (ec.Q - 1) // 2, ec.Q) == 1
            assert square == (cc == c)
            if cc == c:
                assert xx == x
    gens = ec.generators(domain, 8)
    assert len(set(gens)) == 8


def test_commitment_homomorphism():
    domain = hashlib.sha256(b"commit pins").digest()
    gens = ec.generators(domain, 16)
    rng = random.Random(3)
    a = [rng.randrange(-2 ** 31, 2 ** 31) for _ in range(16)]
    b = [rng.randrange(-2 ** 31, 2 ** 31) for _ in range(16)]
    ca, cb = ec.commit(a, gens), ec.commit(b, gens)
    assert ec.add(ca, cb) == ec.commit([x + y for x, y in zip(a, b)], gens)
    assert ec.neg(ca) == ec.commit([-x for x in a], gens)
    assert ec.commit([0] * 16, gens) is None
    for i in (0, 5, 15):
        e = [0] * 16
        e[i] = 1
        assert ec.commit(e, gens) == gens[i]
    assert ec.commit([3] + [0] * 15, gens) == ec.mul(3, gens[0])
    assert ec.decode(ec.encode(ca)) == ca and ec.decode(ec.encode(None)) is None
