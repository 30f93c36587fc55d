"""Pure-Python brute force over F_{p^2} = F_p[i] / (i^2 + 1), for tiny inputs.
Used to pin the oracle's F_{p^2} protocol; shares nothing with it.

Elements are represented by 2 x 2 matrices [[a, -b], [b, a]] over F_p (the
regular representation of a + b i: multiplying by a + b i maps the basis
(1, i) to (a + b i, -b + a i)), and multiplied as matrices, so the field
product is not retyped from the oracle's formula.
"""
from brute import P, bits_msb


class Fp2:
    __slots__ = ("m",)

    def __init__(self, a=0, b=0):
        a %= P
        b %= P
        self.m = ((a, (-b) % P), (b, a))

    @staticmethod
    def _of(x):
        return x if isinstance(x, Fp2) else Fp2(int(x), 0)

    @property
    def pair(self):
        return (self.m[0][0], self.m[1][0])

    def __add__(self, o):
        o = Fp2._of(o)
        return Fp2(self.m[0][0] + o.m[0][0], self.m[1][0] + o.m[1][0])

    __radd__ = __add__

    def __sub__(self, o):
        o = Fp2._of(o)
        return Fp2(self.m[0][0] - o.m[0][0], self.m[1][0] - o.m[1][0])

    def __rsub__(self, o):
        return Fp2._of(o) - self

    def __mul__(self, o):
        o = Fp2._of(o)
        a, b = self.m, o.m
        prod = [[sum(a[r][t] * b[t][c] for t in range(2)) % P for c in range(2)] for r in range(2)]
        assert prod[0][0] == prod[1][1] and (prod[0][1] + prod[1][0]) % P == 0  # stays in the field
        return Fp2(prod[0][0], prod[1][0])

    __rmul__ = __mul__

    def __eq__(self, o):
        return self.pair == Fp2._of(o).pair

    def __pow__(self, e):
        r, base = Fp2(1), self
        while e:
            if e & 1:
                r = r * base
            base = base * base
            e >>= 1
        return r


def eq_point2(z, y):
    acc = Fp2(1)
    for zi, yi in zip(z, y):
        acc = acc * (zi * yi + (1 - zi) * (1 - yi))
    return acc


def mle2(table, z):
    """Eq. (1) over F_{p^2}: sum_y e(y) prod_i (z_i y_i + (1 - z_i)(1 - y_i))."""
    v = len(z)
    assert len(table) == 1 << v
    acc = Fp2(0)
    for y, e in enumerate(table):
        acc = acc + Fp2._of(e) * eq_point2(z, bits_msb(y, v))
    return acc


def round_polys2(v, deg, f_at, rho):
    """Sum-check round polynomials of sum_x f(x) by direct hypercube sums, f_at
    evaluating the extended summand at a point of F_{p^2}^v."""
    out = []
    for j in range(v):
        g = []
        for X in range(deg + 1):
            acc = Fp2(0)
            for rest in range(1 << (v - j - 1)):
                acc = acc + f_at(list(rho[:j]) + [Fp2(X)] + [Fp2(b) for b in bits_msb(rest, v - j - 1)])
            g.append(acc.pair)
        out.append(g)
    return out
