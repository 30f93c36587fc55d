"""Pure-Python brute force written from the paper's definitions, for tiny
inputs only.  Used to pin the oracle; shares nothing with it.

 - multilinear extension by Eq. (1) (sum over the hypercube of the table times
   the product of per-variable Lagrange factors);
 - sum-check round polynomials by direct summation over the hypercube of the
   extended summand (Sec. II-D), evaluating every multilinear factor at the
   partially-bound point by Eq. (1);
 - the rounding operator of Sec. II-A with Python's floor modulo.
"""
P = (1 << 61) - 1


def bits_msb(y, v):
    return [(y >> (v - 1 - i)) & 1 for i in range(v)]


def eq_point(z, y_bits):
    """prod_i (z_i y_i + (1 - z_i)(1 - y_i)) for arbitrary field points y."""
    acc = 1
    for zi, yi in zip(z, y_bits):
        acc = acc * ((zi * yi + (1 - zi) * (1 - yi)) % P) % P
    return acc


def mle(table, z):
    """Eq. (1): e~(z) = sum_y e(y) prod_i (z_i y_i + (1 - z_i)(1 - y_i))."""
    v = len(z)
    assert len(table) == 1 << v
    acc = 0
    for y, e in enumerate(table):
        acc = (acc + (int(e) % P) * eq_point(z, bits_msb(y, v))) % P
    return acc


def rounding(x, s):
    """Operator of Sec. II-A: (x + 2^(s-1) - ((x + 2^(s-1)) mod 2^s)) / 2^s."""
    h = 1 << (s - 1)
    return (x + h - ((x + h) % (1 << s))) // (1 << s)


def round_polys(v, deg, f_at, rho):
    """Round polynomials of the sum-check for sum_{x in {0,1}^v} f(x), where
    f_at(point) evaluates the extended summand at any field point."""
    out = []
    for j in range(v):
        g = []
        for X in range(deg + 1):
            acc = 0
            for rest in range(1 << (v - j - 1)):
                pt = list(rho[:j]) + [X] + bits_msb(rest, v - j - 1)
                acc = (acc + f_at(pt)) % P
            g.append(acc)
        out.append(g)
    return out


def lagrange_eval(evals, x):
    """Value at x of the polynomial through (i, evals[i]), i = 0..d."""
    d = len(evals) - 1
    acc = 0
    for i in range(d + 1):
        num, den = 1, 1
        for j in range(d + 1):
            if j != i:
                num = num * (x - j) % P
                den = den * (i - j) % P
        acc = (acc + evals[i] * num * pow(den, P - 2, P)) % P
    return acc
