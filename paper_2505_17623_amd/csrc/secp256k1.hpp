// secp256k1.hpp -- the group of the commitments: y^2 = x^3 + 7 over F_q,
// q = 2^256 - 2^32 - 977 (the curve Sec. IV names), on the host and the
// device.
//
// Field elements are 8 little-endian 32-bit limbs, canonical in [0, q).  A
// product is the 512-bit schoolbook product reduced with 2^256 = 2^32 + 977
// (mod q), twice.  Points are Jacobian (X, Y, Z) with x = X / Z^2, y = Y /
// Z^3 (Z = 0: the identity); generators are affine.  The doubling and
// addition formulas are the standard ones for a = 0 (Jacobian doubling with
// A = X^2, B = Y^2, C = B^2; mixed and full additions with the
// H = U2 - U1, r = 2 (S2 - S1) form), each checked for the special cases
// (identity, equal points, opposite points).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace secp {

#define SECP_HD __host__ __device__ __forceinline__

struct Fe {
    uint32_t v[8];
};

// q and 2^256 - q = 2^32 + 977
constexpr uint32_t kQ[8] = {0xFFFFFC2Fu, 0xFFFFFFFEu, 0xFFFFFFFFu, 0xFFFFFFFFu,
                            0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
constexpr uint32_t kFold = 977;  // 2^256 = 2^32 + 977 (mod q)

SECP_HD Fe fe_zero()
{
    Fe r;
    for (int i = 0; i < 8; i++) r.v[i] = 0;
    return r;
}
SECP_HD Fe fe_small(uint32_t a)
{
    Fe r = fe_zero();
    r.v[0] = a;
    return r;
}
SECP_HD bool fe_is_zero(const Fe &a)
{
    uint32_t o = 0;
    for (int i = 0; i < 8; i++) o |= a.v[i];
    return o == 0;
}
SECP_HD bool fe_eq(const Fe &a, const Fe &b)
{
    uint32_t o = 0;
    for (int i = 0; i < 8; i++) o |= a.v[i] ^ b.v[i];
    return o == 0;
}

// r + (2^32 + 977) over 256 bits; returns the carry out
SECP_HD uint32_t add_fold(Fe &r, const Fe &a)
{
    uint64_t c = (uint64_t)a.v[0] + kFold;
    r.v[0] = (uint32_t)c;
    c = (c >> 32) + (uint64_t)a.v[1] + 1;
    r.v[1] = (uint32_t)c;
    c >>= 32;
    for (int i = 2; i < 8; i++) {
        c += a.v[i];
        r.v[i] = (uint32_t)c;
        c >>= 32;
    }
    return (uint32_t)c;
}

// s < 2^256 with a possible carry bit above it, s + carry 2^256 < 2q -> [0, q)
SECP_HD Fe fe_canon(const Fe &s, uint32_t carry)
{
    Fe t;
    const uint32_t c2 = add_fold(t, s);  // t = s + 2^256 - q = s - q (mod 2^256)
    return (carry | c2) ? t : s;
}

SECP_HD Fe fe_add(const Fe &a, const Fe &b)
{
    Fe s;
    uint64_t c = 0;
    for (int i = 0; i < 8; i++) {
        c += (uint64_t)a.v[i] + b.v[i];
        s.v[i] = (uint32_t)c;
        c >>= 32;
    }
    return fe_canon(s, (uint32_t)c);
}

SECP_HD Fe fe_sub(const Fe &a, const Fe &b)
{
    Fe d;
    int64_t c = 0;
    for (int i = 0; i < 8; i++) {
        c += (int64_t)a.v[i] - (int64_t)b.v[i];
        d.v[i] = (uint32_t)c;
        c >>= 32;  // arithmetic: 0 or -1
    }
    if (c) {  // borrow: d + q = d - (2^32 + 977) mod 2^256
        int64_t e = (int64_t)d.v[0] - kFold;
        d.v[0] = (uint32_t)e;
        e = (e >> 32) + (int64_t)d.v[1] - 1;
        d.v[1] = (uint32_t)e;
        e >>= 32;
        for (int i = 2; i < 8; i++) {
            e += d.v[i];
            d.v[i] = (uint32_t)e;
            e >>= 32;
        }
    }
    return d;
}

SECP_HD Fe fe_neg(const Fe &a) { return fe_sub(fe_zero(), a); }

SECP_HD Fe fe_mul(const Fe &a, const Fe &b)
{
    uint32_t t[16];
    for (int i = 0; i < 16; i++) t[i] = 0;
    for (int i = 0; i < 8; i++) {
        uint64_t c = 0;
        for (int j = 0; j < 8; j++) {
            c += (uint64_t)a.v[i] * b.v[j] + t[i + j];
            t[i + j] = (uint32_t)c;
            c >>= 32;
        }
        t[i + 8] = (uint32_t)c;
    }
    // L + H (2^32 + 977): limb i gets L_i + 977 H_i + H_{i-1}
    uint32_t r[8];
    uint64_t c = 0;
    for (int i = 0; i < 8; i++) {
        c += (uint64_t)t[i] + (uint64_t)t[8 + i] * kFold + (i ? t[7 + i] : 0);
        r[i] = (uint32_t)c;
        c >>= 32;
    }
    // the part at 2^256: below 2^32 + 978, so it can exceed 32 bits (when H is
    // within about 2^-22 of 2^256, e.g. for (q - 1)^2)
    const uint64_t r8 = c + t[15];
    // fold it again: r8 (2^32 + 977)
    Fe s;
    c = (uint64_t)r[0] + r8 * kFold;
    s.v[0] = (uint32_t)c;
    c = (c >> 32) + (uint64_t)r[1] + r8;
    s.v[1] = (uint32_t)c;
    c >>= 32;
    for (int i = 2; i < 8; i++) {
        c += r[i];
        s.v[i] = (uint32_t)c;
        c >>= 32;
    }
    if (c) {  // one more 2^256: s + 2^32 + 977 cannot carry again
        Fe u;
        add_fold(u, s);
        s = u;
    }
    return fe_canon(s, 0);
}

SECP_HD Fe fe_sqr(const Fe &a) { return fe_mul(a, a); }

// a^e for a 256-bit exponent e (8 little-endian limbs), square-and-multiply
SECP_HD Fe fe_pow(const Fe &a, const uint32_t e[8])
{
    Fe r = fe_small(1);
    for (int i = 255; i >= 0; i--) {
        r = fe_sqr(r);
        if ((e[i >> 5] >> (i & 31)) & 1) r = fe_mul(r, a);
    }
    return r;
}

SECP_HD Fe fe_inv(const Fe &a)  // a^(q - 2)
{
    uint32_t e[8];
    for (int i = 0; i < 8; i++) e[i] = kQ[i];
    e[0] -= 2;
    return fe_pow(a, e);
}

// a^((q + 1) / 4): a square root when a is a square (q = 3 mod 4)
SECP_HD Fe fe_sqrt(const Fe &a)
{
    uint32_t e[8];
    uint64_t c = 1;  // (q + 1) / 4 = q / 4 + 1 / 4 ... computed as (q + 1) >> 2
    uint32_t q1[8];
    for (int i = 0; i < 8; i++) {
        c += kQ[i];
        q1[i] = (uint32_t)c;
        c >>= 32;
    }
    for (int i = 0; i < 8; i++) e[i] = (q1[i] >> 2) | (i < 7 ? (q1[i + 1] << 30) : ((uint32_t)c << 30));
    return fe_pow(a, e);
}

struct Jac {
    Fe X, Y, Z;
};
struct Aff {
    Fe x, y;
};

SECP_HD Jac jac_inf()
{
    Jac r;
    r.X = fe_small(1);
    r.Y = fe_small(1);
    r.Z = fe_zero();
    return r;
}
SECP_HD bool jac_is_inf(const Jac &p) { return fe_is_zero(p.Z); }
SECP_HD Jac jac_neg(const Jac &p)
{
    Jac r = p;
    r.Y = fe_neg(p.Y);
    return r;
}

SECP_HD Jac jac_dbl(const Jac &p)
{
    if (jac_is_inf(p) || fe_is_zero(p.Y)) return jac_inf();
    const Fe A = fe_sqr(p.X), B = fe_sqr(p.Y), C = fe_sqr(B);
    Fe D = fe_sub(fe_sub(fe_sqr(fe_add(p.X, B)), A), C);
    D = fe_add(D, D);
    const Fe E = fe_add(fe_add(A, A), A), F = fe_sqr(E);
    Jac r;
    r.X = fe_sub(F, fe_add(D, D));
    Fe C8 = fe_add(C, C);
    C8 = fe_add(C8, C8);
    C8 = fe_add(C8, C8);
    r.Y = fe_sub(fe_mul(E, fe_sub(D, r.X)), C8);
    const Fe YZ = fe_mul(p.Y, p.Z);
    r.Z = fe_add(YZ, YZ);
    return r;
}

// p + q for an affine q (q is never the identity)
SECP_HD Jac jac_add_aff(const Jac &p, const Aff &q)
{
    if (jac_is_inf(p)) {
        Jac r;
        r.X = q.x;
        r.Y = q.y;
        r.Z = fe_small(1);
        return r;
    }
    const Fe Z1Z1 = fe_sqr(p.Z);
    const Fe U2 = fe_mul(q.x, Z1Z1);
    const Fe S2 = fe_mul(q.y, fe_mul(p.Z, Z1Z1));
    const Fe H = fe_sub(U2, p.X);
    const Fe rr = fe_sub(S2, p.Y);
    if (fe_is_zero(H)) {
        if (fe_is_zero(rr)) return jac_dbl(p);
        return jac_inf();
    }
    const Fe HH = fe_sqr(H);
    Fe I = fe_add(HH, HH);
    I = fe_add(I, I);
    const Fe J = fe_mul(H, I);
    const Fe r2 = fe_add(rr, rr);
    const Fe V = fe_mul(p.X, I);
    Jac o;
    o.X = fe_sub(fe_sub(fe_sqr(r2), J), fe_add(V, V));
    const Fe YJ = fe_mul(p.Y, J);
    o.Y = fe_sub(fe_mul(r2, fe_sub(V, o.X)), fe_add(YJ, YJ));
    o.Z = fe_sub(fe_sub(fe_sqr(fe_add(p.Z, H)), Z1Z1), HH);
    return o;
}

SECP_HD Jac jac_add(const Jac &p, const Jac &q)
{
    if (jac_is_inf(p)) return q;
    if (jac_is_inf(q)) return p;
    const Fe Z1Z1 = fe_sqr(p.Z), Z2Z2 = fe_sqr(q.Z);
    const Fe U1 = fe_mul(p.X, Z2Z2), U2 = fe_mul(q.X, Z1Z1);
    const Fe S1 = fe_mul(p.Y, fe_mul(q.Z, Z2Z2)), S2 = fe_mul(q.Y, fe_mul(p.Z, Z1Z1));
    const Fe H = fe_sub(U2, U1), rr = fe_sub(S2, S1);
    if (fe_is_zero(H)) {
        if (fe_is_zero(rr)) return jac_dbl(p);
        return jac_inf();
    }
    const Fe H2 = fe_add(H, H), I = fe_sqr(H2), J = fe_mul(H, I);
    const Fe r2 = fe_add(rr, rr), V = fe_mul(U1, I);
    Jac o;
    o.X = fe_sub(fe_sub(fe_sqr(r2), J), fe_add(V, V));
    const Fe SJ = fe_mul(S1, J);
    o.Y = fe_sub(fe_mul(r2, fe_sub(V, o.X)), fe_add(SJ, SJ));
    o.Z = fe_mul(fe_sub(fe_sub(fe_sqr(fe_add(p.Z, q.Z)), Z1Z1), Z2Z2), H);
    return o;
}

// affine coordinates as 64 big-endian bytes (x then y); the identity as zeros
SECP_HD void jac_encode(const Jac &p, uint8_t out[64])
{
    if (jac_is_inf(p)) {
        for (int i = 0; i < 64; i++) out[i] = 0;
        return;
    }
    const Fe zi = fe_inv(p.Z), zi2 = fe_sqr(zi);
    const Fe x = fe_mul(p.X, zi2), y = fe_mul(p.Y, fe_mul(zi2, zi));
    for (int i = 0; i < 32; i++) {
        out[i] = (uint8_t)(x.v[7 - i / 4] >> (8 * (3 - i % 4)));
        out[32 + i] = (uint8_t)(y.v[7 - i / 4] >> (8 * (3 - i % 4)));
    }
}

}  // namespace secp
