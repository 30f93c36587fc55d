"""ctypes front end of the CPU oracle (ra_oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline leg call this module; the product library never imports it.  It
compiles ``ra_oracle.c`` with gcc into ``libra_oracle.so`` beside it.

Every function returns plain numpy arrays / Python ints.  Field elements are
canonical integers in [0, p), p = 2^61 - 1.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

P61 = (1 << 61) - 1
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ra_oracle.c")
_SRC2 = os.path.join(_HERE, "ra_oracle_fp2.c")   # the same protocol with challenges in F_{p^2}
_SRC3 = os.path.join(_HERE, "ra_oracle_fs.c")    # the Fiat-Shamir transcript (SHA-256, Merkle root)
_HDR3 = os.path.join(_HERE, "ra_oracle_fs.h")
_LIB = os.path.join(_HERE, "libra_oracle.so")
_lib = None

ERRORS = {-1: "invalid argument", -3: "field too small", -4: "range",
          -5: "challenge stream", -10: "out of memory"}


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle error {code}: {ERRORS.get(code, '?')}")
        self.code = code


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C11, -O2, no OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                        _SRC, _SRC2, _SRC3, "-o", tmp], check=True)
        os.replace(tmp, _LIB)
    return _LIB


class LayerInfo(ctypes.Structure):
    _fields_ = [("t", ctypes.c_int32), ("P", ctypes.c_int32), ("log_p", ctypes.c_int32),
                ("n_mm_rounds", ctypes.c_int32), ("n_rs_rounds", ctypes.c_int32),
                ("n_zc_rounds", ctypes.c_int32), ("challenges_used", ctypes.c_int64),
                ("c0", ctypes.c_uint64), ("a_star", ctypes.c_uint64), ("b_star", ctypes.c_uint64),
                ("r_claim", ctypes.c_uint64), ("rm_claim", ctypes.c_uint64),
                ("y_claim", ctypes.c_uint64), ("z_claim", ctypes.c_uint64),
                ("range_sum", ctypes.c_uint64), ("bits_claim", ctypes.c_uint64),
                ("r_at", ctypes.c_uint64), ("y_at", ctypes.c_uint64)]


class F2(ctypes.Structure):
    _fields_ = [("re", ctypes.c_uint64), ("im", ctypes.c_uint64)]


class LayerInfo2(ctypes.Structure):
    """orc2_layer_info: the scalars of a layer's transcript over F_{p^2}."""
    _fields_ = [("t", ctypes.c_int32), ("P", ctypes.c_int32), ("log_p", ctypes.c_int32),
                ("n_mm_rounds", ctypes.c_int32), ("n_rs_rounds", ctypes.c_int32),
                ("n_zc_rounds", ctypes.c_int32), ("challenges_used", ctypes.c_int64)] + \
        [(k, F2) for k in ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim",
                           "range_sum", "bits_claim", "r_at", "y_at")]


F2_SCALARS = ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim", "range_sum", "bits_claim",
              "r_at", "y_at")


class FsState(ctypes.Structure):
    """orc_fs: the transcript's 32-byte state and the bytes pending since the last draw."""
    _fields_ = [("S", ctypes.c_uint8 * 32), ("qlen", ctypes.c_uint32), ("Q", ctypes.c_uint8 * 1024)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < max(os.path.getmtime(f)
                                                                       for f in (_SRC, _SRC2, _SRC3, _HDR3)):
            build()
        L = ctypes.CDLL(_LIB)
        u64p = ctypes.POINTER(ctypes.c_uint64)
        i64p = ctypes.POINTER(ctypes.c_int64)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        L.orc_fmul.restype = L.orc_fadd.restype = L.orc_fsub.restype = ctypes.c_uint64
        L.orc_fmul.argtypes = L.orc_fadd.argtypes = L.orc_fsub.argtypes = [ctypes.c_uint64] * 2
        L.orc_fint.restype = ctypes.c_uint64
        L.orc_fint.argtypes = [ctypes.c_int64]
        L.orc_chi_at.restype = ctypes.c_uint64
        L.orc_chi_at.argtypes = [u64p, ctypes.c_int, ctypes.c_uint64]
        L.orc_chi_vector.argtypes = [u64p, ctypes.c_int, u64p]
        L.orc_mle_int.argtypes = [i64p, ctypes.c_int, u64p, u64p]
        L.orc_mle_field.argtypes = [u64p, ctypes.c_int, u64p, u64p]
        L.orc_interp.restype = ctypes.c_uint64
        L.orc_interp.argtypes = [u64p, ctypes.c_int, ctypes.c_uint64]
        L.orc_plane_count.argtypes = [ctypes.c_int] * 3
        L.orc_prove_layer.argtypes = [ctypes.c_int64] * 3 + [i64p, i64p] + [ctypes.c_int] * 4 + \
            [u64p, ctypes.c_int64, i64p] + [i64p] * 5 + [u8p, u64p, u64p, u64p,
                                                        ctypes.POINTER(LayerInfo)]
        L.orc_verify_layer.argtypes = [ctypes.c_int64] * 3 + [i64p] * 3 + [ctypes.c_int] * 3 + \
            [i64p] * 4 + [u64p] * 3 + [ctypes.POINTER(LayerInfo), u64p, ctypes.c_int64, i64p]
        L.orc_link_prove.argtypes = [ctypes.c_int64, i64p, u64p, ctypes.c_int64, i64p, u64p, ctypes.c_int64, i64p,
                                     u64p, u64p, u64p, u64p]
        L.orc_link_verify.argtypes = [ctypes.c_int64, i64p, u64p, ctypes.c_int64, i64p, ctypes.c_uint64, u64p,
                                      ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, u64p, ctypes.c_int64, i64p]
        u8p_ = ctypes.c_char_p
        L.orc_sha256.argtypes = [u8p_, ctypes.c_size_t, u8p_]
        L.orc_witness_root.argtypes = [i64p] * 4 + [u64p, ctypes.c_int64, u8p_]
        fsp = ctypes.POINTER(FsState)
        L.orc2_fs_init.argtypes = [fsp, u8p_]
        L.orc2_fs_absorb.argtypes = [fsp, u8p_, ctypes.c_uint32]
        L.orc2_fs_draw.argtypes = [fsp, u64p]
        L.orc2_prove_layer_fs.argtypes = [ctypes.c_int64] * 3 + [i64p, i64p] + [ctypes.c_int] * 4 + \
            [fsp, u8p_] + [i64p] * 5 + [u8p, u64p, u64p, u64p, ctypes.POINTER(LayerInfo2), u64p, ctypes.c_int64]
        L.orc2_verify_layer_fs.argtypes = [ctypes.c_int64] * 3 + [i64p] * 3 + [ctypes.c_int] * 3 + \
            [i64p] * 4 + [u64p] * 3 + [ctypes.POINTER(LayerInfo2), fsp, u8p_]
        L.orc2_mul.argtypes = [u64p, u64p, u64p]
        L.orc2_inv.argtypes = [u64p, u64p]
        L.orc2_mle_int.argtypes = [i64p, ctypes.c_int, u64p, u64p]
        L.orc2_prove_layer.argtypes = [ctypes.c_int64] * 3 + [i64p, i64p] + [ctypes.c_int] * 4 + \
            [u64p, ctypes.c_int64, i64p] + [i64p] * 5 + [u8p, u64p, u64p, u64p, ctypes.POINTER(LayerInfo2)]
        L.orc2_verify_layer.argtypes = [ctypes.c_int64] * 3 + [i64p] * 3 + [ctypes.c_int] * 3 + \
            [i64p] * 4 + [u64p] * 3 + [ctypes.POINTER(LayerInfo2), u64p, ctypes.c_int64, i64p]
        _lib = L
    return _lib


def _u64(a):
    return np.ascontiguousarray(a, dtype=np.uint64)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _ptr(a, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


# --- small helpers exported for pins -------------------------------------
def fmul(a, b): return int(lib().orc_fmul(a, b))
def fadd(a, b): return int(lib().orc_fadd(a, b))
def fsub(a, b): return int(lib().orc_fsub(a, b))
def fint(z): return int(lib().orc_fint(int(z)))


def chi_at(z, y):
    z = _u64(z)
    return int(lib().orc_chi_at(_ptr(z, ctypes.c_uint64), len(z), y))


def chi_vector(z):
    z = _u64(z)
    out = np.zeros(1 << len(z), dtype=np.uint64)
    lib().orc_chi_vector(_ptr(z, ctypes.c_uint64), len(z), _ptr(out, ctypes.c_uint64))
    return out


def mle_int(table, z):
    t = _i64(np.asarray(table).reshape(-1))
    z = _u64(z)
    assert t.size == 1 << len(z)
    out = np.zeros(1, dtype=np.uint64)
    lib().orc_mle_int(_ptr(t, ctypes.c_int64), len(z), _ptr(z, ctypes.c_uint64), _ptr(out, ctypes.c_uint64))
    return int(out[0])


def mle_field(table, z):
    t = _u64(np.asarray(table).reshape(-1))
    z = _u64(z)
    assert t.size == 1 << len(z)
    out = np.zeros(1, dtype=np.uint64)
    lib().orc_mle_field(_ptr(t, ctypes.c_uint64), len(z), _ptr(z, ctypes.c_uint64), _ptr(out, ctypes.c_uint64))
    return int(out[0])


def interp(evals, x):
    e = _u64(evals)
    return int(lib().orc_interp(_ptr(e, ctypes.c_uint64), len(e) - 1, x))


def plane_count(s, t, relu):
    return int(lib().orc_plane_count(s, t, int(bool(relu))))


# --- layer protocol -------------------------------------------------------
def prove_layer(A, B, s, relu, mode, chal, cursor=0, t_in=-1):
    """Prove one layer; returns a dict with the witness tables, the bit table
    (uint8, planes x N), the transcript and the new challenge cursor."""
    A = _i64(A)
    B = _i64(B)
    n, m = A.shape
    m2, k = B.shape
    assert m == m2
    N = n * k
    chal = _u64(chal)
    cur = np.array([cursor], dtype=np.int64)
    C, R, Rm, Y, Z = (np.zeros(N, dtype=np.int64) for _ in range(5))
    bits = np.zeros(128 * N, dtype=np.uint8)
    lm = m.bit_length() - 1
    lN = N.bit_length() - 1
    mm = np.zeros(3 * max(lm, 1), dtype=np.uint64)
    rs = np.zeros(4 * (lN + 7), dtype=np.uint64)
    zc = np.zeros(4 * max(lN, 1), dtype=np.uint64)
    info = LayerInfo()
    i64 = ctypes.c_int64
    rc = lib().orc_prove_layer(n, m, k, _ptr(A, i64), _ptr(B, i64), s, int(bool(relu)), mode, t_in,
                               _ptr(chal, ctypes.c_uint64), len(chal), _ptr(cur, i64),
                               _ptr(C, i64), _ptr(R, i64), _ptr(Rm, i64), _ptr(Y, i64), _ptr(Z, i64),
                               _ptr(bits, ctypes.c_uint8), _ptr(mm, ctypes.c_uint64),
                               _ptr(rs, ctypes.c_uint64), _ptr(zc, ctypes.c_uint64), ctypes.byref(info))
    if rc != 0:
        raise OracleError(rc)
    P = info.P
    out = dict(n=n, m=m, k=k, s=s, relu=int(bool(relu)), mode=mode,
               C=C.reshape(n, k), R=R.reshape(n, k), Rm=Rm.reshape(n, k), Y=Y.reshape(n, k),
               Z=Z.reshape(n, k), bits=bits[:P * N].reshape(P, N).copy(),
               t=info.t, P=P, cursor=int(cur[0]), challenges_used=int(info.challenges_used),
               c0=int(info.c0), mm_evals=[int(v) for v in mm[:3 * info.n_mm_rounds]],
               a_star=int(info.a_star), b_star=int(info.b_star),
               r_claim=int(info.r_claim), rm_claim=int(info.rm_claim),
               y_claim=int(info.y_claim), z_claim=int(info.z_claim),
               range_sum=int(info.range_sum),
               rs_evals=[int(v) for v in rs[:4 * info.n_rs_rounds]], bits_claim=int(info.bits_claim),
               zc_evals=[int(v) for v in zc[:4 * info.n_zc_rounds]],
               r_at=int(info.r_at), y_at=int(info.y_at))
    return out


def verify_layer(A, B, Z, s, relu, mode, R, Rm, Y, bits, tr, chal, cursor=0):
    """Run the oracle's verifier; returns (verdict, new_cursor).  verdict 0 =
    accept, else the number of the first failing check (see ra_oracle.c)."""
    A = _i64(A)
    B = _i64(B)
    n, m = A.shape
    k = B.shape[1]
    N = n * k
    lm = m.bit_length() - 1
    lN = N.bit_length() - 1
    info = LayerInfo()
    info.t = tr["t"]
    info.P = tr["P"]
    for key in ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim",
                "bits_claim", "r_at", "y_at"):
        setattr(info, key, int(tr[key]) & 0xFFFFFFFFFFFFFFFF)
    mm = _u64(np.array(list(tr["mm_evals"]) + [0] * 3, dtype=object).astype(np.uint64))
    rs = _u64(np.array(list(tr["rs_evals"]) + [0] * 4, dtype=object).astype(np.uint64))
    zc = _u64(np.array(list(tr["zc_evals"]) + [0] * 4, dtype=object).astype(np.uint64))
    want_rs = 4 * (int(tr["P"]).bit_length() - 1 + lN)
    if len(tr["mm_evals"]) != 3 * lm or len(tr["rs_evals"]) != want_rs or \
            len(tr["zc_evals"]) != (4 * lN if relu else 0):
        return 13, cursor
    bits = _i64(np.asarray(bits).reshape(-1))
    if bits.size != int(tr["P"]) * N:
        return 12, cursor
    chal = _u64(chal)
    cur = np.array([cursor], dtype=np.int64)
    i64 = ctypes.c_int64
    arrs = [_i64(np.asarray(x).reshape(-1)) for x in (Z, R, Rm, Y)]
    v = lib().orc_verify_layer(n, m, k, _ptr(A, i64), _ptr(B, i64), _ptr(arrs[0], i64), s,
                               int(bool(relu)), mode, _ptr(arrs[1], i64), _ptr(arrs[2], i64),
                               _ptr(arrs[3], i64), _ptr(bits, i64), _ptr(mm, ctypes.c_uint64),
                               _ptr(rs, ctypes.c_uint64), _ptr(zc, ctypes.c_uint64), ctypes.byref(info),
                               _ptr(chal, ctypes.c_uint64), len(chal), _ptr(cur, i64))
    return int(v), int(cur[0])


def link_point(n, m, k, chal, cursor):
    """The point (r1, rho) at which a layer proven from `cursor` claims A~ (its a*)."""
    ln, lm, lk = n.bit_length() - 1, m.bit_length() - 1, k.bit_length() - 1
    c = [int(x) for x in chal[cursor:cursor + ln + lk + lm]]
    return c[:ln] + c[ln + lk:]


def prove_link(Z, src, z, chal, cursor=0):
    """Gather link (ra_oracle.c, orc_link_prove): reduce A~(z) of A[a] =
    Z[src[a]] (0 where src < 0) to Z~(y*) W~_z(y*).  Returns a dict with
    evals (3 per round), claim, z_at, w_at, cursor."""
    Zf = _i64(np.asarray(Z).reshape(-1))
    src = _i64(np.asarray(src).reshape(-1))
    vz = Zf.size.bit_length() - 1
    zz = _u64(list(z) or [0])
    chal = _u64(chal)
    cur = np.array([cursor], dtype=np.int64)
    ev = np.zeros(3 * max(vz, 1), dtype=np.uint64)
    out = np.zeros(3, dtype=np.uint64)
    u64 = ctypes.c_uint64
    rc = lib().orc_link_prove(src.size, _ptr(src, ctypes.c_int64), _ptr(zz, u64), Zf.size, _ptr(Zf, ctypes.c_int64),
                              _ptr(chal, u64), len(chal), _ptr(cur, ctypes.c_int64), _ptr(ev, u64),
                              _ptr(out[0:], u64), _ptr(out[1:], u64), _ptr(out[2:], u64))
    if rc != 0:
        raise OracleError(rc)
    return dict(evals=[int(x) for x in ev[:3 * vz]], claim=int(out[0]), z_at=int(out[1]), w_at=int(out[2]),
                cursor=int(cur[0]))


def verify_link(Z, src, z, a_star, link, chal, cursor=0):
    """Verifier of a gather link: (0 or 15, new cursor)."""
    Zf = _i64(np.asarray(Z).reshape(-1))
    src = _i64(np.asarray(src).reshape(-1))
    vz = Zf.size.bit_length() - 1
    if len(link["evals"]) != 3 * vz:
        return 15, cursor
    zz = _u64(list(z) or [0])
    ev = _u64(np.array(list(link["evals"]) + [0] * 3, dtype=object).astype(np.uint64))
    chal = _u64(chal)
    cur = np.array([cursor], dtype=np.int64)
    u64 = ctypes.c_uint64
    v = lib().orc_link_verify(src.size, _ptr(src, ctypes.c_int64), _ptr(zz, u64), Zf.size, _ptr(Zf, ctypes.c_int64),
                              int(a_star) & 0xFFFFFFFFFFFFFFFF, _ptr(ev, u64), int(link["claim"]) & 0xFFFFFFFFFFFFFFFF,
                              int(link["z_at"]) & 0xFFFFFFFFFFFFFFFF, int(link["w_at"]) & 0xFFFFFFFFFFFFFFFF,
                              _ptr(chal, u64), len(chal), _ptr(cur, ctypes.c_int64))
    return int(v), int(cur[0])


def prove_network(workload, layers_out=None, links=False):
    """Prove every layer of a workload (see paper_2505_17623_amd.inputs) in
    order; a layer's A is the workload's input or the previous output passed
    through the workload's link.  With links=True every gather link (a layer
    whose input is a gather of the previous output) is proven right after its
    layer, from the next challenges (res["link"]).  Returns the list of
    per-layer results."""
    results = []
    cursor = 0
    Z = None
    for li, layer in enumerate(workload.layers):
        A = workload.layer_input(li, Z)
        start = cursor
        res = prove_layer(A, layer.B, layer.s, layer.relu, workload.mode, workload.challenges, cursor)
        cursor = res["cursor"]
        if links and li > 0 and workload.links[li] is not None:
            n, m = A.shape
            z = link_point(n, m, layer.B.shape[1], workload.challenges, start)
            res["link"] = prove_link(Z, workload.link_map(li), z, workload.challenges, cursor)
            res["link_point"] = z
            cursor = res["link"]["cursor"]
            res["cursor"] = cursor
        res["A"] = A
        Z = res["Z"]
        results.append(res)
    return results


# --- the protocol over F_{p^2} (ra_oracle_fp2.c) ----------------------------
# Field elements of F_{p^2} = F_p[i] / (i^2 + 1) are pairs (re, im).
def f2mul(a, b):
    x, y, out = _u64(list(a)), _u64(list(b)), np.zeros(2, dtype=np.uint64)
    lib().orc2_mul(_ptr(x, ctypes.c_uint64), _ptr(y, ctypes.c_uint64), _ptr(out, ctypes.c_uint64))
    return int(out[0]), int(out[1])


def f2inv(a):
    x, out = _u64(list(a)), np.zeros(2, dtype=np.uint64)
    lib().orc2_inv(_ptr(x, ctypes.c_uint64), _ptr(out, ctypes.c_uint64))
    return int(out[0]), int(out[1])


def mle_int_fp2(table, z):
    """MLE of an integer table at a point of F_{p^2}^v (list of pairs)."""
    t = _i64(np.asarray(table).reshape(-1))
    assert t.size == 1 << len(z)
    zz = _u64([c for pair in z for c in pair] or [0])
    out = np.zeros(2, dtype=np.uint64)
    lib().orc2_mle_int(_ptr(t, ctypes.c_int64), len(z), _ptr(zz, ctypes.c_uint64), _ptr(out, ctypes.c_uint64))
    return int(out[0]), int(out[1])


def _pairs(a, n):
    return [(int(a[2 * i]), int(a[2 * i + 1])) for i in range(n)]


def prove_layer_fp2(A, B, s, relu, mode, chal, cursor=0, t_in=-1):
    """Prove one layer with challenges in F_{p^2} (pairs of consecutive words
    of the F_p stream `chal`, from word `cursor`).  Returns a dict like
    prove_layer's, with every transcript element a pair (re, im)."""
    A = _i64(A)
    B = _i64(B)
    n, m = A.shape
    k = B.shape[1]
    N = n * k
    chal = _u64(chal)
    cur = np.array([cursor], dtype=np.int64)
    C, R, Rm, Y, Z = (np.zeros(N, dtype=np.int64) for _ in range(5))
    bits = np.zeros(128 * N, dtype=np.uint8)
    lm = m.bit_length() - 1
    lN = N.bit_length() - 1
    mm = np.zeros(2 * 3 * max(lm, 1), dtype=np.uint64)
    rs = np.zeros(2 * 4 * (lN + 7), dtype=np.uint64)
    zc = np.zeros(2 * 4 * max(lN, 1), dtype=np.uint64)
    info = LayerInfo2()
    i64 = ctypes.c_int64
    rc = lib().orc2_prove_layer(n, m, k, _ptr(A, i64), _ptr(B, i64), s, int(bool(relu)), mode, t_in,
                                _ptr(chal, ctypes.c_uint64), len(chal), _ptr(cur, i64),
                                _ptr(C, i64), _ptr(R, i64), _ptr(Rm, i64), _ptr(Y, i64), _ptr(Z, i64),
                                _ptr(bits, ctypes.c_uint8), _ptr(mm, ctypes.c_uint64),
                                _ptr(rs, ctypes.c_uint64), _ptr(zc, ctypes.c_uint64), ctypes.byref(info))
    if rc != 0:
        raise OracleError(rc)
    P = info.P
    out = dict(n=n, m=m, k=k, s=s, relu=int(bool(relu)), mode=mode,
               C=C.reshape(n, k), R=R.reshape(n, k), Rm=Rm.reshape(n, k), Y=Y.reshape(n, k),
               Z=Z.reshape(n, k), bits=bits[:P * N].reshape(P, N).copy(),
               t=info.t, P=P, cursor=int(cur[0]), challenges_used=int(info.challenges_used),
               mm_evals=_pairs(mm, 3 * info.n_mm_rounds), rs_evals=_pairs(rs, 4 * info.n_rs_rounds),
               zc_evals=_pairs(zc, 4 * info.n_zc_rounds))
    for key in F2_SCALARS:
        v = getattr(info, key)
        out[key] = (int(v.re), int(v.im))
    return out


def verify_layer_fp2(A, B, Z, s, relu, mode, R, Rm, Y, bits, tr, chal, cursor=0):
    """The F_{p^2} verifier (checks numbered as verify_layer); returns (verdict, new_cursor)."""
    A = _i64(A)
    B = _i64(B)
    n, m = A.shape
    k = B.shape[1]
    N = n * k
    lm = m.bit_length() - 1
    lN = N.bit_length() - 1
    info = LayerInfo2()
    info.t = tr["t"]
    info.P = tr["P"]
    for key in F2_SCALARS:
        re, im = tr[key]
        setattr(info, key, F2(int(re) & 0xFFFFFFFFFFFFFFFF, int(im) & 0xFFFFFFFFFFFFFFFF))
    flat = lambda ev, pad: _u64(np.array([c for pair in ev for c in pair] + [0] * pad, dtype=object).astype(np.uint64))
    mm, rs, zc = flat(tr["mm_evals"], 6), flat(tr["rs_evals"], 8), flat(tr["zc_evals"], 8)
    want_rs = 4 * (int(tr["P"]).bit_length() - 1 + lN)
    if len(tr["mm_evals"]) != 3 * lm or len(tr["rs_evals"]) != want_rs or \
            len(tr["zc_evals"]) != (4 * lN if relu else 0):
        return 13, cursor
    bits = _i64(np.asarray(bits).reshape(-1))
    if bits.size != int(tr["P"]) * N:
        return 12, cursor
    chal = _u64(chal)
    cur = np.array([cursor], dtype=np.int64)
    i64 = ctypes.c_int64
    arrs = [_i64(np.asarray(x).reshape(-1)) for x in (Z, R, Rm, Y)]
    v = lib().orc2_verify_layer(n, m, k, _ptr(A, i64), _ptr(B, i64), _ptr(arrs[0], i64), s,
                                int(bool(relu)), mode, _ptr(arrs[1], i64), _ptr(arrs[2], i64),
                                _ptr(arrs[3], i64), _ptr(bits, i64), _ptr(mm, ctypes.c_uint64),
                                _ptr(rs, ctypes.c_uint64), _ptr(zc, ctypes.c_uint64), ctypes.byref(info),
                                _ptr(chal, ctypes.c_uint64), len(chal), _ptr(cur, i64))
    return int(v), int(cur[0])


def prove_network_fp2(workload):
    """Every layer of a workload over F_{p^2}, the stream read in pairs."""
    results = []
    cursor = 0
    Z = None
    chal = fp2_stream(workload)
    for li, layer in enumerate(workload.layers):
        A = workload.layer_input(li, Z)
        res = prove_layer_fp2(A, layer.B, layer.s, layer.relu, workload.mode, chal, cursor)
        cursor = res["cursor"]
        res["A"] = A
        Z = res["Z"]
        results.append(res)
    return results


def fp2_stream(workload):
    """The F_p stream a workload's F_{p^2} proof reads: twice the draws of its F_p proof."""
    from paper_2505_17623_amd import inputs
    return inputs.xorshift64_stream(workload.challenge_seed, 2 * len(workload.challenges))


# --- the non-interactive protocol: Fiat-Shamir over F_{p^2} (ra_oracle_fs.c) ---
def sha256(msg: bytes) -> bytes:
    out = ctypes.create_string_buffer(32)
    lib().orc_sha256(msg, len(msg), out)
    return out.raw


def witness_root(R, Rm, Y, Z, words) -> bytes:
    """Merkle root of the witness tables (R, Rm, Y, Z as integers, the packed bit words)."""
    arrs = [_i64(np.asarray(x).reshape(-1)) for x in (R, Rm, Y, Z)]
    w = _u64(np.asarray(words).reshape(-1))
    out = ctypes.create_string_buffer(32)
    i64 = ctypes.c_int64
    rc = lib().orc_witness_root(*[_ptr(a, i64) for a in arrs], _ptr(w, ctypes.c_uint64), w.size, out)
    if rc != 0:
        raise OracleError(rc)
    return out.raw


def fs_init(domain: bytes) -> FsState:
    assert len(domain) == 32
    st = FsState()
    lib().orc2_fs_init(ctypes.byref(st), domain)
    return st


def fs_absorb(st: FsState, msg: bytes):
    if lib().orc2_fs_absorb(ctypes.byref(st), msg, len(msg)) != 0:
        raise OracleError(-1)


def fs_draw(st: FsState):
    out = np.zeros(2, dtype=np.uint64)
    lib().orc2_fs_draw(ctypes.byref(st), _ptr(out, ctypes.c_uint64))
    return int(out[0]), int(out[1])


def pack_words(planes) -> np.ndarray:
    """(P, N) 0/1 planes -> N uint64 words, bit q = plane q."""
    planes = np.asarray(planes)
    w = np.zeros(planes.shape[1], dtype=np.uint64)
    for q in range(planes.shape[0]):
        w |= planes[q].astype(np.uint64) << np.uint64(q)
    return w


def prove_layer_fs(A, B, s, relu, mode, fs: FsState, pub: bytes, t_in=-1):
    """One layer made non-interactive (orc2_prove_layer_fs): the challenges
    are drawn from the transcript `fs` (updated in place), pub the caller's
    32-byte digest of the public inputs.  Returns a dict like
    prove_layer_fp2's plus "drawn" (every challenge, in order)."""
    assert len(pub) == 32
    A = _i64(A)
    B = _i64(B)
    n, m = A.shape
    k = B.shape[1]
    N = n * k
    C, R, Rm, Y, Z = (np.zeros(N, dtype=np.int64) for _ in range(5))
    bits = np.zeros(128 * N, dtype=np.uint8)
    lm = m.bit_length() - 1
    lN = N.bit_length() - 1
    mm = np.zeros(2 * 3 * max(lm, 1), dtype=np.uint64)
    rs = np.zeros(2 * 4 * (lN + 7), dtype=np.uint64)
    zc = np.zeros(2 * 4 * max(lN, 1), dtype=np.uint64)
    cap = 4 * (lN + 64)
    drawn = np.zeros(2 * cap, dtype=np.uint64)
    info = LayerInfo2()
    i64 = ctypes.c_int64
    rc = lib().orc2_prove_layer_fs(n, m, k, _ptr(A, i64), _ptr(B, i64), s, int(bool(relu)), mode, t_in,
                                   ctypes.byref(fs), pub, _ptr(C, i64), _ptr(R, i64), _ptr(Rm, i64), _ptr(Y, i64),
                                   _ptr(Z, i64), _ptr(bits, ctypes.c_uint8), _ptr(mm, ctypes.c_uint64),
                                   _ptr(rs, ctypes.c_uint64), _ptr(zc, ctypes.c_uint64), ctypes.byref(info),
                                   _ptr(drawn, ctypes.c_uint64), cap)
    if rc != 0:
        raise OracleError(rc)
    P = info.P
    out = dict(n=n, m=m, k=k, s=s, relu=int(bool(relu)), mode=mode,
               C=C.reshape(n, k), R=R.reshape(n, k), Rm=Rm.reshape(n, k), Y=Y.reshape(n, k),
               Z=Z.reshape(n, k), bits=bits[:P * N].reshape(P, N).copy(), t=info.t, P=P,
               challenges_used=int(info.challenges_used),
               mm_evals=_pairs(mm, 3 * info.n_mm_rounds), rs_evals=_pairs(rs, 4 * info.n_rs_rounds),
               zc_evals=_pairs(zc, 4 * info.n_zc_rounds), drawn=_pairs(drawn, info.challenges_used // 2))
    for key in F2_SCALARS:
        v = getattr(info, key)
        out[key] = (int(v.re), int(v.im))
    return out


def verify_layer_fs(A, B, Z, s, relu, mode, R, Rm, Y, bits, tr, fs: FsState, pub: bytes):
    """The Fiat-Shamir verifier (orc2_verify_layer_fs): replays the transcript
    through `fs` (updated in place); returns the verdict (numbers as verify_layer)."""
    A = _i64(A)
    B = _i64(B)
    n, m = A.shape
    k = B.shape[1]
    N = n * k
    lm = m.bit_length() - 1
    lN = N.bit_length() - 1
    info = LayerInfo2()
    info.t = tr["t"]
    info.P = tr["P"]
    for key in F2_SCALARS:
        re, im = tr[key]
        setattr(info, key, F2(int(re) & 0xFFFFFFFFFFFFFFFF, int(im) & 0xFFFFFFFFFFFFFFFF))
    flat = lambda ev, pad: _u64(np.array([c for pair in ev for c in pair] + [0] * pad, dtype=object).astype(np.uint64))
    mm, rs, zc = flat(tr["mm_evals"], 6), flat(tr["rs_evals"], 8), flat(tr["zc_evals"], 8)
    want_rs = 4 * (int(tr["P"]).bit_length() - 1 + lN)
    if len(tr["mm_evals"]) != 3 * lm or len(tr["rs_evals"]) != want_rs or \
            len(tr["zc_evals"]) != (4 * lN if relu else 0):
        return 13
    bits = _i64(np.asarray(bits).reshape(-1))
    if bits.size != int(tr["P"]) * N:
        return 12
    i64 = ctypes.c_int64
    arrs = [_i64(np.asarray(x).reshape(-1)) for x in (Z, R, Rm, Y)]
    return int(lib().orc2_verify_layer_fs(n, m, k, _ptr(A, i64), _ptr(B, i64), _ptr(arrs[0], i64), s,
                                          int(bool(relu)), mode, _ptr(arrs[1], i64), _ptr(arrs[2], i64),
                                          _ptr(arrs[3], i64), _ptr(bits, i64), _ptr(mm, ctypes.c_uint64),
                                          _ptr(rs, ctypes.c_uint64), _ptr(zc, ctypes.c_uint64), ctypes.byref(info),
                                          ctypes.byref(fs), pub))


def prove_network_fs(workload, domain: bytes, pubs):
    """Every layer of a workload made non-interactive, one transcript from
    `domain` through all layers; pubs[li] is layer li's 32-byte public digest."""
    fs = fs_init(domain)
    results = []
    Z = None
    for li, layer in enumerate(workload.layers):
        A = workload.layer_input(li, Z)
        res = prove_layer_fs(A, layer.B, layer.s, layer.relu, workload.mode, fs, pubs[li])
        res["A"] = A
        Z = res["Z"]
        results.append(res)
    return results
