"""Python binding of the C ABI in include/ra.h (libra_mi355x.so).

Argument marshalling only: every step of the prover runs in the HIP library.
torch supplies device memory and the HIP stream.  Field elements are held in
int64 tensors / uint64 numpy arrays (same bits).  The library must be built
(``python -m paper_2505_17623_amd.build``); importing this module without it
raises, there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libra_mi355x.so")
P61 = (1 << 61) - 1

RA_I16, RA_I32, RA_I64, RA_FIELD, RA_U16, RA_U64 = 1, 2, 3, 4, 5, 6
RA_ROUND_NEAREST, RA_ROUND_FLOOR = 0, 1
STATUS = {0: "RA_OK", -1: "RA_E_INVAL", -2: "RA_E_UNSUPPORTED_PRIME", -3: "RA_E_FIELD_TOO_SMALL",
          -4: "RA_E_RANGE", -5: "RA_E_SEED", -6: "RA_E_HIP", -7: "RA_E_STATE",
          -8: "RA_E_BUFSIZE", -9: "RA_E_NOT_IMPLEMENTED", -10: "RA_E_SCRATCH", -11: "RA_E_NOMEM"}
EXPORTS = ["ra_ctx_create", "ra_ctx_create_stream", "ra_ctx_destroy", "ra_ctx_cursor", "ra_status_str",
           "ra_workspace_size", "ra_ctx_set_profiling", "ra_ctx_profile", "ra_ctx_set_deferred", "ra_ctx_sync",
           "ra_mle_bind", "ra_sumcheck_matmul_prove", "ra_rescale_relu_witness", "ra_range_prove", "ra_verify",
           "ra_verify_stream", "ra_witness_plan", "ra_mle_bind_noalloc", "ra_prove_layer_fp2",
           "ra_workspace_size_fp2", "ra_verify_fp2", "ra_link_prove", "ra_link_workspace_size",
           "ra_link_gather", "ra_verify_fs",
           "ra_ctx_create_fs", "ra_prove_layer_fs",
           "ra_commit_generators", "ra_commit_workspace_size", "ra_commit", "ra_commit_open",
           "ra_commit_batch_workspace_size", "ra_commit_batch"]


class RAError(RuntimeError):
    def __init__(self, code, where=""):
        super().__init__(f"{where}: {STATUS.get(code, code)}")
        self.code = code


u64 = ctypes.c_uint64
u64p = ctypes.POINTER(ctypes.c_uint64)


class MatmulProof(ctypes.Structure):
    _fields_ = [("log_m", ctypes.c_uint32), ("c0", u64), ("evals", u64p), ("a_star", u64), ("b_star", u64)]


class WitnessInfo(ctypes.Structure):
    _fields_ = [("s", ctypes.c_uint32), ("relu", ctypes.c_uint32), ("round_mode", ctypes.c_uint32),
                ("t", ctypes.c_int32), ("P", ctypes.c_uint32), ("r_claim", u64), ("rm_claim", u64),
                ("y_claim", u64), ("z_claim", u64)]


class RangeProof(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_uint32), ("evals", u64p), ("range_sum", u64), ("bits_claim", u64),
                ("relu_rounds", ctypes.c_uint32), ("relu_evals", u64p), ("r_at", u64), ("y_at", u64)]


class LayerPublic(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint32), ("m", ctypes.c_uint32), ("k", ctypes.c_uint32),
                ("s", ctypes.c_uint32), ("relu", ctypes.c_uint32), ("round_mode", ctypes.c_uint32),
                ("a_dtype", ctypes.c_int), ("A", ctypes.c_void_p), ("B", ctypes.c_void_p),
                ("Z", ctypes.c_void_p), ("chained", ctypes.c_uint32), ("link_src", ctypes.c_void_p)]


class LayerTables(ctypes.Structure):
    _fields_ = [("R", ctypes.c_void_p), ("Rm", ctypes.c_void_p), ("Y", ctypes.c_void_p),
                ("bits", ctypes.c_void_p)]


class LinkProof(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_uint32), ("evals", u64p), ("claim", u64), ("z_at", u64), ("w_at", u64)]


class LayerTranscript(ctypes.Structure):
    _fields_ = [("mm", MatmulProof), ("wit", WitnessInfo), ("rng", RangeProof), ("link", LinkProof)]


class Fp2(ctypes.Structure):
    """An element re + im i of F_{p^2} = F_p[i] / (i^2 + 1)."""
    _fields_ = [("re", u64), ("im", u64)]


Fp2p = ctypes.POINTER(Fp2)


class LayerProofFp2(ctypes.Structure):
    _fields_ = [("s", ctypes.c_uint32), ("relu", ctypes.c_uint32), ("round_mode", ctypes.c_uint32),
                ("t", ctypes.c_int32), ("P", ctypes.c_uint32), ("log_m", ctypes.c_uint32),
                ("c0", Fp2), ("a_star", Fp2), ("b_star", Fp2), ("mm_evals", Fp2p),
                ("r_claim", Fp2), ("rm_claim", Fp2), ("y_claim", Fp2), ("z_claim", Fp2),
                ("rounds", ctypes.c_uint32), ("rs_evals", Fp2p), ("range_sum", Fp2), ("bits_claim", Fp2),
                ("relu_rounds", ctypes.c_uint32), ("zc_evals", Fp2p), ("r_at", Fp2), ("y_at", Fp2)]


FP2_SCALARS = ("c0", "a_star", "b_star", "r_claim", "rm_claim", "y_claim", "z_claim", "range_sum", "bits_claim",
               "r_at", "y_at")


_lib = None


def lib():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} not built; run python -m paper_2505_17623_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        L.ra_ctx_create.argtypes = [u64, u64, vp, ctypes.POINTER(vp)]
        L.ra_ctx_create_stream.argtypes = [u64, u64p, u64, vp, ctypes.POINTER(vp)]
        L.ra_workspace_size.argtypes = [ctypes.c_uint32] * 4 + [ctypes.POINTER(ctypes.c_size_t)]
        L.ra_ctx_destroy.argtypes = [vp]
        L.ra_ctx_cursor.argtypes = [vp, u64p]
        L.ra_ctx_set_profiling.argtypes = [vp, ctypes.c_int]
        L.ra_ctx_set_deferred.argtypes = [vp, ctypes.c_int]
        L.ra_ctx_sync.argtypes = [vp]
        L.ra_ctx_profile.argtypes = [vp, ctypes.c_uint32, ctypes.POINTER(ctypes.c_char_p),
                                     ctypes.POINTER(ctypes.c_double), u64p]
        L.ra_status_str.restype = ctypes.c_char_p
        L.ra_status_str.argtypes = [ctypes.c_int32]
        L.ra_mle_bind.argtypes = [vp, vp, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int, u64p,
                                  ctypes.c_uint32, vp]
        L.ra_mle_bind_noalloc.argtypes = [vp, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int, u64p,
                                          ctypes.c_uint32, vp, vp]
        L.ra_sumcheck_matmul_prove.argtypes = [vp, vp, ctypes.c_int, vp, ctypes.c_uint32, ctypes.c_uint32,
                                               ctypes.c_uint32, vp, vp, ctypes.c_size_t, ctypes.POINTER(MatmulProof)]
        L.ra_rescale_relu_witness.argtypes = [vp, vp, ctypes.c_uint32, ctypes.c_uint32, vp, vp, vp, vp, vp,
                                              u64, vp, ctypes.c_size_t, ctypes.POINTER(WitnessInfo)]
        L.ra_witness_plan.argtypes = [vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int32, vp, vp,
                                      vp, vp, vp, u64]
        L.ra_range_prove.argtypes = [vp, vp, vp, vp, ctypes.c_uint32, ctypes.c_uint32,
                                     ctypes.POINTER(WitnessInfo), vp, ctypes.c_size_t, ctypes.POINTER(RangeProof)]
        tail = [ctypes.c_uint32, ctypes.POINTER(LayerPublic), ctypes.POINTER(LayerTables),
                ctypes.POINTER(LayerTranscript), ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_uint32)]
        L.ra_verify.argtypes = [u64, u64] + tail
        L.ra_verify_stream.argtypes = [u64, u64p, u64] + tail
        L.ra_prove_layer_fp2.argtypes = [vp, vp, ctypes.c_int, vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                         vp, vp, vp, vp, vp, vp, u64, vp, ctypes.c_size_t,
                                         ctypes.POINTER(LayerProofFp2)]
        L.ra_workspace_size_fp2.argtypes = [ctypes.c_uint32] * 3 + [ctypes.POINTER(ctypes.c_size_t)]
        L.ra_link_prove.argtypes = [vp, vp, u64, vp, u64, vp, ctypes.c_size_t, ctypes.POINTER(LinkProof)]
        L.ra_link_workspace_size.argtypes = [u64, ctypes.c_uint32, ctypes.c_uint32, ctypes.POINTER(ctypes.c_size_t)]
        L.ra_link_gather.argtypes = [vp, vp, u64, vp, u64, vp]
        L.ra_ctx_create_fs.argtypes = [u64, ctypes.c_char_p, vp, ctypes.POINTER(vp)]
        L.ra_commit_generators.argtypes = [vp, ctypes.c_char_p, u64, u64, vp]
        L.ra_commit_workspace_size.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
        L.ra_commit.argtypes = [vp, vp, ctypes.c_int, u64, vp, vp, ctypes.c_size_t, ctypes.c_char_p]
        L.ra_commit_open.argtypes = [vp, ctypes.c_int, u64, vp, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int32)]
        L.ra_commit_batch_workspace_size.argtypes = [vp, ctypes.c_uint32, ctypes.POINTER(ctypes.c_size_t)]
        L.ra_commit_batch.argtypes = [vp, vp, vp, vp, ctypes.c_uint32, vp, vp, ctypes.c_size_t, ctypes.c_char_p]
        L.ra_prove_layer_fs.argtypes = [vp, vp, ctypes.c_int, vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                        vp, vp, vp, vp, vp, vp, u64, ctypes.c_char_p, vp, ctypes.c_size_t,
                                        ctypes.POINTER(LayerProofFp2), ctypes.c_char_p]
        L.ra_verify_fs.argtypes = [u64, ctypes.c_char_p, ctypes.c_uint32, ctypes.POINTER(LayerPublic),
                                   ctypes.POINTER(LayerTables), ctypes.POINTER(LayerProofFp2), ctypes.c_char_p,
                                   ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_uint32)]
        L.ra_verify_fp2.argtypes = [u64, u64, ctypes.c_uint32, ctypes.POINTER(LayerPublic),
                                    ctypes.POINTER(LayerTables), ctypes.POINTER(LayerProofFp2),
                                    ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_uint32)]
        for f in (L.ra_ctx_create, L.ra_ctx_create_stream, L.ra_workspace_size, L.ra_verify_stream,
                  L.ra_prove_layer_fp2, L.ra_workspace_size_fp2, L.ra_verify_fp2, L.ra_link_prove,
                  L.ra_link_workspace_size, L.ra_link_gather, L.ra_verify_fs, L.ra_ctx_create_fs,
                  L.ra_prove_layer_fs, L.ra_commit_generators, L.ra_commit_workspace_size, L.ra_commit,
                  L.ra_commit_open, L.ra_commit_batch_workspace_size, L.ra_commit_batch,
                  L.ra_ctx_destroy, L.ra_ctx_cursor, L.ra_ctx_set_profiling, L.ra_ctx_profile,
                  L.ra_ctx_set_deferred, L.ra_ctx_sync,
                  L.ra_mle_bind, L.ra_sumcheck_matmul_prove,
                  L.ra_rescale_relu_witness, L.ra_range_prove, L.ra_verify, L.ra_witness_plan,
                  L.ra_mle_bind_noalloc):
            f.restype = ctypes.c_int32
        _lib = L
    return _lib


def _check(code, where):
    if code != 0:
        raise RAError(code, where)


def _dptr(t: torch.Tensor):
    assert t.is_cuda and t.is_contiguous(), "device tensors must be contiguous CUDA tensors"
    return ctypes.c_void_p(t.data_ptr())


def _u64_array(vals):
    a = np.ascontiguousarray(np.asarray(vals, dtype=np.uint64))
    return a, a.ctypes.data_as(u64p)


_DT = {torch.int16: RA_I16, torch.int32: RA_I32, torch.int64: RA_I64}


class Context:
    """A prover context: the challenge stream on the device plus per-layer
    state.  Give `seed` (the library draws the stream: ra_ctx_create),
    `challenges` (a given array: ra_ctx_create_stream) or `fs_domain` (32
    bytes: a Fiat-Shamir transcript for non-interactive proofs,
    ra_ctx_create_fs)."""

    def __init__(self, challenges=None, stream: torch.cuda.Stream | None = None, deferred: bool = False,
                 seed: int | None = None, fs_domain: bytes | None = None):
        assert sum(x is not None for x in (challenges, seed, fs_domain)) == 1, "give challenges, seed or fs_domain"
        self.stream = stream or torch.cuda.current_stream()
        h = ctypes.c_void_p()
        sp = ctypes.c_void_p(self.stream.cuda_stream)
        if fs_domain is not None:
            assert len(fs_domain) == 32
            _check(lib().ra_ctx_create_fs(P61, bytes(fs_domain), sp, ctypes.byref(h)), "ra_ctx_create_fs")
        elif seed is not None:
            _check(lib().ra_ctx_create(P61, seed, sp, ctypes.byref(h)), "ra_ctx_create")
        else:
            self._chal, cp = _u64_array(challenges)
            _check(lib().ra_ctx_create_stream(P61, cp, len(self._chal), sp, ctypes.byref(h)),
                   "ra_ctx_create_stream")
        self.h = h
        self._fills = []  # Python-side results completed at sync (deferred mode)
        self.deferred = False
        if deferred:
            self.set_deferred(True)

    def set_deferred(self, on: bool):
        """Deferred mode: proving calls return once enqueued; results are filled by sync()."""
        _check(lib().ra_ctx_set_deferred(self.h, int(bool(on))), "ra_ctx_set_deferred")
        if not on:
            self._run_fills()
        self.deferred = bool(on)

    def _run_fills(self):
        fills, self._fills = self._fills, []
        for f in fills:
            f()

    def later(self, fill):
        """Run `fill` now (synchronous mode) or at the next sync (deferred mode)."""
        if self.deferred:
            self._fills.append(fill)
        else:
            fill()

    def sync(self):
        """Wait for all enqueued work and complete every deferred result."""
        code = lib().ra_ctx_sync(self.h)
        self._run_fills()
        _check(code, "ra_ctx_sync")

    def close(self):
        if self.h:
            lib().ra_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_profiling(self, on: bool):
        _check(lib().ra_ctx_set_profiling(self.h, int(bool(on))), "ra_ctx_set_profiling")

    def profile(self):
        """{group name: (total ms, launches)} accumulated since profiling was turned on."""
        out = {}
        i = 0
        while True:
            name = ctypes.c_char_p()
            ms = ctypes.c_double()
            cnt = u64()
            if lib().ra_ctx_profile(self.h, i, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(cnt)) != 0:
                return out
            out[name.value.decode()] = (float(ms.value), int(cnt.value))
            i += 1

    def cursor(self):
        v = u64()
        _check(lib().ra_ctx_cursor(self.h, ctypes.byref(v)), "ra_ctx_cursor")
        return int(v.value)


def ra_mle_bind(ctx: Context, T: torch.Tensor, bind_rows: bool, point, field: bool = False):
    """d_out[c] = sum_r eq(point, r) T[r, c] (rows) or d_out[r] = sum_c T[r, c] eq(point, c)."""
    rows, cols = T.shape
    dt = RA_FIELD if field else _DT[T.dtype]
    pt, pp = _u64_array(point)
    out = torch.empty(cols if bind_rows else rows, dtype=torch.int64, device=T.device)
    _check(lib().ra_mle_bind(ctx.h, _dptr(T), dt, rows, cols, int(bool(bind_rows)), pp, len(pt), _dptr(out)),
           "ra_mle_bind")
    return out


def ra_mle_bind_noalloc(T: torch.Tensor, bind_rows: bool, point, out: torch.Tensor, field: bool = False,
                        stream: torch.cuda.Stream | None = None):
    """ra_mle_bind without a context or allocation: writes `out` (int64,
    cols or rows entries) on `stream` (default: the current stream) and
    returns without waiting."""
    rows, cols = T.shape
    dt = RA_FIELD if field else _DT[T.dtype]
    pt, pp = _u64_array(point)
    assert out.dtype == torch.int64 and out.numel() == (cols if bind_rows else rows) and out.is_contiguous()
    st = stream or torch.cuda.current_stream()
    _check(lib().ra_mle_bind_noalloc(_dptr(T), dt, rows, cols, int(bool(bind_rows)), pp, len(pt), _dptr(out),
                                     ctypes.c_void_p(st.cuda_stream)), "ra_mle_bind_noalloc")
    return out


def workspace_size(n: int, m: int, k: int, P: int = 64) -> int:
    """Bytes of caller workspace that cover every call of an n x m x k layer (ra_workspace_size)."""
    v = ctypes.c_size_t()
    _check(lib().ra_workspace_size(n, m, k, P, ctypes.byref(v)), "ra_workspace_size")
    return int(v.value)


def _ws(ws):
    """(pointer, bytes) of an optional caller workspace tensor (None: the context's own)."""
    if ws is None:
        return None, 0
    assert ws.is_cuda and ws.is_contiguous()
    return ctypes.c_void_p(ws.data_ptr()), ws.numel() * ws.element_size()


def ra_sumcheck_matmul_prove(ctx: Context, A: torch.Tensor, B: torch.Tensor, C: torch.Tensor | None = None,
                             ws: torch.Tensor | None = None):
    """Returns (C, transcript dict); in deferred mode the dict is filled at ctx.sync().
    C (optional): an int64 n x k device tensor to write the product to.
    ws (optional): caller-owned device workspace (see workspace_size)."""
    n, m = A.shape
    m2, k = B.shape
    assert m == m2 and B.dtype == torch.int16
    if C is None:
        C = torch.empty((n, k), dtype=torch.int64, device=A.device)
    assert C.shape == (n, k) and C.dtype == torch.int64 and C.is_contiguous()
    lm = m.bit_length() - 1
    ev = np.zeros(max(3 * lm, 1), dtype=np.uint64)
    pr = MatmulProof()
    pr.evals = ev.ctypes.data_as(u64p)
    _check(lib().ra_sumcheck_matmul_prove(ctx.h, _dptr(A), _DT[A.dtype], _dptr(B), n, m, k, _dptr(C), *_ws(ws),
                                          ctypes.byref(pr)), "ra_sumcheck_matmul_prove")
    res = {}
    ctx.later(lambda: res.update(c0=int(pr.c0), mm_evals=ev[:3 * lm].tolist(), a_star=int(pr.a_star),
                                 b_star=int(pr.b_star)))
    return C, res


def witness_outputs(n: int, k: int, device):
    """Device tensors (R, Rm, Y, Z, bits) for a witness call on an n x k product."""
    return (torch.empty((n, k), dtype=torch.int32, device=device),
            torch.empty((n, k), dtype=torch.int16, device=device),   # uint16 bits
            torch.empty((n, k), dtype=torch.int32, device=device),
            torch.empty((n, k), dtype=torch.int32, device=device),
            torch.empty(n * k, dtype=torch.int64, device=device))    # uint64 words


def ra_rescale_relu_witness(ctx: Context, C: torch.Tensor, s: int, relu: bool, mode: int = 0, t: int = -1,
                            outs=None, ws: torch.Tensor | None = None):
    """Returns ((R, Rm, Y, Z, bits), info).  info.t and info.P are set on return
    (at once when t is given); the claims in info are final after ctx.sync()
    in deferred mode.  outs (optional): the five output tensors, as made by
    witness_outputs."""
    n, k = C.shape
    R, Rm, Y, Z, bits = witness_outputs(n, k, C.device) if outs is None else outs
    for tsr, dt in ((R, torch.int32), (Rm, torch.int16), (Y, torch.int32), (Z, torch.int32), (bits, torch.int64)):
        assert tsr.dtype == dt and tsr.numel() == n * k and tsr.is_contiguous()
    info = WitnessInfo(s=s, relu=int(bool(relu)), round_mode=mode, t=t)
    _check(lib().ra_rescale_relu_witness(ctx.h, _dptr(C), n, k, _dptr(R), _dptr(Rm), _dptr(Y), _dptr(Z),
                                         _dptr(bits), n * k, *_ws(ws), ctypes.byref(info)),
           "ra_rescale_relu_witness")
    return (R, Rm, Y, Z, bits), info


def ra_witness_plan(ctx: Context, s: int, relu: bool, mode: int, t: int, outs):
    """Announce the next witness call (given t, output tensors as made by
    witness_outputs) so that the next matrix call computes it in its product."""
    R, Rm, Y, Z, bits = outs
    _check(lib().ra_witness_plan(ctx.h, s, int(bool(relu)), mode, t, _dptr(R), _dptr(Rm), _dptr(Y), _dptr(Z),
                                 _dptr(bits), bits.numel()), "ra_witness_plan")


def ra_range_prove(ctx: Context, bits, R, Y, info: WitnessInfo, ws: torch.Tensor | None = None):
    """Returns the range / ReLU transcript dict (filled at ctx.sync() in deferred mode)."""
    n, k = R.shape
    N = n * k
    lN = N.bit_length() - 1
    lP = info.P.bit_length() - 1
    ev = np.zeros(4 * (lP + lN), dtype=np.uint64)
    zev = np.zeros(max(4 * lN, 1), dtype=np.uint64)
    pr = RangeProof()
    pr.evals = ev.ctypes.data_as(u64p)
    pr.relu_evals = zev.ctypes.data_as(u64p)
    _check(lib().ra_range_prove(ctx.h, _dptr(bits), _dptr(R), _dptr(Y), n, k, ctypes.byref(info), *_ws(ws),
                                ctypes.byref(pr)), "ra_range_prove")
    res = {}
    ctx.later(lambda: res.update(rs_evals=ev.tolist(), range_sum=int(pr.range_sum),
                                 bits_claim=int(pr.bits_claim), zc_evals=zev[:4 * pr.relu_rounds].tolist(),
                                 r_at=int(pr.r_at), y_at=int(pr.y_at)))
    return res


def prove_layer(ctx: Context, A: torch.Tensor, B: torch.Tensor, s: int, relu: bool, mode: int = 0, t: int = -1,
                bufs: dict | None = None, plan: bool = True, ws: torch.Tensor | None = None):
    """The three calls of one layer; returns device tensors and the transcript
    (complete at once, or after ctx.sync() in deferred mode).  bufs (optional):
    a dict that keeps the layer's device outputs, made on first use and
    written again by later calls with it (a caller proving the same shapes
    repeatedly saves the allocations).  With t given and plan set, the
    witness is announced (ra_witness_plan) and computed inside the product."""
    n, k = A.shape[0], B.shape[1]
    if bufs is not None and "C" not in bufs:
        bufs["C"] = torch.empty((n, k), dtype=torch.int64, device=A.device)
        bufs["wit"] = witness_outputs(n, k, A.device)
    wit = None if bufs is None else bufs["wit"]
    if t >= 0 and plan:  # t given: the witness is announced and computed inside the product
        if wit is None:
            wit = witness_outputs(n, k, A.device)
        ra_witness_plan(ctx, s, relu, mode, t, wit)
    C, mm = ra_sumcheck_matmul_prove(ctx, A, B, None if bufs is None else bufs["C"], ws)
    (R, Rm, Y, Z, bits), info = ra_rescale_relu_witness(ctx, C, s, relu, mode, t, wit, ws)
    rs = ra_range_prove(ctx, bits, R, Y, info, ws)
    tr = {}

    def fill():
        tr.update(mm)
        tr.update(rs)
        tr.update(t=int(info.t), P=int(info.P), r_claim=int(info.r_claim), rm_claim=int(info.rm_claim),
                  y_claim=int(info.y_claim), z_claim=int(info.z_claim), s=s, relu=int(bool(relu)), mode=mode)
    ctx.later(fill)
    return dict(C=C, R=R, Rm=Rm, Y=Y, Z=Z, bits=bits, transcript=tr)


def to_device(a: np.ndarray, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def link_prove(ctx: Context, Z_prev: torch.Tensor, src: torch.Tensor, ws: torch.Tensor | None = None):
    """The gather link of the layer just proven (ra_link_prove): A[a] =
    Z_prev[src[a]] (-1: zero), src an int32 device tensor of the layer's n m
    entries.  Returns dict(evals, claim, z_at, w_at), filled at ctx.sync() in
    deferred mode."""
    assert Z_prev.dtype == torch.int32 and src.dtype == torch.int32
    nz = Z_prev.numel()
    vz = nz.bit_length() - 1
    ev = np.zeros(max(3 * vz, 1), dtype=np.uint64)
    pr = LinkProof()
    pr.evals = ev.ctypes.data_as(u64p)
    _check(lib().ra_link_prove(ctx.h, _dptr(Z_prev), nz, _dptr(src), src.numel(), *_ws(ws), ctypes.byref(pr)),
           "ra_link_prove")
    res = {}
    ctx.later(lambda: res.update(evals=[int(x) for x in ev[:3 * vz]], claim=int(pr.claim), z_at=int(pr.z_at),
                                 w_at=int(pr.w_at)))
    return res


def link_gather(ctx: Context, Z_prev: torch.Tensor, src: torch.Tensor, out: torch.Tensor | None = None):
    """The gathered input A[a] = Z_prev[src[a]] (0 where src = -1) on the
    device (ra_link_gather; enqueued on the context's stream)."""
    assert Z_prev.dtype == torch.int32 and src.dtype == torch.int32
    if out is None:
        out = torch.empty(src.shape, dtype=torch.int32, device=src.device)
    _check(lib().ra_link_gather(ctx.h, _dptr(Z_prev), Z_prev.numel(), _dptr(src), src.numel(), _dptr(out)),
           "ra_link_gather")
    return out


def link_workspace_size(z_entries: int, n: int, m: int) -> int:
    v = ctypes.c_size_t()
    _check(lib().ra_link_workspace_size(z_entries, n, m, ctypes.byref(v)), "ra_link_workspace_size")
    return int(v.value)


def prove_network(ctx: Context, workload, device="cuda", X=None, Bs=None, ts=None, bufs=None, plan=True, ws=None,
                  links=False):
    """Prove every layer of a workload in order.  A layer's input is the
    previous output on the device (MLP chains) or the workload's link (im2col)
    applied on the host.  X / Bs may hold device copies of the inputs; ts may
    give each layer's range parameter t (else it is derived from the data);
    bufs (optional) is a list of per-layer output dicts (prove_layer), grown
    on first use.  links=True also proves every gather link right after its
    layer (res["link"], res["link_src"] the map on the device)."""
    if bufs is not None:
        while len(bufs) < len(workload.layers):
            bufs.append({})
    X = to_device(workload.X, device) if X is None else X
    Bs = [to_device(L.B, device) for L in workload.layers] if Bs is None else Bs
    outs = []
    Z = None
    for li, layer in enumerate(workload.layers):
        if li == 0:
            A = X
        elif workload.links[li] is None:
            A = Z
        else:   # a gather of the previous output (im2col, flatten), on the device
            keep = bufs[li] if bufs is not None else {}
            if "src" not in keep:
                n, m = workload.shapes()[li][:2]
                keep["src"] = to_device(workload.link_map(li).astype(np.int32).reshape(n, m), device)
            src = keep["src"]
            A = link_gather(ctx, Z, src, keep.get("A"))
            keep["A"] = A
        t = -1 if ts is None else int(ts[li])
        res = prove_layer(ctx, A, Bs[li], layer.s, layer.relu, workload.mode, t,
                          None if bufs is None else bufs[li], plan, ws)
        if links and li > 0 and workload.links[li] is not None:
            res["link"] = link_prove(ctx, Z, src, ws)
            res["link_src"] = src
        res["A"] = A
        Z = res["Z"]
        outs.append(res)
    return outs


def unpack_bits(words: np.ndarray, P: int) -> np.ndarray:
    """(N,) uint64 words -> (P, N) uint8 planes (bit q of word x = plane q)."""
    w = np.asarray(words).view(np.uint64)
    q = np.arange(P, dtype=np.uint64)[:, None]
    return ((w[None, :] >> q) & np.uint64(1)).astype(np.uint8)


def ra_verify(challenges, layers):
    """Host verifier.  `challenges` is a seed (int: ra_verify draws the
    stream) or an array of challenges (ra_verify_stream).  `layers` is a
    list of dicts with numpy arrays A, B, Z, R, Rm, Y, bits (uint64 words)
    and the transcript dict; returns (verdict, failed_layer)."""
    seeded = isinstance(challenges, (int, np.integer))
    if not seeded:
        chal, cp = _u64_array(challenges)
    nl = len(layers)
    pubs = (LayerPublic * nl)()
    tabs = (LayerTables * nl)()
    trs = (LayerTranscript * nl)()
    keep = []
    for i, L in enumerate(layers):
        tr = L["transcript"]
        A = np.ascontiguousarray(L["A"])
        B = np.ascontiguousarray(L["B"], dtype=np.int16)
        n, m = A.shape
        k = B.shape[1]
        arrs = dict(A=A, B=B, Z=np.ascontiguousarray(L["Z"], dtype=np.int32),
                    R=np.ascontiguousarray(L["R"], dtype=np.int32),
                    Rm=np.ascontiguousarray(np.asarray(L["Rm"]).view(np.uint16)),
                    Y=np.ascontiguousarray(L["Y"], dtype=np.int32),
                    bits=np.ascontiguousarray(np.asarray(L["bits"]).view(np.uint64)))
        mm = np.array(tr["mm_evals"] + [0], dtype=np.uint64)
        rs = np.array(tr["rs_evals"] + [0], dtype=np.uint64)
        zc = np.array(tr["zc_evals"] + [0], dtype=np.uint64)
        keep += list(arrs.values()) + [mm, rs, zc]
        lsrc = None
        if L.get("link_src") is not None:
            lsrc = np.ascontiguousarray(L["link_src"], dtype=np.int32)
            keep.append(lsrc)
        pubs[i] = LayerPublic(n, m, k, tr["s"], tr["relu"], tr["mode"],
                              RA_I16 if A.dtype == np.int16 else RA_I32, arrs["A"].ctypes.data,
                              arrs["B"].ctypes.data, arrs["Z"].ctypes.data, int(L.get("chained", 0)),
                              None if lsrc is None else lsrc.ctypes.data)
        tabs[i] = LayerTables(arrs["R"].ctypes.data, arrs["Rm"].ctypes.data, arrs["Y"].ctypes.data,
                              arrs["bits"].ctypes.data)
        t = trs[i]
        t.mm.log_m = m.bit_length() - 1
        t.mm.c0, t.mm.a_star, t.mm.b_star = tr["c0"], tr["a_star"], tr["b_star"]
        t.mm.evals = mm.ctypes.data_as(u64p)
        t.wit = WitnessInfo(tr["s"], tr["relu"], tr["mode"], tr["t"], tr["P"], tr["r_claim"], tr["rm_claim"],
                            tr["y_claim"], tr["z_claim"])
        t.rng.rounds = len(tr["rs_evals"]) // 4
        t.rng.evals = rs.ctypes.data_as(u64p)
        t.rng.range_sum, t.rng.bits_claim = tr["range_sum"], tr["bits_claim"]
        t.rng.relu_rounds = len(tr["zc_evals"]) // 4
        t.rng.relu_evals = zc.ctypes.data_as(u64p)
        t.rng.r_at, t.rng.y_at = tr["r_at"], tr["y_at"]
        if L.get("link") is not None:
            lk = L["link"]
            le = np.array(list(lk["evals"]) + [0], dtype=np.uint64)
            keep.append(le)
            t.link.rounds = len(lk["evals"]) // 3
            t.link.evals = le.ctypes.data_as(u64p)
            t.link.claim, t.link.z_at, t.link.w_at = lk["claim"], lk["z_at"], lk["w_at"]
    verdict = ctypes.c_int32()
    failed = ctypes.c_uint32()
    if seeded:
        _check(lib().ra_verify(P61, int(challenges), nl, pubs, tabs, trs, ctypes.byref(verdict),
                               ctypes.byref(failed)), "ra_verify")
    else:
        _check(lib().ra_verify_stream(P61, cp, len(chal), nl, pubs, tabs, trs, ctypes.byref(verdict),
                                      ctypes.byref(failed)), "ra_verify_stream")
    return int(verdict.value), int(failed.value)



# --- layers with challenges in F_{p^2} ---------------------------------------
def workspace_size_fp2(n: int, m: int, k: int) -> int:
    v = ctypes.c_size_t()
    _check(lib().ra_workspace_size_fp2(n, m, k, ctypes.byref(v)), "ra_workspace_size_fp2")
    return int(v.value)


def _fp2_list(arr, count):
    return [(int(arr[i].re), int(arr[i].im)) for i in range(count)]


def prove_layer_fp2(ctx: Context, A: torch.Tensor, B: torch.Tensor, s: int, relu: bool, mode: int = 0, t: int = -1,
                    bufs: dict | None = None, ws: torch.Tensor | None = None, pub: bytes | None = None):
    """One layer over F_{p^2} (ra_prove_layer_fp2; waits for its work), or,
    with pub (the layer's 32-byte public digest) on a Fiat-Shamir context,
    the non-interactive proof (ra_prove_layer_fs; result["root"] is the
    witness tables' Merkle root).  Returns the device tensors and the
    transcript, every element a pair (re, im)."""
    n, m = A.shape
    k = B.shape[1]
    dev = A.device
    if bufs is not None and "C" in bufs:
        C, (R, Rm, Y, Z, bits) = bufs["C"], bufs["wit"]
    else:
        C = torch.empty((n, k), dtype=torch.int64, device=dev)
        R, Rm, Y, Z, bits = witness_outputs(n, k, dev)
        if bufs is not None:
            bufs["C"], bufs["wit"] = C, (R, Rm, Y, Z, bits)
    N = n * k
    lm, lN = m.bit_length() - 1, N.bit_length() - 1
    mm = (Fp2 * max(3 * lm, 1))()
    rs = (Fp2 * (4 * (6 + lN)))()
    zc = (Fp2 * max(4 * lN, 1))()
    pr = LayerProofFp2(s=s, relu=int(bool(relu)), round_mode=mode, t=t)
    pr.mm_evals, pr.rs_evals, pr.zc_evals = mm, rs, zc
    root = None
    if pub is None:
        _check(lib().ra_prove_layer_fp2(ctx.h, _dptr(A), _DT[A.dtype], _dptr(B), n, m, k, _dptr(C), _dptr(R),
                                        _dptr(Rm), _dptr(Y), _dptr(Z), _dptr(bits), N, *_ws(ws), ctypes.byref(pr)),
               "ra_prove_layer_fp2")
    else:
        assert len(pub) == 32
        rb = ctypes.create_string_buffer(32)
        _check(lib().ra_prove_layer_fs(ctx.h, _dptr(A), _DT[A.dtype], _dptr(B), n, m, k, _dptr(C), _dptr(R),
                                       _dptr(Rm), _dptr(Y), _dptr(Z), _dptr(bits), N, bytes(pub), *_ws(ws),
                                       ctypes.byref(pr), rb), "ra_prove_layer_fs")
        root = rb.raw
    tr = dict(t=int(pr.t), P=int(pr.P), s=s, relu=int(bool(relu)), mode=mode,
              mm_evals=_fp2_list(mm, 3 * pr.log_m), rs_evals=_fp2_list(rs, 4 * pr.rounds),
              zc_evals=_fp2_list(zc, 4 * pr.relu_rounds))
    for key in FP2_SCALARS:
        v = getattr(pr, key)
        tr[key] = (int(v.re), int(v.im))
    return dict(C=C, R=R, Rm=Rm, Y=Y, Z=Z, bits=bits, transcript=tr, root=root)


def prove_network_fp2(ctx: Context, workload, device="cuda", X=None, Bs=None, ts=None, bufs=None, ws=None,
                      pubs=None):
    """Every layer of a workload over F_{p^2}, inputs as in prove_network;
    with pubs (one 32-byte public digest per layer) on a Fiat-Shamir context,
    the non-interactive proof."""
    if bufs is not None:
        while len(bufs) < len(workload.layers):
            bufs.append({})
    X = to_device(workload.X, device) if X is None else X
    Bs = [to_device(L.B, device) for L in workload.layers] if Bs is None else Bs
    outs, Z = [], None
    for li, layer in enumerate(workload.layers):
        if li == 0:
            A = X
        elif workload.links[li] is None:
            A = Z
        else:
            A = to_device(workload.links[li](Z.cpu().numpy()), device)
        t = -1 if ts is None else int(ts[li])
        res = prove_layer_fp2(ctx, A, Bs[li], layer.s, layer.relu, workload.mode, t,
                              None if bufs is None else bufs[li], ws, None if pubs is None else pubs[li])
        res["A"] = A
        Z = res["Z"]
        outs.append(res)
    return outs


def _fp2_layer_structs(layers):
    """ctypes arrays (public data, tables, transcripts) of layers proven over F_{p^2}."""
    nl = len(layers)
    pubs = (LayerPublic * nl)()
    tabs = (LayerTables * nl)()
    trs = (LayerProofFp2 * nl)()
    keep = []
    for i, L in enumerate(layers):
        tr = L["transcript"]
        A = np.ascontiguousarray(L["A"])
        B = np.ascontiguousarray(L["B"], dtype=np.int16)
        n, m = A.shape
        k = B.shape[1]
        arrs = dict(A=A, B=B, Z=np.ascontiguousarray(L["Z"], dtype=np.int32),
                    R=np.ascontiguousarray(L["R"], dtype=np.int32),
                    Rm=np.ascontiguousarray(np.asarray(L["Rm"]).view(np.uint16)),
                    Y=np.ascontiguousarray(L["Y"], dtype=np.int32),
                    bits=np.ascontiguousarray(np.asarray(L["bits"]).view(np.uint64)))

        def fp2_array(ev):
            a = (Fp2 * max(len(ev), 1))()
            for j, (re, im) in enumerate(ev):
                a[j].re, a[j].im = re, im
            return a
        mm, rs, zc = fp2_array(tr["mm_evals"]), fp2_array(tr["rs_evals"]), fp2_array(tr["zc_evals"])
        keep += list(arrs.values()) + [mm, rs, zc]
        pubs[i] = LayerPublic(n, m, k, tr["s"], tr["relu"], tr["mode"], RA_I16 if A.dtype == np.int16 else RA_I32,
                              arrs["A"].ctypes.data, arrs["B"].ctypes.data, arrs["Z"].ctypes.data,
                              int(L.get("chained", 0)))
        tabs[i] = LayerTables(arrs["R"].ctypes.data, arrs["Rm"].ctypes.data, arrs["Y"].ctypes.data,
                              arrs["bits"].ctypes.data)
        t = trs[i]
        t.s, t.relu, t.round_mode, t.t, t.P = tr["s"], tr["relu"], tr["mode"], tr["t"], tr["P"]
        t.log_m = len(tr["mm_evals"]) // 3
        t.rounds = len(tr["rs_evals"]) // 4
        t.relu_rounds = len(tr["zc_evals"]) // 4
        t.mm_evals, t.rs_evals, t.zc_evals = mm, rs, zc
        for key in FP2_SCALARS:
            re, im = tr[key]
            setattr(t, key, Fp2(re, im))
    return pubs, tabs, trs, keep


def ra_verify_fp2(seed: int, layers):
    """Host verifier for layers proven over F_{p^2}; `layers` as for ra_verify
    with the transcripts of prove_layer_fp2.  Returns (verdict, failed_layer)."""
    nl = len(layers)
    pubs, tabs, trs, keep = _fp2_layer_structs(layers)
    verdict = ctypes.c_int32()
    failed = ctypes.c_uint32()
    _check(lib().ra_verify_fp2(P61, int(seed), nl, pubs, tabs, trs, ctypes.byref(verdict), ctypes.byref(failed)),
           "ra_verify_fp2")
    return int(verdict.value), int(failed.value)


def ra_verify_fs(domain: bytes, pub_digests, layers):
    """Host verifier of non-interactive proofs (Fiat-Shamir over F_{p^2}):
    domain the transcript's 32 bytes, pub_digests one 32-byte digest per
    layer, layers as for ra_verify_fp2.  Returns (verdict, failed_layer)."""
    assert len(domain) == 32 and len(pub_digests) == len(layers)
    nl = len(layers)
    pubs, tabs, trs, keep = _fp2_layer_structs(layers)
    digests = b"".join(bytes(d) for d in pub_digests)
    assert len(digests) == 32 * nl
    verdict = ctypes.c_int32()
    failed = ctypes.c_uint32()
    _check(lib().ra_verify_fs(P61, bytes(domain), nl, pubs, tabs, trs, digests, ctypes.byref(verdict),
                              ctypes.byref(failed)), "ra_verify_fs")
    return int(verdict.value), int(failed.value)


# --- Pedersen vector commitments on secp256k1 ---------------------------------
_CDT = {torch.int16: RA_I16, torch.int32: RA_I32}
_NDT = {np.dtype(np.int16): RA_I16, np.dtype(np.uint16): RA_U16, np.dtype(np.int32): RA_I32,
        np.dtype(np.uint64): RA_U64}


def commit_generators(ctx: Context, domain: bytes, count: int, first: int = 0, out: torch.Tensor | None = None):
    """Generators first .. first + count - 1 (ra_commit_generators): a device
    uint32 tensor of count x 16 limbs (x then y, little-endian)."""
    assert len(domain) == 32
    if out is None:
        out = torch.empty((count, 16), dtype=torch.int32, device="cuda")
    _check(lib().ra_commit_generators(ctx.h, bytes(domain), first, count, _dptr(out)), "ra_commit_generators")
    return out


def commit(ctx: Context, values: torch.Tensor, gens: torch.Tensor, dtype: int | None = None,
           ws: torch.Tensor | None = None) -> bytes:
    """sum_i values[i] G_i as 64 big-endian bytes (ra_commit).  values: an
    int16 / int32 device tensor, or another 2- or 8-byte tensor with dtype
    RA_U16 / RA_U64 given."""
    d = dtype if dtype is not None else _CDT[values.dtype]
    out = ctypes.create_string_buffer(64)
    _check(lib().ra_commit(ctx.h, _dptr(values), d, values.numel(), _dptr(gens), *_ws(ws), out), "ra_commit")
    return out.raw


def commit_batch(ctx: Context, tables, gens: torch.Tensor, ws: torch.Tensor | None = None) -> list:
    """Commitments to several tables in one call (ra_commit_batch): tables is
    a list of device tensors or (tensor, dtype) pairs as for commit; returns
    one 64-byte commitment per table."""
    vals, dts, ns = [], [], []
    for tb in tables:
        v, d = tb if isinstance(tb, tuple) else (tb, None)
        vals.append(_dptr(v))
        dts.append(d if d is not None else _CDT[v.dtype])
        ns.append(v.numel())
    cnt = len(vals)
    pv = (ctypes.c_void_p * cnt)(*vals)
    pd = (ctypes.c_int32 * cnt)(*dts)
    pn = (ctypes.c_uint64 * cnt)(*ns)
    out = ctypes.create_string_buffer(64 * cnt)
    _check(lib().ra_commit_batch(ctx.h, pv, pd, pn, cnt, _dptr(gens), *_ws(ws), out), "ra_commit_batch")
    return [out.raw[64 * t:64 * (t + 1)] for t in range(cnt)]


def commit_open(values: np.ndarray, gens_limbs: np.ndarray, commitment: bytes) -> bool:
    """Host opening check (ra_commit_open) of a commitment to host values."""
    v = np.ascontiguousarray(values)
    g = np.ascontiguousarray(gens_limbs, dtype=np.uint32)
    ok = ctypes.c_int32()
    _check(lib().ra_commit_open(v.ctypes.data, _NDT[v.dtype], v.size, g.ctypes.data, bytes(commitment),
                                ctypes.byref(ok)), "ra_commit_open")
    return bool(ok.value)


def point_limbs(points) -> np.ndarray:
    """Affine points (x, y) as the generator layout: 16 little-endian uint32 limbs each."""
    out = np.zeros((len(points), 16), dtype=np.uint32)
    for i, (x, y) in enumerate(points):
        for l in range(8):
            out[i, l] = (x >> (32 * l)) & 0xFFFFFFFF
            out[i, 8 + l] = (y >> (32 * l)) & 0xFFFFFFFF
    return out
