"""Test helpers: conversions between the oracle's plain tables and the
library's ABI layout, and transcript comparison."""
import numpy as np

TRANSCRIPT_KEYS = ["t", "P", "c0", "mm_evals", "a_star", "b_star", "r_claim", "rm_claim", "y_claim",
                   "z_claim", "range_sum", "rs_evals", "bits_claim", "zc_evals", "r_at", "y_at"]


def pack_planes(planes: np.ndarray) -> np.ndarray:
    """(P, N) 0/1 planes -> (N,) uint64 words with bit q = plane q."""
    P, N = planes.shape
    w = np.zeros(N, dtype=np.uint64)
    for q in range(P):
        w |= planes[q].astype(np.uint64) << np.uint64(q)
    return w


def oracle_layer_for_abi(res, B, chained=False):
    """An oracle layer result as the dict ra.ra_verify expects."""
    A = res["A"]
    a_dtype = np.int16 if (np.abs(A).max(initial=0) < 2 ** 15 and not chained) else np.int32
    return dict(A=np.ascontiguousarray(A, dtype=a_dtype), B=np.ascontiguousarray(B, dtype=np.int16),
                Z=res["Z"].astype(np.int32), R=res["R"].astype(np.int32), Rm=res["Rm"].astype(np.uint16),
                Y=res["Y"].astype(np.int32), bits=pack_planes(res["bits"]), transcript=res, chained=chained)


def diff_transcripts(a: dict, b: dict):
    """Keys whose values differ (every transcript word must match)."""
    bad = []
    for key in TRANSCRIPT_KEYS:
        if list(np.atleast_1d(a[key])) != list(np.atleast_1d(b[key])):
            bad.append(key)
    return bad
