"""Every-row comparison of a device result against the oracle, streamed in row chunks.

The oracle's SpMM is plain single-threaded C; the comparison runs it on independent row
chunks from worker threads (the C call releases the interpreter lock), so a full-size
result (tens of millions of entries times F features) is checked in seconds.  Nothing
here computes an expected value: each chunk's reference and bound come from the oracle.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

BF16_U = 2.0 ** -8              # unit roundoff of bfloat16 (8 significand bits), nearest-even


def workers():
    """Worker threads: the host cores this process may use, at most 16."""
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    return max(1, min(16, cores))


def spmm_judge(tol=1e-5):
    """|y - y_ref| <= tol * sum |a||x| (exactly 0 where the bound is 0)."""
    def judge(rows, Yc, Yr, B):
        err = np.abs(Yc - Yr)
        lim = tol * B
        return err, lim
    return judge


def act_bf16_judge(tol=1e-5):
    """Output stored as bfloat16 after ReLU: the float32 sum is within tol * B of the oracle,
    ReLU is 1-Lipschitz, and the rounding to bfloat16 adds at most 2^-8 of the float32 value:
    |out - relu(y_ref)| <= tol B (1 + 2^-8) + 2^-8 |relu(y_ref)|."""
    def judge(rows, Yc, Yr, B):
        R = np.maximum(Yr, 0.0)
        err = np.abs(Yc - R)
        lim = tol * B * (1.0 + BF16_U) + BF16_U * R
        return err, lim
    return judge


def fused_judge(W, tol=1e-2):
    """T = bf16(relu(A X)) bf16(W) with float32 accumulation, against the float64
    H W with H = relu(A X): |T - H W| <= tol ((|H| + B) |W|).  The bound covers the SpMM's
    float32 error (1e-5 B), the two bfloat16 roundings of each product (at most
    2 * 2^-8 + 2^-16 relative) and the float32 accumulation over F_in terms."""
    Wd = np.asarray(W, dtype=np.float64)
    Wa = np.abs(Wd)

    def judge(rows, Tc, Yr, B):
        H = np.maximum(Yr, 0.0)
        err = np.abs(Tc - H @ Wd)
        lim = tol * ((np.abs(H) + B) @ Wa)
        return err, lim
    return judge


def compare_all_rows(g, X, Y, judge, chunk=1 << 16, what=""):
    """Checks every row of Y (host array, n x F or n x F_out) with `judge` on the oracle's
    SpMM of X.  Raises AssertionError naming the first element outside the bound and the
    number of such elements; returns the largest err / bound ratio."""
    n = g.n
    Xc = np.ascontiguousarray(X, dtype=np.float32)
    starts = list(range(0, n, chunk))

    def one(s):
        rows = np.arange(s, min(n, s + chunk), dtype=np.int32)
        Yr, B = oracle.spmm(g, Xc, rows)
        Yc = np.asarray(Y[s:s + rows.size], dtype=np.float64)
        err, lim = judge(rows, Yc, Yr, B)
        bad = ~(err <= lim)            # NaN (an unwritten element of a poisoned output) is bad
        nbad = int(bad.sum())
        first = None
        if nbad:
            i = np.argwhere(bad)[0]
            first = (int(rows[i[0]]), int(i[1]), float(Yc[tuple(i)]), float(lim[tuple(i)]))
        with np.errstate(divide="ignore", invalid="ignore"):
            ratio = np.where(lim > 0, err / np.where(lim > 0, lim, 1.0), np.where(err > 0, np.inf, 0.0))
        worst = float(np.nanmax(ratio)) if ratio.size else 0.0
        return nbad, first, worst

    with ThreadPoolExecutor(workers()) as ex:
        results = list(ex.map(one, starts))
    nbad = sum(r[0] for r in results)
    if nbad:
        first = next(r[1] for r in results if r[0])
        raise AssertionError(f"{what}: {nbad} elements outside the bound; first (row, feature, "
                             f"got, bound) = {first}")
    return max(r[2] for r in results)
