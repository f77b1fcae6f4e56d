"""fp64 CPU oracle for attention forward/backward and the schedule model.

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP path (``paper_2601_21824_amd``) and neither imports the
other; both are fed by the seeded generators in ``paper_2601_21824_amd.synth``,
which hold none of the method's arithmetic.

The arithmetic lives in ``attn_oracle.c`` (plain C, fp64, definitions written
out; see its header for the formulas and the paper passages they follow).
This module converts inputs exactly to float64, calls it head by head, and
returns numpy arrays.  ``schedule.py`` holds the schedule enumeration and the
DAG model of Section 3.

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
(finite differences, closed forms, invariants, a torch fp64 autograd
cross-check, and the paper's closed-form makespans for the schedules).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "attn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile attn_oracle.c into liboracle.so with gcc (fp64, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                        "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        ip = ctypes.POINTER(ctypes.c_int)
        ci, cd = ctypes.c_int, ctypes.c_double
        lib.oracle_fwd_rows.argtypes = [dp, dp, dp, ci, ci, ci, cd, ip, ci, dp, dp]
        lib.oracle_bwd_dq_rows.argtypes = [dp, dp, dp, dp, ci, ci, ci, cd, ip, ci, dp, dp, dp]
        lib.oracle_bwd_dkdv_cols.argtypes = [dp, dp, dp, dp, ci, ci, ci, cd, dp, dp, ip, ci, dp, dp]
        lib.oracle_probs.argtypes = [dp, dp, ci, ci, ci, cd, dp]
        for f in (lib.oracle_fwd_rows, lib.oracle_bwd_dq_rows, lib.oracle_bwd_dkdv_cols,
                  lib.oracle_probs):
            f.restype = None
        _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    """Exact promotion to a C-contiguous float64 array (bf16/fp32 -> fp64 is exact)."""
    if hasattr(x, "detach"):  # a torch tensor
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _ip(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))


def _rows(sel, n):
    if sel is None:
        return np.arange(n, dtype=np.int32)
    return np.ascontiguousarray(np.asarray(sel, dtype=np.int32))


def _scale(d, scale):
    return 1.0 / np.sqrt(d) if scale is None else float(scale)


def attn_fwd(q, k, v, causal: bool, scale=None, rows=None):
    """O [.., N, d] and L [.., N] (natural-log logsumexp of the scaled scores).

    q, k, v: [..., N, d] (any leading dims, each slice one head).  ``rows``
    restricts the work to those query rows (others are left at NaN).
    """
    lib = _load()
    q, k, v = _f64(q), _f64(k), _f64(v)
    *lead, n, d = q.shape
    s = _scale(d, scale)
    heads = int(np.prod(lead)) if lead else 1
    qf, kf, vf = q.reshape(heads, n, d), k.reshape(heads, n, d), v.reshape(heads, n, d)
    o = np.full((heads, n, d), np.nan)
    lse = np.full((heads, n), np.nan)
    r = _rows(rows, n)
    for h in range(heads):
        qh, kh, vh = (np.ascontiguousarray(a[h]) for a in (qf, kf, vf))
        oh, lh = np.full((n, d), np.nan), np.full(n, np.nan)
        lib.oracle_fwd_rows(_p(qh), _p(kh), _p(vh), n, d, int(causal), s, _ip(r), len(r), _p(oh), _p(lh))
        o[h], lse[h] = oh, lh
    return o.reshape(*lead, n, d), lse.reshape(*lead, n)


def lse_and_d(q, k, v, do, causal: bool, scale=None, block=512):
    """L and D of every query row of one head ([N, d] inputs), fp64.

    The two row vectors the backward needs besides Q, K, V and dO (the
    Background section's logsumexp vector L and Algorithm 1's preprocessing
    D = rowsum(dO o O)), from their definitions, for query rows taken ``block``
    at a time: S = scale * Q_b K^T (a library fp64 matrix product), masked
    entries -inf, L = m + log sum exp(S - m) with m the row maximum,
    P = exp(S - L), O_b = P V (a library product), D = sum over columns of
    dO_b o O_b.  No blocking over keys, so each row's sums are the plain
    definitions; it exists because the C row functions take minutes for
    every row of a 32768-row head, which sampled dK/dV rows need.  With a
    causal mask only the keys up to the block's last row enter, and P is
    formed as exp(S - m) / sum exp(S - m), which equals exp(S - L).
    """
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    n, d = q.shape
    s = _scale(d, scale)
    lse = np.empty(n)
    dvec = np.empty(n)
    for r0 in range(0, n, block):
        r1 = min(n, r0 + block)
        nk = r1 if causal else n  # keys past the block's last row are masked for all its rows
        sc = s * (q[r0:r1] @ k[:nk].T)
        if causal:  # query r0 + a sees key r0 + b iff b <= a
            diag = sc[:, r0:r1]
            diag[np.triu(np.ones((r1 - r0, r1 - r0), dtype=bool), 1)] = -np.inf
        m = sc.max(axis=1, keepdims=True)
        e = np.exp(sc - m)
        z = e.sum(axis=1, keepdims=True)
        lb = m + np.log(z)
        ob = (e / z) @ v[:nk]
        lse[r0:r1] = lb[:, 0]
        dvec[r0:r1] = np.sum(do[r0:r1] * ob, axis=1)
    return lse, dvec


def attn_bwd(q, k, v, do, causal: bool, scale=None, dq_rows=None, kv_rows=None):
    """dQ, dK, dV (fp64) of attention, plus the L and D vectors used.

    ``dq_rows`` / ``kv_rows`` restrict which rows of dQ / dK,dV are produced
    (others NaN).  Computing any dK/dV row needs L and D of every query row:
    with every dQ row requested they come from the same row-by-row pass;
    with only some dQ rows, from ``lse_and_d`` (all rows) while dQ is
    computed for the requested rows only.
    """
    lib = _load()
    q, k, v, do = _f64(q), _f64(k), _f64(v), _f64(do)
    *lead, n, d = q.shape
    s = _scale(d, scale)
    heads = int(np.prod(lead)) if lead else 1
    arrs = [a.reshape(heads, n, d) for a in (q, k, v, do)]
    dq = np.full((heads, n, d), np.nan)
    dk = np.full((heads, n, d), np.nan)
    dv = np.full((heads, n, d), np.nan)
    lse = np.full((heads, n), np.nan)
    dvec = np.full((heads, n), np.nan)
    qr = _rows(dq_rows, n)
    kr = _rows(kv_rows, n)
    for h in range(heads):
        qh, kh, vh, doh = (np.ascontiguousarray(a[h]) for a in arrs)
        dqh = np.full((n, d), np.nan)
        lh, Dh = np.full(n, np.nan), np.full(n, np.nan)
        if len(qr):
            lib.oracle_bwd_dq_rows(_p(qh), _p(kh), _p(vh), _p(doh), n, d, int(causal), s,
                                   _ip(qr), len(qr), _p(dqh), _p(lh), _p(Dh))
        if len(kr) and dq_rows is not None:  # L and D of the rows dQ did not cover
            lh, Dh = lse_and_d(qh, kh, vh, doh, causal, scale)
        dkh, dvh = np.full((n, d), np.nan), np.full((n, d), np.nan)
        if len(kr):
            lib.oracle_bwd_dkdv_cols(_p(qh), _p(kh), _p(vh), _p(doh), n, d, int(causal), s,
                                     _p(lh), _p(Dh), _ip(kr), len(kr), _p(dkh), _p(dvh))
        dq[h], dk[h], dv[h], lse[h], dvec[h] = dqh, dkh, dvh, lh, Dh
    shp = (*lead, n, d)
    return (dq.reshape(shp), dk.reshape(shp), dv.reshape(shp),
            lse.reshape(*lead, n), dvec.reshape(*lead, n))


def probs(q, k, causal: bool, scale=None):
    """Full P matrix of one head ([N, d] inputs), tiny problems only."""
    lib = _load()
    q, k = _f64(q), _f64(k)
    n, d = q.shape
    out = np.zeros((n, n))
    lib.oracle_probs(_p(q), _p(k), n, d, int(causal), _scale(d, scale), _p(out))
    return out


def ordered_sum_f32(partials):
    """fp32 sum of a list of fp32 arrays, strictly in list order, first term stored.

    The deterministic reduction's definition: dQacc starts as the rank-0
    partial and each later partial is added with one fp32 rounding per element
    (Algorithm 1, dQ-writer: wait for the turn, add, advance the order).
    """
    acc = np.array(partials[0], dtype=np.float32, copy=True)
    for p in partials[1:]:
        acc = (acc + np.asarray(p, dtype=np.float32)).astype(np.float32)
    return acc
