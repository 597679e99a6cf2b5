"""Comparison helpers shared by the parity tests (no method arithmetic here).

Floating-point parity is judged per element against the oracle's tolerance
scale `mag` (the sum of the absolute values of the terms that make up the
result, computed by the oracle in fp64):

    |gpu - oracle| <= rtol * mag

so an element whose terms cancel is judged on the size of what cancelled, not
on the (possibly tiny) result.  NaN or inf from the GPU where the oracle is
finite always fails.  The plain maximum relative error and the norm-relative
error are reported alongside but are not the gate.
"""
from __future__ import annotations

import numpy as np

FWD_RTOL = 1e-5   # forward outputs
BWD_RTOL = 1e-4   # backward outputs and meta-gradients


def stats(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    diff = np.abs(got - ref)
    nz = ref != 0
    plain = float(np.max(diff[nz] / np.abs(ref[nz]))) if nz.any() else 0.0
    den = float(np.linalg.norm(ref))
    normrel = float(np.linalg.norm(got - ref) / den) if den > 0 else float(np.linalg.norm(got - ref))
    return plain, normrel


def assert_mag_close(got, ref, mag, rtol, what=""):
    got = np.asarray(got, np.float64).reshape(-1)
    ref = np.asarray(ref, np.float64).reshape(-1)
    mag = np.asarray(mag, np.float64).reshape(-1)
    err = np.abs(got - ref)
    ok = err <= rtol * mag
    if not ok.all():
        bad = np.flatnonzero(~ok)
        i = bad[0]
        worst = bad[np.nanargmax(np.where(np.isfinite(err[bad]), err[bad] / np.maximum(mag[bad], 1e-300), np.inf))]
        raise AssertionError(
            "%s: %d of %d elements exceed %.0e x mag; first at %d: got %r ref %r mag %r; "
            "worst at %d: got %r ref %r mag %r"
            % (what, bad.size, got.size, rtol, i, got[i], ref[i], mag[i], worst, got[worst], ref[worst],
               mag[worst]))
    return stats(got, ref)


def assert_bits_equal(got, ref, what=""):
    got = np.ascontiguousarray(got)
    ref = np.ascontiguousarray(ref)
    assert got.dtype.itemsize == ref.dtype.itemsize and got.size == ref.size, what
    u = {1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[got.dtype.itemsize]
    gv, rv = got.view(u), ref.view(u)
    if not np.array_equal(gv, rv):
        bad = np.flatnonzero(gv != rv)
        raise AssertionError("%s: %d of %d elements differ; first at %d: got %#x ref %#x"
                             % (what, bad.size, gv.size, bad[0], int(gv[bad[0]]), int(rv[bad[0]])))
