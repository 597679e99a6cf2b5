"""CPU fp64 oracle for the differentiable Adam step and tree pack/unpack.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the CPU-baseline leg of the benchmark, never by the product path.  It shares
no code with the HIP library.  The arithmetic lives in ``oracle.c`` (plain C,
fp64, single thread, no FMA contraction); this module only marshals numpy
arrays into it.  The header of ``oracle.c`` lists the paper passages each
function follows, the readings taken where the paper is silent, and the pins
that tie each function to something other than itself.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# Plain C, no fast-math, no contraction: every operation is one IEEE double op.
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so next to it (gcc)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        build()
        _lib = _configure(ctypes.CDLL(_LIB))
    return _lib


def _configure(lib):
    """Declare the C signatures on a loaded copy of the oracle library (the
    tests also load deliberately altered builds of it, to show that their
    pins catch a planted mistake)."""
    d = ctypes.POINTER(ctypes.c_double)
    i64 = ctypes.c_int64
    f64 = ctypes.c_double
    hyper = [i64, f64, f64, f64, f64, f64]  # count, lr, b1, b2, eps, eps_root
    lib.oracle_adam_fwd.argtypes = [i64, d, d, d, d, *hyper, d, d, d, d]
    lib.oracle_adam_bwd.argtypes = [i64, d, d, d, d, d, d, *hyper, d, d, d, d]
    lib.oracle_adam_fwd_mag.argtypes = [i64, d, d, d, d, *hyper, d, d, d, d]
    lib.oracle_adam_bwd_mag.argtypes = [i64, d, d, d, d, d, d, *hyper, d, d, d]
    lib.oracle_unrolled_fwd.argtypes = [i64, i64, d, d, d, d, *hyper, d, d, d]
    lib.oracle_unrolled_bwd.argtypes = [i64, i64, d, d, d, d, *hyper, d, d, d, d]
    vp = ctypes.c_void_p
    lib.oracle_pack.argtypes = [i64, ctypes.POINTER(i64), ctypes.POINTER(i64), i64,
                                ctypes.POINTER(vp), vp]
    lib.oracle_unpack.argtypes = [i64, ctypes.POINTER(i64), ctypes.POINTER(i64), i64,
                                  vp, ctypes.POINTER(vp)]
    lib.oracle_sgd_fwd.argtypes = [i64, d, d, d, f64, f64, i64, d, d]
    lib.oracle_sgd_bwd.argtypes = [i64, d, d, f64, f64, i64, d, d]
    rms = [f64, f64, f64, f64, f64]  # lr, alpha, eps, eps_root, mu
    lib.oracle_rmsprop_fwd.argtypes = [i64, d, d, d, d, *rms, d, d, d]
    lib.oracle_rmsprop_bwd.argtypes = [i64, d, d, d, d, d, *rms, d, d, d]
    lib.oracle_rmsprop_fwd_mag.argtypes = [i64, d, d, d, d, *rms, d, d, d]
    lib.oracle_rmsprop_bwd_mag.argtypes = [i64, d, d, d, d, d, *rms, d, d, d]
    for f in ("oracle_sgd_fwd", "oracle_sgd_bwd", "oracle_rmsprop_fwd", "oracle_rmsprop_bwd",
              "oracle_rmsprop_fwd_mag", "oracle_rmsprop_bwd_mag",
              "oracle_adam_fwd", "oracle_adam_bwd", "oracle_adam_fwd_mag",
              "oracle_adam_bwd_mag", "oracle_unrolled_fwd", "oracle_unrolled_bwd",
              "oracle_pack", "oracle_unpack"):
        getattr(lib, f).restype = None
    lib.oracle_es_perturb.argtypes = [i64, i64, d, d, f64, i64, d]
    lib.oracle_es_perturb.restype = None
    lib.oracle_es_estimate.argtypes = [i64, i64, d, d, f64, d]
    lib.oracle_es_estimate.restype = None
    u64p = ctypes.POINTER(ctypes.c_uint64)
    lib.oracle_philox4x64_10.argtypes = [u64p, u64p, u64p]
    lib.oracle_philox4x64_10.restype = None
    lib.oracle_box_muller.argtypes = [ctypes.c_uint64, d, d]
    lib.oracle_box_muller.restype = None
    lib.oracle_es_gaussian_noise.argtypes = [i64, i64, ctypes.c_uint64, d]
    lib.oracle_es_gaussian_noise.restype = None
    lib.oracle_es_gaussian_noise_radius.argtypes = [i64, i64, ctypes.c_uint64, d]
    lib.oracle_es_gaussian_noise_radius.restype = None
    lib.oracle_es_gaussian_noise_cols.argtypes = [i64, i64, ctypes.POINTER(i64), ctypes.c_uint64, d, d]
    lib.oracle_es_gaussian_noise_cols.restype = None
    lib.oracle_es_weights.argtypes = [i64, d, f64, i64, f64, d, d]
    lib.oracle_es_weights.restype = None
    return lib


def _f64(x, n=None):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64).reshape(-1))
    if n is not None and a.size != n:
        raise ValueError("expected %d elements, got %d" % (n, a.size))
    return a


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _hyper(count, lr, b1, b2, eps, eps_root):
    return [int(count), float(lr), float(b1), float(b2), float(eps), float(eps_root)]


def adam_fwd(p, g, m, v, count, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, eps_root=0.0):
    """One Adam step; returns (p', m', v', u) as fp64 arrays."""
    p = _f64(p)
    n = p.size
    g, m, v = _f64(g, n), _f64(m, n), _f64(v, n)
    outs = [np.empty(n) for _ in range(4)]
    _load().oracle_adam_fwd(n, _ptr(p), _ptr(g), _ptr(m), _ptr(v),
                            *_hyper(count, lr, b1, b2, eps, eps_root), *map(_ptr, outs))
    return tuple(outs)


def adam_bwd(dP, dM, dV, g, m, v, count, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, eps_root=0.0):
    """VJP of one Adam step; dM/dV may be None (zero).  Returns (dp, dg, dm, dv)."""
    dP = _f64(dP)
    n = dP.size
    dM = None if dM is None else _f64(dM, n)
    dV = None if dV is None else _f64(dV, n)
    g, m, v = _f64(g, n), _f64(m, n), _f64(v, n)
    outs = [np.empty(n) for _ in range(4)]
    _load().oracle_adam_bwd(n, _ptr(dP), _ptr(dM), _ptr(dV), _ptr(g), _ptr(m), _ptr(v),
                            *_hyper(count, lr, b1, b2, eps, eps_root), *map(_ptr, outs))
    return tuple(outs)


def adam_fwd_mag(p, g, m, v, count, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, eps_root=0.0):
    """Tolerance scales (mag_p, mag_m, mag_v, mag_u) of the forward outputs."""
    p = _f64(p)
    n = p.size
    g, m, v = _f64(g, n), _f64(m, n), _f64(v, n)
    outs = [np.empty(n) for _ in range(4)]
    _load().oracle_adam_fwd_mag(n, _ptr(p), _ptr(g), _ptr(m), _ptr(v),
                                *_hyper(count, lr, b1, b2, eps, eps_root), *map(_ptr, outs))
    return tuple(outs)


def adam_bwd_mag(dP, dM, dV, g, m, v, count, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8,
                 eps_root=0.0):
    """Tolerance scales (mag_dg, mag_dm, mag_dv) of the backward outputs."""
    dP = _f64(dP)
    n = dP.size
    dM = None if dM is None else _f64(dM, n)
    dV = None if dV is None else _f64(dV, n)
    g, m, v = _f64(g, n), _f64(m, n), _f64(v, n)
    outs = [np.empty(n) for _ in range(3)]
    _load().oracle_adam_bwd_mag(n, _ptr(dP), _ptr(dM), _ptr(dV), _ptr(g), _ptr(m), _ptr(v),
                                *_hyper(count, lr, b1, b2, eps, eps_root), *map(_ptr, outs))
    return tuple(outs)


def unrolled_fwd(p0, grads, m0, v0, count0, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8,
                 eps_root=0.0):
    """K steps from (p0, m0, v0) with grads [K, n].  Returns (pK, m_traj, v_traj),
    the trajectories shaped [K+1, n] with entry 0 equal to m0 / v0."""
    p0 = _f64(p0)
    n = p0.size
    grads = np.ascontiguousarray(np.asarray(grads, dtype=np.float64).reshape(-1, n))
    K = grads.shape[0]
    m0, v0 = _f64(m0, n), _f64(v0, n)
    pK = np.empty(n)
    mt = np.empty((K + 1, n))
    vt = np.empty((K + 1, n))
    _load().oracle_unrolled_fwd(K, n, _ptr(p0), _ptr(grads), _ptr(m0), _ptr(v0),
                                *_hyper(count0, lr, b1, b2, eps, eps_root),
                                _ptr(pK), _ptr(mt), _ptr(vt))
    return pK, mt, vt


def unrolled_bwd(dpK, grads, m_traj, v_traj, count0, lr=1e-3, b1=0.9, b2=0.999, eps=1e-8,
                 eps_root=0.0):
    """Reverse pass through K steps.  Returns (dp0, dg [K, n], dm0, dv0)."""
    dpK = _f64(dpK)
    n = dpK.size
    grads = np.ascontiguousarray(np.asarray(grads, dtype=np.float64).reshape(-1, n))
    K = grads.shape[0]
    mt = np.ascontiguousarray(np.asarray(m_traj, dtype=np.float64).reshape(K + 1, n))
    vt = np.ascontiguousarray(np.asarray(v_traj, dtype=np.float64).reshape(K + 1, n))
    dp0, dm0, dv0 = np.empty(n), np.empty(n), np.empty(n)
    dg = np.empty((K, n))
    _load().oracle_unrolled_bwd(K, n, _ptr(dpK), _ptr(grads), _ptr(mt), _ptr(vt),
                                *_hyper(count0, lr, b1, b2, eps, eps_root),
                                _ptr(dp0), _ptr(dg), _ptr(dm0), _ptr(dv0))
    return dp0, dg, dm0, dv0


def _seg_args(numel, offsets):
    numel = np.ascontiguousarray(np.asarray(numel, dtype=np.int64).reshape(-1))
    offs = None if offsets is None else np.ascontiguousarray(
        np.asarray(offsets, dtype=np.int64).reshape(-1))
    p64 = ctypes.POINTER(ctypes.c_int64)
    return numel, offs, numel.ctypes.data_as(p64), (None if offs is None else offs.ctypes.data_as(p64))


def pack(leaves, flat_len=None, offsets=None, dtype=None):
    """Pack a list of numpy arrays (same dtype) into a new flat array by byte copy.
    Gaps (explicit offsets) are left zero."""
    leaves = [np.ascontiguousarray(x) for x in leaves]
    if dtype is None:
        dtype = leaves[0].dtype if leaves else np.float32
    dtype = np.dtype(dtype)
    numel = [x.size for x in leaves]
    for x in leaves:
        if x.dtype.itemsize != dtype.itemsize:
            raise ValueError("all leaves must share the element size")
    if flat_len is None:
        flat_len = (sum(numel) if offsets is None else
                    max([o + k for o, k in zip(offsets, numel)] + [0]))
    flat = np.zeros(flat_len, dtype=dtype)
    numel_a, offs_a, pn, po = _seg_args(numel, offsets)
    ptrs = (ctypes.c_void_p * max(len(leaves), 1))(*[x.ctypes.data for x in leaves])
    _load().oracle_pack(len(leaves), pn, po, dtype.itemsize, ptrs, flat.ctypes.data)
    return flat


def unpack(flat, shapes, offsets=None):
    """Split a flat numpy array into new arrays of the given shapes by byte copy."""
    flat = np.ascontiguousarray(flat)
    leaves = [np.empty(s, dtype=flat.dtype) for s in shapes]
    numel = [x.size for x in leaves]
    numel_a, offs_a, pn, po = _seg_args(numel, offsets)
    ptrs = (ctypes.c_void_p * max(len(leaves), 1))(*[x.ctypes.data for x in leaves])
    _load().oracle_unpack(len(leaves), pn, po, flat.dtype.itemsize, flat.ctypes.data, ptrs)
    return leaves


def _opt(x, n):
    return None if x is None else _f64(x, n)


def sgd_fwd(p, g, t, lr, momentum=0.0, nesterov=False):
    """SGD with momentum; t may be None (zero trace).  Returns (p', t')."""
    p = _f64(p)
    n = p.size
    g, t = _f64(g, n), _opt(t, n)
    po, to = np.empty(n), np.empty(n)
    _load().oracle_sgd_fwd(n, _ptr(p), _ptr(g), _ptr(t), float(lr), float(momentum), int(bool(nesterov)),
                           _ptr(po), _ptr(to))
    return po, to


def sgd_bwd(dP, dT, lr, momentum=0.0, nesterov=False):
    """VJP of sgd_fwd; dT may be None.  Returns (dp, dg, dt)."""
    dP = _f64(dP)
    n = dP.size
    dT = _opt(dT, n)
    dg, dt = np.empty(n), np.empty(n)
    _load().oracle_sgd_bwd(n, _ptr(dP), _ptr(dT), float(lr), float(momentum), int(bool(nesterov)), _ptr(dg),
                           _ptr(dt))
    return dP.copy(), dg, dt


def rmsprop_fwd(p, g, v, b, lr, alpha=0.99, eps=1e-8, eps_root=0.0, momentum=0.0):
    """RMSProp; b may be None.  Returns (p', v', b') (b' is zeros when momentum == 0)."""
    p = _f64(p)
    n = p.size
    g, v, b = _f64(g, n), _f64(v, n), _opt(b, n)
    po, vo, bo = np.empty(n), np.empty(n), np.zeros(n)
    _load().oracle_rmsprop_fwd(n, _ptr(p), _ptr(g), _ptr(v), _ptr(b), float(lr), float(alpha), float(eps),
                               float(eps_root), float(momentum), _ptr(po), _ptr(vo), _ptr(bo))
    return po, vo, bo


def rmsprop_bwd(dP, dV, dB, g, v, lr, alpha=0.99, eps=1e-8, eps_root=0.0, momentum=0.0):
    """VJP of rmsprop_fwd; dV, dB may be None.  Returns (dp, dg, dv, db)."""
    dP = _f64(dP)
    n = dP.size
    dV, dB = _opt(dV, n), _opt(dB, n)
    g, v = _f64(g, n), _f64(v, n)
    dg, dv, db = np.empty(n), np.empty(n), np.zeros(n)
    _load().oracle_rmsprop_bwd(n, _ptr(dP), _ptr(dV), _ptr(dB), _ptr(g), _ptr(v), float(lr), float(alpha),
                               float(eps), float(eps_root), float(momentum), _ptr(dg), _ptr(dv), _ptr(db))
    return dP.copy(), dg, dv, db


def rmsprop_fwd_mag(p, g, v, b, lr, alpha=0.99, eps=1e-8, eps_root=0.0, momentum=0.0):
    """Tolerance scales (mag_p, mag_v, mag_b) of rmsprop_fwd."""
    p = _f64(p)
    n = p.size
    g, v, b = _f64(g, n), _f64(v, n), _opt(b, n)
    out = [np.empty(n) for _ in range(3)]
    _load().oracle_rmsprop_fwd_mag(n, _ptr(p), _ptr(g), _ptr(v), _ptr(b), float(lr), float(alpha), float(eps),
                                   float(eps_root), float(momentum), *map(_ptr, out))
    return tuple(out)


def rmsprop_bwd_mag(dP, dV, dB, g, v, lr, alpha=0.99, eps=1e-8, eps_root=0.0, momentum=0.0):
    """Tolerance scales (mag_dg, mag_dv, mag_db) of rmsprop_bwd."""
    dP = _f64(dP)
    n = dP.size
    dV, dB = _opt(dV, n), _opt(dB, n)
    g, v = _f64(g, n), _f64(v, n)
    out = [np.empty(n) for _ in range(3)]
    _load().oracle_rmsprop_bwd_mag(n, _ptr(dP), _ptr(dV), _ptr(dB), _ptr(g), _ptr(v), float(lr), float(alpha),
                                   float(eps), float(eps_root), float(momentum), *map(_ptr, out))
    return tuple(out)


def sgd_fwd_mag(p, g, t, lr, momentum=0.0, nesterov=False):
    """Tolerance scales (mag_p, mag_t) of sgd_fwd: sums of |terms|."""
    p, g = _f64(p), _f64(g)
    at = np.zeros_like(p) if t is None else np.abs(_f64(t, p.size))
    mag_t = momentum * at + np.abs(g)
    mag_u = abs(lr) * (np.abs(g) + momentum * mag_t) if nesterov else abs(lr) * mag_t
    return np.abs(p) + mag_u, mag_t


def sgd_bwd_mag(dP, dT, lr, momentum=0.0, nesterov=False):
    """Tolerance scales (mag_dg, mag_dt) of sgd_bwd: sums of |terms|."""
    dP = np.abs(_f64(dP))
    adT = np.zeros_like(dP) if dT is None else np.abs(_f64(dT, dP.size))
    mag_T = adT + abs(lr * momentum if nesterov else lr) * dP
    mag_dg = mag_T + (abs(lr) * dP if nesterov else 0.0)
    return mag_dg, momentum * mag_T


def es_perturb(theta, noise, sigma, antithetic=False):
    """Rows theta + sigma z_i (then theta - sigma z_i if antithetic), fp64 [N or 2N, n]."""
    theta = _f64(theta)
    n = theta.size
    Z = np.ascontiguousarray(np.asarray(noise, dtype=np.float64).reshape(-1, n))
    N = Z.shape[0]
    out = np.empty(((2 if antithetic else 1) * N, n))
    _load().oracle_es_perturb(N, n, _ptr(theta), _ptr(Z), float(sigma), int(bool(antithetic)), _ptr(out))
    return out


def es_estimate(noise, weights, scale):
    """grad = scale * sum_i w_i z_i (sample order), fp64 [n]."""
    w = _f64(weights)
    N = w.size
    Z = np.ascontiguousarray(np.asarray(noise, dtype=np.float64).reshape(N, -1))
    n = Z.shape[1]
    g = np.empty(n)
    _load().oracle_es_estimate(N, n, _ptr(Z), _ptr(w), float(scale), _ptr(g))
    return g


def es_estimate_mag(noise, weights, scale):
    """Tolerance scale of es_estimate: |scale| * sum_i |w_i z_ij|."""
    w = np.abs(_f64(weights))
    Z = np.abs(np.asarray(noise, dtype=np.float64).reshape(w.size, -1))
    return abs(scale) * (w @ Z)


def philox4x64_10(counter, key):
    """One Philox-4x64-10 block: counter (4 uint64 words), key (2 words) -> 4 words."""
    c = np.ascontiguousarray(np.asarray(counter, dtype=np.uint64).reshape(4))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint64).reshape(2))
    out = np.empty(4, dtype=np.uint64)
    u64p = ctypes.POINTER(ctypes.c_uint64)
    _load().oracle_philox4x64_10(c.ctypes.data_as(u64p), k.ctypes.data_as(u64p), out.ctypes.data_as(u64p))
    return out


def box_muller(word):
    """The two normals the transform makes of one 64-bit word."""
    za, zb = ctypes.c_double(), ctypes.c_double()
    _load().oracle_box_muller(ctypes.c_uint64(int(word)), ctypes.byref(za), ctypes.byref(zb))
    return za.value, zb.value


ES_METHODS = {"plain": 0, "baseline": 1, "antithetic": 2}


def es_gaussian_noise(N, n, seed):
    """The seeded N x n noise matrix of the zero-order estimator, fp64."""
    z = np.empty((int(N), int(n)))
    _load().oracle_es_gaussian_noise(int(N), int(n), ctypes.c_uint64(int(seed)), _ptr(z))
    return z


def es_gaussian_noise_radius(N, n, seed):
    """Tolerance scale of each noise element: the Box-Muller radius of its pair."""
    r = np.empty((int(N), int(n)))
    _load().oracle_es_gaussian_noise_radius(int(N), int(n), ctypes.c_uint64(int(seed)), _ptr(r))
    return r


def es_gaussian_noise_cols(N, cols, seed):
    """(z, r) of the noise at the given parameter indices only: [N, len(cols)] each."""
    cols = np.ascontiguousarray(np.asarray(cols, dtype=np.int64).reshape(-1))
    z = np.empty((int(N), cols.size))
    r = np.empty((int(N), cols.size))
    _load().oracle_es_gaussian_noise_cols(int(N), cols.size, cols.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                          ctypes.c_uint64(int(seed)), _ptr(z), _ptr(r))
    return z, r


def es_weights(fvals, method, sigma, f0=0.0):
    """(w, scale) of the estimate from the evaluations: plain, baseline (f0 =
    f(theta)) or antithetic (fvals holds the N plus-points, then the N minus-points)."""
    m = ES_METHODS[method]
    f = _f64(fvals)
    N = f.size // 2 if m == 2 else f.size
    if m == 2 and f.size != 2 * N:
        raise ValueError("antithetic needs 2N evaluations")
    w = np.empty(N)
    scale = ctypes.c_double()
    _load().oracle_es_weights(N, _ptr(f), float(f0), m, float(sigma), _ptr(w), ctypes.byref(scale))
    return w, scale.value


def es_weight_terms(fvals, method, f0=0.0):
    """|terms| of each weight (tolerance scales): |f_i|, |f_i| + |f0| or |f_i| + |f_{N+i}|."""
    f = np.abs(_f64(fvals))
    m = ES_METHODS[method]
    if m == 0:
        return f
    if m == 1:
        return f + abs(float(f0))
    N = f.size // 2
    return f[:N] + f[N:]
