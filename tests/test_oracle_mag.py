"""The oracle's tolerance scales pinned from above.

Every floating-point parity bar in the GPU tests is |gpu - oracle| <= rtol *
mag, where mag is the oracle's sum of the absolute values of the additive
terms that make up a result.  The triangle inequality pins mag from below
(mag >= |value|, tests/test_oracle_adam.py and test_oracle_optim.py).  This
file pins it from above: on inputs where every additive term of a result has
the same sign, the sum of absolute values IS the absolute value of the sum,
so mag must equal |value| up to rounding.  A term counted twice, an extra
term, or a term of the wrong size breaks that equality.

The second half shows that the pins have teeth: it plants such mistakes in
copies of the oracle built on the CPU (each term of each scale doubled in
turn, in the C source or in the Python helpers) and requires every copy to
fail at least one pin.
"""
import concurrent.futures
import ctypes
import inspect
import os
import subprocess
import textwrap

import numpy as np
import pytest

import oracle

REL = 1e-12  # fp64 rounding of a handful of operations, with margin


def _same(val, mag):
    """mag == |val| elementwise, to REL of mag (both may be zero)."""
    val, mag = np.asarray(val, np.float64), np.asarray(mag, np.float64)
    return bool(np.all(np.abs(mag - np.abs(val)) <= REL * mag))


def _mags(n, seed, **scales):
    rng = np.random.default_rng(seed)
    return {k: np.abs(rng.normal(0.0, s, n)) + 0.1 * s for k, s in scales.items()}


N = 500
ADAM_HYPER = [  # count, lr, b1, b2, eps, eps_root: every term of every scale is significant in one of them
    (0, 1e-3, 0.9, 0.999, 1e-8, 0.0),
    (7, 1e-3, 0.9, 0.999, 1e-3, 1e-4),
    (100, -2e-3, 0.8, 0.99, 1e-4, 1e-6),
]
RMS_HYPER = [  # lr, alpha, eps, eps_root, momentum
    (1e-2, 0.99, 1e-8, 0.0, 0.0),
    (1e-3, 0.9, 1e-3, 1e-4, 0.9),
    (-5e-3, 0.5, 1e-4, 1e-6, 0.5),
]
SGD_HYPER = [(0.1, 0.0, False), (0.05, 0.9, False), (0.05, 0.9, True), (-0.02, 0.5, True)]


def adam_pins():
    """(name, holds) for every Adam output on its same-sign inputs."""
    out = []
    for h, (count, lr, b1, b2, eps, er) in enumerate(ADAM_HYPER):
        sg = np.sign(lr)
        x = _mags(N, 10 + h, p=0.05, g=0.01, m=0.01, v=1e-4, dP=1.0, dM=1.0, dV=1.0)
        hy = (count, lr, b1, b2, eps, er)
        # forward: m, g > 0 makes m' > 0 and the update -lr m^/d of sign -sg;
        # p of the update's sign makes p' = p + u a same-sign sum
        for flip in (1.0, -1.0):
            p, g, m, v = -sg * flip * x["p"], flip * x["g"], flip * x["m"], x["v"]
            vals = oracle.adam_fwd(p, g, m, v, *hy)
            mags = oracle.adam_fwd_mag(p, g, m, v, *hy)
            for name, a, b in zip(("p'", "m'", "v'", "u"), vals, mags):
                out.append(("adam fwd %s h%d flip%+d" % (name, h, flip), _same(a, b)))
        # backward, dg and dm: with g m < 0 every term of the reduced form's
        # numerator N is negative, so dP lr N / (s d^2) has sign -sg; dM and
        # g dV take that sign too
        g, m, v = x["g"], -x["m"], x["v"]
        dP, dM, dV = x["dP"], -sg * x["dM"], -sg * x["dV"]
        _, dg, dm, dv = oracle.adam_bwd(dP, dM, dV, g, m, v, *hy)
        mg, mm, mv = oracle.adam_bwd_mag(dP, dM, dV, g, m, v, *hy)
        out += [("adam bwd dg h%d" % h, _same(dg, mg)), ("adam bwd dm h%d" % h, _same(dm, mm))]
        # backward, dv: m, g > 0 makes m^ > 0, so dP lr m^ / (2 c2 s d^2) has sign sg; dV too
        m, dV = x["m"], sg * x["dV"]
        _, dg, dm, dv = oracle.adam_bwd(dP, dM, dV, g, m, v, *hy)
        mg, mm, mv = oracle.adam_bwd_mag(dP, dM, dV, g, m, v, *hy)
        out.append(("adam bwd dv h%d" % h, _same(dv, mv)))
        # the 0/0 point (s = 0: eps_root = 0, v = 0, g = 0): dg = (1-b1) dM - dP lr a / d
        if er == 0.0:
            z = np.zeros(N)
            m0 = np.where(np.arange(N) % 2, 1.0, -1.0) * x["m"]
            _, dg, dm, dv = oracle.adam_bwd(dP, dM, dV, z, m0, z, *hy)
            mg, mm, mv = oracle.adam_bwd_mag(dP, dM, dV, z, m0, z, *hy)
            out += [("adam bwd 0/0 dg h%d" % h, _same(dg, mg)), ("adam bwd 0/0 dm h%d" % h, _same(dm, mm)),
                    ("adam bwd 0/0 dv h%d" % h, _same(dv, mv))]
    return out


def rmsprop_pins():
    out = []
    for h, (lr, alpha, eps, er, mu) in enumerate(RMS_HYPER):
        sg = np.sign(lr)
        x = _mags(N, 20 + h, p=0.05, g=0.01, v=1e-4, b=0.1, dP=1.0, dV=1.0, dB=1.0)
        hy = (lr, alpha, eps, er, mu)
        b = x["b"] if mu > 0 else None
        # forward: g, b > 0 makes b' (or g/d) > 0 and the update of sign -sg
        p, g, v = -sg * x["p"], x["g"], x["v"]
        vals = oracle.rmsprop_fwd(p, g, v, b, *hy)
        mags = oracle.rmsprop_fwd_mag(p, g, v, b, *hy)
        out += [("rms fwd p' h%d" % h, _same(vals[0], mags[0])), ("rms fwd v' h%d" % h, _same(vals[1], mags[1]))]
        if mu > 0:
            out.append(("rms fwd b' h%d" % h, _same(vals[2], mags[2])))
        # backward, dg and db: Bt = dB - lr dP of sign -sg, and g dV of that sign
        dP = x["dP"]
        dB = -sg * x["dB"] if mu > 0 else None
        dV = -sg * x["dV"]
        _, dg, dv, db = oracle.rmsprop_bwd(dP, dV, dB, g, v, *hy)
        mg, mv, mb = oracle.rmsprop_bwd_mag(dP, dV, dB, g, v, *hy)
        out.append(("rms bwd dg h%d" % h, _same(dg, mg)))
        if mu > 0:
            out.append(("rms bwd db h%d" % h, _same(db, mb)))
        # backward, dv: dv = alpha (dV - Bt g / (2 s d^2)), the second term of sign sg
        dV = sg * x["dV"]
        _, dg, dv, db = oracle.rmsprop_bwd(dP, dV, dB, g, v, *hy)
        mg, mv, mb = oracle.rmsprop_bwd_mag(dP, dV, dB, g, v, *hy)
        out.append(("rms bwd dv h%d" % h, _same(dv, mv)))
        if er == 0.0:  # s = 0: dg = Bt / d
            z = np.zeros(N)
            _, dg, dv, db = oracle.rmsprop_bwd(dP, dV, dB, z, z, *hy)
            mg, mv, mb = oracle.rmsprop_bwd_mag(dP, dV, dB, z, z, *hy)
            out += [("rms bwd 0/0 dg h%d" % h, _same(dg, mg)), ("rms bwd 0/0 dv h%d" % h, _same(dv, mv))]
    return out


def sgd_pins():
    out = []
    for h, (lr, mu, nest) in enumerate(SGD_HYPER):
        sg = np.sign(lr)
        x = _mags(N, 30 + h, p=0.05, g=0.01, t=0.01, dP=1.0, dT=1.0)
        for t in (None, x["t"]):
            tag = "h%d %s" % (h, "fresh" if t is None else "trace")
            p, g = -sg * x["p"], x["g"]
            po, to = oracle.sgd_fwd(p, g, t, lr, mu, nest)
            mp, mt = oracle.sgd_fwd_mag(p, g, t, lr, mu, nest)
            out += [("sgd fwd p' " + tag, _same(po, mp)), ("sgd fwd t' " + tag, _same(to, mt))]
        # backward: Tt = dT - c dP with c = lr mu (Nesterov) or lr, of sign -sg; dg adds -lr dP
        dP, dT = x["dP"], -sg * x["dT"]
        for dTx in (None, dT):
            _, dg, dt = oracle.sgd_bwd(dP, dTx, lr, mu, nest)
            mg, mt = oracle.sgd_bwd_mag(dP, dTx, lr, mu, nest)
            tag = "h%d %s" % (h, "no dT" if dTx is None else "dT")
            out += [("sgd bwd dg " + tag, _same(dg, mg)), ("sgd bwd dt " + tag, _same(dt, mt))]
    return out


def es_pins():
    rng = np.random.default_rng(40)
    Nn, n = 9, 300
    sgn = np.where(rng.random(Nn) < 0.5, -1.0, 1.0)
    w = sgn * (np.abs(rng.normal(0, 1, Nn)) + 0.1)
    Z = sgn[:, None] * (np.abs(rng.normal(0, 1, (Nn, n))) + 0.1)  # every w_i z_ij > 0
    out = []
    for scale in (0.3, -2.0):
        out.append(("es estimate scale %g" % scale,
                    _same(oracle.es_estimate(Z, w, scale), oracle.es_estimate_mag(Z, w, scale))))
    # weights formed from evaluations: f_i of the sign of z_i, and the
    # subtracted f0 or f_{N+i} of the other sign
    Zp = np.abs(Z)
    f = np.abs(rng.normal(0, 1, 2 * Nn)) + 0.1
    f[Nn:] *= -1.0
    for method, fv, f0 in (("plain", f[:Nn], 0.0), ("baseline", f[:Nn], -0.7), ("antithetic", f, 0.0)):
        wm, sc = oracle.es_weights(fv, method, 0.05, f0=f0)
        terms = oracle.es_weight_terms(fv, method, f0=f0)
        out.append(("es weights %s" % method, _same(wm, terms)))
        out.append(("es estimate %s" % method,
                    _same(oracle.es_estimate(Zp, wm, sc), oracle.es_estimate_mag(Zp, terms, sc))))
    return out


ALL_PINS = (adam_pins, rmsprop_pins, sgd_pins, es_pins)


@pytest.mark.parametrize("pins", ALL_PINS, ids=lambda f: f.__name__)
def test_mag_equals_abs_value_when_terms_share_a_sign(pins):
    res = pins()
    assert res
    bad = [name for name, ok in res if not ok]
    assert not bad, bad


# ---------------------------------------------------------------- planted mistakes


def _body(src, fname):
    """Start and end offsets of the body of C function `fname` in src."""
    i = src.index("void %s(" % fname)
    j = src.index("{", i)
    depth, k = 0, j
    while True:
        if src[k] == "{":
            depth += 1
        elif src[k] == "}":
            depth -= 1
            if depth == 0:
                return j, k
        k += 1


def _double_terms(stmt, terms):
    """One planted mistake per term: `term` -> `2.0 * term` inside statement `stmt`."""
    out = []
    for t in terms:
        assert stmt.count(t) == 1, (stmt, t)
        out.append((stmt, stmt.replace(t, "2.0 * " + t)))
    return out


C_MUTANTS = {
    "oracle_adam_fwd_mag": (
        _double_terms("double am = b1 * fabs(m[i]) + (1.0 - b1) * fabs(g[i]);",
                      ["b1 * fabs(m[i])", "(1.0 - b1) * fabs(g[i])"])
        + _double_terms("double av = b2 * fabs(v[i]) + (1.0 - b2) * g[i] * g[i];",
                        ["b2 * fabs(v[i])", "(1.0 - b2) * g[i] * g[i]"])
        + _double_terms("double v1 = b2 * v[i] + (1.0 - b2) * g[i] * g[i];", ["b2 * v[i]", "(1.0 - b2) * g"])
        + _double_terms("double s = sqrt(v1 / c2 + eps_root);", ["eps_root"])
        + _double_terms("double d = s + eps;", ["eps"])
        + _double_terms("double au = fabs(lr) * am / (c1 * d);", ["fabs(lr)"])
        + _double_terms("mag_p[i] = fabs(p[i]) + au;", ["fabs(p[i])", "au;"])),
    "oracle_adam_bwd_mag": (
        _double_terms("double v1 = b2 * v[i] + (1.0 - b2) * g[i] * g[i];", ["b2 * v[i]", "(1.0 - b2) * g"])
        + _double_terms("double s = sqrt(v1 / c2 + eps_root);", ["eps_root"])
        + _double_terms("double d = s + eps;", ["eps"])
        + _double_terms("double amh = (b1 * fabs(m[i]) + (1.0 - b1) * fabs(g[i])) / c1;",
                        ["b1 * fabs(m[i])", "(1.0 - b1) * fabs(g[i])"])
        + _double_terms("double num = b * b1 * fabs(g[i] * m[i]) / c1 + a * b2 * fabs(v[i]) / c2 +\n"
                        "                   a * (eps_root + s * eps);",
                        ["b * b1", "a * b2", "a * (eps_root", "eps_root + s", "s * eps)"])
        + _double_terms("t3 = adP * fabs(lr) * num / (s * d * d);", ["adP"])
        + _double_terms("tv = adP * fabs(lr) * amh / (2.0 * c2 * s * d * d);", ["adP"])
        + _double_terms("t3 = adP * fabs(lr) * a / d;", ["adP"])
        + _double_terms("mag_dg[i] = (1.0 - b1) * adM + 2.0 * (1.0 - b2) * fabs(g[i]) * adV + t3;",
                        ["(1.0 - b1) * adM", "(1.0 - b2) * fabs", "t3;"])
        + _double_terms("mag_dm[i] = b1 * (adM + adP * fabs(lr) / (c1 * d));", ["adM", "adP"])
        + _double_terms("mag_dv[i] = b2 * (adV + tv);", ["adV", "tv)"])),
    "oracle_rmsprop_fwd_mag": (
        _double_terms("double v1 = alpha * fabs(v[i]) + (1.0 - alpha) * g[i] * g[i];",
                      ["alpha * fabs", "(1.0 - alpha)"])
        + _double_terms("double s = sqrt(alpha * v[i] + (1.0 - alpha) * g[i] * g[i] + eps_root);",
                        ["alpha * v[i]", "(1.0 - alpha)", "eps_root"])
        + _double_terms("double d = s + eps;", ["eps"])
        + _double_terms("double aq = fabs(g[i]) / d;", ["fabs(g[i])"])
        + _double_terms("double ab = mu > 0.0 ? mu * fabs(b ? b[i] : 0.0) + aq : aq;",
                        ["mu * fabs", "aq :", "aq;"])
        + _double_terms("mag_p[i] = fabs(p[i]) + fabs(lr) * ab;", ["fabs(p[i])", "fabs(lr)"])),
    "oracle_rmsprop_bwd_mag": (
        _double_terms("double s = sqrt(alpha * v[i] + (1.0 - alpha) * g[i] * g[i] + eps_root);",
                      ["alpha * v[i]", "(1.0 - alpha)", "eps_root"])
        + _double_terms("double d = s + eps;", ["eps"])
        + _double_terms("double aBt = (mu > 0.0 ? fabs(dB ? dB[i] : 0.0) : 0.0) + fabs(lr) * fabs(dP[i]);",
                        ["fabs(dB ?", "fabs(lr)"])
        + _double_terms("double t3 = s > 0.0 ? aBt * (alpha * fabs(v[i]) + eps_root + s * eps) / (s * d * d) "
                        ": aBt / d;", ["alpha * fabs", "eps_root +", "s * eps", "aBt / d"])
        + _double_terms("double tv = s > 0.0 ? aBt * fabs(g[i]) / (2.0 * s * d * d) : 0.0;", ["aBt"])
        + _double_terms("mag_dg[i] = 2.0 * (1.0 - alpha) * fabs(g[i]) * adV + t3;", ["(1.0 - alpha)", "t3"])
        + _double_terms("mag_dv[i] = alpha * (adV + tv);", ["adV", "tv)"])
        + _double_terms("if (mag_db) mag_db[i] = mu * aBt;", ["mu * aBt"])),
}

PY_MUTANTS = {
    "sgd_fwd_mag": (
        _double_terms("mag_t = momentum * at + np.abs(g)", ["momentum * at", "np.abs(g)"])
        + _double_terms("mag_u = abs(lr) * (np.abs(g) + momentum * mag_t) if nesterov else abs(lr) * mag_t",
                        ["np.abs(g) +", "momentum * mag_t", "abs(lr) * mag_t"])
        + _double_terms("return np.abs(p) + mag_u, mag_t", ["np.abs(p)", "mag_u,"])),
    "sgd_bwd_mag": (
        _double_terms("mag_T = adT + abs(lr * momentum if nesterov else lr) * dP", ["adT", "abs(lr * momentum"])
        + _double_terms("mag_dg = mag_T + (abs(lr) * dP if nesterov else 0.0)", ["abs(lr) * dP"])
        + _double_terms("return mag_dg, momentum * mag_T", ["momentum * mag_T"])),
    "es_estimate_mag": [("return abs(scale) * (w @ Z)", "return abs(scale) * (w @ Z + w[0] * Z[0])")],
    "es_weight_terms": [("return f + abs(float(f0))", "return f + 2.0 * abs(float(f0))"),
                        ("return f[:N] + f[N:]", "return 2.0 * f[:N] + f[N:]"),
                        ("return f[:N] + f[N:]", "return f[:N] + 2.0 * f[N:]")],
}


def _any_pin_fails():
    return any(not ok for pins in ALL_PINS for _, ok in pins())


@pytest.fixture(scope="module")
def oracle_source():
    with open(oracle._SRC) as f:
        return f.read()


@pytest.mark.parametrize("fname", sorted(C_MUTANTS))
def test_pins_catch_a_doubled_term_in_the_c_scales(fname, oracle_source, tmp_path, monkeypatch):
    src = oracle_source
    j, k = _body(src, fname)
    builds = []
    for idx, (old, new) in enumerate(C_MUTANTS[fname]):
        assert src[j:k].count(old) == 1, (fname, old)
        c = tmp_path / ("m%d.c" % idx)
        c.write_text(src[:j] + src[j:k].replace(old, new) + src[k:])
        builds.append((c, tmp_path / ("m%d.so" % idx)))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        list(ex.map(lambda b: subprocess.check_call(["gcc", *oracle.CFLAGS, str(b[0]), "-o", str(b[1]), "-lm"]),
                    builds))
    for (old, new), (_, so) in zip(C_MUTANTS[fname], builds):
        monkeypatch.setattr(oracle, "_lib", oracle._configure(ctypes.CDLL(str(so))))
        assert _any_pin_fails(), "planted mistake not caught: %s: %r -> %r" % (fname, old, new)
    monkeypatch.undo()
    assert not _any_pin_fails()  # the real oracle passes again


@pytest.mark.parametrize("fname", sorted(PY_MUTANTS))
def test_pins_catch_a_doubled_term_in_the_python_scales(fname, monkeypatch):
    src = textwrap.dedent(inspect.getsource(getattr(oracle, fname)))
    for old, new in PY_MUTANTS[fname]:
        assert src.count(old) == 1, (fname, old)
        ns = dict(vars(oracle))
        exec(compile(src.replace(old, new), "<mutant %s>" % fname, "exec"), ns)
        monkeypatch.setattr(oracle, fname, ns[fname])
        assert _any_pin_fails(), "planted mistake not caught: %s: %r -> %r" % (fname, old, new)
        monkeypatch.undo()
    assert not _any_pin_fails()


def test_mutants_cover_every_scale_statement(oracle_source):
    # every statement of a C scale that adds terms is mutated at least once
    for fname, muts in C_MUTANTS.items():
        j, k = _body(oracle_source, fname)
        stmts = {old for old, _ in muts}
        body = oracle_source[j:k]
        for line in body.split(";"):
            line = line.strip()
            if " + " in line and not line.startswith("for"):
                assert any(line in s or s.rstrip(";") in line for s in stmts), (fname, line)
    assert os.path.exists(oracle._SRC)
