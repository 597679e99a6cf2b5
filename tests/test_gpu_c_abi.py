"""The C ABI used from plain C, without PyTorch: tests/c_abi/caller (built by
__graft_entry__.build()) allocates leaves with hipMalloc, packs the params
tree and K gradient trees in one batched call, runs the K-step driver forward
and VJP with only the final moment state stored, and unpacks p_K and the
gradient cotangents.  Its outputs are checked against the oracle: p_K per
element within 1e-5 of its term scale, the final moments within 1e-5 and the
meta-gradients within 1e-4, norm-relative (end to end from the fp32 inputs).
The tree has empty and odd-sized leaves and spans several copy tiles."""
import os
import struct
import subprocess

import numpy as np
import pytest

import oracle
from tests.support import BWD_RTOL, FWD_RTOL, assert_mag_close, stats
from workloads import HYPER, normal

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
CALLER = os.path.join(HERE, "c_abi", "caller")


@pytest.mark.parametrize("K,count0,eps_root", [(3, 0, 0.0), (8, 4, 1e-8)])
def test_plain_c_caller_matches_oracle(tmp_path, K, count0, eps_root):
    assert os.path.exists(CALLER), "tests/c_abi/caller is not built: run __graft_entry__.build()"
    numel = [5, 0, 4096 * 3 + 7, 1, 0, 999, 65536, 13]
    n = sum(numel)
    p = normal(n, 0.05, "cabi", "p0", K)
    grads = [normal(n, 1e-2, "cabi", "grad", 10 * K + k) for k in range(K)]
    cot = normal(n, 1.0, "cabi", "cot_p", K)
    lr, b1, b2, eps = HYPER["lr"], HYPER["b1"], HYPER["b2"], HYPER["eps"]
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(src, "wb") as f:
        f.write(struct.pack("<3q5d", len(numel), K, count0, lr, b1, b2, eps, eps_root))
        f.write(np.asarray(numel, "<i8").tobytes())
        for arr in [p, *grads, cot]:  # trees as their leaves back to back, i.e. the dense flat order
            f.write(np.asarray(arr, "<f4").tobytes())
    r = subprocess.run([CALLER, str(src), str(dst)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    out = np.fromfile(dst, dtype="<f4").astype(np.float64)
    assert out.size == n * (3 + K + 2)
    pK, muK, nuK = out[:n], out[n:2 * n], out[2 * n:3 * n]
    dg = [out[(3 + k) * n:(4 + k) * n] for k in range(K)]
    dm0, dv0 = out[(3 + K) * n:(4 + K) * n], out[(4 + K) * n:]

    G = np.stack([g.astype(np.float64) for g in grads])
    z = np.zeros(n)
    h = (lr, b1, b2, eps, eps_root)
    pK_r, mt_r, vt_r = oracle.unrolled_fwd(p.astype(np.float64), G, z, z, count0, *h)
    mag_p = np.abs(p.astype(np.float64))
    for k in range(1, K + 1):
        mag_p = mag_p + oracle.adam_fwd_mag(p, G[k - 1], mt_r[k - 1], vt_r[k - 1], count0 + k - 1, *h)[3]
    assert_mag_close(pK, pK_r, mag_p, FWD_RTOL, "p_K")
    assert stats(muK, mt_r[K])[1] < FWD_RTOL
    assert stats(nuK, vt_r[K])[1] < FWD_RTOL
    _, dg_r, dm0_r, dv0_r = oracle.unrolled_bwd(cot.astype(np.float64), G, mt_r, vt_r, count0, *h)
    for k in range(K):
        assert stats(dg[k], dg_r[k])[1] < BWD_RTOL, k
    assert stats(dm0, dm0_r)[1] < BWD_RTOL
    assert stats(dv0, dv0_r)[1] < BWD_RTOL
