"""Python binding of the diffopt C ABI (include/diffopt.h).

Argument marshalling only: every function here is the C entry point
``diffopt_<name>`` with the same arguments, taking torch tensors (device
memory) or raw device addresses, and enqueuing on the current torch stream
unless a stream is given.  All arithmetic and data movement happens in the
HIP library; importing this module fails loudly if the library is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdiffopt.so")

DIFFOPT_OK = 0
DIFFOPT_EINVAL = -1
DIFFOPT_ENOMEM = -2
DIFFOPT_EHIP = -3
REMAT_SPAN = 8  # DIFFOPT_REMAT_SPAN: longest run of steps the K-step backward recomputes


class DiffoptError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__("diffopt error %d: %s" % (code, message))
        self.code = code


def _load_library():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            "libdiffopt.so is not built (%s); run `python paper_2211_06934_amd/build.py`" % _LIB_PATH)
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i64, i32, f64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    pp = ctypes.POINTER(ctypes.c_void_p)
    p64 = ctypes.POINTER(ctypes.c_int64)
    hyper = [i64, f64, f64, f64, f64, f64]  # count, lr, b1, b2, eps, eps_root
    sig = {
        "diffopt_last_error": (ctypes.c_char_p, []),
        "diffopt_segtable_create": (ctypes.c_int, [i64, p64, p64, i32, ctypes.POINTER(vp)]),
        "diffopt_segtable_destroy": (None, [vp]),
        "diffopt_segtable_total": (i64, [vp]),
        "diffopt_segtable_nseg": (i64, [vp]),
        "diffopt_tree_flatten": (ctypes.c_int, [vp, vp, vp, vp]),
        "diffopt_tree_unflatten": (ctypes.c_int, [vp, vp, vp, vp]),
        "diffopt_tree_flatten_batch": (ctypes.c_int, [vp, i64, pp, pp, vp]),
        "diffopt_tree_unflatten_batch": (ctypes.c_int, [vp, i64, pp, pp, vp]),
        "diffopt_adam_fwd": (ctypes.c_int, [vp, vp, vp, vp, i64, *hyper, vp, vp, vp, vp, vp]),
        "diffopt_adam_bwd": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, i64, *hyper, vp, vp, vp, vp, vp]),
        "diffopt_adam_unrolled_fwd": (ctypes.c_int, [i64, i64, vp, pp, pp, pp, vp, *hyper, vp]),
        "diffopt_adam_unrolled_bwd": (ctypes.c_int, [i64, i64, vp, pp, pp, pp, pp, vp, vp, *hyper, vp]),
        "diffopt_adam_fwd_tree": (ctypes.c_int, [vp, vp, vp, vp, vp, *hyper, vp, vp, vp, vp]),
        "diffopt_adam_bwd_tree": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, vp, *hyper, vp, vp, vp, vp]),
        "diffopt_adam_unrolled_fwd_tree": (ctypes.c_int, [vp, i64, vp, pp, pp, pp, vp, *hyper, vp]),
        "diffopt_adam_unrolled_bwd_tree": (ctypes.c_int, [vp, i64, vp, pp, pp, pp, pp, vp, vp, *hyper, vp]),
        "diffopt_sgd_fwd": (ctypes.c_int, [vp, vp, vp, i64, f64, f64, i32, vp, vp, vp]),
        "diffopt_sgd_bwd": (ctypes.c_int, [vp, vp, i64, f64, f64, i32, vp, vp, vp]),
        "diffopt_rmsprop_fwd": (ctypes.c_int, [vp, vp, vp, vp, i64, f64, f64, f64, f64, f64, vp, vp, vp, vp]),
        "diffopt_rmsprop_bwd": (ctypes.c_int, [vp, vp, vp, vp, vp, i64, f64, f64, f64, f64, f64, vp, vp, vp, vp]),
        "diffopt_sgd_fwd_tree": (ctypes.c_int, [vp, vp, vp, vp, f64, f64, i32, vp, vp, vp]),
        "diffopt_sgd_bwd_tree": (ctypes.c_int, [vp, vp, vp, f64, f64, i32, vp, vp, vp]),
        "diffopt_rmsprop_fwd_tree": (ctypes.c_int, [vp, vp, vp, vp, vp, f64, f64, f64, f64, f64, vp, vp, vp, vp]),
        "diffopt_rmsprop_bwd_tree": (ctypes.c_int, [vp, vp, vp, vp, vp, vp, f64, f64, f64, f64, f64, vp, vp, vp,
                                                    vp]),
        "diffopt_es_perturb": (ctypes.c_int, [vp, vp, i64, i64, f64, i32, vp, vp]),
        "diffopt_es_estimate": (ctypes.c_int, [vp, vp, i64, i64, f64, vp, vp]),
        "diffopt_es_perturb_gaussian": (ctypes.c_int, [vp, i64, i64, ctypes.c_uint64, f64, i32, vp, vp]),
        "diffopt_es_estimate_gaussian": (ctypes.c_int, [vp, vp, i64, i32, i64, ctypes.c_uint64, f64, vp, vp]),
        "diffopt_es_weights": (ctypes.c_int, [vp, vp, i64, i32, f64, vp, vp]),
    }
    for name, (res, args) in sig.items():
        if not hasattr(lib, name):
            raise ImportError("%s lacks %s: it is older than its sources; rebuild with "
                              "`python paper_2211_06934_amd/build.py`" % (_LIB_PATH, name))
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load_library()
LIBRARY_PATH = _LIB_PATH


def last_error() -> str:
    """diffopt_last_error(): message of the last failing call on this thread."""
    return _lib.diffopt_last_error().decode()


def _check(rc: int) -> None:
    if rc != DIFFOPT_OK:
        raise DiffoptError(rc, last_error())


def _addr(x, what: str, dtype=torch.float32, n: Optional[int] = None) -> Optional[int]:
    """Device address of a tensor (checked) or a raw integer address."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not isinstance(x, torch.Tensor):
        raise TypeError("%s: expected a torch.Tensor or an int address" % what)
    if not x.is_cuda:
        raise ValueError("%s: tensor must live in device memory" % what)
    if dtype is not None and x.dtype != dtype:
        raise ValueError("%s: expected dtype %s, got %s" % (what, dtype, x.dtype))
    if not x.is_contiguous():
        raise ValueError("%s: tensor must be contiguous" % what)
    if n is not None and x.numel() != n:
        raise ValueError("%s: expected %d elements, got %d" % (what, n, x.numel()))
    return x.data_ptr()


# torch's current raw stream without building a Stream object (the public
# torch.cuda.current_stream() costs about as much as a kernel launch)
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_cur_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream) -> Optional[int]:
    if stream is None:
        if _raw_stream is not None and _cur_device is not None:
            return _raw_stream(_cur_device())
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr_array(items, what, n):
    arr = (ctypes.c_void_p * len(items))()
    for i, t in enumerate(items):
        arr[i] = _addr(t, "%s[%d]" % (what, i), n=n)
    return arr


class SegTable:
    """Owner of a diffopt_segtable handle (freed on close() or collection).

    Keep it alive while calls that use it may still run, and outside graph
    capture: freeing its device memory is not a capturable operation.  The
    tree module caches one table per structure for the life of the process."""

    def __init__(self, handle: int, numel: Sequence[int], offsets, elem_bytes: int, total: Optional[int] = None):
        self.handle = handle
        self.numel = list(numel)
        self.offsets = None if offsets is None else list(offsets)
        self.elem_bytes = elem_bytes
        self._total = total

    @property
    def total(self) -> int:
        """Flat length in elements (read once from the library at creation)."""
        if self._total is None:
            self._total = segtable_total(self)
        return self._total

    @property
    def nseg(self) -> int:
        return segtable_nseg(self)

    def close(self) -> None:
        if self.handle:
            _lib.diffopt_segtable_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def segtable_create(numel: Sequence[int], offsets: Optional[Sequence[int]] = None,
                    elem_bytes: int = 4) -> SegTable:
    """diffopt_segtable_create on the current device."""
    k = len(numel)
    n_arr = (ctypes.c_int64 * max(k, 1))(*[int(x) for x in numel])
    o_arr = None
    if offsets is not None:
        if len(offsets) != k:
            raise ValueError("offsets must have one entry per leaf")
        o_arr = (ctypes.c_int64 * max(k, 1))(*[int(x) for x in offsets])
    h = ctypes.c_void_p()
    _check(_lib.diffopt_segtable_create(k, n_arr, o_arr, int(elem_bytes), ctypes.byref(h)))
    return SegTable(h.value, numel, offsets, elem_bytes, int(_lib.diffopt_segtable_total(h.value)))


def segtable_destroy(table: SegTable) -> None:
    table.close()


def segtable_total(table: SegTable) -> int:
    return int(_lib.diffopt_segtable_total(table.handle))


def segtable_nseg(table: SegTable) -> int:
    return int(_lib.diffopt_segtable_nseg(table.handle))


def _tree_sizes(table: SegTable, leaf_ptrs, flat, what: str = "") -> None:
    """Size checks of one tree's (leaf_ptrs, flat) for the copy kernels.

    A tensor leaf_ptrs must hold one int64 address per leaf of the table, and
    a tensor flat must have the table's element width and at least
    table.total elements: the kernels read that many addresses and write or
    read that many flat elements.  Raw integer addresses are passed through
    unchecked."""
    if isinstance(leaf_ptrs, torch.Tensor):
        if leaf_ptrs.dtype != torch.int64 or leaf_ptrs.numel() != len(table.numel):
            raise ValueError("%sleaf_ptrs: expected %d int64 leaf addresses, got %d of %s"
                             % (what, len(table.numel), leaf_ptrs.numel(), leaf_ptrs.dtype))
    if isinstance(flat, torch.Tensor):
        if flat.element_size() != table.elem_bytes:
            raise ValueError("%sflat: the table copies %d-byte elements, flat has %d-byte %s"
                             % (what, table.elem_bytes, flat.element_size(), flat.dtype))
        if flat.numel() < table.total:
            raise ValueError("%sflat: the table needs %d elements, flat has %d" % (what, table.total, flat.numel()))


def _tree_operands(table: SegTable, leaf_ptrs, flat, what: str = ""):
    """Checked addresses of one tree's (leaf_ptrs, flat)."""
    _tree_sizes(table, leaf_ptrs, flat, what)
    return _addr(leaf_ptrs, what + "leaf_ptrs", torch.int64), _addr(flat, what + "flat", None)


def tree_flatten(table: SegTable, leaf_ptrs, flat, stream=None) -> None:
    """diffopt_tree_flatten: leaf_ptrs is a device int64 tensor of leaf addresses."""
    lp, fl = _tree_operands(table, leaf_ptrs, flat)
    _check(_lib.diffopt_tree_flatten(table.handle, lp, fl, _stream(stream)))


def tree_unflatten(table: SegTable, flat, leaf_ptrs, stream=None) -> None:
    """diffopt_tree_unflatten."""
    lp, fl = _tree_operands(table, leaf_ptrs, flat)
    _check(_lib.diffopt_tree_unflatten(table.handle, fl, lp, _stream(stream)))


def _batch_operands(table: SegTable, leaf_ptrs: Sequence, flats: Sequence):
    if len(leaf_ptrs) != len(flats):
        raise ValueError("leaf_ptrs and flats need one entry per tree")
    for t, (lp, fl) in enumerate(zip(leaf_ptrs, flats)):  # every size before any device check
        _tree_sizes(table, lp, fl, "tree %d: " % t)
    ops = [_tree_operands(table, lp, fl, "tree %d: " % t) for t, (lp, fl) in enumerate(zip(leaf_ptrs, flats))]
    lp_arr = (ctypes.c_void_p * max(len(ops), 1))(*[o[0] for o in ops])
    fl_arr = (ctypes.c_void_p * max(len(ops), 1))(*[o[1] for o in ops])
    return len(ops), lp_arr, fl_arr


def tree_flatten_batch(table: SegTable, leaf_ptrs: Sequence, flats: Sequence, stream=None) -> None:
    """diffopt_tree_flatten_batch: tree t is (leaf_ptrs[t], flats[t])."""
    k, lp, fl = _batch_operands(table, leaf_ptrs, flats)
    _check(_lib.diffopt_tree_flatten_batch(table.handle, k, lp, fl, _stream(stream)))


def tree_unflatten_batch(table: SegTable, flats: Sequence, leaf_ptrs: Sequence, stream=None) -> None:
    """diffopt_tree_unflatten_batch."""
    k, lp, fl = _batch_operands(table, leaf_ptrs, flats)
    _check(_lib.diffopt_tree_unflatten_batch(table.handle, k, fl, lp, _stream(stream)))


def adam_fwd(params, grad, mu, nu, count, lr, b1, b2, eps, eps_root,
             params_out, mu_out, nu_out, update_out=None, stream=None, n: Optional[int] = None) -> None:
    """diffopt_adam_fwd; n defaults to params.numel()."""
    if n is None:
        n = params.numel()
    _check(_lib.diffopt_adam_fwd(
        _addr(params, "params", n=n), _addr(grad, "grad", n=n), _addr(mu, "mu", n=n), _addr(nu, "nu", n=n),
        int(n), int(count), float(lr), float(b1), float(b2), float(eps), float(eps_root),
        _addr(params_out, "params_out", n=n), _addr(mu_out, "mu_out", n=n), _addr(nu_out, "nu_out", n=n),
        _addr(update_out, "update_out", n=n), _stream(stream)))


def adam_bwd(dupdate, dmu, dnu, grad, mu, nu, count, lr, b1, b2, eps, eps_root,
             dparams, dgrad, dmu_in, dnu_in, stream=None, n: Optional[int] = None) -> None:
    """diffopt_adam_bwd; dmu/dnu/dparams may be None."""
    if n is None:
        n = dupdate.numel()
    _check(_lib.diffopt_adam_bwd(
        _addr(dupdate, "dupdate", n=n), _addr(dmu, "dmu", n=n), _addr(dnu, "dnu", n=n),
        _addr(grad, "grad", n=n), _addr(mu, "mu", n=n), _addr(nu, "nu", n=n),
        int(n), int(count), float(lr), float(b1), float(b2), float(eps), float(eps_root),
        _addr(dparams, "dparams", n=n), _addr(dgrad, "dgrad", n=n), _addr(dmu_in, "dmu_in", n=n),
        _addr(dnu_in, "dnu_in", n=n), _stream(stream)))


def adam_unrolled_fwd(p0, grads, mu_traj, nu_traj, pK, count0, lr, b1, b2, eps, eps_root,
                      stream=None) -> None:
    """diffopt_adam_unrolled_fwd; grads has K entries, mu_traj/nu_traj K+1.

    Intermediate trajectory entries (0 < k < K) may be None: that state is not
    stored, and adam_unrolled_bwd recomputes it (at most REMAT_SPAN - 1
    consecutive None entries for the backward)."""
    K = len(grads)
    n = p0.numel()
    if len(mu_traj) != K + 1 or len(nu_traj) != K + 1:
        raise ValueError("mu_traj and nu_traj need K+1 entries")
    _check(_lib.diffopt_adam_unrolled_fwd(
        K, n, _addr(p0, "p0", n=n), _ptr_array(grads, "grads", n), _ptr_array(mu_traj, "mu_traj", n),
        _ptr_array(nu_traj, "nu_traj", n), _addr(pK, "pK", n=n), int(count0), float(lr), float(b1),
        float(b2), float(eps), float(eps_root), _stream(stream)))


def adam_unrolled_bwd(dpK, grads, mu_traj, nu_traj, dgrads, dmu0, dnu0, count0, lr, b1, b2, eps,
                      eps_root, stream=None) -> None:
    """diffopt_adam_unrolled_bwd; mu_traj/nu_traj may hold K or K+1 entries,
    None where the forward did not store the state."""
    K = len(grads)
    n = dpK.numel()
    if len(dgrads) != K or len(mu_traj) < K or len(nu_traj) < K:
        raise ValueError("dgrads needs K entries, mu_traj/nu_traj at least K")
    _check(_lib.diffopt_adam_unrolled_bwd(
        K, n, _addr(dpK, "dpK", n=n), _ptr_array(grads, "grads", n), _ptr_array(mu_traj[:K], "mu_traj", n),
        _ptr_array(nu_traj[:K], "nu_traj", n), _ptr_array(dgrads, "dgrads", n), _addr(dmu0, "dmu0", n=n),
        _addr(dnu0, "dnu0", n=n), int(count0), float(lr), float(b1), float(b2), float(eps), float(eps_root),
        _stream(stream)))


# ---- leaf-direct ("tree map") form: every operand is a device int64 tensor of
# leaf addresses in table order (see tree.leaf_pointer_tensors)


def _leaf_array(x, what, nseg):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return _addr(x, what, torch.int64, n=nseg)


def _leaf_array_list(items, what, nseg):
    arr = (ctypes.c_void_p * len(items))()
    for i, t in enumerate(items):
        arr[i] = _leaf_array(t, "%s[%d]" % (what, i), nseg)
    return arr


def adam_fwd_tree(table: SegTable, params, grad, mu, nu, count, lr, b1, b2, eps, eps_root,
                  params_out, mu_out, nu_out, stream=None) -> None:
    """diffopt_adam_fwd_tree."""
    k = len(table.numel)
    _check(_lib.diffopt_adam_fwd_tree(
        table.handle, *[_leaf_array(x, w, k) for x, w in ((params, "params"), (grad, "grad"), (mu, "mu"),
                                                           (nu, "nu"))],
        int(count), float(lr), float(b1), float(b2), float(eps), float(eps_root),
        *[_leaf_array(x, w, k) for x, w in ((params_out, "params_out"), (mu_out, "mu_out"), (nu_out, "nu_out"))],
        _stream(stream)))


def adam_bwd_tree(table: SegTable, dupdate, dmu, dnu, grad, mu, nu, count, lr, b1, b2, eps, eps_root,
                  dgrad, dmu_in, dnu_in, stream=None) -> None:
    """diffopt_adam_bwd_tree; dmu/dnu may be None."""
    k = len(table.numel)
    _check(_lib.diffopt_adam_bwd_tree(
        table.handle, *[_leaf_array(x, w, k) for x, w in ((dupdate, "dupdate"), (dmu, "dmu"), (dnu, "dnu"),
                                                           (grad, "grad"), (mu, "mu"), (nu, "nu"))],
        int(count), float(lr), float(b1), float(b2), float(eps), float(eps_root),
        *[_leaf_array(x, w, k) for x, w in ((dgrad, "dgrad"), (dmu_in, "dmu_in"), (dnu_in, "dnu_in"))],
        _stream(stream)))


def adam_unrolled_fwd_tree(table: SegTable, p0, grads, mu_traj, nu_traj, pK, count0, lr, b1, b2, eps, eps_root,
                           stream=None) -> None:
    """diffopt_adam_unrolled_fwd_tree; grads has K entries, mu_traj/nu_traj K+1."""
    K = len(grads)
    k = len(table.numel)
    if len(mu_traj) != K + 1 or len(nu_traj) != K + 1:
        raise ValueError("mu_traj and nu_traj need K+1 entries")
    _check(_lib.diffopt_adam_unrolled_fwd_tree(
        table.handle, K, _leaf_array(p0, "p0", k), _leaf_array_list(grads, "grads", k),
        _leaf_array_list(mu_traj, "mu_traj", k), _leaf_array_list(nu_traj, "nu_traj", k), _leaf_array(pK, "pK", k),
        int(count0), float(lr), float(b1), float(b2), float(eps), float(eps_root), _stream(stream)))


def adam_unrolled_bwd_tree(table: SegTable, dpK, grads, mu_traj, nu_traj, dgrads, dmu0, dnu0, count0, lr, b1, b2,
                           eps, eps_root, stream=None) -> None:
    """diffopt_adam_unrolled_bwd_tree; mu_traj/nu_traj may hold K or K+1 entries."""
    K = len(grads)
    k = len(table.numel)
    if len(dgrads) != K or len(mu_traj) < K or len(nu_traj) < K:
        raise ValueError("dgrads needs K entries, mu_traj/nu_traj at least K")
    _check(_lib.diffopt_adam_unrolled_bwd_tree(
        table.handle, K, _leaf_array(dpK, "dpK", k), _leaf_array_list(grads, "grads", k),
        _leaf_array_list(mu_traj[:K], "mu_traj", k), _leaf_array_list(nu_traj[:K], "nu_traj", k),
        _leaf_array_list(dgrads, "dgrads", k), _leaf_array(dmu0, "dmu0", k), _leaf_array(dnu0, "dnu0", k),
        int(count0), float(lr), float(b1), float(b2), float(eps), float(eps_root), _stream(stream)))


# ---- SGD-momentum and RMSProp (flat fp32 buffers)


def sgd_fwd(params, grad, trace, lr, momentum, nesterov, params_out, trace_out=None, stream=None,
            n: Optional[int] = None) -> None:
    """diffopt_sgd_fwd; trace may be None (zero), trace_out is needed when momentum > 0."""
    if n is None:
        n = params.numel()
    _check(_lib.diffopt_sgd_fwd(_addr(params, "params", n=n), _addr(grad, "grad", n=n),
                                _addr(trace, "trace", n=n), int(n), float(lr), float(momentum),
                                int(bool(nesterov)), _addr(params_out, "params_out", n=n),
                                _addr(trace_out, "trace_out", n=n), _stream(stream)))


def sgd_bwd(dparams_out, dtrace_out, lr, momentum, nesterov, dgrad, dtrace_in=None, stream=None,
            n: Optional[int] = None) -> None:
    """diffopt_sgd_bwd; dtrace_out may be None (zero)."""
    if n is None:
        n = dparams_out.numel()
    _check(_lib.diffopt_sgd_bwd(_addr(dparams_out, "dparams_out", n=n), _addr(dtrace_out, "dtrace_out", n=n),
                                int(n), float(lr), float(momentum), int(bool(nesterov)),
                                _addr(dgrad, "dgrad", n=n), _addr(dtrace_in, "dtrace_in", n=n), _stream(stream)))


def rmsprop_fwd(params, grad, nu, mom, lr, alpha, eps, eps_root, momentum, params_out, nu_out, mom_out=None,
                stream=None, n: Optional[int] = None) -> None:
    """diffopt_rmsprop_fwd; mom may be None (zero), mom_out is needed when momentum > 0."""
    if n is None:
        n = params.numel()
    _check(_lib.diffopt_rmsprop_fwd(_addr(params, "params", n=n), _addr(grad, "grad", n=n), _addr(nu, "nu", n=n),
                                    _addr(mom, "mom", n=n), int(n), float(lr), float(alpha), float(eps),
                                    float(eps_root), float(momentum), _addr(params_out, "params_out", n=n),
                                    _addr(nu_out, "nu_out", n=n), _addr(mom_out, "mom_out", n=n), _stream(stream)))


def rmsprop_bwd(dparams_out, dnu_out, dmom_out, grad, nu, lr, alpha, eps, eps_root, momentum, dgrad, dnu_in,
                dmom_in=None, stream=None, n: Optional[int] = None) -> None:
    """diffopt_rmsprop_bwd; dnu_out / dmom_out may be None (zero)."""
    if n is None:
        n = dparams_out.numel()
    _check(_lib.diffopt_rmsprop_bwd(_addr(dparams_out, "dparams_out", n=n), _addr(dnu_out, "dnu_out", n=n),
                                    _addr(dmom_out, "dmom_out", n=n), _addr(grad, "grad", n=n),
                                    _addr(nu, "nu", n=n), int(n), float(lr), float(alpha), float(eps),
                                    float(eps_root), float(momentum), _addr(dgrad, "dgrad", n=n),
                                    _addr(dnu_in, "dnu_in", n=n), _addr(dmom_in, "dmom_in", n=n), _stream(stream)))


def sgd_fwd_tree(table: SegTable, params, grad, trace, lr, momentum, nesterov, params_out, trace_out=None,
                 stream=None) -> None:
    """diffopt_sgd_fwd_tree; every operand a device int64 array of leaf addresses (trace may be None)."""
    k = len(table.numel)
    _check(_lib.diffopt_sgd_fwd_tree(
        table.handle, _leaf_array(params, "params", k), _leaf_array(grad, "grad", k), _leaf_array(trace, "trace", k),
        float(lr), float(momentum), int(bool(nesterov)), _leaf_array(params_out, "params_out", k),
        _leaf_array(trace_out, "trace_out", k), _stream(stream)))


def sgd_bwd_tree(table: SegTable, dparams_out, dtrace_out, lr, momentum, nesterov, dgrad, dtrace_in=None,
                 stream=None) -> None:
    """diffopt_sgd_bwd_tree (dtrace_out may be None)."""
    k = len(table.numel)
    _check(_lib.diffopt_sgd_bwd_tree(
        table.handle, _leaf_array(dparams_out, "dparams_out", k), _leaf_array(dtrace_out, "dtrace_out", k),
        float(lr), float(momentum), int(bool(nesterov)), _leaf_array(dgrad, "dgrad", k),
        _leaf_array(dtrace_in, "dtrace_in", k), _stream(stream)))


def rmsprop_fwd_tree(table: SegTable, params, grad, nu, mom, lr, alpha, eps, eps_root, momentum, params_out, nu_out,
                     mom_out=None, stream=None) -> None:
    """diffopt_rmsprop_fwd_tree (mom may be None)."""
    k = len(table.numel)
    _check(_lib.diffopt_rmsprop_fwd_tree(
        table.handle, *[_leaf_array(x, w, k) for x, w in ((params, "params"), (grad, "grad"), (nu, "nu"),
                                                           (mom, "mom"))],
        float(lr), float(alpha), float(eps), float(eps_root), float(momentum),
        *[_leaf_array(x, w, k) for x, w in ((params_out, "params_out"), (nu_out, "nu_out"), (mom_out, "mom_out"))],
        _stream(stream)))


def rmsprop_bwd_tree(table: SegTable, dparams_out, dnu_out, dmom_out, grad, nu, lr, alpha, eps, eps_root, momentum,
                     dgrad, dnu_in, dmom_in=None, stream=None) -> None:
    """diffopt_rmsprop_bwd_tree (dnu_out / dmom_out may be None)."""
    k = len(table.numel)
    _check(_lib.diffopt_rmsprop_bwd_tree(
        table.handle, *[_leaf_array(x, w, k) for x, w in ((dparams_out, "dparams_out"), (dnu_out, "dnu_out"),
                                                           (dmom_out, "dmom_out"), (grad, "grad"), (nu, "nu"))],
        float(lr), float(alpha), float(eps), float(eps_root), float(momentum),
        *[_leaf_array(x, w, k) for x, w in ((dgrad, "dgrad"), (dnu_in, "dnu_in"), (dmom_in, "dmom_in"))],
        _stream(stream)))


# ---- zero-order (ES) gradient estimation


def es_perturb(params, noise, sigma, antithetic, out, stream=None) -> None:
    """diffopt_es_perturb: noise is [N, n]; out is [N, n] (or [2N, n] if antithetic)."""
    n = params.numel()
    N = noise.numel() // n if n else 0
    if noise.numel() != N * n or out.numel() != (2 if antithetic else 1) * N * n:
        raise ValueError("noise must be [N, n] and out [N or 2N, n]")
    _check(_lib.diffopt_es_perturb(_addr(params, "params"), _addr(noise, "noise"), int(N), int(n), float(sigma),
                                   int(bool(antithetic)), _addr(out, "out"), _stream(stream)))


def es_estimate(noise, weights, scale, grad, stream=None) -> None:
    """diffopt_es_estimate: grad = scale * weights @ noise (noise [N, n], weights [N] on the device)."""
    n = grad.numel()
    N = weights.numel()
    if noise.numel() != N * n:
        raise ValueError("noise must be [N, n] with N = weights.numel(), n = grad.numel()")
    _check(_lib.diffopt_es_estimate(_addr(noise, "noise"), _addr(weights, "weights"), int(N), int(n), float(scale),
                                    _addr(grad, "grad"), _stream(stream)))


ES_METHODS = {"plain": 0, "baseline": 1, "antithetic": 2}


def _es_method(method) -> int:
    if method not in ES_METHODS:
        raise ValueError("method must be one of %s" % sorted(ES_METHODS))
    return ES_METHODS[method]


def es_perturb_gaussian(params, num_samples: int, seed: int, sigma, antithetic, out, stream=None) -> None:
    """diffopt_es_perturb_gaussian: out is [N, n] (or [2N, n] if antithetic); the noise is generated in the kernel."""
    n = params.numel()
    if out.numel() != (2 if antithetic else 1) * num_samples * n:
        raise ValueError("out must be [N or 2N, n]")
    _check(_lib.diffopt_es_perturb_gaussian(_addr(params, "params"), int(n), int(num_samples),
                                            int(seed) & ((1 << 64) - 1), float(sigma), int(bool(antithetic)),
                                            _addr(out, "out"), _stream(stream)))


def es_estimate_gaussian(fvals, method: str, num_samples: int, seed: int, sigma, grad, f0=None, stream=None) -> None:
    """diffopt_es_estimate_gaussian: fvals [N] (plain, baseline) or [2N] (antithetic), f0 a device scalar
    (baseline); the weights, the scale and the noise are formed in the kernel."""
    m = _es_method(method)
    if fvals.numel() != (2 if m == 2 else 1) * num_samples:
        raise ValueError("fvals must hold %s evaluations" % ("2N" if m == 2 else "N"))
    if m == 1 and f0 is None:
        raise ValueError("the baseline method needs f0 = f(theta)")
    _check(_lib.diffopt_es_estimate_gaussian(_addr(fvals, "fvals"), _addr(f0, "f0", n=1) if m == 1 else None,
                                             int(num_samples), m, int(grad.numel()), int(seed) & ((1 << 64) - 1),
                                             float(sigma), _addr(grad, "grad"), _stream(stream)))


def es_weights(fvals, method: str, num_samples: int, sigma, weights, f0=None, stream=None) -> None:
    """diffopt_es_weights: weights [N] = scale * w for diffopt_es_estimate with scale 1."""
    m = _es_method(method)
    if fvals.numel() != (2 if m == 2 else 1) * num_samples or weights.numel() != num_samples:
        raise ValueError("fvals must hold N (2N antithetic) evaluations and weights N entries")
    if m == 1 and f0 is None:
        raise ValueError("the baseline method needs f0 = f(theta)")
    _check(_lib.diffopt_es_weights(_addr(fvals, "fvals"), _addr(f0, "f0", n=1) if m == 1 else None,
                                   int(num_samples), m, float(sigma), _addr(weights, "weights"), _stream(stream)))
