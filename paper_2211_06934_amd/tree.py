"""Tensor-tree flatten / unflatten over the device segment table.

The host part of a tree operation (Sec. 2.3 "PyTree"; Appendix D, Table 2)
is a walk over nested Python containers that lists the leaf tensors and
records the structure.  The device part moves the leaf data into one flat
buffer (or back) in a single kernel through ``diffopt_tree_flatten`` /
``diffopt_tree_unflatten``.  A segment table depends only on the leaf shapes
and dtype, so it is built once per structure and cached.

Leaf order: dicts by sorted key, lists and tuples by index, a torch.nn.Module's
parameters in registration order (``named_parameters``).  The paper does not
fix an order; any fixed order works as long as flatten and unflatten agree.
"""
from __future__ import annotations

import contextlib

import dataclasses
from typing import Any, Dict, List, Optional, Sequence, Tuple

import torch

from . import diffopt as _d


@dataclasses.dataclass(frozen=True)
class TreeDef:
    """Structure of a tree: container kinds and keys, with leaf slots."""
    kind: str                      # "leaf", "dict", "list", "tuple", "none"
    keys: Tuple[Any, ...] = ()
    children: Tuple["TreeDef", ...] = ()

    @property
    def num_leaves(self) -> int:
        if self.kind == "leaf":
            return 1
        return sum(c.num_leaves for c in self.children)


LEAF = TreeDef("leaf")
NONE = TreeDef("none")


def tree_leaves(tree) -> Tuple[List[torch.Tensor], TreeDef]:
    """Flatten the container structure: returns (leaves, treedef)."""
    leaves: List[torch.Tensor] = []

    def walk(x) -> TreeDef:
        if isinstance(x, torch.Tensor):
            leaves.append(x)
            return LEAF
        if x is None:
            return NONE
        if isinstance(x, torch.nn.Module):
            x = dict(x.named_parameters())
            keys = tuple(x.keys())  # registration order
            return TreeDef("dict", keys, tuple(walk(x[k]) for k in keys))
        if isinstance(x, dict):
            keys = tuple(sorted(x.keys()))
            return TreeDef("dict", keys, tuple(walk(x[k]) for k in keys))
        if isinstance(x, (list, tuple)):
            return TreeDef("list" if isinstance(x, list) else "tuple", (),
                           tuple(walk(v) for v in x))
        raise TypeError("unsupported tree node of type %s" % type(x).__name__)

    td = walk(tree)
    return leaves, td


def tree_build(td: TreeDef, leaves: Sequence[torch.Tensor]):
    """Inverse of tree_leaves: rebuild containers around the given leaves."""
    it = iter(leaves)

    def build(t: TreeDef):
        if t.kind == "leaf":
            return next(it)
        if t.kind == "none":
            return None
        if t.kind == "dict":
            return {k: build(c) for k, c in zip(t.keys, t.children)}
        vals = [build(c) for c in t.children]
        return vals if t.kind == "list" else tuple(vals)

    return build(td)


@dataclasses.dataclass
class FlatSpec:
    """Everything needed to split a flat buffer back into a tree."""
    treedef: TreeDef
    shapes: Tuple[Tuple[int, ...], ...]
    dtype: torch.dtype
    table: _d.SegTable

    @property
    def total(self) -> int:
        return self.table.total


_TABLES: Dict[Tuple, _d.SegTable] = {}


def segment_table(shapes: Sequence[Tuple[int, ...]], dtype: torch.dtype,
                  device: Optional[torch.device] = None) -> _d.SegTable:
    """Cached dense segment table for leaves of these shapes and dtype."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    key = (tuple(tuple(int(d) for d in s) for s in shapes), dtype, dev.index)
    t = _TABLES.get(key)
    if t is None:
        numel = [int(torch.Size(s).numel()) for s in shapes]
        elem = torch.empty((), dtype=dtype).element_size()
        with torch.cuda.device(dev):
            t = _d.segtable_create(numel, None, elem)
        _TABLES[key] = t
    return t


def _stream_context(stream):
    """Make `stream` (a torch stream, a raw hipStream_t address or None) current."""
    if stream is None:
        return contextlib.nullcontext()
    if isinstance(stream, int):
        stream = torch.cuda.ExternalStream(stream)
    return torch.cuda.stream(stream)


def leaf_pointer_tensors(groups: Sequence[Optional[Sequence[torch.Tensor]]], device,
                         stream=None) -> List[Optional[torch.Tensor]]:
    """One device int64 array of leaf addresses (table order) per group of
    leaves; None for a group that is None.

    All arrays are slices of one device buffer, filled by a single
    asynchronous copy from pinned host memory, so building them neither waits
    for the device nor costs one transfer per operand.  The buffer is
    allocated on `stream` (default: the current one), the stream whose kernels
    read it: torch's caching allocator hands a freed block only to later work
    on the stream it was allocated on, so the arrays may be dropped as soon as
    the kernels are enqueued (the pinned staging block is likewise held until
    the copy has run)."""
    ptrs: List[int] = []
    for g in groups:
        if g is None:
            continue
        for i, x in enumerate(g):
            if not x.is_contiguous():
                raise ValueError("leaf %d is not contiguous" % i)
            ptrs.append(x.data_ptr())
    with _stream_context(stream):
        host = torch.tensor(ptrs, dtype=torch.int64).pin_memory()
        dev = host.to(device, non_blocking=True)
    out: List[Optional[torch.Tensor]] = []
    o = 0
    for g in groups:
        if g is None:
            out.append(None)
            continue
        out.append(dev[o:o + len(g)])
        o += len(g)
    return out


def leaf_pointer_tensor(leaves: Sequence[torch.Tensor], device, stream=None) -> torch.Tensor:
    """Device int64 array of leaf addresses, in table order (one group of
    leaf_pointer_tensors)."""
    return leaf_pointer_tensors([leaves], device, stream)[0]


def flatten(tree, out: Optional[torch.Tensor] = None, stream=None) -> Tuple[torch.Tensor, FlatSpec]:
    """Pack every leaf of `tree` into one flat device buffer (one kernel)."""
    leaves, td = tree_leaves(tree)
    if not leaves:
        raise ValueError("tree has no tensor leaves")
    dtype = leaves[0].dtype
    device = leaves[0].device
    for x in leaves:
        if x.dtype != dtype or x.device != device:
            raise ValueError("all leaves must share dtype and device")
    shapes = tuple(tuple(x.shape) for x in leaves)
    table = segment_table(shapes, dtype, device)
    if out is None:
        out = torch.empty(table.total, dtype=dtype, device=device)
    elif out.numel() < table.total or out.dtype != dtype:
        raise ValueError("out is too small or of the wrong dtype")
    _d.tree_flatten(table, leaf_pointer_tensor(leaves, device, stream), out, stream)
    return out, FlatSpec(td, shapes, dtype, table)


def unflatten(flat: torch.Tensor, spec: FlatSpec, out_leaves: Optional[Sequence[torch.Tensor]] = None,
              stream=None):
    """Split a flat buffer into new (or given) leaf tensors and rebuild the tree."""
    if out_leaves is None:
        out_leaves = [torch.empty(s, dtype=spec.dtype, device=flat.device) for s in spec.shapes]
    _d.tree_unflatten(spec.table, flat, leaf_pointer_tensor(out_leaves, flat.device, stream), stream)
    return tree_build(spec.treedef, out_leaves)
