"""Pins of the oracle's tree pack/unpack (flatten/unflatten, Appendix D,
Table 2) against numpy's concatenation and slicing, bit for bit."""
import numpy as np
import pytest

import oracle
from workloads import random_shapes, random_bits, special_f32


def _bits(a):
    a = np.ascontiguousarray(a)
    return a.view({1: np.uint8, 2: np.uint16, 4: np.uint32, 8: np.uint64}[a.dtype.itemsize])


@pytest.mark.parametrize("dtype", [np.float32, np.float64, np.float16, np.uint8])
def test_pack_equals_concatenate(dtype):
    shapes = random_shapes(300, 5000, seed=1)
    leaves = []
    for i, s in enumerate(shapes):
        n = int(np.prod(s))
        leaves.append(random_bits(n, dtype, seed=1000 + i).reshape(s))
    flat = oracle.pack(leaves, dtype=dtype)
    ref = np.concatenate([x.reshape(-1) for x in leaves]) if leaves else np.zeros(0, dtype)
    assert flat.dtype == np.dtype(dtype)
    assert np.array_equal(_bits(flat), _bits(ref))


def test_unpack_inverts_pack_special_values():
    sp = special_f32()
    leaves = [sp, sp[:1], np.zeros(0, np.float32), np.tile(sp, 7)[:37], sp[::-1].copy()]
    flat = oracle.pack(leaves)
    back = oracle.unpack(flat, [x.shape for x in leaves])
    for a, b in zip(leaves, back):
        assert np.array_equal(_bits(a), _bits(b))
    # and a direct slice check of where each leaf landed
    off = 0
    for a in leaves:
        assert np.array_equal(_bits(flat[off:off + a.size]), _bits(a))
        off += a.size


def test_explicit_offsets_with_gaps():
    rng = np.random.default_rng(5)
    leaves = [random_bits(k, np.float32, seed=k) for k in (5, 0, 1, 17, 64, 3)]
    offsets = []
    pos = 3
    for x in leaves:
        offsets.append(pos)
        pos += x.size + int(rng.integers(0, 9))
    flat = oracle.pack(leaves, offsets=offsets, flat_len=pos + 2)
    expect = np.zeros(pos + 2, np.float32)
    for o, x in zip(offsets, leaves):
        expect[o:o + x.size] = x
    assert np.array_equal(_bits(flat), _bits(expect))
    back = oracle.unpack(flat, [x.shape for x in leaves], offsets=offsets)
    for a, b in zip(leaves, back):
        assert np.array_equal(_bits(a), _bits(b))


def test_single_segment_is_memcpy():
    x = random_bits(100003, np.float32, seed=9)
    assert np.array_equal(_bits(oracle.pack([x])), _bits(x))
