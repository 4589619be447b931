"""CPU checks of the C ABI: the library loads, exports every symbol the
headers declare, and its host-side tree metadata agrees with the oracle."""
import os
import re

import numpy as np
import pytest

from oracle import oracle as O
from paper_2510_26843_amd import cas, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in ("cas.h", "cas_ops.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(cas_[a-z0-9_]+)\s*\(", src))
    return names


@pytest.mark.parametrize("debug", [False, True], ids=["release", "device_checks"])
def test_library_exports_every_declared_symbol(debug):
    L = cas.lib(debug)
    declared = _declared()
    assert len(declared) >= 20
    for n in sorted(declared):
        assert hasattr(L, n), n
    assert declared == set(cas.EXPORTS)
    assert L.cas_debug_build() == (1 if debug else 0)


@pytest.mark.parametrize("branching,n", [((3, 2, 1), 15), ((4, 2, 2, 1, 1), 32), ((4, 4, 4, 4), 64),
                                         ((2,) * 7, 128), ((), 1)])
def test_tree_info_matches_oracle(branching, n):
    parents = synth.tree_from_branching(branching, n) if branching else [-1]
    depth, anc = cas.tree_info(parents)
    d_ref, a_ref = O.tree_metadata(parents)
    assert list(depth) == d_ref
    for i in range(n):
        assert int(anc[i, 0]) | (int(anc[i, 1]) << 64) == a_ref[i]


def test_tree_info_rejects_invalid_parents():
    for bad in ([0], [-1, 1], [-1, 0, 3, 1], [-1, -1], [-1, 0, 2]):
        with pytest.raises(cas.CasError) as e:
            cas.tree_info(bad)
        assert e.value.status == cas.ERR_TREE
    with pytest.raises(cas.CasError):
        cas.tree_info(list(range(-1, 128)))  # 129 nodes: beyond the 128-bit masks


def test_create_without_device_fails_cleanly():
    """Creating a context where no GPU is visible returns a status, not a crash."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    with pytest.raises(cas.CasError) as e:
        cas.Model(synth.SHAPES["tiny"], max_ctx=256)
    assert e.value.status == cas.ERR_DEVICE


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=96), cas.ERR_UNSUPPORTED), (dict(n_kv_heads=3), cas.ERR_ARG),
    (dict(d_model=250), cas.ERR_UNSUPPORTED), (dict(vocab=2050), cas.ERR_UNSUPPORTED)])
def test_create_validates_shape_before_the_device(change, status):
    import dataclasses
    shape = dataclasses.replace(synth.SHAPES["tiny"], **change)
    with pytest.raises(cas.CasError) as e:
        cas.Model(shape, max_ctx=256)
    assert e.value.status == status
    with pytest.raises(cas.CasError) as e:
        cas.Model(synth.SHAPES["tiny"], max_ctx=256, max_tree=129)
    assert e.value.status == cas.ERR_UNSUPPORTED
