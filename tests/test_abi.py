"""The C ABI without a GPU: the library loads, exports every symbol the
header declares, and rejects invalid configurations on the host before any
device call.  Also checks that the product code never reaches the oracle."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rheo.h")
PKG = os.path.join(ROOT, "paper_2609_21827_amd")
LIB = os.path.join(PKG, "librheo.so")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|int32_t|const char\*)\s+(rheo_\w+)\(", text, re.M)))


needs_lib = pytest.mark.skipif(not os.path.exists(LIB), reason="librheo.so not built")


@needs_lib
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    from paper_2609_21827_amd import binding
    assert sorted(binding.EXPORTS) == names


def _cfg(**kw):
    from paper_2609_21827_amd.binding import RheoConfig
    base = dict(batch=2, vocab=1000, pool=4, leads=1, depth=3, n_expand=0,
                support=128, construct_tempered=0, dtype=1, method=0,
                construct_full=0, row_stride=1000, eps_m0=0.0)
    base.update(kw)
    return RheoConfig(**base)


BAD = [
    dict(batch=0), dict(vocab=1), dict(vocab=262144), dict(pool=0), dict(pool=16),
    dict(leads=4), dict(leads=-1), dict(depth=0), dict(depth=16),
    dict(n_expand=5), dict(dtype=7), dict(method=3), dict(method=-1), dict(support=0, vocab=3, row_stride=8),
    dict(construct_full=2), dict(construct_full=-1),
    dict(support=3), dict(vocab=5000, row_stride=5000, support=2000), dict(row_stride=999),
    dict(row_stride=1001), dict(eps_m0=-1.0),
    dict(vocab=3, support=3, pool=4),
]


@needs_lib
@pytest.mark.parametrize("bad", BAD)
def test_invalid_configs_rejected_on_host(bad):
    from paper_2609_21827_amd import binding
    lib = binding.load_library()
    h = ctypes.c_void_p()
    rc = lib.rheo_create(ctypes.byref(_cfg(**bad)), ctypes.byref(h))
    assert rc == binding.RHEO_EINVAL, (bad, rc)
    assert not h.value
    assert lib.rheo_last_error().decode()


@needs_lib
def test_null_handles_rejected():
    from paper_2609_21827_amd import binding
    lib = binding.load_library()
    assert lib.rheo_begin_step(None) == binding.RHEO_EINVAL
    assert lib.rheo_prune(None, 1, None) == binding.RHEO_EINVAL
    assert lib.rheo_verify(None, None, 1.0, 0, None, None, None, None) == binding.RHEO_EINVAL
    assert lib.rheo_create(None, None) == binding.RHEO_EINVAL


def test_binding_fails_loudly_without_library(tmp_path):
    import importlib
    from paper_2609_21827_amd import binding
    saved = binding._LIB
    binding._LIB = None
    try:
        with pytest.raises(ImportError):
            binding.load_library(str(tmp_path / "missing.so"))
    finally:
        binding._LIB = saved


def test_product_never_imports_the_oracle():
    for dirpath, _, files in os.walk(PKG):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle", text, re.M), f
                assert "oracle/" not in text, f
    for f in os.listdir(os.path.join(ROOT, "synth")):
        if f.endswith(".py"):
            text = open(os.path.join(ROOT, "synth", f)).read()
            assert not re.search(r"^\s*(import|from)\s+(oracle|paper_2609)", text, re.M)


@needs_lib
def test_static_tree_size_limit_on_host():
    """rheo_create_static refuses a tree larger than its static scratch
    array before any device call."""
    from paper_2609_21827_amd import binding
    lib = binding.load_library()
    cfg = _cfg(batch=128, vocab=128256, row_stride=128256, pool=10, depth=8, support=1024)
    h = ctypes.c_void_p()
    assert lib.rheo_create_static(ctypes.byref(cfg), ctypes.byref(h)) == binding.RHEO_EINVAL
    assert "static scratch" in lib.rheo_last_error().decode()
