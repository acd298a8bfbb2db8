"""Host-side checks of the C ABI that need no GPU: the library loads,
exports every function include/bgmf.h declares, and rejects bad shapes
before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "bgmf.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bgmf_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    from paper_2304_13724_amd import bgmf
    lib = ctypes.CDLL(bgmf.LIB_PATH)
    names = _declared()
    assert len(names) >= 16
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(bgmf.EXPORTED) == names


@pytest.mark.parametrize("n,m,k,p,needle", [
    (0, 10, 16, 1, "n and m"),
    (10, 10, 24, 1, "multiple of 16"),
    (10, 10, 272, 1, "multiple of 16"),
    (10, 10, 16, 0, "p must be"),
    (10, 5, 16, 6, "p must be"),
    (10_000_000, 10, 16, 10, "blocks too large"),
    # one past the widest block a record can index (65,536 local rows or columns)
    (65_537, 10, 16, 1, "blocks too large"),
    (10, 65_537, 16, 1, "blocks too large"),
    (131_073, 131_072, 16, 2, "blocks too large"),
    (131_072, 131_073, 16, 2, "blocks too large"),
])
def test_create_rejects_bad_shapes(n, m, k, p, needle):
    from paper_2304_13724_amd import bgmf
    with pytest.raises(bgmf.BgmfError) as ei:
        bgmf.bgmf_create(n, m, k, p)
    assert needle in str(ei.value)
