"""The C-ABI library loads and exports every entry point include/*.h declares
(no GPU needed: no compute call is made)."""
import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ro.h")


def _declared(paths=None):
    names = set()
    for path in paths or sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        text = re.sub(r"/\*.*?\*/", "", open(path).read(), flags=re.S)
        names.update(re.findall(r"\bint\s+(ro_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_header_declares_the_boundary():
    names = _declared([HEADER])
    for must in ("ro_expand", "ro_batch", "ro_gather", "ro_stream_create", "ro_stream_report",
                 "ro_stream_emit", "ro_stream_destroy", "ro_ctx_create", "ro_ctx_status"):
        assert must in names


def test_library_exports_every_declared_symbol():
    import paper_2609_18703_amd as R
    if not os.path.exists(R.LIB_PATH):
        pytest.skip("libro.so not built")
    lib = ctypes.CDLL(R.LIB_PATH)
    names = _declared()
    assert "ro_debug_epochs" in names       # the test aid, from its own header
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_loads_and_fails_loudly_without_library(tmp_path):
    import paper_2609_18703_amd as R
    with pytest.raises(RuntimeError):
        R.load(str(tmp_path / "missing.so"))


def test_status_codes_match_header():
    import paper_2609_18703_amd as R
    text = open(HEADER).read()
    for name, val in [("RO_OK", R.OK), ("RO_EINVAL", R.EINVAL), ("RO_ERANGE", R.ERANGE), ("RO_EDUP", R.EDUP),
                      ("RO_ECAP", R.ECAP), ("RO_EOVERFLOW", R.EOVERFLOW), ("RO_ESTATE", R.ESTATE),
                      ("RO_EHIP", R.EHIP), ("RO_SUCCESS", R.SUCCESS), ("RO_FAILED", R.FAILED),
                      ("RO_SKIPPED", R.SKIPPED), ("RO_PENDING", R.PENDING)]:
        m = re.search(name + r"\s*=\s*(-?\d+)", text)
        assert m and int(m.group(1)) == val, name


def test_kernel_names_match_header_enum():
    import paper_2609_18703_amd as R
    text = open(HEADER).read()
    m = re.search(r"enum \{\s*(RO_K_EXPAND_SCAN.*?RO_K_COUNT)\s*\}", text, flags=re.S)
    names = [x.strip().split("=")[0].strip() for x in m.group(1).split(",")]
    names = [n for n in names if n and n != "RO_K_COUNT"]
    assert [n[len("RO_K_"):].lower() for n in names] == R.KERNELS
