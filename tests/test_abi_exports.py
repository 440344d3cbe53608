"""The C-ABI library loads on any host and exports every function include/asyncstage.h declares
(no compute calls: this runs without a GPU)."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "asyncstage.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(?:int|size_t|void|const char\*)\s+(\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    from paper_2606_30634_amd import binding
    lib = ctypes.CDLL(binding.LIB_PATH)
    names = _declared()
    assert len(names) >= 10, names
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(binding.EXPORTS) == names


def test_shape_validation_on_host():
    from paper_2606_30634_amd import binding as B
    ok = B.StageShape(2, 128, 4, 4, 32, 512, 512, 1, 1, 1, 64, 2, 1, 0, 1e-5, 10000.0)
    assert B.stage_required_bytes(ok) > 0
    for field, bad in [("head_dim", 48), ("n_kv_heads", 3), ("d_model", 100), ("dtype", 7)]:
        s = B.StageShape(2, 128, 4, 4, 32, 512, 512, 1, 1, 1, 64, 2, 1, 0, 1e-5, 10000.0)
        setattr(s, field, bad)
        assert B.stage_required_bytes(s) == 0
        assert B.last_error()
    # a last stage without the tied embedding is rejected
    s = B.StageShape(2, 128, 4, 4, 32, 512, 0, 0, 1, 0, 64, 2, 1, 1, 1e-5, 10000.0)
    assert B.stage_required_bytes(s) == 0
