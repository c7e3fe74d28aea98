"""Host-side contracts that need no GPU: the bench refuses more than one GPU,
the library loader has no fallback, and the graft entry points exist."""
import importlib
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_missing_library_raises(monkeypatch, tmp_path):
    from paper_2607_15650_amd import _lib
    monkeypatch.setattr(_lib, "_handle", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "libditango.so"))
    try:
        _lib.lib()
    except RuntimeError as e:
        assert "no fallback" in str(e)
    else:
        raise AssertionError("loading a missing library must raise")


def test_graft_entry_points_exist():
    sys.path.insert(0, ROOT)
    m = importlib.import_module("__graft_entry__")
    assert callable(m.build) and callable(m.smoke)


def test_product_modules_do_not_import_the_oracle():
    """Only tests, the smoke check and the bench's CPU baseline may use the
    oracle: the package's sources never import it."""
    pkg = os.path.join(ROOT, "paper_2607_15650_amd")
    for name in os.listdir(pkg):
        if name.endswith(".py"):
            text = open(os.path.join(pkg, name)).read()
            assert "import oracle" not in text and "from oracle" not in text, name
