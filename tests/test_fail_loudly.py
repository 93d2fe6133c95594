"""Without libcheb.so the package does not import: there is no CPU fallback
anywhere on the product path."""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def test_missing_library_is_an_import_error(tmp_path):
    pkg = os.path.join(ROOT, "paper_2608_23429_amd")
    dst = os.path.join(tmp_path, "paper_2608_23429_amd")
    shutil.copytree(pkg, dst, ignore=shutil.ignore_patterns("*.so", "__pycache__", "csrc"))
    assert not any(f.endswith(".so") for f in os.listdir(dst))
    code = ("import sys; sys.path.insert(0, %r)\n"
            "try:\n    import paper_2608_23429_amd\nexcept ImportError as e:\n"
            "    print('IMPORT ERROR:', e); sys.exit(3)\nsys.exit(0)\n") % str(tmp_path)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 3, r.stdout + r.stderr
    assert "not built" in r.stdout
