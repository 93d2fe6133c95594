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


def test_build_script_loads_without_the_library(tmp_path):
    """build() must work in a tree where nothing is built yet: it reaches the
    build scripts without importing the package (which would need the
    library it is about to build)."""
    for rel in ("__graft_entry__.py", "paper_2608_23429_amd", "oracle"):
        src = os.path.join(ROOT, rel)
        if os.path.isdir(src):
            shutil.copytree(src, os.path.join(tmp_path, rel),
                            ignore=shutil.ignore_patterns("*.so", "__pycache__"))
        else:
            shutil.copy(src, tmp_path)
    code = ("import sys; sys.path.insert(0, %r)\n"
            "import __graft_entry__ as g\n"
            "m = g._load_build_script('paper_2608_23429_amd/build.py')\n"
            "o = g._load_build_script('oracle/build.py')\n"
            "assert 'paper_2608_23429_amd' not in sys.modules\n"
            "assert m.LIB.endswith('libcheb.so') and o.LIB.endswith('liboracle.so')\n"
            "print('ok')\n") % str(tmp_path)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120,
                       cwd=str(tmp_path))
    assert r.returncode == 0 and "ok" in r.stdout, r.stdout + r.stderr
