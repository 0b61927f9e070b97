"""The product path has no CPU fallback and does not reach the oracle.

- A copy of the binding next to no built library raises ImportError at import
  time (run in a fresh interpreter, so the real package is never loaded).
- No source of the package or of the C ABI names the oracle: the Python
  binding, the HIP kernels and the ABI share no code with it.
"""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_09208_amd")


def test_binding_without_library_fails_at_import(tmp_path):
    dst = tmp_path / "paper_2609_09208_amd"
    dst.mkdir()
    shutil.copy(os.path.join(PKG, "__init__.py"), dst / "__init__.py")
    code = ("import sys\n"
            f"sys.path.insert(0, {str(tmp_path)!r})\n"
            "try:\n"
            "    import paper_2609_09208_amd\n"
            "except ImportError as e:\n"
            "    print('IMPORT-ERROR', e)\n"
            "    sys.exit(0)\n"
            "sys.exit(3)\n")
    res = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         timeout=300, cwd=str(tmp_path))
    assert res.returncode == 0, res.stdout + res.stderr
    assert "IMPORT-ERROR" in res.stdout and "not built" in res.stdout


def test_product_sources_do_not_name_the_oracle():
    roots = [PKG, os.path.join(ROOT, "include")]
    offenders = []
    for root in roots:
        for dirpath, _, files in os.walk(root):
            if "__pycache__" in dirpath:
                continue
            for f in files:
                if not f.endswith((".py", ".hip", ".cpp", ".hpp", ".h")):
                    continue
                p = os.path.join(dirpath, f)
                text = open(p, encoding="utf-8").read()
                if "import oracle" in text or "from oracle" in text or "liboracle" in text \
                        or "pot_oracle" in text:
                    offenders.append(p)
    assert not offenders, offenders
