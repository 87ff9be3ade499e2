"""The product path stands alone: importing the package loads no part of the
CPU oracle, and without the built HIP library every entry point raises
instead of computing anything another way."""
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]


def test_package_import_loads_no_oracle():
    code = ("import sys; sys.path.insert(0, %r); import paper_2609_33586_amd as p; "
            "import paper_2609_33586_amd.synth; "
            "print(sorted(m for m in sys.modules if m == 'oracle' or m.startswith('oracle.')))") % str(ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "[]"


def test_missing_library_raises(monkeypatch, tmp_path):
    import paper_2609_33586_amd as pkg
    monkeypatch.setattr(pkg, "_lib", None)
    monkeypatch.setattr(pkg, "LIB_PATH", tmp_path / "libh15attn.so")
    with pytest.raises(RuntimeError, match="missing"):
        pkg.lib()
    with pytest.raises(RuntimeError, match="missing"):
        pkg.attn_tile_bc()


def test_product_sources_do_not_reference_the_oracle():
    pkgdir = ROOT / "paper_2609_33586_amd"
    for f in list(pkgdir.glob("*.py")) + list((pkgdir / "csrc").glob("*")) + list((ROOT / "include").glob("*.h")):
        text = f.read_text()
        assert "import oracle" not in text and "from oracle" not in text and "attn_oracle" not in text, f.name
