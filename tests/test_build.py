"""The build's housekeeping: objects that no source produces are removed
from the build folder, and a library that leaves one of its own symbols
undefined is refused."""

import os

from paper_2211_17111_amd import build as b


def test_remove_stale_objects(tmp_path, monkeypatch):
    monkeypatch.setattr(b, "BUILD", str(tmp_path))
    for name in ("prepare.o", "forward_old.o", "notes.txt", "api.o"):
        (tmp_path / name).write_text("x")
    removed = b.remove_stale_objects()
    assert removed == ["forward_old.o"]
    assert sorted(os.listdir(tmp_path)) == ["api.o", "notes.txt", "prepare.o"]


def test_check_defined(tmp_path):
    """A shared library that leaves one of its own symbols undefined links
    without complaint; the build refuses it."""
    import shutil
    import subprocess

    import pytest

    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no host C compiler")
    src = tmp_path / "lib.c"
    src.write_text("void bevpool_missing_stub(void);\n"
                   "void bevpool_caller(void) { bevpool_missing_stub(); }\n")
    bad = tmp_path / "libbad.so"
    subprocess.run([gcc, "-shared", "-fPIC", str(src), "-o", str(bad)], check=True)
    with pytest.raises(RuntimeError, match="undefined"):
        b.check_defined(str(bad))
    src.write_text("int bevpool_ok(void) { return 1; }\n")
    good = tmp_path / "libgood.so"
    subprocess.run([gcc, "-shared", "-fPIC", str(src), "-o", str(good)], check=True)
    b.check_defined(str(good))
