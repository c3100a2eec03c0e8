"""The build's housekeeping (no compiler run): objects that no source
produces are removed from the build folder."""

import os

from paper_2211_17111_amd import build as b


def test_remove_stale_objects(tmp_path, monkeypatch):
    monkeypatch.setattr(b, "BUILD", str(tmp_path))
    for name in ("prepare.o", "forward_old.o", "notes.txt", "api.o"):
        (tmp_path / name).write_text("x")
    removed = b.remove_stale_objects()
    assert removed == ["forward_old.o"]
    assert sorted(os.listdir(tmp_path)) == ["api.o", "notes.txt", "prepare.o"]
