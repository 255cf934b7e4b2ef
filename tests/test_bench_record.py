"""Host checks of bench.py's traffic record: the figure is keyed by the
megakernel's sources, and only an edit of the code (not of its comments)
makes a stored measurement stale."""
import os
import shutil

import bench


def _copy_sources(tmp_path):
    for p in bench.KERNEL_SOURCES:
        dst = tmp_path / p
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(bench.ROOT, p), dst)


def test_comment_edits_keep_the_hash_and_code_edits_change_it(tmp_path, monkeypatch):
    _copy_sources(tmp_path)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_sources_hash()
    gemm = tmp_path / "paper_2609_21483_amd/csrc/gemm.h"
    src = gemm.read_text()
    gemm.write_text(src + "\n// a new comment line\n/* and a block\n   comment */\n")
    assert bench.kernel_sources_hash() == h0
    assert "NSTAGE = 4;" in src
    gemm.write_text(src.replace("NSTAGE = 4;", "NSTAGE = 2;"))
    assert bench.kernel_sources_hash() != h0

