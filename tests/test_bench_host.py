"""Host-side pieces of bench.py: the kernel-source hash that ties the
recorded HBM counters (profiles/traffic.json) to the code they were taken
on follows the code and ignores its comments."""
from __future__ import annotations

import os
import shutil

import bench

SRC = ("ks_kernels.hip", "ks_expand.hip", "ks_internal.h", "ks_sched.inc")


def _tree(tmp_path, edit=None):
    d = tmp_path / "paper_2606_28565_amd" / "csrc"
    d.mkdir(parents=True)
    for f in SRC:
        shutil.copy(os.path.join(bench.ROOT, "paper_2606_28565_amd", "csrc", f), d / f)
    if edit:
        p = d / "ks_kernels.hip"
        p.write_text(edit(p.read_text()))
    return str(tmp_path)


def _hash(monkeypatch, root):
    monkeypatch.setattr(bench, "ROOT", root)
    return bench.kernel_source_hash()


def test_source_hash_ignores_comments_and_blank_lines(tmp_path, monkeypatch):
    base = _hash(monkeypatch, _tree(tmp_path / "a"))
    commented = _hash(monkeypatch, _tree(tmp_path / "b", lambda s: "// note\n\n/* block\n comment */\n" +
                                         s.replace("\n}\n", "\n}  // end\n\n", 3)))
    assert commented == base


def test_source_hash_follows_code(tmp_path, monkeypatch):
    base = _hash(monkeypatch, _tree(tmp_path / "a"))
    changed = _hash(monkeypatch, _tree(tmp_path / "b", lambda s: s.replace("kStreamR * lane", "kStreamR*lane", 1)))
    assert changed != base
