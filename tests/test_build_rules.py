"""CPU checks of the build's object rules: objects that no current source
produces are deleted before the link, and the link names exactly the current
sources' objects (an object left behind by an older source, with kernels built
for an older argument layout, once won the link and faulted)."""

import os

from paper_2203_14685_amd import build as b


def test_stale_objects_are_pruned(tmp_path):
    objdir = str(tmp_path)
    keep = [src.replace(".hip", ".o") for src in b.SOURCES]
    for name in keep + ["old_route.o", "layout_v1.o", "notes.txt"]:
        open(os.path.join(objdir, name), "w").close()
    removed = b.prune_stale_objects(objdir)
    assert removed == ["layout_v1.o", "old_route.o"]
    assert sorted(os.listdir(objdir)) == sorted(keep + ["notes.txt"])


def test_link_names_exactly_the_source_objects(tmp_path):
    objdir = str(tmp_path)
    open(os.path.join(objdir, "stale.o"), "w").close()
    cmd = b.link_command("hipcc", objdir, "lib.so")
    objs = [a for a in cmd if a.endswith(".o")]
    assert objs == [os.path.join(objdir, src.replace(".hip", ".o")) for src in b.SOURCES]
    assert not any("*" in a for a in cmd)
    assert cmd[-2:] == ["-o", "lib.so"] and "--offload-arch=gfx950" in cmd


def test_every_source_file_exists():
    for src in b.SOURCES:
        assert os.path.exists(os.path.join(b.CSRC, src)), src
