"""The build script compiles every kernel source, each with the packed-fp32
switch, and its per-source code-generation options name real sources (CPU
tests; nothing is compiled)."""
import os

from paper_2609_13612_amd import build


def test_every_source_is_built():
    on_disk = sorted(f for f in os.listdir(build.CSRC) if f.endswith((".hip", ".cpp")))
    assert sorted(build.SOURCES) == on_disk


def test_source_flags_name_built_hip_sources():
    for src, flags in build.SOURCE_FLAGS.items():
        assert src in build.SOURCES and src.endswith(".hip"), src
        # backend options only: each is an -mllvm pair, and none re-enables packed fp32
        assert len(flags) % 2 == 0 and all(f == "-mllvm" for f in flags[::2]), flags
        assert not any("packed-fp32" in f for f in flags)


def test_packed_fp32_is_off_for_every_device_source(monkeypatch):
    seen = {}

    class Done:
        returncode, stderr = 0, ""

    def fake_run(cmd, **kw):
        seen[os.path.basename(cmd[2])] = cmd
        return Done()

    monkeypatch.setattr(build.subprocess, "run", fake_run)
    for src in build.SOURCES:
        build._compile(src)
    for src, cmd in seen.items():
        has = any(a == "-packed-fp32-ops" for a in cmd)
        assert has == src.endswith(".hip"), src
        for f in build.SOURCE_FLAGS.get(src, []):
            assert f in cmd, (src, f)
