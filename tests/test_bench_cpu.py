"""Host-side checks of bench.py that need no GPU: the kernel-source hash that
guards the committed rocprofv3 figures follows the code and not its comments,
and a multi-GPU request is refused with a message."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def sources():
    out = {}
    for name in bench.KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_24089_amd", "csrc", name)) as f:
            out[name] = f.read()
    return out


def test_hash_ignores_comments_and_layout():
    src = sources()
    base = bench.kernel_source_hash(lambda n: src[n])
    assert base == bench.kernel_source_hash()
    edited = dict(src)
    edited["fb_kernels.h"] = "// a new comment line\n" + src["fb_kernels.h"].replace("\n", "\n  ", 3)
    edited["fb_common.h"] = src["fb_common.h"] + "\n/* trailing\n   block comment */\n"
    assert bench.kernel_source_hash(lambda n: edited[n]) == base


def test_hash_follows_code():
    src = sources()
    base = bench.kernel_source_hash(lambda n: src[n])
    edited = dict(src)
    edited["fb_launch.h"] = src["fb_launch.h"].replace("kP1{1, 8,", "kP1{1, 4,", 1)
    assert edited["fb_launch.h"] != src["fb_launch.h"]
    assert bench.kernel_source_hash(lambda n: edited[n]) != base


def test_hash_follows_build_flags(monkeypatch):
    from paper_2609_24089_amd import build
    base = bench.kernel_source_hash()
    monkeypatch.setattr(build, "SOURCES", [(n, []) for n, _ in build.SOURCES])
    assert bench.kernel_source_hash() != base


def test_code_tokens():
    assert bench.code_tokens("a /* x\n y */ b // z\n  c") == "a b c"


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode != 0
    assert "one GPU" in res.stdout + res.stderr
