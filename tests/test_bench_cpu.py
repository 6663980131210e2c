"""bench.py's host logic: the HBM traffic of a counter summary is reported only
while the kernel sources it was taken with are unchanged."""
import importlib.util
import os
import shutil

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(root):
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    b.ROOT = root
    return b


@pytest.fixture
def tree(tmp_path):
    src = os.path.join(ROOT, "paper_2609_26425_amd", "csrc")
    dst = tmp_path / "paper_2609_26425_amd" / "csrc"
    shutil.copytree(src, dst)
    (tmp_path / "profiles").mkdir()
    return tmp_path


def _write_summary(b, tree, name, attend_bytes, append_bytes):
    (tree / "profiles" / f"traffic_{name}.md").write_text(
        "# HBM traffic\n\n"
        f"attend_traffic_bytes_per_launch: {attend_bytes}\n"
        f"attend_source_sha256: {b.source_digest('attend')}\n"
        f"append_traffic_bytes_per_launch: {append_bytes}\n"
        f"append_source_sha256: {b.source_digest('append')}\n")


def test_traffic_reported_while_sources_match(tree):
    b = _bench(str(tree))
    _write_summary(b, tree, "w", 123456, 789)
    assert b.measured_traffic("attend", "w") == 123456
    assert b.measured_traffic("append", "w") == 789
    assert b.measured_traffic("attend", "missing") is None


def test_traffic_withdrawn_when_a_kernel_source_changes(tree):
    b = _bench(str(tree))
    _write_summary(b, tree, "w", 123456, 789)
    # an edit to an append source retires the append figure only
    f = tree / "paper_2609_26425_amd" / "csrc" / "append_bf16.hip"
    f.write_text(f.read_text() + "\n// edited\n")
    assert b.measured_traffic("append", "w") is None
    assert b.measured_traffic("attend", "w") == 123456
    # a header both kernels include retires both
    h = tree / "paper_2609_26425_amd" / "csrc" / "qwm_common.h"
    h.write_text(h.read_text() + "\n// edited\n")
    assert b.measured_traffic("attend", "w") is None


def test_committed_summaries_parse():
    b = _bench(ROOT)
    names = [f[len("traffic_"):-3] for f in os.listdir(os.path.join(ROOT, "profiles")) if f.startswith("traffic_")]
    assert names, "no traffic summaries under profiles/"
    for n in names:
        for k in ("attend", "append"):
            v = b.measured_traffic(k, n)
            assert v is None or (isinstance(v, int) and v > 0), (n, k, v)
