"""Host-side pieces of bench.py: the gate that keeps a measured HBM-traffic
figure only while the kernel's code is the one it was measured on."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_code_digest_ignores_comments_not_code(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("int f() {\n  return 1;  // one\n}\n")
    b = tmp_path / "b.hip"
    b.write_text("// header\n\nint f() {\n  return 1;\n}\n   // trailing\n")
    c = tmp_path / "c.hip"
    c.write_text("int f() {\n  return 2;\n}\n")
    assert bench.code_digest(a) == bench.code_digest(b)
    assert bench.code_digest(a) != bench.code_digest(c)


def test_traffic_records_name_existing_sources():
    for (workload, kernel), (nbytes, src, digest) in bench.MEASURED_TRAFFIC.items():
        assert os.path.exists(os.path.join(ROOT, src))
        assert nbytes > 0 and len(digest) == 16
