"""The benchmark reports HBM traffic from a committed counter summary only
while the GEMM sources hash to the value recorded with the counters; the
hash covers code, not comments or layout."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402

SRC = """// a kernel
/* block
   comment */
__global__ void k(float* y, const float* x) {  // trailing
  y[threadIdx.x] = 2.0f * x[threadIdx.x];
}
"""


def _hash(tmp_path, text):
    p = tmp_path / "k.hip"
    p.write_text(text)
    return bench.source_hash([str(p)])


def test_comments_and_layout_keep_the_hash(tmp_path):
    h = _hash(tmp_path, SRC)
    edited = SRC.replace("// a kernel", "// a kernel, reworded\n// and longer").replace("/* block", "/* other")
    edited = edited.replace("  y[threadIdx.x]", "\n      y[threadIdx.x]")
    assert _hash(tmp_path, edited) == h


def test_code_changes_alter_the_hash(tmp_path):
    h = _hash(tmp_path, SRC)
    assert _hash(tmp_path, SRC.replace("2.0f", "3.0f")) != h
    assert _hash(tmp_path, SRC.replace("y[threadIdx.x] =", "y[threadIdx.x + 1] =")) != h

