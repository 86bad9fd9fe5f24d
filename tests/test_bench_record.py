"""The counter record's source hash (bench.gemm_code_sha): it survives edits of
comments and layout, and changes with any edit of the code."""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402

SRC = """// header
__global__ void k(float* p) {  // trailing
  /* block
     comment */ p[threadIdx.x] = 1.f;
}
"""


def _sha(tmp_path, text, name):
    f = tmp_path / name
    f.write_text(text)
    return bench.gemm_code_sha(str(f))


def test_comment_and_layout_edits_keep_the_hash(tmp_path):
    base = _sha(tmp_path, SRC, "a.hip")
    edited = SRC.replace("// header", "// another header").replace("/* block", "/* other block")
    relaid = SRC.replace("  /* block", "\n\n    /* block").replace("{  //", "{ //")
    assert _sha(tmp_path, edited, "b.hip") == base
    assert _sha(tmp_path, relaid, "c.hip") == base


def test_code_edits_change_the_hash(tmp_path):
    base = _sha(tmp_path, SRC, "a.hip")
    assert _sha(tmp_path, SRC.replace("1.f", "2.f"), "b.hip") != base
    assert _sha(tmp_path, SRC.replace("threadIdx.x", "threadIdx.y"), "c.hip") != base


def test_library_source_hashes():
    assert len(bench.gemm_code_sha()) == 64


def test_traffic_record_is_for_the_b7_step_only():
    # the committed counters were taken on the 1,920-row b7 verify step; other
    # workloads (stress, small) get no traffic figure from them
    assert bench.gemm_traffic("gate/up GEMM", "stress") is None
    assert bench.gemm_traffic("gate/up GEMM", "small") is None
    assert bench.gemm_traffic("no such kernel", "b7") is None
