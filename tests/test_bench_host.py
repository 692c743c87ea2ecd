"""Host logic of bench.py: the source hash that keys recorded HBM counters
ignores comments and blank lines but not code.  CPU only."""
import os

import bench

CSRC = os.path.join(os.path.dirname(bench.__file__), "paper_2609_19242_amd", "csrc")


def test_strip_comments_keeps_code_and_string_literals():
    src = 'int a = 1; // tail\n/* block\n   comment */ const char* s = "x//y\\"z";\n\n  int b; /* inline */ int c;\n'
    assert bench.strip_comments(src) == 'int a = 1;\n const char* s = "x//y\\"z";\n  int b;  int c;'


def test_comment_edit_leaves_the_stripped_source_alone_and_code_edit_does_not():
    with open(os.path.join(CSRC, "bwd_dkdv.hip"), encoding="utf-8") as f:
        src = f.read()
    base = bench.strip_comments(src)
    commented = src.replace("namespace bdlm {", "// a new comment\nnamespace bdlm {  /* and another */\n\n", 1)
    assert commented != src
    assert bench.strip_comments(commented) == base
    edited = src.replace("constexpr int kStages = 4;", "constexpr int kStages = 3;", 1)
    assert edited != src
    assert bench.strip_comments(edited) != base


def test_every_timed_kernel_has_a_source_list_that_exists():
    for kernel, files in bench.KERNEL_SOURCES.items():
        assert files, kernel
        for f in files:
            assert os.path.exists(os.path.join(CSRC, f)), (kernel, f)
        assert len(bench.kernel_source_hash(kernel)) == 16
