"""Host-side parts of bench.py that decide whether committed traffic
summaries still describe the kernels: the source hash ignores comments and
layout but not code."""
import bench


def test_code_only_strips_comments_and_layout():
    a = 'int a = 1; // note\n/* block\n comment */  int b = 2;\n'
    b = 'int a = 1;\n\n   int b = 2;'
    assert bench._code_only(a) == bench._code_only(b)


def test_code_only_keeps_literals_and_code():
    assert bench._code_only('s = "a // b /* c */";') == 's = "a // b /* c */";'
    assert bench._code_only("c = '/';  d = '\\'';") == "c = '/'; d = '\\'';"
    assert bench._code_only("x = a / b;") != bench._code_only("x = a * b;")


def test_kernel_source_sha_is_stable():
    assert bench.kernel_source_sha() == bench.kernel_source_sha()
    assert len(bench.kernel_source_sha()) == 16
