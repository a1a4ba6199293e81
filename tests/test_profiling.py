"""Host logic of the measurement: the kernel-source hash that ties the stored
traffic counters to the code they were taken on, and the counter scaling."""
from paper_2501_12162_amd import profiling


def test_hash_ignores_comments_and_whitespace_only():
    code = "int f(int a) {\n  return a + 1;  // one more\n}\n/* block\n comment */\n"
    same = "int f(int a) { return a + 1; }   // another comment\n"
    changed = "int f(int a) { return a + 2; }\n"
    assert profiling._code_only(code) == profiling._code_only(same)
    assert profiling._code_only(code) != profiling._code_only(changed)
    assert profiling._code_only("a/*x*/b") == "a b"


def test_source_hash_is_stable_and_short():
    h = profiling.kernel_source_hash()
    assert h == profiling.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0

