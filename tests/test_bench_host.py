"""Host-side pieces of bench.py: the kernel-source stamp that decides whether
a committed counter summary still applies."""
import bench


def test_code_only_drops_comments_and_blank_lines():
    src = ("// header\n#include <x>\n\nint f() {  // trailing\n  return 1; /* inline */\n}\n"
           "/* block\n   comment */\nint g;\n")
    assert bench._code_only(src) == "#include <x>\nint f() {\n  return 1;\n}\nint g;"


def test_comment_edit_keeps_the_stamp_and_code_edit_changes_it():
    a = "int f(int x) {\n  return x + 1;  // add one\n}\n"
    b = "// adds one\nint f(int x) {\n\n  return x + 1;\n}\n"
    c = "int f(int x) {\n  return x + 2;  // add one\n}\n"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)


def test_every_kernel_kind_has_a_stamp():
    for kind in bench.KERNEL_SOURCES:
        assert len(bench.kernel_sha(kind)) == 64
