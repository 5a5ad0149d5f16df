"""The benchmark matches committed counter summaries to the kernel code by a
hash of the sources with comments left out: a comment-only edit keeps the
counters, a code edit voids them."""
import bench


def test_strip_comments_keeps_code_and_literals():
    src = ('int a = 1; // note\n/* block\n comment */ const char *s = "a//b /* c */";\n'
           "char q = '\"';\n\n   // only a comment\nint b;  \n")
    assert bench.strip_comments(src) == ('int a = 1;\n const char *s = "a//b /* c */";\n'
                                         "char q = '\"';\nint b;")


def test_hash_ignores_comments_only():
    a = bench.strip_comments("x = 1; // one\n")
    b = bench.strip_comments("// header\nx = 1;    /* two */\n")
    c = bench.strip_comments("x = 2;\n")
    assert a == b and a != c
