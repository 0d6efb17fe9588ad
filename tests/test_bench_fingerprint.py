"""The bench's fingerprint of the copy kernels' code, which decides whether its
recorded HBM traffic still applies (else it reports the traffic as null):
comments and blank space do not change it, code does."""
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_module", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_comments_and_spacing_do_not_change_the_fingerprint():
    b = _bench()
    base = ["int f(int a) {\n  return a + 1;  // one more\n}\n", "/* header */\n#define K 2\n"]
    same = ["// a new comment\nint   f(int a)\n{\n  return a + 1;\n}\n", "#define K 2 /* two */\n"]
    assert b.kernels_sha256(base) == b.kernels_sha256(same)


def test_code_changes_the_fingerprint():
    b = _bench()
    base = ["int f(int a) { return a + 1; }\n", "#define K 2\n"]
    assert b.kernels_sha256(base) != b.kernels_sha256(["int f(int a) { return a + 2; }\n", "#define K 2\n"])
    assert b.kernels_sha256(base) != b.kernels_sha256(["int f(int a) { return a + 1; }\n", "#define K 3\n"])

