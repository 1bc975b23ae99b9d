"""Host logic of bench.py that decides which committed counter summary applies to the kernel being timed."""
import importlib.util
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    argv = sys.argv
    sys.argv = ["bench.py"]
    try:
        spec.loader.exec_module(mod)
    finally:
        sys.argv = argv
    return mod


def _hash_of(bench, text, tmp_path):
    src = tmp_path / "attn.hip"
    src.write_text(text)
    old = bench.ATTN_SRC
    bench.ATTN_SRC = str(src)
    try:
        return bench.kernel_source_hash()
    finally:
        bench.ATTN_SRC = old


CODE = '''// header comment
#define WAIT() asm volatile("s_waitcnt lgkmcnt(0) // not a comment" ::: "memory")
__global__ void k(int* p) {  /* block
   comment */
  p[0] = 1;  // trailing
}
'''


def test_comment_and_whitespace_edits_keep_the_key(tmp_path):
    b = _bench()
    base = _hash_of(b, CODE, tmp_path)
    edited = CODE.replace("// header comment", "// another header\n// with two lines") \
                 .replace("/* block\n   comment */", "/* reworded */").replace("  p[0] = 1;", "    p[0]   =   1;")
    assert _hash_of(b, edited, tmp_path) == base


def test_code_edits_change_the_key(tmp_path):
    b = _bench()
    base = _hash_of(b, CODE, tmp_path)
    assert _hash_of(b, CODE.replace("p[0] = 1;", "p[0] = 2;"), tmp_path) != base
    # text inside a string literal is code, even when it looks like a comment
    assert _hash_of(b, CODE.replace("// not a comment", "// changed"), tmp_path) != base


def test_committed_summary_matches_the_current_kernel():
    """The committed counter summary of the default workload is keyed to the current attention source,
    so the bench line reports its traffic (a kernel change must come with new counters)."""
    import json
    b = _bench()
    with open(os.path.join(ROOT, "profiles", "attn_traffic.json")) as f:
        entry = json.load(f)["long-720p-401f"]["auto"]
    assert entry["kernel_sha"] == b.kernel_source_hash()
