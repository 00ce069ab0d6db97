"""Host logic of bench.py that needs no GPU: the counter profiles apply only to
the kernel they were taken on (its sources, code only, and the flags its
.hip files compile with), and the committed mid profile matches the current
sources."""
import bench
from paper_2608_12146_amd import build as B


def test_profile_hash_ignores_comments_only():
    src = "int a; // note\n\n  int b;  \n"
    assert bench._code_text(src) == "int a;\n  int b;"
    assert bench._code_text('const char *s = "//x";') == 'const char *s = "//x";'


def test_profile_hash_covers_compile_flags(monkeypatch):
    h0 = bench.kernel_source_hash("chain_run")
    monkeypatch.setitem(B.FILE_FLAGS, "rp_anneal_chain.hip", ["-mllvm", "-amdgpu-sched-strategy=max-ilp"])
    assert bench.kernel_source_hash("chain_run") != h0
    monkeypatch.setitem(B.FILE_FLAGS, "rp_anneal_chain.hip", [])
    assert bench.kernel_source_hash("chain_run") != h0


def test_committed_mid_profile_matches_the_sources():
    pmc = bench.read_pmc("chain_run", "mid")
    assert pmc is not None and pmc > 0
