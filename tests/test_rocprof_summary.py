"""Host logic of the profile summaries: the recorded HBM traffic and VALU
instruction counts are used only while the sources their kernel is built from
are unchanged."""
import os

from paper_2202_01258_amd import rocprof_summary as R

VARY = "k_vary_eval<2, false, false, 4>"
ROLL = "k_rollout<64, false, false>"


def test_digest_covers_the_rollout_header_only_for_policy_kernels():
    assert R.sources_digest(VARY) == R.sources_digest("k_insert<1, 2>")
    assert R.sources_digest(VARY) != R.sources_digest(ROLL)
    assert R.sources_digest(ROLL) == R.sources_digest("k_regen_mlp<false>")


def test_recorded_traffic_matches_kernel_and_digest(tmp_path):
    f = tmp_path / "t.txt"
    f.write_text("header line\n"
                 f"{R.TRAFFIC_TAG} 1234 {R.sources_digest(VARY)} {VARY}\n"
                 f"{R.TRAFFIC_TAG} 99 {'0' * 64} {ROLL}\n")
    assert R.recorded_traffic(str(f), VARY) == 1234.0
    assert R.recorded_traffic(str(f), ROLL) is None          # other sources
    assert R.recorded_traffic(str(f), "k_other") is None     # not recorded
    assert R.recorded_traffic(str(tmp_path / "absent.txt"), VARY) is None


def test_recorded_valu_matches_kernel_and_digest(tmp_path):
    f = tmp_path / "sq.txt"
    f.write_text(f"{R.TRAFFIC_TAG} 5 {R.sources_digest(VARY)} {VARY}\n"
                 f"{R.VALU_TAG} 49168434 {R.sources_digest(VARY)} {VARY}\n"
                 f"{R.VALU_TAG} 7 {'f' * 64} {ROLL}\n")
    assert R.recorded_valu(str(f), VARY) == 49168434.0   # its own tag, not traffic's
    assert R.recorded_traffic(str(f), VARY) == 5.0
    assert R.recorded_valu(str(f), ROLL) is None
    assert R.recorded_valu(str(tmp_path / "absent.txt"), VARY) is None


def test_committed_summaries_name_their_kernel():
    root = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles")
    for name in os.listdir(root):
        if not name.endswith("_hbm_traffic.txt"):
            continue
        with open(os.path.join(root, name)) as fh:
            tagged = [ln.split(maxsplit=3) for ln in fh if ln.startswith(R.TRAFFIC_TAG)]
        assert len(tagged) == 1, name
        assert name.startswith(tagged[0][3].split("<")[0].strip()), name


def test_digest_ignores_comments_and_layout_but_not_code(tmp_path):
    a = tmp_path / "a.hpp"
    b = tmp_path / "b.hpp"
    c = tmp_path / "c.hpp"
    a.write_text('// note\nint f(int x) { return x + 1; }  /* one */\nconst char* s = "// kept";\n')
    b.write_text('int f(int x) {\n  return x + 1;   // a different note\n}\nconst char* s = "// kept";\n')
    c.write_text('int f(int x) { return x + 2; }\nconst char* s = "// kept";\n')
    assert R._code_text(str(a)) == R._code_text(str(b))
    assert R._code_text(str(a)) != R._code_text(str(c))
    assert b'"// kept"' in R._code_text(str(a))


def test_split_per_archive():
    rows = [("copy", 0, 5), ("k_clear_archive(a)", 10, 11), ("k_vary_eval<2>", 12, 20),
            ("k_vary_eval<2>", 21, 25), ("k_clear_archive(a)", 30, 31), ("k_vary_eval<2>", 32, 42)]
    runs = R.split_per_archive(list(reversed(rows)))
    assert [len(r) for r in runs] == [1, 3, 2]
    assert runs[1][1:] == [("k_vary_eval<2>", 8), ("k_vary_eval<2>", 4)]
    assert runs[2] == [("k_clear_archive(a)", 1), ("k_vary_eval<2>", 10)]
