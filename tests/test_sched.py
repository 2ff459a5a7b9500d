"""The MFMA group schedules compiled into the bf16 heads: the committed
include is what gen_sched.py writes, and every table passes its dependency
check (layer-2 chunks read packed halves, accumulator pairs are free before
reuse, epilogues start after their block's last MFMA and end before the
accumulators are overwritten)."""
import importlib.util
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_28565_amd", "csrc")


def _gen():
    spec = importlib.util.spec_from_file_location("gen_sched", os.path.join(CSRC, "gen_sched.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def test_tables_pass_their_checks_and_cover_every_mfma():
    g = _gen()
    for mb in (4, 8):
        for kc1 in (1, 2):
            t = g.gen_sched(mb, kc1)          # runs check()
            l1 = sorted((x[1], x[2]) for x in t if x[0] == 1)
            l2 = sorted((x[1], x[2]) for x in t if x[0] == 2)
            assert l1 == [(b, k) for b in range(mb) for k in range(kc1)]
            assert l2 == [(b, k) for b in range(mb) for k in range(2 * mb)]
            packs = sorted((x[4], x[5]) for x in t if x[3] == 1)
            assert packs == [(b, h) for b in range(mb) for h in (0, 1)]
            pairs = sorted((x[4], j) for x in t if x[3] == 2 for j in range(x[5], x[5] + x[6]))
            assert pairs == [(b, j) for b in range(mb - 1) for j in range(8)]


def test_committed_include_is_current(tmp_path):
    g = _gen()
    committed = open(os.path.join(CSRC, "ks_sched.inc")).read()
    g_dir = tmp_path / "csrc"
    g_dir.mkdir()
    import shutil
    shutil.copy(os.path.join(CSRC, "gen_sched.py"), g_dir / "gen_sched.py")
    spec = importlib.util.spec_from_file_location("gen_sched_copy", str(g_dir / "gen_sched.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    m.emit()
    assert (g_dir / "ks_sched.inc").read_text() == committed
