"""bench.py's command line on the host: more than one GPU is refused with a
message (this build measures one GPU), and the per-layer dispatch rule picks
the compacting / skipping calls only where an earlier call could skip."""
import os
import subprocess
import sys
import types

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_adaptive_choice():
    import bench
    st = lambda live, total: types.SimpleNamespace(rows_live=live, rows_total=total)
    wt = lambda skipped, total: types.SimpleNamespace(blocks_skipped=skipped, blocks_total=total)
    assert bench.adaptive_choice(st(100, 100), wt(0, 100)) == (False, False)     # nothing to skip
    assert bench.adaptive_choice(st(90, 100), wt(5, 100)) == (True, True)        # at the thresholds
    assert bench.adaptive_choice(st(91, 100), wt(4, 100)) == (False, False)
    assert bench.adaptive_choice(None, wt(50, 100)) == (False, True)             # no data gradient
