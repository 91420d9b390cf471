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


def test_alternate_rotates_the_order():
    import bench
    calls = []
    out = bench.alternate({"a": "a", "b": "b"}, lambda f: calls.append(f) or len(calls), 4)
    assert calls == ["a", "b", "b", "a", "a", "b", "b", "a"]
    assert out["a"] == [1, 4, 5, 8] and out["b"] == [2, 3, 6, 7]
    calls.clear()
    bench.alternate({"a": "a", "b": "b", "c": "c"}, lambda f: calls.append(f), 3)
    assert calls == ["a", "b", "c", "b", "c", "a", "c", "a", "b"]


def test_step_bytes_of_the_bench_layer():
    """Algorithmic bytes of the benchmark layer: dX 107.2 MB (dY, W, footprint
    bits, dX) and dW 105.1 MB (X, dY, fp32 dW)."""
    import bench
    import workloads as wl
    spec = wl.config2()[0]
    act = 32 * 56 * 56 * 256 * 2
    w = 256 * 9 * 256
    assert bench.step_bytes(spec) == (act + 2 * w + act // 16 + act) + (act + act + 4 * w)
    assert abs(bench.step_bytes(spec) / 1e6 - 212.27) < 0.01
