"""Host-side contract checks that need no GPU: the package refuses to load
without its HIP library (there is no CPU fallback), shares torch's HIP
runtime whatever the import order, and bench.py measures one GPU only."""
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_package_import_fails_without_the_library(tmp_path):
    pkg = tmp_path / "paper_2404_09544_amd"
    pkg.mkdir()
    for f in ("__init__.py", "step.py"):
        shutil.copy(os.path.join(ROOT, "paper_2404_09544_amd", f), pkg / f)
    r = subprocess.run([sys.executable, "-c", "import paper_2404_09544_amd"], cwd=tmp_path,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "is not built" in r.stderr


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr


def test_one_hip_runtime_whatever_the_import_order():
    """Importing the package before torch must not load a second HIP runtime
    next to the copy that ships with torch."""
    code = ("import paper_2404_09544_amd, torch\n"
            "libs = {l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}\n"
            "print(len(libs)); print(sorted(libs))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.splitlines()[0] == "1", r.stdout


def test_bench_pipeline_choice():
    """bench.py's pipelined legs: forced settings are taken as given, and in
    auto mode every candidate is timed and the fastest kept (a stand-in
    pipeline whose batches take a known time per setting)."""
    import argparse
    import time as _time
    sys.path.insert(0, ROOT)
    import bench

    class FakeCuda:
        @staticmethod
        def synchronize():
            pass

    class FakeTorch:
        cuda = FakeCuda

    cost = {(False, 3): 0.004, (True, 2): 0.001, (True, 3): 0.003}
    made = []

    class FakePipe:
        def __init__(self, depth, part):
            self.key = (part, depth)
            made.append(self)

        def enqueue(self, b):
            _time.sleep(cost[self.key])

        def synchronize(self):
            pass

    def run(**kw):
        a = argparse.Namespace(cu_partition="auto", depth=None)
        for k, v in kw.items():
            setattr(a, k, v)
        return bench.pick_pipeline(a, lambda d, p: FakePipe(d, p), lambda p, b: p.enqueue(b), 4, FakeTorch,
                                   n_time=3)

    assert run(cu_partition="on")[:2] == (True, 2)
    assert run(cu_partition="off")[:2] == (False, 3)
    assert run(cu_partition="on", depth=4)[:2] == (True, 4)
    made.clear()
    part, depth, trial = run()
    assert (part, depth) == (True, 2)
    assert set(trial) == {"all_units_3", "shares_2", "shares_3"}
    assert min(trial, key=trial.get) == "shares_2"
    assert len(made) == 3
    made.clear()
    part, depth, trial = run(depth=3)
    assert depth == 3 and set(trial) == {"all_units_3", "shares_3"} and part is True
