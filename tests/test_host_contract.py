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
