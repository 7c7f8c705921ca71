"""One mini-batch through the C ABI from a plain C program (no Python, no
torch in the process that runs it): tests/c_consumer/consumer.c builds the
CSR and the degree-ranked cache, samples (Eq. 2), gathers F_L's rows
(Section 3.2's cache step) and runs the 2-layer SAGE forward (Eq. 1).
Frontier sizes and hit/miss counts must equal the oracle's exactly, the
logits within the fp32 bound."""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W
from parity_util import FP32_TOL, assert_rows_close

HERE = os.path.dirname(os.path.abspath(__file__))
BIN = os.path.join(HERE, "c_consumer", "consumer")


def say(*a):
    print("[c consumer]", *a, flush=True)
    sys.stdout.flush()


def write_problem(path, n, src, dst, feats, fanouts, dims, seeds, ws, r, rng_seed):
    with open(path, "wb") as f:
        np.array([n, src.size, feats.shape[1], len(fanouts), seeds.size], np.int64).tofile(f)
        np.array([r], np.float64).tofile(f)
        np.array([rng_seed], np.uint64).tofile(f)
        src.astype(np.int32).tofile(f)
        dst.astype(np.int32).tofile(f)
        np.ascontiguousarray(feats, np.float32).tofile(f)
        np.array(fanouts, np.int32).tofile(f)
        np.array(dims, np.int32).tofile(f)
        seeds.astype(np.int32).tofile(f)
        for w in ws:
            np.ascontiguousarray(w, np.float32).tofile(f)


@pytest.mark.gpu
@pytest.mark.parametrize("fanouts,r", [([7, 3], 0.3), ([25, 10], 0.0), ([5, 70], 1.0)])
def test_c_program_matches_oracle(tmp_path, fanouts, r):
    assert os.path.exists(BIN), "tests/c_consumer/consumer is not built (python tests/c_consumer/build.py)"
    n, d = 3000, 64
    n, src, dst = W.random_graph(n, 40000, 11)
    feats = W.features(n, d, "f32", seed=12)
    dims = [d, 48, 16]
    ws = [W.glorot(dims[l], dims[l + 1], "f32", seed=13 + l) for l in range(2)]
    seeds = np.random.default_rng(14).integers(0, n, 300).astype(np.int32)   # with repeats
    rng_seed = W.rng_seed_for_batch(3)
    prob, out = str(tmp_path / "problem.bin"), str(tmp_path / "out.bin")
    write_problem(prob, n, src, dst, feats, fanouts, dims, seeds, ws, r, rng_seed)
    say("run", fanouts, r)
    res = subprocess.run([BIN, prob, out], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, f"consumer exited {res.returncode}: {res.stderr}"
    raw = np.fromfile(out, np.int64, count=len(fanouts) + 1 + 3)
    sizes, counts = raw[:len(fanouts) + 1].tolist(), raw[len(fanouts) + 1:]
    logits = np.fromfile(out, np.float32, offset=8 * raw.size).reshape(sizes[0], dims[-1])

    csr = O.build_csr(n, src, dst)
    ref_b = O.sample_blocks(csr, seeds, fanouts, rng_seed)
    _, slot, _ = O.rank_cache(csr, r)
    h0, ref_counts = O.gather(feats, slot, ref_b.nodes)
    assert sizes == list(ref_b.sizes)
    assert np.array_equal(counts, ref_counts)
    ref = O.sage_forward(ref_b, O.to_f64(h0, "f32"), [O.to_f64(w, "f32") for w in ws])
    worst = assert_rows_close(logits, ref, FP32_TOL, "logits")
    say("ok", sizes, counts.tolist(), f"worst row {worst:.2e}")


def test_c_program_built_against_the_tree_library():
    """The consumer links this tree's libgnnav.so and the HIP runtime, and
    rejects a bad command line before any device work.  (On the CPU the
    program is compiled here if the build step has not made it yet.)"""
    if not os.path.exists(BIN):
        subprocess.run([sys.executable, os.path.join(HERE, "c_consumer", "build.py")], check=True, timeout=300)
    ldd = subprocess.run(["ldd", BIN], capture_output=True, text=True, timeout=60).stdout
    lib = [l for l in ldd.splitlines() if "libgnnav.so" in l]
    assert lib and os.path.realpath(lib[0].split("=>")[1].split("(")[0].strip()) == os.path.realpath(
        os.path.join(os.path.dirname(HERE), "paper_2404_09544_amd", "libgnnav.so"))
    assert any("libamdhip64" in l for l in ldd.splitlines())
    res = subprocess.run([BIN], capture_output=True, text=True, timeout=60)
    assert res.returncode == 2 and "usage" in res.stderr
