"""Which code may touch the oracle, and bench.py's single-GPU contract (no GPU needed).

The oracle is test infrastructure: the library package, the bench's timed path and
the stored-value reader must not import it (only tests, smoke() and the bench's
CPU-baseline leg run it).
"""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _imports_oracle(stmt: str) -> bool:
    code = f"import sys; {stmt}; print('oracle' in sys.modules)"
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, check=True)
    return out.stdout.strip().splitlines()[-1] == "True"


def test_library_and_bench_path_do_not_import_the_oracle():
    assert not _imports_oracle("import paper_2607_07508_amd")
    assert not _imports_oracle("import bench")
    assert not _imports_oracle("from tests.golden.make_full_logprobs import load, path_for")


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True, text=True)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
