"""One HIP runtime per process: the library binds to torch's HIP runtime
whichever of the two is imported first (two HSA runtimes in one process
cannot both open the device). Runs the import orders in child processes."""

import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SCRIPT = """
import sys
sys.path.insert(0, {root!r})
{first}
{second}
x = torch.ones(4, device="cuda")
torch.cuda.synchronize()
p = flowpool.pool_create(hidden=64, page_tokens=4, hbm_pages=4, vocab=10)
flowpool.pool_destroy(p)
maps = open("/proc/self/maps").read()
print("runtimes", len(set(l.split()[-1] for l in maps.splitlines() if "libhsa-runtime64" in l)))
"""


@pytest.mark.parametrize("library_first", [True, False])
def test_one_runtime_either_import_order(library_first):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = "from paper_2606_23087_amd import flowpool"
    tor = "import torch"
    code = SCRIPT.format(root=ROOT, first=lib if library_first else tor, second=tor if library_first else lib)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "runtimes 1" in r.stdout, r.stdout
