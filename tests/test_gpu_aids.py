"""The library's measurement kernels (fp_copy_bytes, fp_gather_rows), which
give the benchmark its same-run ceilings, do what they claim: byte-exact
copies and gathers at sizes that end in every chunk stage (full chunks, both
shrinking tail sizes, a ragged last chunk), for rows that take 12 KiB and
8 KiB chunks, with and without table-row marks on the gathered rows."""

import numpy as np
import pytest

from gpu_common import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def fp():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_23087_amd import flowpool
    return flowpool


@pytest.mark.parametrize("nbytes,row_bytes", [(16, 16), (4096, 7168), (12288 * 5 + 48, 7168),
                                              (117_000_000 // 16 * 16, 7168), (64_000_000, 16384)])
def test_copy_bytes(fp, nbytes, row_bytes):
    say(f"case copy aid: {nbytes} bytes, rows of {row_bytes}")
    g = torch.Generator(device="cuda").manual_seed(nbytes)
    src = torch.randint(-128, 128, (nbytes + 64,), dtype=torch.int8, device="cuda", generator=g)
    dst = torch.zeros(nbytes + 64, dtype=torch.int8, device="cuda")
    fp.fp_copy_bytes(src.data_ptr() + 16, dst, nbytes, row_bytes)
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src[16:16 + nbytes]) and not bool(dst[nbytes:].any())


@pytest.mark.parametrize("n_rows,hidden", [(1, 8), (333, 3584), (16000, 3584), (16001, 3584), (2500, 8192), (7, 5120)])
def test_gather_rows(fp, n_rows, hidden):
    say(f"case gather aid: {n_rows} rows, H={hidden}")
    rng = np.random.default_rng(n_rows)
    table = torch.from_numpy(rng.integers(-2 ** 15, 2 ** 15, size=(4096, hidden), dtype=np.int16)).to("cuda")
    pick = rng.integers(0, 4096, size=n_rows)
    addr = table.data_ptr() + pick.astype(np.int64) * 2 * hidden
    addr |= rng.integers(0, 2, size=n_rows) * (n_rows % 2)      # table-row marks (bit 0) on odd cases
    out = torch.zeros((n_rows + 2, hidden), dtype=torch.int16, device="cuda")
    fp.fp_gather_rows(torch.from_numpy(addr).to("cuda"), n_rows, 2 * hidden, out)
    torch.cuda.synchronize()
    assert torch.equal(out[:n_rows], table[torch.from_numpy(pick).to("cuda")]) and not bool(out[n_rows:].any())
