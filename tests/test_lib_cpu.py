"""The C-ABI library without a GPU: it loads, exports every entry point the
header declares, and its host-only greedy partition equals the oracle's."""

import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from oracle.plan import cost_scaled, greedy_partition, zigzag_partition

fp = pytest.importorskip("paper_2606_23087_amd.flowpool",
                         reason="libflowpool.so not built (run __graft_entry__.build())")


def _declared():
    src = open(os.path.join(ROOT, "include", "flowpool.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:fp_status|int32_t|const char\s*\*|void)\s+(\w+)\s*\(", src, flags=re.M)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert {"pool_create", "pool_write_sample", "pool_free_sample", "plan_microbatches",
            "pack_microbatch"} <= set(names)
    lib = ctypes.CDLL(fp.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(fp.EXPORTED)
    assert fp.fp_abi_version() == fp.ABI_VERSION == 5


def test_constants_match_header():
    """Every FP_* enumerator of the header has the same value in the bindings."""
    src = open(os.path.join(ROOT, "include", "flowpool.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    consts = {}
    for body in re.findall(r"enum\s*\{(.*?)\}", src, flags=re.S):
        for name, val in re.findall(r"(FP_\w+)\s*=\s*(-?\d+)", body):
            consts[name] = int(val)
    assert len(consts) == 17
    for name, val in consts.items():
        assert getattr(fp, name) == val, name
    assert int(re.search(r"#define FP_ABI_VERSION (\d+)", src).group(1)) == fp.ABI_VERSION


def test_config_struct_matches_header():
    # fp_pool_config: 2*i32, 2*i64, 2*i32, i64, u64, 2*i32, 2*i64, u64, i64, 2 ptrs, 2*i32
    assert ctypes.sizeof(fp.fp_pool_config) == 8 + 16 + 8 + 8 + 8 + 8 + 16 + 8 + 8 + 16 + 8


@pytest.mark.parametrize("policy", ["lpt", "zigzag"])
@pytest.mark.parametrize("seed", range(30))
def test_plan_partition_equals_oracle(seed, policy):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 300))
    M = int(rng.integers(1, 70))
    K = int(rng.integers(1, 9000))
    lengths = rng.integers(1, 5000, size=n)
    if seed % 3 == 0 and n:
        lengths = rng.choice([100, 200, 300], size=n)       # many ties
    C = int(rng.integers(5000, 40000))
    costs = [cost_scaled(int(l), K) for l in lengths]
    if policy == "lpt":
        got = fp.plan_partition(lengths, costs, C, M)
        assign, tok, cst = greedy_partition([int(x) for x in lengths], K, C, M)
    else:
        got = fp.plan_partition(lengths, costs, C, M, fp.FP_PLAN_ZIGZAG)
        assign, tok, cst = zigzag_partition([int(x) for x in lengths], K, C, M)
    assert got["assign"].tolist() == assign
    assert got["mb_tokens"].tolist() == tok and got["mb_cost_scaled"].tolist() == cst
    mx = [max([int(lengths[i]) for i in range(n) if assign[i] == j], default=0) for j in range(M)]
    assert got["mb_max_len"].tolist() == mx


def test_plan_partition_errors():
    with pytest.raises(fp.FlowPoolError) as e:
        fp.plan_partition([1, 2], [1, 2], 10, 0)
    assert e.value.code == "EINVAL"
    with pytest.raises(fp.FlowPoolError) as e:
        fp.plan_partition([0], [0], 10, 1)
    assert e.value.code == "EINVAL"
    assert fp.plan_partition([], [], 10, 2)["mb_tokens"].tolist() == [0, 0]
    with pytest.raises(fp.FlowPoolError) as e:
        fp.plan_dynamic_packing([5, 6], 10, (1 << 20) + 1, 2)
    assert e.value.code == "EINVAL"
    for bad in (dict(policy=2), dict(policy=-1), dict(n_mb=(1 << 20) + 1)):
        args = dict(lengths=[1], costs_scaled=[1], capacity=10, n_mb=2)
        args.update(bad)
        with pytest.raises(fp.FlowPoolError) as e:
            fp.plan_partition(**args)
        assert e.value.code == "EINVAL"


def test_pool_create_rejects_bad_config_without_gpu():
    # Argument checks come before any device call.
    for kw in [dict(hidden=4), dict(hidden=12), dict(page_tokens=0), dict(hbm_pages=0),
               dict(alloc=7), dict(world_size=2), dict(pack_cus=-1), dict(meta_bytes=(1 << 33) + 16)]:
        args = dict(hidden=256, page_tokens=16, hbm_pages=4)
        args.update(kw)
        with pytest.raises(fp.FlowPoolError) as e:
            fp.pool_create(**args)
        assert e.value.code == "EINVAL"


def test_null_pool_is_rejected_by_every_pool_call():
    """Every call taking a pool answers EINVAL for a null pool (no device use)."""
    lib = ctypes.CDLL(fp.LIB_PATH)
    n = ctypes.c_int64()
    assert lib.pool_reclaim(None, 0, ctypes.byref(n)) == fp.FP_EINVAL
    assert lib.pool_migrate(None, None, 0, 0, None, None) == fp.FP_EINVAL
    assert lib.plan_pool_packing(None, None, 0, 10, 1, 1, None, None, None, None, None, None, None,
                                 None) == fp.FP_EINVAL
    assert lib.pool_free_sample(None, ctypes.c_uint64(1)) == fp.FP_EINVAL
    assert lib.pack_microbatch(None, None, 0, None, ctypes.c_int64(0), None, ctypes.c_int64(0), None, None,
                               None, None, 3, None) == fp.FP_EINVAL
    assert lib.pack_microbatch_noalloc(None, None, 0, None, ctypes.c_int64(0), None, ctypes.c_int64(0), None, None,
                                       None, None, 3, None) == fp.FP_EINVAL
    assert lib.pool_release_captured(None, None, 0) == fp.FP_EINVAL
    assert lib.pool_forget_stream(None, None) == fp.FP_EINVAL
    assert "null" in fp.fp_last_error()
    assert fp.pool_destroy(0) is None                          # NULL is accepted


def test_measurement_aids_check_arguments_before_the_device():
    """fp_copy_bytes and fp_gather_rows refuse bad sizes and alignments
    before any HIP call (so this runs without a GPU)."""
    lib = ctypes.CDLL(fp.LIB_PATH)
    lib.fp_copy_bytes.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
    lib.fp_gather_rows.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    a, b = 1 << 20, 2 << 20                                    # addresses are never dereferenced here
    assert lib.fp_copy_bytes(a, b, 24, 16, None) == fp.FP_EINVAL           # not a multiple of 16
    assert lib.fp_copy_bytes(a, b, -16, 16, None) == fp.FP_EINVAL
    assert lib.fp_copy_bytes(a, b, (1 << 35), 16, None) == fp.FP_EINVAL     # more than 2^31 - 1024 vectors
    assert lib.fp_copy_bytes(a, b, 32, 8, None) == fp.FP_EINVAL            # row_bytes not a multiple of 16
    assert lib.fp_copy_bytes(None, b, 32, 16, None) == fp.FP_EINVAL
    assert lib.fp_copy_bytes(a + 8, b, 32, 16, None) == fp.FP_EALIGN
    assert lib.fp_gather_rows(a, -1, 16, b, None) == fp.FP_EINVAL
    assert lib.fp_gather_rows(a, 4, 24, b, None) == fp.FP_EINVAL
    assert lib.fp_gather_rows(a, 1 << 30, 1024, b, None) == fp.FP_EINVAL   # too many vectors
    assert lib.fp_gather_rows(None, 4, 16, b, None) == fp.FP_EINVAL
    assert lib.fp_gather_rows(a + 4, 4, 16, b, None) == fp.FP_EALIGN
    assert lib.fp_gather_rows(a, 4, 16, b + 8, None) == fp.FP_EALIGN


def test_bindings_refuse_ordinary_host_tensors():
    """Tensors handed to a kernel must be device or pinned memory; an ordinary
    CPU tensor is refused before the library is called."""
    torch = pytest.importorskip("torch")
    with pytest.raises(ValueError):
        fp._ptr(torch.zeros(8, dtype=torch.int16))
    assert fp._ptr(None) is None and fp._ptr(4096) == 4096
    x = torch.zeros((4, 8), dtype=torch.int16)
    with pytest.raises(ValueError, match="contiguous"):
        fp._buf(x.t(), 64, "out_emb")
    with pytest.raises(ValueError, match="needs 65"):
        fp._buf(x, 65, "out_emb")


def test_pool_create_checks_backing_tensors_before_the_library():
    torch = pytest.importorskip("torch")
    small = torch.zeros(4 * 16 * 512 - 1, dtype=torch.uint8)       # one byte short of 4 pages
    with pytest.raises(ValueError, match="hbm_backing"):
        fp.pool_create(hidden=256, page_tokens=16, hbm_pages=4, hbm_backing=small)
    with pytest.raises(ValueError, match="host_backing"):
        fp.pool_create(hidden=256, page_tokens=16, hbm_pages=4, host_pages=4, host_backing=small)


def test_pool_create_rejects_gva_span_beyond_2_52():
    with pytest.raises(fp.FlowPoolError) as e:
        fp.pool_create(hidden=1 << 20, page_tokens=1 << 20, hbm_pages=1 << 20)
    assert e.value.code == "EINVAL"


def test_c_driver_fails_loudly_without_a_device(tmp_path):
    """The plain-C driver of the C ABI links and runs; with no usable GPU its
    first pool call fails and it exits 1 with the library's message."""
    import os
    import struct
    import subprocess
    drv = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "c_abi", "pack_driver")
    if not os.path.exists(drv):
        pytest.skip("driver not built")
    r = subprocess.run([drv], capture_output=True, text=True, timeout=60)
    assert r.returncode == 1 and "usage" in r.stderr
    import torch
    if torch.cuda.device_count() > 0:
        pytest.skip("a GPU is present (the GPU test drives it)")
    src = tmp_path / "in.bin"
    src.write_bytes(struct.pack("<7i", 8, 4, 1, 1, 16, 1, 16) + bytes(16) + struct.pack("<3i", 1, 0, 0))
    r = subprocess.run([drv, str(src), str(tmp_path / "out.bin")], capture_output=True, text=True, timeout=60)
    assert r.returncode == 1 and "pool_create failed" in r.stderr
