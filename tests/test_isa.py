"""Checks on the gfx950 assembly the compiler makes of the library's kernels
(CPU only: hipcc cross-compiles).

- Every inline-asm 16-byte store is followed, inside its asm block, by the
  two wait states gfx940-class parts need before a VALU instruction may
  overwrite the store's data registers (the compiler cannot see into asm,
  so it does not insert them).
- The pack kernels spill nothing to scratch and stay within the registers
  that keep 8 waves per SIMD resident.
- The pack kernels' leading scalar arguments (13 dwords) arrive preloaded in
  scalar registers, and the first loads of the row lookup (the bucket's run and
  index entry) are issued before the wait for the other kernel arguments, so the two are in
  flight together.
"""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_23087_amd", "csrc")


@pytest.fixture(scope="module")
def isa(tmp_path_factory):
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    if not os.path.exists(hipcc) and not shutil.which("hipcc"):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "kernels.s"
    from paper_2606_23087_amd.build import HIPCC_FLAGS
    flags = [f for f in HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    cmd = [hipcc, *flags, "--cuda-device-only", "-S",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, "kernels.hip"), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def _kernels(text):
    """name -> (body lines, metadata text) for every kernel in the assembly."""
    out = {}
    for m in re.finditer(r"^(_ZN2fp\w+):\s*;", text, re.M):
        name = m.group(1)
        body = text[m.end():text.index("s_endpgm", m.end())]
        meta = text[text.index(f".amdhsa_kernel {name}"):]
        meta = meta[:meta.index(".end_amdhsa_kernel")]
        out[name] = (body.splitlines(), meta)
    return out


def test_asm_stores_carry_their_wait_states(isa):
    kernels = _kernels(isa)
    assert any("k_pack" in k for k in kernels) and any("k_write" in k for k in kernels)
    n = 0
    for name, (lines, _) in kernels.items():
        for i, line in enumerate(lines):
            if "global_store_dwordx4" in line and "sc1 nt" in line:
                n += 1
                nxt = lines[i + 1].strip()
                assert nxt.startswith("s_nop") and int(nxt.split()[1]) >= 1, (name, line, nxt)
    assert n >= 4


def test_pack_kernels_keep_full_occupancy(isa):
    packs = {k: v for k, v in _kernels(isa).items() if "k_pack" in k}
    assert len(packs) == 4                      # 2 and 3 vectors per thread; general and compact arguments
    for name, (_, meta) in packs.items():
        vgpr = int(re.search(r"\.amdhsa_next_free_vgpr (\d+)", meta).group(1))
        scratch = int(re.search(r"\.amdhsa_private_segment_fixed_size (\d+)", meta).group(1))
        assert scratch == 0, name
        assert vgpr <= 64, (name, vgpr)         # 512 VGPRs per lane / 8 waves


def test_pack_kernels_preload_their_head_arguments(isa):
    packs = {k: v for k, v in _kernels(isa).items() if "k_pack" in k}
    assert len(packs) == 4
    for name, (lines, meta) in packs.items():
        assert re.search(r"\.amdhsa_user_sgpr_kernarg_preload_length 13\b", meta), name
        # Entry with preloaded arguments: 256 bytes past the kernel symbol,
        # after the compatibility prologue that loads them for firmware that
        # does not preload. There, the first scalar load that is not a
        # kernel-argument load (the bucket entry) comes before the first wait.
        entry = next(i for i, l in enumerate(lines) if l.startswith(".LBB") and "_0:" in l)
        body = [l.strip() for l in lines[entry:]]
        first_wait = next(i for i, l in enumerate(body) if l.startswith("s_waitcnt"))
        loads = [l for l in body[:first_wait] if l.startswith("s_load")]
        assert loads and not loads[0].split(",")[1].strip().startswith("s[0:1]"), (name, loads[:3])
