import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def golden_path(name: str) -> str:
    return os.path.join(ROOT, "tests", "golden", name)


def read_golden(name: str):
    """Non-comment, non-empty lines of a golden fixture."""
    with open(golden_path(name)) as f:
        return [ln.rstrip("\n") for ln in f if ln.strip() and not ln.lstrip().startswith("#")]


def golden_solves():
    """The hand-worked flow-matching cases of allocator_flow_example.txt:
    (modules, budget, expected) with modules a list of [(tau, r), ...] per
    module (encoders, then the backbone) and expected either None (nothing
    fits) or (choice, G, F, devices)."""
    out = []
    for ln in read_golden("allocator_flow_example.txt"):
        head, _, tail = ln.partition("->")
        f = head.split()
        if f[0] != "solve":
            continue
        mods = []
        for w in f[3:]:
            if w in ("enc", "bb"):
                mods.append([])
            else:
                t, r = w.split(":")
                mods[-1].append((int(t), int(r)))
        t = tail.split()
        if t == ["NONE"]:
            out.append((mods, int(f[2]), None))
        else:
            gi = t.index("G")
            out.append((mods, int(f[2]), ([int(x) for x in t[:gi]], int(t[gi + 1]), int(t[gi + 3]), int(t[gi + 5]))))
    return out
