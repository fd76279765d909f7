"""The oracle's pins catch plausible mistakes (CPU only).

Each mutant below edits one expression of an oracle module's source: the kind
of slip a hand-written oracle could carry (a dropped term, an index or bound
off by one, a comparison made strict, a tie sent the other way, an order
reversed, two operands swapped). The edited source is executed as a module of
its own and put in place of the real one in the pin modules
(tests/test_oracle_*.py), whose tests are then run: every mutant must make at
least one of them fail. The real source, executed the same way, must pass
them all, so that a mutant's failure comes from its edit. These tests plant
mistakes in the oracle only, and run on the CPU.
"""

import importlib
import inspect
import itertools
import os
import types

import pytest

import oracle

ORACLE_DIR = os.path.dirname(os.path.abspath(oracle.__file__))
PIN_MODULES = ["test_oracle_pack", "test_oracle_pool", "test_oracle_plan", "test_oracle_schedule",
               "test_oracle_allocate"]

# (oracle module, text of the real source, its mutated form, the slip)
MUTANTS = [
    # Definitional pack (Sec. 3.1 pairing, Sec. 4.1 interleaving).
    ("pack", "bounds = [0] + [int(p) for p in img_pos] + [int(n_text)]",
     "bounds = [0] + [int(p) + 1 for p in img_pos] + [int(n_text)]", "placeholder one text token late"),
    ("pack", 'segs.append(("text", bounds[j], bounds[j + 1] - bounds[j]))',
     'segs.append(("text", bounds[j], bounds[j + 1] - bounds[j] - 1))', "text run one token short"),
    ("pack", "vis_start += int(img_ntok[j])", "vis_start += 0", "every image read from visual row 0"),
    ("pack", "sample_parts.append(table[ids])", "sample_parts.append(table[ids - 1])", "table row off by one"),
    ("pack", "sample_parts.append(vis_rows[s][start:start + count])",
     "sample_parts.append(vis_rows[s][start:start + count][::-1])", "image rows reversed"),
    ("pack", "cu.append(cu[-1] + length)", "cu.append(length)", "cu_seqlens without the running sum"),
    ("pack", "pos.extend(range(length))", "pos.extend(range(1, length + 1))", "position ids from 1"),
    ("pack", "max_len = max(max_len, length)", "max_len = length", "max_seqlen of the last sample"),
    ("pack", "for s, spec in enumerate(samples):\n        sample_parts = []",
     "for s, spec in enumerate(samples[::-1]):\n        sample_parts = []", "samples packed in reverse order"),
    ("pack", 'out.append(("vis", s, i))', 'out.append(("vis", s, i + 1))', "symbolic image row one off"),
    ("pack", 'out.append(("text", s, int(spec.text_ids[i])))', 'out.append(("text", s, i))',
     "symbolic text row names its position, not its id"),
    # Pool: GVA addressing, page table, allocators, walk, tiers (Sec. 3.2).
    ("pool", "base = self.gva_start + ((gva - self.gva_start) // self.pb) * self.pb",
     "base = self.gva_start + ((gva - self.gva_start) // self.pb + 1) * self.pb", "translation to the next page"),
    ("pool", "gva = s.pages[v // self.P] + (v % self.P) * self.rb\n        tier, frame, off = self.translate(gva)\n"
             "        page = self.frames[tier].get(frame)\n        if page is None:\n            return",
     "gva = s.pages[v // self.P] + (v % self.P) * self.hidden\n        tier, frame, off = self.translate(gva)\n"
     "        page = self.frames[tier].get(frame)\n        if page is None:\n            return",
     "row offset in elements instead of bytes"),
    ("pool", "while j < k and s.img_pos[j] == t:", "while j < k and s.img_pos[j] == t + 1:",
     "walk places images one text token early"),
    ("pool", "            i = self.stack[t].pop()\n            self.used[t][i] = True\n            out.append",
     "            i = self.stack[t].pop(0)\n            self.used[t][i] = True\n            out.append",
     "scatter allocator FIFO instead of LIFO"),
    ("pool", "        for gva in reversed(s.pages):\n            t, i = self._page_of(gva)\n            self.used[t][i] = False\n"
             "            if self.alloc",
     "        for gva in s.pages:\n            t, i = self._page_of(gva)\n            self.used[t][i] = False\n"
     "            if self.alloc", "free gives its pages back first page first"),
    ("pool", "first = i - n + 1", "first = i - n", "contiguous run starts one page early"),
    ("pool", "        for t in (0, 1):\n            used = self.used[t]", "        for t in (1, 0):\n            used = self.used[t]",
     "contiguous pages taken from the host tier first"),
    ("pool", "for i in range(self.n_pages[t]):\n                run = 0 if used[i] else run + 1",
     "for i in range(self.n_pages[t] - 1, -1, -1):\n                run = 0 if used[i] else run + 1",
     "first fit searched from the highest page"),
    ("pool", "run = 0 if used[i] else run + 1", "run = 0 if used[i] else run + 2", "contiguous run counted twice"),
    ("pool", "want = MASK_HBM if tier == TIER_HBM else MASK_HOST", "want = MASK_HOST if tier == TIER_HBM else MASK_HBM",
     "tier mask bits swapped"),
    ("pool", "if tier_mask & MASK_HBM:\n                        out[r] = table[x]",
     "if tier_mask & MASK_HOST:\n                        out[r] = table[x]", "text rows taken as host-tier rows"),
    ("pool", "pos.append(local)", "pos.append(r)", "position ids that do not restart per sample"),
    ("pool", "        for gva in reversed(old):", "        for gva in old:", "migration returns its pages first page first"),
    ("pool", "t = int(wish[j]) if wish is not None else TIER_HBM", "t = 1 - int(wish[j]) if wish is not None else TIER_HBM",
     "tier wishes inverted"),
    ("pool", "return t, (gva - self.seg_start[t]) // self.pb", "return t, (gva - self.seg_start[t]) // self.rb",
     "page index from a row size"),
    ("pool", "moving = [k for k, gva in enumerate(s.pages) if self._page_of(gva)[0] != tier]",
     "moving = [k for k, gva in enumerate(s.pages) if self._page_of(gva)[0] == tier]", "migration moves the wrong pages"),
    ("pool", "self.frames[nt][nf] = self.frames[ot][of].copy()", "self.frames[nt][nf] = self.frames[ot][of] * 0",
     "migration drops the bytes"),
    ("pool", "max_len = max((s.length for s in recs), default=0)", "max_len = sum((s.length for s in recs))",
     "max_seqlen as the total"),
    ("pool", "if out_rows_cap is not None and total > out_rows_cap:", "if out_rows_cap is not None and total >= out_rows_cap:",
     "a microbatch that exactly fills the output refused"),
    ("pool", "if p < 0 or p > T or (j and p < img_pos[j - 1]):", "if p < 0 or p >= T or (j and p < img_pos[j - 1]):",
     "an image after the last text token refused"),
    ("pool", "page[off // self.rb] = vis_rows[v]", "page[(off // self.rb) ^ 1] = vis_rows[v]",
     "producer rows swapped in pairs inside a page"),
    ("pool", "self.region_start = [gva_start, gva_start + world_size * self.max_size[0]]",
     "self.region_start = [gva_start, gva_start + self.max_size[0]]", "DRAM region after one rank's HBM segment"),
    ("pool", "self.seg_start = [self.region_start[t] + rank * self.max_size[t] for t in (0, 1)]",
     "self.seg_start = [self.region_start[t] + rank * self.max_size[0] for t in (0, 1)]",
     "rank segments sized by the HBM tier"),
    ("pool", "self.pb = page_tokens * self.rb", "self.pb = page_tokens * self.hidden", "page size in elements"),
    ("pool", "n_pages = -(-n_vis // self.P)", "n_pages = n_vis // self.P", "partial last page not allocated"),
    ("pool", "if len(moving) > len(self.stack[tier]):", "if len(moving) >= len(self.stack[tier]):",
     "a migration that exactly fits refused"),
    ("pool", "self.stack = [list(range(self.n_pages[0] - 1, -1, -1)),",
     "self.stack = [list(range(self.n_pages[0])),", "HBM stack pops the highest page first"),
    ("pool", "if self.vocab is not None and T and (text_ids.min() < 0 or text_ids.max() >= self.vocab):",
     "if self.vocab is not None and T and (text_ids.min() < 0 or text_ids.max() > self.vocab):",
     "a text id equal to the vocabulary size accepted"),
    ("pool", "self.page_table[self.seg_start[t] + i * self.pb] = (t, order[i])",
     "self.page_table[self.seg_start[t] + i * self.pb] = (t, i)", "frame order ignored"),
    # Planner: per-sample cost, Eq. 3, greedy and zig-zag partitions.
    ("plan", "return k * length + length * length", "return k * length + length", "cost without the square"),
    ("plan", "return sum(lengths) / capacity + (max(lengths) ** 2) / (capacity ** 2)",
     "return sum(lengths) / capacity + (max(lengths) ** 2) / capacity", "Eq. 3 with L instead of L squared"),
    ("plan", "            if tokens[j] + int(lengths[i]) <= capacity:\n                if best < 0",
     "            if tokens[j] + int(lengths[i]) < capacity:\n                if best < 0", "capacity made strict"),
    ("plan", "if best < 0 or mb_cost[j] < mb_cost[best]:", "if best < 0 or mb_cost[j] <= mb_cost[best]:",
     "cost ties go to the higher microbatch"),
    ("plan", "if best < 0 or mb_cost[j] < mb_cost[best]:", "if best < 0 or mb_cost[j] > mb_cost[best]:",
     "most-loaded instead of least-loaded microbatch"),
    ("plan", "    order = sorted(range(n), key=lambda i: (-costs[i], i))\n    tokens = [0] * n_mb\n    mb_cost = [0] * n_mb\n"
             "    assign = [-1] * n\n    for i in order:",
     "    order = sorted(range(n), key=lambda i: (costs[i], i))\n    tokens = [0] * n_mb\n    mb_cost = [0] * n_mb\n"
     "    assign = [-1] * n\n    for i in order:", "greedy takes the samples cheapest first"),
    ("plan", "    order = sorted(range(n), key=lambda i: (-costs[i], i))\n    tokens = [0] * n_mb\n    mb_cost = [0] * n_mb\n"
             "    assign = [-1] * n\n    for i in order:",
     "    order = sorted(range(n), key=lambda i: (-costs[i], -i))\n    tokens = [0] * n_mb\n    mb_cost = [0] * n_mb\n"
     "    assign = [-1] * n\n    for i in order:", "equal-cost samples taken last index first"),
    ("plan", "return q if q < n_mb else 2 * n_mb - 1 - q", "return q if q < n_mb else 2 * n_mb - q",
     "snake turns one position late"),
    ("plan", "j = snake(p + q, n_mb)", "j = snake(p + q + 1, n_mb)", "snake starts one position late"),
    ("plan", "out[j].append(i)", "out[j].insert(0, i)", "microbatch members in reverse input order"),
    ("plan", "return (max(mb_cost) / mean) if mean > 0 else 1.0", "return (min(mb_cost) / mean) if mean > 0 else 1.0",
     "imbalance from the cheapest microbatch"),
    ("plan", "for q in range(2 * n_mb):", "for q in range(n_mb):", "zig-zag tries half the snake"),
    ("plan", "if tok[j] > capacity:", "if tok[j] >= capacity:", "brute force with a strict capacity"),
    ("plan", "        if all(j < n_mb for j in combo):", "        if any(j < n_mb for j in combo):",
     "brute-force optimum over assignments that defer"),
    ("plan", "key = (packed, -mx)", "key = (packed, mx)", "brute force prefers the costlier maximum"),
    # Alg. 1: best-fit packing, Eq. 3 cost, k-means buckets, zig-zag dealing.
    ("schedule", "if best < 0 or residual[j] < residual[best]:", "if best < 0 or residual[j] > residual[best]:",
     "worst fit instead of best fit"),
    ("schedule", "if best < 0 or residual[j] < residual[best]:", "if best < 0 or residual[j] <= residual[best]:",
     "best-fit ties go to the newer microbatch"),
    ("schedule", "if residual[best] < l_min:", "if residual[best] <= l_min:",
     "a microbatch closed while the shortest sequence still fits"),
    ("schedule", "if is_open[j] and residual[j] >= l:", "if is_open[j] and residual[j] > l:",
     "an exact fit refused"),
    ("schedule", "return capacity * sum(int(x) for x in mb_lengths) + max(int(x) for x in mb_lengths) ** 2",
     "return sum(int(x) for x in mb_lengths) + max(int(x) for x in mb_lengths) ** 2", "Eq. 3 without the factor L"),
    ("schedule", "return capacity * sum(int(x) for x in mb_lengths) + max(int(x) for x in mb_lengths) ** 2",
     "return capacity * sum(int(x) for x in mb_lengths) + sum(int(x) for x in mb_lengths) ** 2",
     "Eq. 3 with the sum squared instead of the longest"),
    ("schedule", "centroid[k] = Fraction(sum(pts), len(pts))", "centroid[k] = Fraction(sum(pts), len(pts) + 1)",
     "k-means centroid is not the mean"),
    ("schedule", "new.append(min(range(k_n), key=lambda k: (dist[k], k)))",
     "new.append(max(range(k_n), key=lambda k: (-dist[k], k)))", "k-means distance ties to the higher bucket"),
    ("schedule", "        forward = not forward", "        forward = True", "dealing round-robin instead of zig-zag"),
    ("schedule", "for b in range(n_b - 1, -1, -1):", "for b in range(n_b):", "buckets dealt cheapest first"),
    ("schedule", "key=lambda j: (-costs[j], j))\n        for j, r in zip",
     "key=lambda j: (costs[j], j))\n        for j, r in zip", "a bucket dealt cheapest first"),
    ("schedule", "centroid = [Fraction(costs[order[(2 * k + 1) * m // (2 * k_n)]]) for k in range(k_n)]",
     "centroid = [Fraction(costs[order[k * m // k_n]]) for k in range(k_n)]", "k-means started at other positions"),
    ("schedule", "            next_slot[r] += 1", "            next_slot[r] += 0", "slots not advanced"),
    ("schedule", "return Fraction(cost_scaled(mb_lengths, capacity), capacity * capacity)",
     "return Fraction(cost_scaled(mb_lengths, capacity), capacity)", "exact Eq. 3 over L"),
    ("schedule", "if bins[b] + ls[i] <= capacity and bins[b] not in seen:",
     "if bins[b] + ls[i] < capacity and bins[b] not in seen:", "optimal bin count with a strict capacity"),
    # Allocator: candidate pruning and the flow matching of Eq. 1-2.
    ("allocate", "g, f = min(t_enc, t_bb), abs(t_enc - t_bb)", "g, f = max(t_enc, t_bb), abs(t_enc - t_bb)",
     "throughput of the faster side instead of the slower"),
    ("allocate", "key = (-g, f, cost, choice)", "key = (-g, -f, cost, choice)", "mismatch maximised"),
    ("allocate", "key = (-g, f, cost, choice)", "key = (f, -g, cost, choice)", "criteria in the wrong order"),
    ("allocate", "key = (-g, f, cost, choice)", "key = (-g, f, -cost, choice)", "more devices preferred on ties"),
    ("allocate", "if cost > budget:", "if cost >= budget:", "budget made strict"),
    ("allocate", "t_enc = sum(enc[i][c][0] for i, c in enumerate(choice[:-1]))",
     "t_enc = max(enc[i][c][0] for i, c in enumerate(choice[:-1]))", "encoder throughputs not summed"),
    ("allocate", "if dp * tp * pp <= devices:", "if dp * tp * pp < devices:", "device bound made strict"),
    ("allocate", "pps = divisors(layers)", "pps = divisors(devices)", "PP degree not tied to the layers"),
    ("allocate", "for tp in divisors(per_node):", "for tp in divisors(devices):", "TP degree across nodes"),
    ("allocate", "return [d for d in range(1, n + 1) if n % d == 0]", "return [d for d in range(1, n) if n % d == 0]",
     "divisors without the number itself"),
    ("allocate", "t_bb = bb[choice[-1]][0]", "t_bb = bb[choice[0]][0]", "backbone throughput read from an encoder's choice"),
    ("allocate", "cost = sum(modules[i][c][1] for i, c in enumerate(choice))",
     "cost = max(modules[i][c][1] for i, c in enumerate(choice))", "resources not summed over the modules"),
]


def _source(name: str) -> str:
    with open(os.path.join(ORACLE_DIR, f"{name}.py")) as f:
        return f.read()


def _module(name: str, src: str) -> types.ModuleType:
    mod = types.ModuleType(f"oracle_mutant_{name}")
    mod.__file__ = os.path.join(ORACLE_DIR, f"{name}.py")
    exec(compile(src, mod.__file__, "exec"), mod.__dict__)
    return mod


def _cases(fn):
    """Argument sets of a pin test from its parametrize marks (tests that need
    other fixtures are left out)."""
    names, sets = [], [()]
    for mark in getattr(fn, "pytestmark", []):
        if mark.name != "parametrize":
            continue
        argnames = mark.args[0]
        argnames = [a.strip() for a in argnames.split(",")] if isinstance(argnames, str) else list(argnames)
        values = [v.values if type(v).__name__ == "ParameterSet" else v for v in mark.args[1]]
        values = [v if len(argnames) > 1 else (v[0] if isinstance(v, tuple) and len(v) == 1 else v,)
                  for v in values]
        names += argnames
        sets = [a + tuple(b) for a, b in itertools.product(sets, values)]
    if set(inspect.signature(fn).parameters) - set(names):
        return []
    return [dict(zip(names, s)) for s in sets]


def _first_failure(replaced, monkeypatch):
    """Runs every pin with the oracle modules in `replaced` (name -> module)
    standing in for the real ones; returns the first failing pin, or None."""
    with monkeypatch.context() as m:
        pins = [importlib.import_module(p) for p in PIN_MODULES]
        for name, mod in replaced.items():
            real = getattr(oracle, name)
            by_id = {id(v): k for k, v in vars(real).items()}
            for pin in pins:
                for attr, val in list(vars(pin).items()):
                    if id(val) in by_id and not attr.startswith("__"):
                        m.setattr(pin, attr, getattr(mod, by_id[id(val)]))
        for pin in pins:
            for tname, fn in sorted(vars(pin).items()):
                if not tname.startswith("test_") or not callable(fn):
                    continue
                for kwargs in _cases(fn):
                    try:
                        fn(**kwargs)
                    except pytest.skip.Exception:
                        pass
                    except (Exception, pytest.fail.Exception) as e:   # noqa: BLE001 - any failure of a pin counts
                        return f"{pin.__name__}.{tname}({kwargs}): {type(e).__name__}"
    return None


def test_real_sources_pass_every_pin(monkeypatch):
    replaced = {name: _module(name, _source(name)) for name in sorted({m[0] for m in MUTANTS})}
    assert _first_failure(replaced, monkeypatch) is None


@pytest.mark.parametrize("name,old,new,slip", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_pins_catch_mutant(name, old, new, slip, monkeypatch):
    src = _source(name)
    assert src.count(old) == 1, f"the text to mutate is not found once in oracle/{name}.py"
    caught = _first_failure({name: _module(name, src.replace(old, new))}, monkeypatch)
    assert caught is not None, f"no pin fails for the mutant '{slip}' of oracle/{name}.py"
