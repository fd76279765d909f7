"""Shared helpers for the GPU parity tests: moving uint16 arrays to and from
the device and replaying a workload in the oracle pool."""

import sys

import numpy as np

from oracle.plan import greedy_partition, members
from oracle.pool import OraclePool
from paper_2606_23087_amd.workloads import churn_ops, page_tier_draws


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda")


def to_host(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def oracle_pool_for(cfg, seed, specs, vis_np=None, churn=True, with_bytes=True):
    """Replay the same churn and writes in the oracle pool. Returns (pool, ids)."""
    pool = OraclePool(cfg.hidden, cfg.page_tokens, cfg.hbm_pages, cfg.host_pages, cfg.alloc, cfg.vocab)
    keys = {}
    if churn and cfg.churn_steps:
        for op in churn_ops(cfg, seed):
            if op.kind == "write":
                s = op.spec
                keys[op.key] = pool.write(s.text_ids, s.img_pos, s.img_ntok)
            else:
                pool.free(keys.pop(op.key))
    ids = []
    for i, s in enumerate(specs):
        wish = page_tier_draws(seed, i, -(-s.n_vis // cfg.page_tokens)) if cfg.tier_split else None
        rows = vis_np[i] if (with_bytes and vis_np is not None) else None
        ids.append(pool.write(s.text_ids, s.img_pos, s.img_ntok, rows, tier_wish=wish))
    return pool, ids


def oracle_plan(cfg, specs):
    assign, tok, cst = greedy_partition([s.length for s in specs], cfg.cost_k, cfg.capacity, cfg.n_mb)
    return assign, tok, cst, members(assign, cfg.n_mb)
