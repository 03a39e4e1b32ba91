"""Drives an agent episode (synth.trajectory.schedule) through the oracle's
lifecycle driver and, on a GPU, through the library's (shared test helpers)."""
import numpy as np

from oracle.lifecycle import Agent as OracleAgent
from synth.trajectory import kv_rows, query_rows, schedule


def oracle_agent(cfg, **over):
    kw = dict(n_layers=cfg.n_layers, n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
              page_size=cfg.page_size, budget=cfg.budget, eta=cfg.eta,
              max_pending_pages=cfg.max_pending_pages, max_scan_pages=cfg.max_scan_pages,
              keep_recent=cfg.keep_recent, score_layer=cfg.score_layer, pool_kernel=cfg.pool_kernel,
              pool_mode=cfg.pool_mode)
    kw.update(over)
    return OracleAgent(**kw)


def window(traj, p0):
    """Queries of the scoring layer at [p0, p0 + W) and their positions."""
    W = traj.cfg.window
    return query_rows(traj, traj.cfg.score_layer, p0, p0 + W), np.arange(p0, p0 + W)


def run_oracle(traj, agent, hook=None):
    """Every action of the schedule on the oracle agent; ``hook(action, report)``
    sees each step's report."""
    cfg = traj.cfg
    for act in schedule(traj):
        if act[0] == "append":
            _, kind, p0, p1, dec, first = act
            kv = [kv_rows(traj, l, p0, p1) for l in range(cfg.n_layers)]
            agent.append(kind, p0, p1, [x[0] for x in kv], [x[1] for x in kv], dec, first)
            rep = None
        else:
            Q, qpos = window(traj, act[1])
            rep = getattr(agent, act[0])(Q, qpos)
        if hook:
            hook(act, rep)
    return agent
