"""Host-side logic of bench.py (no GPU): the one-GPU refusal, the workload
shapes, and the pool plan against the stores the oracle fills."""

import os
import subprocess
import sys
from dataclasses import replace

import numpy as np
import pytest

import bench
import oracle
from workload import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_refuses_more_than_one_gpu():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


@pytest.mark.parametrize("idx", range(len(CONFIGS)))
def test_workload_shapes(idx):
    cfg, P, tags, pol, ptags = bench.build_workload(idx)
    assert P.shape == (cfg.batch,) and tags.shape == (cfg.batch, cfg.gen_tokens)
    assert P.min() >= cfg.prompt_min and P.max() <= cfg.prompt_max
    assert pol.n_layers == cfg.n_layers and pol.n_groups == cfg.n_groups
    if cfg.prompt_tagged:
        assert ptags.shape == (cfg.batch, int(P.max())) and pol.n_tags == 12 and pol.n_sink == cfg.n_sink
        assert ptags.max() < 12 and tags.max() < 6
    else:
        assert ptags is None and pol.n_tags == 6


def _store_pages(cfg, P, tags, pol, ptags, layers):
    """Pages the oracle's stores hold after every token of every sequence."""
    pd = dict(action=pol.action, floor=pol.floor, group_of_layer=pol.group_of_layer, n_sink=pol.n_sink)
    oc = oracle.OracleCache(pd, 1, 32)
    hi = lo = 0
    z = np.zeros((1, 1, 32), np.uint16)
    for b in range(cfg.batch):
        for layer in layers:
            p = int(P[b])
            if ptags is None:
                oc.append(layer, b, np.zeros(p, np.uint8), np.repeat(z, p, 0), np.repeat(z, p, 0), keep_all=True)
            else:
                oc.append(layer, b, ptags[b, :p], np.repeat(z, p, 0), np.repeat(z, p, 0))
            t = tags[b, :cfg.gen_tokens]
            oc.append(layer, b, t, np.repeat(z, t.size, 0), np.repeat(z, t.size, 0))
            c = oc.counts(b, layer)
            hi += (c["hi"] + 15) // 16
            lo += (c["lo"] + 15) // 16
    return hi, lo


@pytest.mark.parametrize("idx,beta", [(0, None), (1, None), (3, 0.25), (3, 1.0)])
def test_pool_plan_covers_the_stores(idx, beta):
    cfg, P, tags, pol, ptags = bench.build_workload(idx, beta)
    if cfg.batch > 8:                      # a slice of the batch keeps the oracle fast
        keep = slice(0, 4)
        cfg = replace(cfg, batch=4)
        P, tags = P[keep], tags[keep]
        ptags = None if ptags is None else ptags[keep]
    hi, lo = bench.plan_pool_pages(cfg, P, tags, pol, ptags, online=False)
    need_hi, need_lo = _store_pages(cfg, P, tags, pol, ptags, range(cfg.layers_resident))
    assert need_hi <= hi and need_lo <= lo
    assert hi - need_hi <= cfg.layers_resident * cfg.batch       # the plan's only slack: a spare page per store
    assert lo - need_lo <= cfg.layers_resident * cfg.batch


def test_traffic_record_only_for_its_workload_and_sources(monkeypatch):
    """The committed counter summary is used only for the workload it was
    taken on (a run from another start position names itself apart) and
    only while the attention sources are the ones it was taken with."""
    name = "qwen3_4b_b64_p1k-8k_g1024"
    assert bench.traffic_record(name + "+t0") is None
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 16)
    assert bench.traffic_record(name) is None
