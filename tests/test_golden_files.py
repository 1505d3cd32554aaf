"""The stored expected values match the current generators and oracle.

Each stored file is keyed by the generator version and a digest of the
trace and configuration arrays; these checks regenerate the smaller traces
on the CPU and compare the digests, and recompute the tiny workload's counts
with the literal (non-memo) oracle, so a drifted generator or a corrupted
file is caught without a GPU.
"""
import os
import sys

import numpy as np
import pytest

import tracegen as tg
from tracegen.digest import configs_digest, trace_digest

HERE = os.path.dirname(os.path.abspath(__file__))


def _gold(name):
    return np.load(os.path.join(HERE, "golden", f"counts_{name}.npz"))


@pytest.mark.parametrize("name", ["tiny", "chat", "tenant"])
def test_digests_match_generators(name):
    g = _gold(name)
    assert int(g["generator_version"]) == tg.GENERATOR_VERSION
    t = tg.recipe(name).to_trace()
    assert trace_digest(t.hash, t.req, t.group, t.weight, t.req_time) == str(g["trace_sha"])
    c = tg.configs_for(name, t)
    assert configs_digest(c) == str(g["configs_sha"])
    assert int(g["n"]) == t.n and int(g["n_cfg_total"]) == c.n
    assert g["counts"].shape == (len(g["idx"]), t.n_groups, 3, 8)


@pytest.mark.parametrize("name", ["longctx", "full", "full_ttl", "longctx_leaf"])
def test_large_files_present(name):
    g = _gold(name)
    assert int(g["generator_version"]) == tg.GENERATOR_VERSION
    # the stored configurations are the documented seeded subset
    sys.path.insert(0, os.path.join(HERE, "golden"))
    import make_golden
    assert np.array_equal(g["idx"], make_golden.subset(name, int(g["n_cfg_total"])))
    c = g["counts"].astype(np.int64)
    assert c.shape[0] == len(g["idx"]) > 0
    # every access reaches the first present tier: its hits + misses count
    # all of the group's accesses, and no other tier counts more
    n = int(g["n"])
    for i in range(c.shape[0]):
        reach = [int(c[i, 0, k, 0] + c[i, 0, k, 1]) for k in range(3)]
        live = [r for r in reach if r]
        assert live and live[0] == n and max(live) <= n


def test_tiny_counts_recomputed_literally(oracle_mod):
    g = _gold("tiny")
    t = tg.recipe("tiny").to_trace()
    c = tg.configs_for("tiny", t).subset(g["idx"])
    assert np.array_equal(oracle_mod.replay(t, c), g["counts"])
