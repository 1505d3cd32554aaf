"""The stored expected values match the current generators and oracle.

Each stored file is keyed by the generator version and a digest of the
trace and configuration arrays; these checks regenerate the smaller traces
on the CPU and compare the digests, and recompute the tiny workload's counts
with the literal (non-memo) oracle, so a drifted generator or a corrupted
file is caught without a GPU.
"""
import os

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


def test_tiny_counts_recomputed_literally(oracle_mod):
    g = _gold("tiny")
    t = tg.recipe("tiny").to_trace()
    c = tg.configs_for("tiny", t).subset(g["idx"])
    assert np.array_equal(oracle_mod.replay(t, c), g["counts"])
