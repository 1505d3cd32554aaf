"""Host logic of the benchmark: which replay jobs a batch creates (one per
distinct order, group, policy and capacity below the distinct weight), the
accesses they walk and the workgroups a replay launch runs."""
from types import SimpleNamespace

import bench
import tracegen as tg


def stats(n, n_g, u_w_g):
    return SimpleNamespace(n_groups=len(n_g), n_g=n_g, u_w_g=u_w_g, distinct_w=sum(u_w_g))


def test_shared_jobs_dedupe_capacities_and_skip_closed_form():
    st = stats(1000, [600, 400], [300, 200])
    cfgs = tg.from_list([
        {"cap": (64, 128, 0), "policy": tg.POLICY_LFU},
        {"cap": (64, 256, 0), "policy": tg.POLICY_LFU},    # 64 again: one job
        {"cap": (32, 500, 900), "policy": tg.POLICY_FIFO},  # >= 500 distinct weight: closed form
        {"cap": (32, 0, 0), "policy": tg.POLICY_LRU},       # LRU: the stack pass
    ])
    acc, cnt = bench.replay_job_accesses(cfgs, st, 1000)
    assert cnt == {"lfu": 3, "fifo": 1}
    assert acc == {"lfu": 3 * 1000, "fifo": 1000}


def test_partitioned_jobs_walk_their_group():
    st = stats(1000, [600, 400], [300, 200])
    cg = [[16, 16], [0, 250], [0, 0]]   # tier x group: group 1's DRAM holds all of it
    cfgs = tg.from_list([{"cap": (32, 250, 0), "partitioned": 1,
                          "policy": [tg.POLICY_LFU, tg.POLICY_FIFO], "cap_group": cg}])
    acc, cnt = bench.replay_job_accesses(cfgs, st, 1000)
    assert cnt == {"lfu": 1, "fifo": 1}
    assert acc == {"lfu": 600, "fifo": 400}
