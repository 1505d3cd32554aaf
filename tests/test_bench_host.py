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


def test_stage_table_groups_and_rates():
    n = 1_000_000
    timing = {"load_validate": (1, 1.0), "load_sort": (1, 6.0), "load_links": (1, 3.0),
              "stack_matrix": (4, 2.0), "stack_local": (1, 4.0), "stack_assemble": (1, 1.0),
              "stack_final": (2, 1.0), "replay_lfu": (1, 100.0), "replay_fifo": (1, 50.0),
              "replay_combine": (2, 2.0)}
    t = bench.stage_table("nowhere", timing, 1, n, {"lfu": 3 * n, "fifo": 2 * n},
                          {"lfu": 3, "fifo": 2})
    # the load: 18 B per access over the three load stages' 10 ms
    assert abs(t["load"]["achieved"] - 18 * n / 0.010 / 1e9) < 1e-9
    # the stack pass: 5 B per access over its four stages' 8 ms
    assert abs(t["stack_pass"]["avg_launch_ms"] - 8.0) < 1e-12
    assert abs(t["stack_pass"]["achieved"] - 5 * n / 0.008 / 1e9) < 1e-9
    # a replay: 5 B per (job, access) per launch, one workgroup per job
    assert t["replay_lfu"]["algorithmic_bytes_per_launch"] == 5 * 3 * n
    assert t["replay_lfu"]["workgroups"] == 3
    # two combine launches per step: each reads the jobs' hit bits and 8 planes once
    assert t["replay_combine"]["avg_launch_ms"] == 1.0
    assert t["replay_combine"]["algorithmic_bytes_per_launch"] == (5 + 16) * n / 8 / 2
    for rec in t.values():
        assert rec["frac"] == rec["achieved"] / bench.HBM_PEAK_GBS
        assert rec["traffic"] is None   # no counter record for this workload name


def test_counter_records_are_tied_to_the_kernel_sources(tmp_path, monkeypatch):
    import json
    src = tmp_path / "paper_2603_08739_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "k.hip").write_text("kernel v1")
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    sha = bench.source_sha(["k.hip"])
    assert sha == bench.source_sha("k.hip")
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps(
        {"w": {"replay_lfu": {"source": ["k.hip"], "source_sha": sha, "bytes_per_launch": 7.0}}}))
    (tmp_path / "profiles" / "valu.json").write_text(json.dumps(
        {"w": {"replay_lfu": {"source": ["k.hip"], "source_sha": sha,
                              "valu_insts_per_launch": 4.8e9}}}))
    assert bench.traffic_for("w", "replay_lfu") == 7.0
    assert bench.traffic_for("other", "replay_lfu") is None
    lim = bench.limiter_for("w", "replay_lfu", 1000.0, 48)
    # 4.8e9 wave64 instructions in 1 s against one per cycle per compute unit
    assert abs(lim["achieved"] - 4.8e9) < 1e-3
    assert abs(lim["frac_chip"] - 4.8e9 / (256 * 2.4e9)) < 1e-15
    assert abs(lim["frac_occupied_cus"] - 4.8e9 / (48 * 2.4e9)) < 1e-15
    # a changed kernel source voids both records
    (src / "k.hip").write_text("kernel v2")
    assert bench.traffic_for("w", "replay_lfu") is None
    assert bench.limiter_for("w", "replay_lfu", 1000.0, 48) is None


def test_more_than_one_gpu_is_refused():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
