"""Seeded synthetic inputs for the KV-tier configuration evaluator.

Traces (:mod:`tracegen.workloads`), candidate configuration batches and the
cost-model inputs (:mod:`tracegen.configs`).  Both the GPU library's tests
and benchmark and the CPU oracle draw their inputs from here; the module
holds none of the cache-evaluation arithmetic.
"""
from .workloads import (Trace, Recipe, recipe, make, tiny, chat, tenant, longctx, full, from_blocks,
                        random_trace, WORKLOADS, GENERATOR_VERSION)
from .configs import (ConfigBatch, configs_for, trace_of, grid, from_list, empty, split_capacity,
                      random_configs,
                      DEFAULT_COST, MODE_INCLUSIVE, MODE_EXCLUSIVE_DEMOTE, MODE_INCLUSIVE_PREFIX, POLICY_LRU,
                      POLICY_FIFO, POLICY_LFU, POLICY_LEAF, MAX_GROUPS, GIB, TIB)

__all__ = [
    "Trace", "Recipe", "recipe", "make", "tiny", "chat", "tenant", "longctx", "full", "from_blocks",
    "random_trace", "WORKLOADS", "GENERATOR_VERSION", "ConfigBatch", "configs_for", "trace_of", "grid", "from_list",
    "empty", "split_capacity", "random_configs", "DEFAULT_COST", "MODE_INCLUSIVE", "MODE_EXCLUSIVE_DEMOTE", "MODE_INCLUSIVE_PREFIX",
    "POLICY_LRU", "POLICY_FIFO", "POLICY_LFU", "POLICY_LEAF", "MAX_GROUPS", "GIB", "TIB",
]
