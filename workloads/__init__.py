"""Seeded synthetic inputs shared by the CPU oracle and the HIP path.

Only input generation lives here (activation schedules, distance estimates,
per-agent memory sizes and byte contents); none of the memory manager's
arithmetic does.
"""
from .traces import (SENTINEL, PoolSpec, Trace, Content, CONFIGS, make_trace,
                     exact_distances, noisy_distances, random_tiny_trace,
                     shrink_planes, subsample_agents, splitmix64, lora_chunk_bytes,
                     prefix_tree_objects, prefix_forest)
