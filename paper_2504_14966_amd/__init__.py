"""MI355X-native hot path of the SLO-aware LLM request scheduler (arxiv 2504.14966).

The GPU library (libsloanneal.so, C-ABI in include/sloanneal.h) is loaded lazily by
``paper_2504_14966_amd.sloanneal``; ``workloads`` draws the seeded synthetic queues.
"""
__all__ = ["sloanneal", "workloads"]
