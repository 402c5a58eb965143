"""CPU oracles for the MoE expert-shard layer and for ViBE's placement control
path. TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. It shares no code with the HIP path
(``paper_2606_00735_amd``) and the HIP path never imports it.
"""
from . import moe_oracle, bruteforce, placement_oracle, mx_oracle  # noqa: F401
