"""CPU oracle of the PC-MoE expert layer — test infrastructure only.

Importable only from tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg.
The HIP library never imports, links or calls anything here.

Parity status of every function is pinned by tests/test_oracle_pins.py (finite differences,
closed forms, brute force, invariants) and, for the expert update, tests/test_update_oracle.py
(PyTorch's AdamW and SGD, a closed form, invariants); none is "parity unpinned".
"""
from . import moe_layer, brute, moe_update  # noqa: F401
