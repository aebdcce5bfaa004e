"""CPU oracle for decode attention over token-range KV partitions.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code
with the HIP path, and the HIP path never calls it.

Every function here is the plain fp64 definition of one step of the
weightless attention node's decode work in KernelFlume (arXiv 2606.29207):
the tail append (Section 3.2, step 3; Section 5.1), local attention over one
token range producing a partial (Section 3.2, step 3), and the log-sum-exp
merge of partials (Section 3.2, step 4; Section 5.1).  All functions are
pinned by tests in ``tests/test_oracle_pins.py``; none is "parity unpinned".

``oracle.kf_policy`` is the attention-node scaling policy (Section 4.2:
Algorithm 1, Eqs. (1) and (2)), pinned by ``tests/test_policy_pins.py``.
"""
from .kf_oracle import (  # noqa: F401
    EFLAG_TAIL_FULL,
    EFLAG_BAD_ROUTE,
    EFLAG_BAD_PAGE,
    bf16_to_f64,
    e4m3_table,
    e4m3_to_f64,
    e4m3_encode_rne,
    gather_kv,
    attend,
    route_partial,
    partial_attn,
    merge,
    merge_partials,
    kv_append,
    kv_footprint_bytes,
)
