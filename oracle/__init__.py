"""fp64 CPU oracle for paged-KV append and extend attention.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP library (no kernels, headers, helpers or constants) and
imports nothing from it.

What it computes (the problem the paper frames and the definition it implies):

* ``oracle_append`` -- the KV of newly prefilled tokens only exists once they
  took part in inference and is written back at that boundary (§5.1, §6.2);
  the new tokens of each sequence occupy logical positions P_b .. P_b+S_b-1
  and each position lives in the fixed-size page named by the sequence's block
  table (paged residency, §2.3 / §2.5).
* ``oracle_extend`` -- KV reuse exists to avoid re-prefilling a long reusable
  prefix (§1, §2.2); with a prefix of P_b reused tokens, the S_b new tokens
  attend causally over all P_b+S_b positions.  The result is by definition the
  plain dense causal attention of those rows, so the oracle writes that
  definition out: gather, scaled scores, mask, exact two-pass softmax, weighted
  sum of values.
* ``brute_force_extend`` -- the same definition in pure-Python loops over the
  un-paged logical sequence, used to pin ``oracle_extend`` on tiny inputs.
* ``oracle_to_host`` / ``oracle_to_device`` -- whole pages moved between the
  HBM tier and a packed host buffer (tiered cache, §6; local GPU <-> CPU
  engine, §7): a bitwise copy in page-list order.
* ``OracleManager`` -- the lifecycle states of message versions (§5.2), the
  aggregate state of shared KV and Algorithm 1's state-prioritized admission
  (§6.1), MRU eviction inside the Suspended tier (§6.2), written as a plain
  list-scanning model.

Every function here is pinned by ``tests/test_oracle_pins.py`` (the manager
by ``tests/test_manager.py``) against brute force, closed forms, a library
routine, hand-worked traces and invariants; none is "parity unpinned".
"""
from .attention import (  # noqa: F401
    storage_to_f64,
    oracle_append,
    oracle_extend,
    brute_force_extend,
    gather_logical,
)
from .blocks import oracle_to_device, oracle_to_host  # noqa: F401
from .manager import OracleManager  # noqa: F401
