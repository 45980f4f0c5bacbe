"""Oracle: a plain, slow, float64 CPU executor of primitive graphs.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.
The GPU library never imports, links or calls it, and it shares no code with
the GPU library: the only thing both sides consume is the seeded input
generator in ``synthetic/``.

What it computes (Korch, Sections 3 and 4): a primitive graph is a DAG whose
nodes are elementwise, reduce/broadcast, layout-transformation and
linear-transformation primitives.  The oracle runs the *unfused* graph one
primitive at a time in float64, each primitive materializing its full output
(``graph.run_unfused``).  Orchestration changes cost, never the result, so
every valid kernel orchestration plan must reproduce these outputs
(``graph.run_plan`` executes a plan under the same primitive semantics).

Modules:
  primitives     the semantics of every primitive, in float64
  graph          graph container, shape rules, unfused executor, plan executor
  orchestration  Definitions 1-3, Theorem 1 and the state search of Algorithm 1,
                 written as plain set computations
  configs        the oracle's own builders of the five workload graphs

Parity pins: every function here is pinned by a CPU test against something
other than itself (closed forms, brute-force loops, invariants, library
routines); see ``tests/test_oracle_*.py``.  No function is "parity unpinned".
"""

from . import primitives, graph, orchestration, configs  # noqa: F401
