"""CPU oracle for the EasyBalance hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct NumPy (float64) statement of what the hot
path computes, used to check the HIP path.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it; the product package never does, and this package imports nothing
from the product (it shares no code, tables or helpers with it).

Modules and the passages they follow (EasyBalance, arXiv 2608.07964):

* ``numerics``  -- bf16 round-to-nearest-even, SiLU, softmax.
* ``model``     -- the MoE layer of Section 2.1, Eq. (1) (gate -> top-k ->
                   weighted sum of experts), preceded by RMSNorm and followed by
                   the residual add of Section 2.1; per-device workload vectors
                   (Section 2.3); a plain layer-by-layer run of a stack.
* ``permute``   -- the (layer, expert)-keyed stable permutation that stands in
                   for the all-to-all dispatch / gather of Section 2.2.
* ``sched``     -- Algorithm 1 (EasyBalance loop) with the MaxUtil scheduler and
                   minimum combination size m of Section 4.2, and the CumUtil /
                   DiffPeak heuristics of Section 5.2.
* ``metrics``   -- effective workload (Eq. 2), utilization (Eq. 3), the
                   per-step maximum vs effective workload of Section 5.3.

Readings of points the paper leaves open are listed in each function's
docstring.
"""
