"""CPU oracle for the Oscars local-SGD hot path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
reference of what the GPU path computes, written from the paper (Problem
Formulation, Eq. 1-3; Approach, Algorithm 1 and Eq. 4).  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with ``paper_2102_08550_amd`` (the HIP path) and
imports nothing from it; the only module both sides use is ``workload``, which
draws seeded inputs and holds none of the method's arithmetic.

Precision: float64 everywhere the paper does not fix a precision.  For the
bf16 workloads the oracle rounds to bf16 at the points the GPU rounds, and
keeps float64 elsewhere.  The aggregation tree runs in the dtype of its inputs
so that float32 replicas can be compared bit for bit.

Parity status of each function is given in its module docstring.
"""
from .load_balance import (InfeasibleBarrier, barrier_constraint, load_balance,  # noqa: F401
                           local_steps_from_barrier, max_wait, plan_from_measured,
                           quantize_iteration_times, wait_times)
from .sampler import (SplitMix64, batch_rows, epoch_permutation,  # noqa: F401
                      shard_offsets)
from .aggregate import paper_weights, tree_aggregate  # noqa: F401
from .mlp import bf16_round, evaluate, loss_and_grads, sgd_step  # noqa: F401
from .local_sgd import OracleRun, run_rounds, worker_local_steps  # noqa: F401
from . import cnn  # noqa: F401
