"""CPU oracle for the FedOptima server hot path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, deliberately
unoptimised NumPy implementation of what the server computes:

* the server-side training iteration of Algorithm 4 (forward of M_s, the
  loss f_s of Eq. 5, the backward pass and the SGD update),
* the device-side training iteration of Algorithm 1 (device network, its
  output activations, auxiliary network, local loss f_d, backward, SGD),
* the staleness-weighted asynchronous aggregation of Algorithm 4,
* the Task Scheduler of Algorithms 2 and 3 together with the activation
  flow control of Sec. 3.4.1,
* the pre-processor of the initialization stage: layer profiles, the
  split-point rule of Eq. 6-8 and the default auxiliary network (Sec. 3.2).

It is used by the tests, by the smoke check and by the benchmark's CPU
baseline leg only; the product library never imports, links or calls it,
and it shares no code with the HIP path (inputs come from ``fo_synth``,
which holds draws, not arithmetic).  Floating point runs in fp64 by default
(``dt=np.float32`` gives the CPU-baseline mode).

Parity status: every function here is pinned by the ``-m "not gpu"`` tests
(finite differences, closed forms, invariants, brute force and an
independent autograd library on tiny inputs).  No function is unpinned.
"""
from . import layers, nets, aggregate, scheduler, preproc  # noqa: F401
from .nets import server_step, server_forward, device_step, param_layout, sgd_update  # noqa: F401
from .aggregate import mix, mix_sequence  # noqa: F401
from .scheduler import TaskScheduler  # noqa: F401
