"""CPU oracle for pattern- and connectivity-pruned convolution.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The GPU library
(``paper_2004_11250_amd``) never imports it and shares no code with it; both
take their inputs from the seeded generators in ``workloads.py``.

What it computes follows the paper (Niu et al., "Towards Real-Time DNN
Inference on Mobile Platforms with Model Pruning and Compiler Optimization"):

* ``conv``   -- the plain definition of a pruned 3x3 layer: a direct
  convolution over the dense weights with the pruned taps zeroed (pattern and
  connectivity pruning, Sec. 2), fp64 accumulation; plus the dense ops the
  evaluated networks need (k x k conv, transposed conv, pooling, upsampling,
  pixel shuffle).
* ``ppk1``   -- an independent writer of the compact packed weight format
  (Sec. 3, "sparse model storage" and "matrix reorder") and an interpreter that
  evaluates a layer by walking a packed blob.
* ``net``    -- runs the op lists of ``workloads.py`` with the functions above.
* ``bf16``   -- round-to-nearest-even conversion to bfloat16.

Every function says which passage it follows and the tests in
``tests/test_oracle*.py`` pin it against values fixed by the paper or by
mathematics (hand-computed examples, closed forms, brute force, independent
library routines).
"""
from . import bf16, conv, net, ppk1  # noqa: F401
