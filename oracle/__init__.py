"""fp64 CPU oracle of the MagmaDNN-style minibatch SGD step (test infrastructure).

THIS PACKAGE IS TEST INFRASTRUCTURE ONLY.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The product path (``paper_2011_11188_amd``) never calls it and
fails loudly when its HIP library is missing; the two share no code.

It is a plain, slow, obviously correct restatement of what the step computes
(Archibald et al., "Integrating Deep Learning in Domain Sciences at Exascale"):

* tensors, ops and backpropagation of a fixed layer chain (section 2.1);
* minibatch SGD (section 3.1, the classical algorithm the asynchronous
  variants relax);
* fp16 / bf16 storage with bf16 keeping fp32's exponent range (section 3.2);
* products of low-precision operands accumulated in fp32, D = C + A*B
  (section 3.2); the oracle accumulates in fp64, i.e. exactly up to the
  final storage rounding;
* convolution defined by its sum, independent of the algorithm used to
  evaluate it (section 2.1: convolution algorithms are swappable).

All arithmetic is fp64 over the exact values of fp16 / bf16 / fp32 inputs.
Storage roundings (round-to-nearest-even) happen only where the step stores a
tensor in a narrower type (``rounding.round_to``).  Library primitives used as
steps: numpy's float64 matmul and reductions.

Pins: ``tests/test_oracle_*.py`` check every function against brute force,
closed forms, invariants and library routines (none re-types the oracle's own
formula).  Whole-step numbers have no worked example in the paper:
"parity unpinned" beyond those invariants and finite-difference checks.
"""
from .rounding import round_to, decode, FORMATS  # noqa: F401
from . import ops, train  # noqa: F401
