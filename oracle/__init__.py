"""fp64 CPU oracle for the JAB joint attention-block loss.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``, never by the product package.  It
shares no code with the GPU path; both sides only consume the seeded inputs.

``reference`` composes the C routines of ``jab_oracle.c`` (the plain loop form
of each step) into the loss, the sweep and the gradients; ``brute`` is a second,
independent numpy implementation that materialises the full attention matrix
and searches the quantization grid exhaustively, for tiny inputs.
"""
from . import reference  # noqa: F401
