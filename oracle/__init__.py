"""FP64 CPU oracle for the MACE layer hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything in this
package.  The product path (the HIP library and its Python binding) never
imports it, and it shares no code, table or helper with that path: the only
thing both sides use is the seeded input generator module ``synth``.

Every function cites the passage of the paper (arXiv 2510.23621, "Speeding Up
MACE: Low-Precision Tricks for Equivariant Force Fields") that it follows:
the graph problem statement, the two-body edge embedding (Eq. 26), the
node-local product basis (Eq. 27), the message/update/readout paragraph, the
energy and force equations, and the architecture breakdown table in the
appendix.  Where the paper is silent the oracle takes a fixed reading; each
reading is listed in ``oracle/mace.py``'s module docstring.

Modules
  so3        real spherical harmonics, real Clebsch-Gordan couplings, the
             generalised-CG (U) tensors of the symmetric contraction
  neighbors  brute-force periodic neighbour list
  mace       model layout, forward energies and autograd forces

Parity status: every function is pinned by tests under ``tests/`` (closed
forms, library routines, invariances, finite differences, brute force, the
parameter counts printed in the appendix table).  Absolute energies for
seeded random weights have no printed worked example in the paper; they are
pinned only through those properties (see the test files).
"""
