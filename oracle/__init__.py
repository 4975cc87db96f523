"""CPU oracle for the RNN-T / W-RNNT loss and gradient (float64).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` use it.  It shares no code with the HIP library.

Modules
-------
rnnt_ref     the grid recursion written out from the paper (Eq. 1, Fig. 1,
             Section 2.3 Grid-Transducer, Section 3.2 W-Transducer)
lattice_dag  the same quantities over an explicit arc list (the composed
             lattice view of Section 2.2), a second, independent formulation
brute_force  enumeration of every alignment on tiny lattices
"""
