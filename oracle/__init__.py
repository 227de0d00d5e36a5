"""Reference oracle for the compressed se_a descriptor (test infrastructure).

This package is a plain, slow and deliberately unoptimised CPU implementation
of what the GPU library computes, written from the paper (DP Compress,
arXiv:2107.02103, Sec. II) in float64:

* ``net``   -- the embedding net G(s^) and its first and second derivatives
               (forward mode), the functions that are tabulated;
* ``table`` -- the piecewise fifth-order Hermite table (the coefficient
               closed forms of Sec. II) and its evaluation;
* ``se_a``  -- forward T = G^T R~ and D = T T<^T, the backward pass
               dE/dR~ from dE/dT, evaluated naively pair by pair, and the
               descriptor backward dE/dT from dE/dD;
* ``cref``  -- the same forward/backward as plain C loops (OpenMP over atoms)
               for the large workloads;
* ``env``   -- the environment matrix R~ from positions (Eq. (1) and the
               normalisation) and the forces and virials from dE/dR~;
* ``fitting`` -- the fitting net D -> E and its backward dE/dD;
* ``nlist`` -- the neighbour list (type blocks of sel slots, nearest first)
               by brute force over all atom pairs, as plain C loops.

It is test infrastructure only: the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it; the product path never does.
It shares no code with the GPU library (``paper_2107_02103_amd``) and never
imports it.  Every function is pinned by tests in ``tests/test_oracle_*.py``
against closed forms, invariants, brute force on tiny inputs and finite
differences.
"""
