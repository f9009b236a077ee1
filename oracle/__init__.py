"""Oracle: plain, slow, obviously correct CPU implementations of what the
convolution path computes -- TEST INFRASTRUCTURE ONLY.

* ``oracle.conv``       -- Eq. (1) in fp64 (C source ``conv_ref.c``).
* ``oracle.cost_model`` -- the data-movement model of Sec. 3-5 in exact rationals.

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's cpu_baseline
leg may import, call or link anything here.  The product library never does,
and it shares no code with this package.
"""
