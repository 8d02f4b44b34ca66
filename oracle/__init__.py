"""CPU oracle for restructured batch normalisation -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package.  It shares no code with the HIP
product path and never imports it.

``prims``    -- fp64 primitives (ctypes over ``liboracle.so``, built from
               ``oracle.c``) with numpy arrays in and out.
``compose``  -- the training compositions (one BN-ReLU-CONV unit, a DenseNet
               composite layer, dense block 1 + transition, ...) built from
               the primitives, with an optional bf16 storage model.
"""
