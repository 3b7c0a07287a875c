"""CPU oracle for the learner step: test infrastructure, not part of the product.

Only tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package."""
