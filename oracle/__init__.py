"""CPU fp64 reference oracle for the COUNTDOWN sparse Gated-MLP FFN.

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` are its only users. The product path
(``paper_2505_17701_amd``) never imports it and shares no code with it.
"""
from .oracle import *  # noqa: F401,F403
