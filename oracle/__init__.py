"""CPU oracle for the grouped-absmean ternary linear layer.

TEST INFRASTRUCTURE ONLY: ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product path
(``paper_2606_18114_amd``) never does, and the two share no code.

``ternary`` is the vectorized float64 oracle; ``brute`` is its pure-Python
twin for tiny inputs; ``variants`` covers the threshold-multiplier and
group-magnitude variants of the paper's appendix.
"""
from . import ternary, brute, variants  # noqa: F401
