"""Brute-force oracle for grammar-constrained decoding masks.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The product library never loads
it.  See ``oracle.c`` for what is computed and the readings it takes.

Functions and their pins (tests/test_oracle_pins.py):
  * ``Oracle.masks``       eq. simp over every token; pinned by exhaustive
    enumeration of the arithmetic language, worked examples derived by hand
    from the grammar, an independent JSON recogniser, and invariants
    (EOS <=> membership, non-empty masks, prefix closure, teacher forcing,
    state equivalence).
  * ``Oracle.token_bits``  the same rule for selected tokens.
"""
from .oracle import Oracle, build  # noqa: F401
