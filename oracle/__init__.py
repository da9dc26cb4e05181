"""CPU oracle of the sparsity-preserved LoRA linear -- TEST INFRASTRUCTURE ONLY.

This package is the slow, obviously-correct reference that the GPU library is
checked against.  Only the tests, the smoke check and the benchmark's CPU
baseline leg may import it; the library itself never does, and it shares no
code, tables or helpers with the HIP path.

Contents
--------
``lors``    fp64 numpy definition of the forward and of both backward forms
            (exact masked gradient and the straight-through rearranged one),
            plus one-entry-at-a-time evaluators for large problems.
``loops``   pure-Python loop twin of ``lors`` for tiny shapes.
``masks``   the packed mask layouts (1 bit per element, and 2:4 index codes),
            written out bit by bit.
``bf16``    exact decode of bf16 bit patterns to fp64.

Notation (kept identical across the repository): W is R x C (out x in), M the
R x C 0/1 mask, B the R x r adapter and A the r x C adapter, s the scale, X is
L x C (one token per row), Y and dY are L x R.  The paper writes the R x r
adapter as calligraphic A and the r x C one as calligraphic B, and stores
tokens as columns (X is C x L); the formulas here are the same ones with
those names and that transpose applied.

Parity status: every function is pinned by the CPU tests (finite differences,
special cases, closed forms, brute force); no function is "parity unpinned".
"""

from . import bf16, lors, loops, masks  # noqa: F401
