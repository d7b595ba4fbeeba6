"""RIS sparse attention for AMD Instinct MI355X (gfx950).

The hot path -- on-device geometry generation (CSR of the seed-ensemble
union), RoPE with long-context scaling, and one softmax over each row's
unified key set -- is hand-written HIP behind the C ABI in ``include/ris.h``
(``libris.so``).  ``paper_2607_21927_amd.ris`` is its Python binding.
"""

from . import ris  # noqa: F401
