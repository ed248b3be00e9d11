"""Plain fp64 CPU oracle for shared-prefix paged attention.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (the HIP library and its Python binding) never
imports it, and this package imports nothing from the product path: the two
share no kernels, helpers, tables or pre/post-processing.  Inputs reach both
sides only through the seeded generators, which hold none of the method's
arithmetic.
"""

from .attention import (  # noqa: F401
    PAGE_SIZE,
    bf16_bits_to_f64,
    gather_tokens,
    attend_rows,
    prefix_shared_attention,
    split_attention,
    merge_partials,
    append_kv,
    page_copy,
    pages_needed,
)
from . import movement  # noqa: F401,E402
from . import service  # noqa: F401,E402
