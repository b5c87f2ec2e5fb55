"""Plain, slow CPU oracle for role-conditional KV-cache eviction.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or link
anything in this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers or constants): it restates the paper's
definitions in NumPy float64 so that a reader can check each step by eye.

Modules
-------
``reference``  NumPy float64 definitions: causal softmax, H2O and SnapKV mass,
               max-pool, role allocation (role-conditional, fair, No-X),
               per-role selection, compaction, decoding through the keep-set
               and the per-role mass diagnostics.
``brute``      pure-Python loops over tiny inputs (an independent second
               reading used to pin ``reference``).

Every function names the passage of the paper it follows (section, equation,
algorithm or table).  The readings taken where the paper is silent are listed
in the module docstring of ``reference``.

Parity status: every exported function is pinned by ``tests/test_oracle_*.py``
(directly, or through the function that calls it: ``quest_page_bounds``
through ``quest_mass``, ``rank_key`` through ``select_keep``) against closed
forms, invariants, library routines, brute force or numbers the paper prints.
The whole-tensor wrappers ``snapkv_score``, ``h2o_score`` and ``quest_score``,
which group query heads into KV heads, have their own grouping pins.
"""

from .reference import *  # noqa: F401,F403
