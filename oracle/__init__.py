"""CPU oracle for the iFVS filtered-search hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this
package.  The product path (the HIP library and its Python binding) never
imports it and shares no code with it.
"""
from .ifvs_oracle import *  # noqa: F401,F403
from .ifvs_oracle import __all__  # noqa: F401
from .ifvs_encoder_oracle import encode_predicate  # noqa: F401
