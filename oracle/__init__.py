"""CPU oracle of the DecoMoE RCEP MoE layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute anything in this package: only the test suite, the smoke check in
``__graft_entry__.py`` and the ``cpu_baseline`` leg of ``bench.py`` use it.
It shares no code with the HIP path and imports nothing from it.
"""

from .moe import *  # noqa: F401,F403
