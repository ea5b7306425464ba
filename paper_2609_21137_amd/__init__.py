"""MI355X-native compressed-MoE decode layer (CARDAN hot path).

``configs`` and ``synth`` describe and generate workloads; ``cardan`` is the
binding to the HIP library ``libcardan.so`` built from ``csrc/``.
"""

from . import configs  # noqa: F401
