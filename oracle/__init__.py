"""Float64 CPU oracle of PnP-Nystra -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library
in ``paper_2506_08520_amd``; neither imports the other.
"""
from .reference import (  # noqa: F401
    geometry,
    landmark_map,
    pinv,
    unit_trace,
    forward,
    exact,
    max_threads,
)
