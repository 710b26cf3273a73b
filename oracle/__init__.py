"""Plain float64 CPU oracle of the factorized-cache decode path.

TEST INFRASTRUCTURE.  It exists to check the GPU library and is never part of
it: only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import it.  It shares no code with the library (no kernels, headers,
helpers or table generators); both sides only read the same seeded synthetic
inputs.

* ``factorized``: Eq. 1 reconstruction, softmax decode attention, Eq. 3 probe
  error and the dense residual map.
* ``router``: Eq. 2 rank routing (multi-level reading) and residual offsets,
  for the whole packed axis or a token range continuing an existing table.
* ``compress``: the storage half of Eq. 1 for new tokens: projection onto the
  window basis, routed residual channels, int4 codes, gate-folded scale.
* ``features``: the router's attention-mass and attention-spike features of a
  decode.
* ``control``: probe-feedback threshold updates and budget-driven selection.
* ``sketch``: the randomized-sketch initialization of a window's bases.

Every function is pinned by the CPU tests (brute force in exact arithmetic,
closed forms, reductions to library attention, invariants); none is marked
"parity unpinned".
"""
from . import factorized, router, compress, features, control, sketch
from .factorized import (attention, decode, probe, probe_error, probe_positions, reconstruct,
                         residual_map, int4_from_nibble, entry_codes, q_to_f64,
                         default_scale)
from .router import route, route_range, router_score, level_index, theta_from_tau
from .compress import compress_vectors
