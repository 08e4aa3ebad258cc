"""Reference oracle for projected per-example gradients and attribution scores.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may use it.  It is a plain, slow, obviously-correct CPU
implementation in float64 (numpy), written from the paper's definitions, and it
shares no code, constants or tables with the HIP library under
``paper_2609_38767_amd/``.

Modules
-------
``rng``        counter-based generator for the Gaussian projection maps
               (SplitMix64 seed derivation, Philox4x32-10, Box-Muller), written
               from the published definitions of those algorithms.
``gradients``  per-example weight gradient (Eq. 1), factored and materialized
               projections (Eq. 2), concatenation into one feature vector per
               example, and the factorized inner product (Eq. 4).
``scoring``    gradient-similarity scores with an optional diagonal
               preconditioner, and per-query top-k.
``cost``       closed-form FLOP / byte / storage counts of the two routes
               (Sec. 3.2 "FLOP-aware routing", App. A.4).
``crossgram``  cross-Gram matrices and squared norms of unprojected per-example
               gradients summed over layers, by the factorized route (Eq. 4)
               and through dense gradients (Eq. 1).
``kfac``       K-FAC / EK-FAC curvature on projected factors: factor
               covariances, eigenbases, EK-FAC's eigenvalue correction,
               damping and preconditioned scores (Sec. 3.2, App. A.2, App. B).
``mask``       random coordinate masks of DW gathered from the factors
               (App. A.2 "Random maps").
``token``      token-level attribution: per-token contributions g_t^T R a_t
               whose sum is the sequence score (App. D).

Parity status of each function is stated in its docstring; the functions
with no pin to the paper are the seed/counter layouts of the generator and of
the mask draw, which the paper leaves unspecified ("parity unpinned" w.r.t. the paper, pinned to the
published Philox / SplitMix64 definitions instead).
"""

from . import rng, gradients, scoring, cost, crossgram, kfac, mask, token  # noqa: F401
