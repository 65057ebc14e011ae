"""Plain CPU oracle for the DensityKV hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or call it.  It shares no code with the HIP library
(no kernels, headers, helpers, tables or constants) and imports nothing from
``paper_2608_27922_amd``.

Every function follows the paper's definitions step by step in NumPy:

* Soft-Riesz weight and density (Sec. 3.3, Eqs. 2-3; Supp. B),
* the online bank update for one layer (Sec. 3.4, Eqs. 4-12; Supp. C,
  Algorithm 1, "Insertion hysteresis", "Exact density maintenance"),
* the native attention over the retained bank plus the local window
  (Sec. 3.2 logit; Sec. 1 / Fig. 1 caption: native attention reads the bank).

The arithmetic contract that makes every discrete decision reproducible (keys
on the 1/64 grid, fp32 per-pair weights, Q23 fixed-point integer sums) is
documented in ``densitykv_ref``'s module docstring.
"""

from .densitykv_ref import (  # noqa: F401
    Q23,
    Params,
    BankState,
    UpdateRecord,
    pair_d2,
    pair_d2_bruteforce,
    soft_riesz_weight,
    weight_q23,
    density_from_scratch,
    candidate_scores,
    update_layer,
    attention,
)
