"""fp64 CPU oracle for the KVpop future-attention target.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's CPU
baseline may import this package. The library's GPU path never calls it, and the
two share no code: the oracle decodes bf16 bit patterns itself and evaluates the
paper's definitions directly in float64.

What it computes (paper, App. D.1, eqs. dense_logit_app .. future_mass_app):

* logits   l(d, t) = scale * <q_d, k_t> + bias_t           (t <= d, causal)
* LSE_d    = log sum_{t <= d} exp l(d, t)                   (row log-normaliser)
* p_{d->t} = exp(l(d, t) - LSE_d)                           (causal probability)
* m_t      = sum_{d = t + window}^{min(T-1, t + horizon)} p_{d->t}
             (unnormalised future mass; horizon < 0 means up to T-1)

plus the transposed log-space form of App. D.2 (eq. future_mass_lse_app), used as an
independent cross-check of the same quantity.

The running top-k policy pieces (static priorities, ranks, cutoffs, the sparse
mask and the sparse log-normaliser of App. C and App. D.3) are in
``oracle.running_topk``.

The running top-k sparse attention forward (App. C.1, C.3) with its sparse LSE,
and the token lifetimes [t, e_t) that the running mask reduces to, are in
``oracle.sparse_attention``.

The target epilogue of App. D.4 step 5 (aggregation over the G query heads and
count normalisation, App. B.1-B.2) is in ``oracle.target``.

Every function here is pinned by tests against closed forms, hand enumeration and
brute force (tests/test_oracle_pins.py); no function is "parity unpinned".
"""
from .future_mass import (  # noqa: F401
    bf16_bits_to_f64,
    causal_logits,
    future_mass,
    future_mass_blocked,
    future_mass_columns,
    future_mass_transposed,
    row_lse,
    row_lse_blocked,
    row_lse_rows,
)
from .target import future_count, target_scores  # noqa: F401
from .running_topk import (  # noqa: F401
    ranks_from_priority,
    running_cutoff_bruteforce,
    running_cutoff_fenwick,
    running_topk_mask,
    sparse_row_lse,
    static_priority,
    static_priority_f32,
    teacher_labels,
)
from .sparse_attention import (  # noqa: F401
    eviction_times,
    eviction_times_bruteforce,
    lifetime_mask,
    running_topk_mask_rows,
    sparse_attention,
)
