"""Plain, slow CPU oracle of ParisKV's retrieval path (arXiv 2602.07721).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the smoke check in ``__graft_entry__``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code,
tables or constants with the HIP library; the two meet only at the seeded
synthetic inputs produced by the separate ``workloads`` package.

Everything here is NumPy float64 (plus mpmath for the one offline constant
that needs more than double precision to round correctly), written to be
checked against the paper by eye, not to be fast.

Modules
-------
quantizer   Beta prior of a rotated subspace coordinate and the 3-bit
            Lloyd-Max magnitude quantizer (Appendix: offline quantizer
            derivation, Prop. "rotation-induced Beta priors").
rotation    Sylvester Hadamard matrix, SRHT rotation R = H diag(s)/sqrt(D),
            and an in-place fast Walsh-Hadamard transform.
encode      Key summarisation: centroid ids, 4-bit sign+magnitude codes and
            the per-subspace weight w (Sec. "Prefill Phase", Alg. 1 encode).
retrieve    Query transform, tier-weighted collision scores (Eq.
            collision_score), top-beta candidate selection, the RSQ-IP
            estimator (Eq. rsqip_raw_weighted) and the final top-k.
attention   Exact and candidate-restricted softmax attention
            (Eqs. full_attention, approx_weight, approx_output).
window      The four decode-time KV regions (Sink, Retrieval, Local, Update
            Buffer) replayed token by token from Sec. "Buffer Update", and
            attention over Sink + retrieved + Local + Buffer rows.

Parity status: every function is pinned by a ``-m "not gpu"`` test against
something other than itself (worked examples, closed forms, brute force,
hand-computed fixtures or distributional facts).  None is "parity unpinned".
"""

from . import quantizer, rotation, encode, retrieve, attention, window  # noqa: F401
