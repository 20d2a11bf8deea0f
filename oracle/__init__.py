"""CPU oracle of the HAMburger macro-step decode loop (arXiv 2505.20438).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package; the library under
``paper_2505_20438_amd`` never does, and this package imports nothing from it.

A plain, slow, float64 numpy transcription of what the decode loop computes:
the compositional embedder (Sec. 3.2), the base decoder forward writing one KV
entry per fused group (Sec. 3.1, Sec. 3.7 "Token Fusion"), and the micro-step
decoder with its stop test (Sec. 3.3, Sec. 3.4, Sec. 4.4).  Weights, prompts and
schedules come from :mod:`synth`.

Parity status: every function here is pinned by the ``-m "not gpu"`` tests
(brute force, closed forms, the reduction to plain greedy decoding, prefill
equal to incremental steps, KV counting).  Fidelity of the module readings to
the paper's unreleased trained model (which layers feed the micro decoder, the
exact embedder projections) has no numeric source to pin against: parity
unpinned for that question, by construction of the paper.
"""
from .ham import OracleHam, SeqResult  # noqa: F401
