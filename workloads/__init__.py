"""Seeded synthetic workloads for the shallow-fusion decode step.

This package only draws inputs: a Zipf token corpus, a Kneser-Ney n-gram
language model estimated from it (the model is an *input* of the fusion step,
exactly as a user-supplied ARPA file would be), phrase lists and joint logits.
It holds none of the fusion arithmetic (no backoff evaluation, no trie, no
scoring).  Both the CPU oracle and the GPU library read what it produces.
"""

from .gen import (  # noqa: F401
    CONFIGS,
    LMArrays,
    Phrases,
    Workload,
    make_corpus,
    estimate_kn,
    make_phrases,
    make_logits,
    make_projection,
    make_keyword_lm,
    to_bf16_bits,
    load_workload,
    tiny_random_lm,
    tiny_random_phrases,
)
from .keyword import (  # noqa: F401,E402
    KEYWORD,
    CONDITIONS,
    KeywordWorkload,
    make_keyword_workload,
    hypotheses,
    keyword_recall,
    token_error_rate,
    edit_distance,
    count_occurrences,
)
