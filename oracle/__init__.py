"""fp64 CPU oracle of SpeechKV (arXiv 2607.06827, Sec. III-B Eq. 4-5, Sec. III-C).

TEST INFRASTRUCTURE ONLY: the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this package; the product path never
does.  It shares no code with the GPU library.
"""
from .oracle import (  # noqa: F401
    attention,
    attention_bwd,
    build,
    compressed_len,
    decode,
    num_threads,
    pool,
    pool_bwd,
)
