"""Reference oracle for shared-prefix paged attention (TEST INFRASTRUCTURE ONLY).

This package is a plain, slow, fp64 CPU statement of what the GPU library
computes. It exists to check the library; it is never part of the product
path. Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark may import it. It shares no code with the HIP library or its Python
binding, and it imports neither.

What it follows (arXiv 2509.02121, "Halo"):
  * §3 "Scope" (semantic preserving) and §6.8 "Limitations": sharing a KV cache
    must give strictly the result of the original, unshared execution. So the
    oracle is the unshared definition: every query attends over the full,
    concatenated key sequence of its own request, with no sharing at all.
  * §2 "Background and Motivation" (locality: context reuse; intra-batch
    prefix sharing): requests reuse the KV cache of shared prefixes. In the
    oracle a request's keys are simply the concatenation of the segments on its
    root-to-leaf path.
  * §4.1 "Cost Modeling" (prefix-caching discount): prefill of new tokens over a
    cached prefix. The oracle's prefill lets chunk query i see every prefix key
    and the chunk keys up to and including position i.

The paper never writes out the attention formula; it is the textbook scaled
dot-product attention, softmax(scale * q k^T) v, with grouped heads (q head h
reads kv head h // (H_q / H_kv)).

``paged_kv`` holds the reference of the paged-KV write path (token scatter
into the pool layouts, page copy for copy-on-write); ``forest`` the prefix
forest of a batch of token-id prompts, by brute force.
"""

from .attention import (  # noqa: F401
    attend,
    attention_probs,
    decode,
    prefill,
    gather_tokens,
    merge_partials,
)
from . import paged_kv  # noqa: F401,E402
from . import forest  # noqa: F401,E402
