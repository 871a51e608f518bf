"""CPU fp64 oracle for batched paged-KV attention with per-request segment masks.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call, link
or execute anything in this package: only the test suite, the smoke check and
the benchmark's CPU-baseline leg use it.  It shares no code with the HIP path
(no kernels, headers, helpers, tables or pre/post-processing); the only inputs
both sides share come from the seeded generators in ``workloads``.

What it computes (the plain definition, no blocking, fusion or reordering):
for every request, query head and query row, the softmax-weighted average of
the value rows of the keys that row may see, read through the request's block
table, plus the natural-log log-sum-exp of the scaled scores.  The paper runs
this computation through a paged-attention library inside its
``KVCacheEngine`` (Sec. 3.3, Runtime) over one shared page pool whose page
tables are read in place (Sec. 4.1); it does not define the masks, so the
mask semantics are the reading stated in ``attention.py``.  ``append.py``
holds the paged KV append (the step's new K/V rows written into their pages
before attention reads them).

Pins (tests marked ``not gpu``): brute-force visibility predicates written from
each workload's wording, torch's CPU float64 ``scaled_dot_product_attention``
(causal, unmasked and explicit-mask special cases), closed forms (one visible
key, equal scores), bitwise invariance under physical page permutation, GQA as
repeated-KV MHA, the fp64 split/merge identity, and a second scalar oracle in
plain Python on tiny inputs.  The paper prints no worked attention example, so
no value here is pinned to a number printed in the paper.
"""
from .attention import (  # noqa: F401
    SEG_BLOCKS,
    SEG_CAUSAL,
    SEG_FULL,
    attend,
    block_ids,
    gather_kv,
    merge_partials,
    oracle_attention,
    oracle_rows,
    useful_work,
    visible_matrix,
)
from .append import append_targets, kv_append  # noqa: F401
