"""Oracle — TEST INFRASTRUCTURE ONLY.

A plain, slow fp64 CPU implementation of the VIA-SD verification step
(verifier forward, slim routing, tier rule, accept/rollback loop, paged KV
index model) written from the paper.  Only tests/, __graft_entry__.smoke()
and bench.py's cpu_baseline leg may import it; the HIP library and its
binding never do, and this package imports nothing from them.
"""
