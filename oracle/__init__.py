"""Test infrastructure: the fp64 CPU oracle of the KV-translation operator.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  The product path (``paper_2608_30963_amd``) never imports it.
"""
