"""CPU oracle of mixed chunked-prefill + decode paged attention.

Test infrastructure only: used by the tests, the smoke check and the benchmark's
CPU-baseline leg; the library never imports it.
"""
