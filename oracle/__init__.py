"""CPU oracle for the mixed-batch attention step: TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously correct reference implementations, written from the
definitions they cite, that the HIP library is checked against:

* ``codecs``    - bf16 and OCP FP8 E4M3FN bit patterns to float64
* ``attention`` - paged, GQA, causal attention over materialised K/V (numpy, float64)
* ``brute``     - the same attention as scalar Python loops (tiny shapes only)
* ``kvpark``    - the byte image of parked KV blocks, and the resume scatter
* ``kvappend``  - the step's new K/V rows written into the paged cache
* ``former``    - the token-budget batch former (pure Python, float64)

Only the test suite, the smoke check and the benchmark's CPU-baseline leg
import this package. The product path (the C ABI library and its binding)
never imports, links or calls it, and this package imports nothing from the
product path.
"""
