"""CPU oracle for the CubicQuant hot path.

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, fp64/int64 restatement
of what the CubicQuant paper (arXiv 2608.06763) defines: the packed code stream,
the cubic level function, the Dynamic-A8 activation quantizer and INT8 weight
carriers, the reference products, the continuous groupwise fitter and the
population-distortion theory used to pin the rest.

Only the test suite, the smoke check of the package entry point and the
``cpu_baseline`` leg of ``bench.py`` may import it.  The product library never
imports, links or calls anything here, and nothing here imports the product.
The one shared dependency is ``workloads``, which only draws seeded random
inputs and holds none of the method's arithmetic.
"""
