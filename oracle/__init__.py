"""CPU oracle of the DiffKV hot path -- test infrastructure only.

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The product library never loads it.
"""
