"""CPU oracle of the ABCD active-block step -- test infrastructure only.

Imported by the tests, the smoke check and the CPU-baseline leg of the
benchmark; never by the product package.
"""
