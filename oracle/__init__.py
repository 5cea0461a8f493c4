"""CPU oracle for the HUGE embedding training step -- test infrastructure only.

Imported by the tests, the smoke check and the benchmark's CPU baseline; the
product library never imports, links or executes anything in this package.
"""
