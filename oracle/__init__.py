"""CPU oracle of DAMP's decode-step update - test infrastructure only.

Only tests, the smoke check and the benchmark's CPU-baseline leg import this
package. ``oracle.oracle`` wraps the plain-C fp32 oracle; ``oracle.brute`` is
an independent float64 brute force of the recurrence used to pin it.
"""
