"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package produces *inputs only*: simulation parameters X, the time input
t, temperature fields u, and the put/sample schedule that streams them.  It
holds none of the arithmetic of the method under test (the training
reservoir and the surrogate train step); both the oracle and the HIP path
consume what it produces.
"""
