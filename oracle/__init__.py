"""CPU oracle of sequential ASGD (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package. It shares no code with the GPU library: the per-push arithmetic is
plain C (asgd_oracle.c), the protocol (queue, timestamp, staleness, pull
skip) is plain Python (server.py). The product path never imports it.
"""
