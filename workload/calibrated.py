"""Temperatures fixed by tests/golden/calibrate_temperature.py (oracle only).

The 1B-shape workload scales logits so that about half of the drafted
positions clear the accept threshold; the value below is the one that
script found by bisection and is frozen as an fp32 literal.
"""
TEMPERATURE = {
    "1b_bf16": 1.0,
}
