"""Temperatures fixed by tests/golden/calibrate_temperature.py (oracle only).

TEMPERATURE: the 1B-shape and the 8B chain and tree workloads scale their
logits so that about half of the drafted positions (teacher-forced greedy
windows) clear the accept threshold; the long-context batch runs at its
mixed-tier temperature.
MIXED_TEMPERATURE: the temperature maximising the smallest of the three
tier fractions over drafted positions (greedy drafts mixed with the
workload's rate of uniformly random tokens).  Values are frozen as fp32
literals.
"""
TEMPERATURE = {
    '1b_bf16': 28.40304946899414,
    '8b_bf16_chain': 33.97911834716797,
    '8b_bf16_long': 8.428129196166992,
    '8b_bf16_tree': 33.97911834716797,
}
MIXED_TEMPERATURE = {
    '8b_bf16_chain': 8.306769371032715,
    '8b_bf16_long': 8.428129196166992,
}
