"""Temperatures fixed by tests/golden/calibrate_temperature.py (oracle only).

Each bf16 workload scales its logits so that about half of the drafted
positions (teacher-forced greedy windows) clear the accept threshold;
the 8B-shape workloads share one model and one temperature.  Values are
frozen as fp32 literals.
"""
TEMPERATURE = {
    '1b_bf16': 28.40304946899414,
    '8b_bf16_chain': 33.97911834716797,
    '8b_bf16_long': 33.97911834716797,
    '8b_bf16_tree': 33.97911834716797,
}
