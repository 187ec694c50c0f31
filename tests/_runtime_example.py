"""The paper's runtime example (App. A.5) as a pool-level replay.

Printed values (tests/golden/runtime_example_app_a5.json): the founder
tau_p was branched from its root at decoding step 13,934 and inherited
14,004 tokens, so the root held a 70-token prompt plus its 13,934 generated
tokens; tau_p later generated 20,669 tokens of its own.  Its child tau_B
inherited 31,404 tokens, i.e. tau_p had generated 17,400 when that branch
happened, and tau_B generated 3,649 of its own.

The replay uses three slots (root 0, tau_p 1, tau_B 2) and grows traces
with allocations (one trace at a time, so the blocks are those a run of
single-token decode steps would take).
"""
import json
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "runtime_example_app_a5.json")
BS = 16


def load():
    with open(GOLDEN) as f:
        return json.load(f)


def schedule(g):
    """[(op, args)] of the replay: alloc / fork in order."""
    p, b = g["tau_p"], g["tau_B"]
    prompt = p["inherited_tokens"] - p["created_at_step"]
    p_before_b = b["inherited_tokens"] - p["inherited_tokens"]
    return [
        ("alloc", [0], [prompt + p["created_at_step"]]),
        ("fork", [0], [1]),
        ("alloc", [1], [p_before_b]),
        ("fork", [1], [2]),
        ("alloc", [1, 2], [p["generated_tokens"] - p_before_b, b["generated_tokens"]]),
    ]


def expected_lengths(g):
    p, b = g["tau_p"], g["tau_B"]
    return {
        0: p["inherited_tokens"],
        1: p["inherited_tokens"] + p["generated_tokens"],
        2: b["inherited_tokens"] + b["generated_tokens"],
    }
