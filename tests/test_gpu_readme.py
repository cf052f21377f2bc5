"""The Python example of README.md runs as written.

The CPU test checks that the block compiles and names only what the binding
defines.  The GPU test (needs an MI355X) executes the block and compares its
outputs with the oracle's on the same inputs, bit for bit; the inputs are
drawn again from the block's seeded generator, in the block's order.
"""
import ast
import os
import re
import sys

import numpy as np
import pytest

from paper_2608_12123_amd import rc_cohort as rc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KEYS = ("state", "outcome", "eff_sid", "eff_tool", "eff_payload", "n_taken")


def readme_block() -> str:
    path = os.path.join(ROOT, "README.md")
    if not os.path.exists(path):  # a copy of the tree without its documentation
        pytest.skip("README.md is not in this copy of the tree")
    with open(path) as f:
        text = f.read()
    sec = text.index("## Use from Python")
    m = re.compile(r"```python\n(.*?)```", re.S).search(text, sec)
    assert m is not None, "no python block under 'Use from Python'"
    return m.group(1)


def test_readme_block_names_the_binding():
    tree = ast.parse(readme_block())
    used = {n.attr for n in ast.walk(tree)
            if isinstance(n, ast.Attribute) and isinstance(n.value, ast.Name) and n.value.id == "rc"}
    assert used, "the block calls nothing of the binding"
    for name in used:
        assert hasattr(rc, name), name
    methods = {n.func.attr for n in ast.walk(tree)
               if isinstance(n, ast.Call) and isinstance(n.func, ast.Attribute)
               and isinstance(n.func.value, ast.Name) and n.func.value.id == "co"}
    for name in methods:
        assert hasattr(rc.Cohort, name), name


@pytest.mark.gpu
def test_readme_block_matches_oracle():
    import oracle
    print("readme block: N=1000 W=32 R=256 T=16 (mod routes, p = 0.5)", flush=True)
    sys.stdout.flush()
    ns = {}
    exec(compile(readme_block(), "README.md", "exec"), ns)
    N, W, R, T = ns["N"], ns["W"], ns["R"], ns["T"]
    rng = np.random.default_rng(0)
    table = rng.integers(0, 2**32, size=(R, 16), dtype=np.uint32)
    state = rng.integers(0, 2**32, size=(W, N), dtype=np.uint32)
    outcome = rng.integers(0, 2**32, size=N, dtype=np.uint32)
    assert np.array_equal(table, ns["table"]), "the inputs were not redrawn in the block's order"
    oracle.build(force=False)
    want = oracle.load().run_chain(n_words=W, n_routes=R, cohort_offsets=ns["offsets"],
                                   table=table, route_mode=rc.RC_ROUTE_MOD, route_cdf=None,
                                   decide_thr=32768, state=state, outcome=outcome, n_steps=T)
    got = ns["out"]
    for k in KEYS:
        assert np.array_equal(got[k], want[k]), k
