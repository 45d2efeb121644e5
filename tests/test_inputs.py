"""The seeded input recipe: the four-block stack's Q, K and V read one block
input, every other array is drawn per projection."""

import numpy as np

from paper_2603_06492_amd import inputs as inp


def test_stack_shares_the_block_input_across_q_k_v():
    name = "llm1p5b_stack4_r128"
    src = inp.workload_x_source(name)
    assert src == [6 * (i // 6) if i % 6 in (1, 2) else i for i in range(24)]
    q, k, v, o = (inp.draw_workload_projection(name, i, T=16) for i in range(4))
    assert np.array_equal(q["x"], k["x"]) and np.array_equal(q["x"], v["x"])
    assert not np.array_equal(q["x"], o["x"])
    # the rest of K is K's own draw
    assert not np.array_equal(q["W"], k["W"]) and not np.array_equal(q["dy"], k["dy"])
    # block 1's Q has its own input
    assert not np.array_equal(q["x"], inp.draw_workload_projection(name, 6, T=16)["x"])


def test_draw_x_is_the_first_draw():
    p = inp.draw_projection("t", 5, 24, 16, 8, "bf16", seed=9)
    assert np.array_equal(inp.draw_x(5, 24, "bf16", 9), p["x"])
    p = inp.draw_projection("t", 5, 24, 16, 8, "f32", seed=9)
    assert np.array_equal(inp.draw_x(5, 24, "f32", 9), p["x"])


def test_other_workloads_read_their_own_input():
    for name in inp.WORKLOADS:
        if name != "llm1p5b_stack4_r128":
            assert inp.workload_x_source(name) == list(range(len(inp.WORKLOADS[name]["projections"])))
