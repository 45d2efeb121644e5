"""Concurrent calls: the library keeps no shared state between calls (each
call brings its own reserve and scratch), so layers driven from several host
threads, each on its own stream, give the results of the same layers run one
after another on the default stream."""

import numpy as np
import pytest

from paper_2603_06492_amd import inputs as inp

from _parity import TOL, parity_report

pytestmark = pytest.mark.gpu

LAYERS = [
    # name, T, d_in, d_out, r, groups, dtype
    ("bf16_a", 700, 256, 264, 64, 1, "bf16"),
    ("bf16_g3", 300, 128, 192, 40, 3, "bf16"),
    ("bf16_r0", 513, 200, 136, 0, 1, "bf16"),
    ("f32_b", 257, 96, 80, 24, 1, "f32"),
]


def test_threads_on_their_own_streams():
    import threading
    import torch
    from paper_2603_06492_amd.runner import DeviceProblem
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    print("[streams] sequential reference", flush=True)
    probs = [inp.draw_projection(n, T, di, do, r, dt, seed=501 + i, bias_std=0.5, groups=G)
             for i, (n, T, di, do, r, G, dt) in enumerate(LAYERS)]
    dps = [DeviceProblem(p) for p in probs]
    for dp in dps:
        dp.fwd()
        dp.bwd()
    ref = [dp.outputs() for dp in dps]
    for dp in dps:
        for t in [dp.y] + [v for v in dp.g.values() if v is not None]:
            t.fill_(float("nan"))
    torch.cuda.synchronize()

    print("[streams] four threads, four streams", flush=True)
    errors = []
    start = threading.Barrier(len(dps))

    def run(dp):
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.default_stream())
            start.wait()
            with torch.cuda.stream(s):
                for _ in range(5):
                    dp.fwd(stream=s)
                    dp.bwd(stream=s)
            s.synchronize()
        except Exception as e:   # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=run, args=(dp,)) for dp in dps]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for (name, *_, dt), dp, want in zip(LAYERS, dps, ref):
        got = dp.outputs()
        for k in ("y", "dx", "dW"):
            np.testing.assert_array_equal(got[k], want[k], err_msg=f"{name} {k}")
        rep = parity_report(got, want)
        print(name, rep, flush=True)
        for k, e in rep.items():
            assert e <= TOL[dt] / 10, (name, k, e)
