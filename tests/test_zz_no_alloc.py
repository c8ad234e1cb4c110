"""The allocation-free scoring entry point (ps_score_window_dev_fixed)
against the allocating one (ps_score_window_dev), through the C ABI (needs
an MI355X): byte-identical results and set sizes on two calls in a row, the
second smaller, on windows that take every scoring path, then the limit."""
import sys

import numpy as np
import pytest

import synth
from tests.gpu_util import DeviceWindow, load_window

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ps():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_33224_amd as ps
    return ps


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# c3: 65,536 requests (the fixed scratch's limit) on 1,024 instances, with
# popular groups (the general scorer's class path); c2: 64 instances (the
# small-pool kernels); c5's first 20,000 requests on 4,096 instances.
@pytest.mark.parametrize("name,n_big,n_small", [("c3", 65536, 5000), ("c2", 16384, 700),
                                                ("c5", 20000, 3)])
def test_fixed_scratch_matches_allocating_entry(ps, name, n_big, n_small):
    _say(f"no-alloc {name}: {n_big} then {n_small} requests")
    w = synth.generate(name)
    sc = ps.Scorer(0)
    try:
        load_window(sc, w)
        wins = [DeviceWindow(w.subset(range(n))) for n in (n_big, n_small)]
        want = []
        for dw in wins:
            res, sizes = dw.score(sc)
            res_ns, _ = dw.score(sc, with_sizes=False)
            want.append((res.tobytes(), sizes.copy(), res_ns.tobytes()))
        # two calls in a row of each kind, the second with the smaller window
        got = [dw.score(sc, fixed=True) for dw in wins]
        got_ns = [dw.score(sc, with_sizes=False, fixed=True)[0] for dw in wins]
        for k, dw in enumerate(wins):
            assert got[k][0].tobytes() == want[k][0], f"{name} call {k}: results differ"
            assert (got[k][1] == want[k][1]).all(), f"{name} call {k}: set sizes differ"
            assert got_ns[k].tobytes() == want[k][2], f"{name} call {k}: results without sizes differ"
        _say(f"no-alloc {name}: identical")
    finally:
        sc.close()


def test_fixed_scratch_limit(ps):
    import torch
    w = synth.generate("c1")
    sc = ps.Scorer(0)
    try:
        load_window(sc, w)
        n = 65537
        idx = np.arange(n) % w.n_req
        dw = DeviceWindow(w.subset(idx))
        with pytest.raises(ps.PackServeError) as e:
            dw.score(sc, fixed=True)
        assert e.value.code == ps.binding.PS_E_RANGE
        # a call after the refused one works
        dw = DeviceWindow(w)
        a, sa = dw.score(sc)
        b, sb = dw.score(sc, fixed=True)
        assert a.tobytes() == b.tobytes() and (sa == sb).all()
    finally:
        sc.close()
