"""The committed oracle against every pin in oracle_pins.py (CPU only)."""
import pytest

import os, sys
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle_pins as P  # noqa: E402


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(olib, pin):
    pin(olib)


def test_digest_of_empty_trace(olib):
    import numpy as np
    s, dg, fin = olib.simulate_job(np.zeros(0), np.zeros(0, np.int32), np.ones(1), np.array([1], np.int32),
                                   np.ones((1, 1, 1)), np.zeros(1, np.int32), np.ones(1, np.uint64), 5.0,
                                   want_finish=True)
    assert s == 0 and dg == (0, 0) and len(fin) == 0


def test_oracle_refuses_inputs_outside_the_model(olib):
    import numpy as np
    args = dict(t=np.zeros(2), model=np.array([0, 1], np.int32), d_single=np.ones(2),
                cfg_stages=np.array([1], np.int32), stage_lat=np.ones((2, 1, 1)),
                group_cfg=np.array([0, -1], np.int32), host_mask=np.array([1, 2], np.uint64),
                slo_scale=5.0)
    with pytest.raises(ValueError):  # model 1 hosted on an unused group
        olib.simulate_job(**args)
    args["host_mask"] = np.array([1, 1], np.uint64)
    args["model"] = np.array([0, 2], np.int32)
    with pytest.raises(ValueError):  # model id out of range
        olib.simulate_job(**args)
