"""The oracle against its stored outputs on config 1 (tests/golden/, written
by tests/golden/make_golden.py from the oracle alone): any change of the
oracle's arithmetic shows up here and has to be justified and re-recorded."""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden"))
import make_golden  # noqa: E402


def test_oracle_matches_stored_config1_outputs():
    stored = make_golden.read()
    now = make_golden.compute()
    assert set(stored) == set(now)
    for k in ("visual_index", "budget", "keep_idx", "cu_out"):
        assert [int(x) for x in stored[k]] == now[k], k
    for k in ("score", "img_sum"):
        np.testing.assert_allclose(now[k], stored[k], rtol=1e-12, atol=0.0, err_msg=k)
