"""The measured cost model: one small grid point timed on the GPU, fed to the
library's Eq. 1-4, agrees with the oracle's cost model on the same times."""
import pytest

import oracle.costmodel as ref
from gpu_util import say
from paper_2408_11049_amd import costmodel

pytestmark = pytest.mark.gpu


def test_measured_point_through_the_cost_model():
    m = costmodel.measure(B=4, S=4096, max_gamma=4, reps=2)
    say(f"  B=4 S=4096: T_T {m['t_target']:.1f} us, T_V {[round(x, 1) for x in m['t_verify']]}, "
        f"T_D {m['t_draft_streaming']:.1f} / {m['t_draft_listed']:.1f} / "
        f"{m['t_draft_gathered']:.1f} us")
    assert len(m["t_verify"]) == 4 and all(t > 0 for t in m["t_verify"])
    assert m["t_target"] > 0 and m["t_draft_streaming"] > 0 and m["t_draft_listed"] > 0
    assert m["t_draft_gathered"] > 0
    model = costmodel.analyse(m)
    for name, td in (("streaming", m["t_draft_streaming"]), ("listed", m["t_draft_listed"]),
                     ("gathered", m["t_draft_gathered"])):
        for a in costmodel.ALPHAS:
            g, r = ref.best_gamma(a, m["t_target"], td, m["t_verify"])
            got = model[f"{name}@{a}"]
            assert got["gamma"] == g and abs(got["ratio"] - r) <= 1e-12 * r
