"""The minimal-staleness bound on measured stage durations (Sec. 3.2;
App. D.1 profiles a few iterations): the stage times of a sequential run on
the GPU, then the library's solver against the oracle's on those times."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle.staleness_schedule import min_staleness  # noqa: E402
from workloads import make_weights, make_workload  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2402_15113_amd import tgm
    tgm.lib()


@pytest.mark.parametrize("mitigation", [None, dict(p=0.6, lam=0.95, K=4)])
def test_bound_from_measured_stage_times(mitigation):
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import (from_workload, minimal_staleness,
                                            stage_durations_us)
    wl = make_workload("tiny", E=8000)
    st = from_workload(wl, make_weights(wl.M, wl.D_e, wl.D_t), mitigation=mitigation)
    for i in range(3):
        st.step(i)
    torch.cuda.synchronize()
    tgm.tgm_profile_reset()
    tgm.tgm_profile_enable(True)
    n = 12
    for i in range(3, 3 + n):
        st.step(i)
    torch.cuda.synchronize()
    tgm.tgm_profile_enable(False)
    tau = stage_durations_us(tgm.tgm_profile_read(), n)
    print("stage durations (us):", [round(t, 2) for t in tau], flush=True)
    assert tau[1] == 0.0 and all(tau[j] > 0 for j in (0, 2, 3, 4))
    res = minimal_staleness(tau, k_max=16, n=64)
    ref = min_staleness(tau, 64, 16)
    assert res["k_min"] == ref[-1][0] >= 1
    assert res["stall_free"] == (ref[-1][2] == 0.0)
    st.close()


def test_calibrated_staleness_drives_the_run(orc):
    """The online schedule: the bound solved from a calibration stage's
    profiled steps sets the s of a fresh run, which matches the oracle at that
    s (and the pipelined executor runs it as well)."""
    from paper_2402_15113_amd.stage import calibrate_staleness, from_workload
    from test_gpu_parity import run_pair
    wl = make_workload("tiny", E=8000)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    cal_stage = from_workload(wl, w)
    cal = calibrate_staleness(cal_stage)
    cal_stage.close()
    print("calibrated:", cal, flush=True)
    assert cal["s"] == cal["k_min"] - 1 >= 0
    assert cal["calibration"] == {"first": 0, "warm": 3, "iters": 12}
    assert min_staleness([cal["tau_us"][k] for k in ("sample", "feature_fetch", "memory_fetch",
                                                     "compute", "memory_update")],
                         64, 16)[-1][0] == cal["k_min"]
    run_pair(orc, make_workload("tiny", E=8000, s=cal["s"]), w, s=cal["s"])
