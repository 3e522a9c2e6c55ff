"""The hand-off latency calibration behind the pipelined passes' latency
roofline: one LDS hand-off between two waves and device-scope hand-offs
between workgroups, measured through the C ABI."""
import pytest

from paper_2509_21221_amd import mcf

pytestmark = pytest.mark.gpu


def test_handoff_calibration_reports_plausible_latencies():
    import torch

    torch.cuda.init()
    out = mcf.gwtf_mcf_calibrate_handoff(0, torch.cuda.current_stream().cuda_stream, 4)
    print(out, flush=True)
    # every bounded wait completed, and each hand-off takes between one
    # cycle-scale event and a few microseconds
    for key in ("lds_wave_ns", "device_neighbour_ns", "device_same_xcd_ns"):
        assert 1.0 < out[key] < 20000.0, (key, out)
    # crossing between CUs costs more than staying in one CU's LDS
    assert out["lds_wave_ns"] < out["device_neighbour_ns"]


def test_handoff_calibration_rejects_bad_arguments():
    with pytest.raises(mcf.GwtfError):
        mcf.gwtf_mcf_calibrate_handoff(0, 0, 8)
    with pytest.raises(mcf.GwtfError):
        mcf.gwtf_mcf_calibrate_handoff(0, 0, 0)
    with pytest.raises(mcf.GwtfError):
        mcf.gwtf_mcf_calibrate_handoff(-1, 0, 4)
