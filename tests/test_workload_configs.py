"""Every configuration the benchmark, the smoke run and the workloads use is
one the library accepts: with anomaly elimination on, a warm-up of at least
edit_outer_min_warmup(alpha, delta) rounds (Sec. 3.2, Eq. 1 from the zero EMA
state).  CPU only: the check is the library's host-side function."""
import pytest

import __graft_entry__
from paper_2412_07210_amd import min_warmup, synth


@pytest.mark.parametrize("name", sorted(synth.WORKLOADS))
def test_workload_warmup_is_accepted(name):
    h = synth.get(name).hyper()
    assert h["warmup_rounds"] >= min_warmup(h["ema_alpha"], h["z_threshold"]), name


def test_smoke_workload_warmup_is_accepted():
    wl = __graft_entry__.smoke_workload()
    h = wl.hyper()
    assert h["warmup_rounds"] == min_warmup(h["ema_alpha"], h["z_threshold"])
    assert wl.num_workers == 4 and wl.num_units == 3
