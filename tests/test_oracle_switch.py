"""Pins of the oracle's storage switch and periodic schedule (Sec. 4.3 and the
appendix's implementation details): the optimizer only ever sees the expert
storage, bit for bit; the simulated view shows the latest simulate; offload
mode refills the buffer with the frozen base on restore; one simulated step
closes each cycle of t steps."""
import numpy as np
import pytest

import oracle
from oracle import EXPERT, SIMULATED, StateError, StorageSwitch


def _lists():
    rng = np.random.default_rng(0)
    th = [rng.standard_normal(n).astype(np.float32) for n in (3, 100)]
    t0 = [rng.standard_normal(n).astype(np.float32) for n in (3, 100)]
    return th, t0


def test_resident_cycle():
    th, t0 = _lists()
    sw = StorageSwitch(th, t0)
    assert sw.state == EXPERT
    with pytest.raises(StateError):
        sw.switch(SIMULATED)                 # nothing simulated yet
    sim = [x + 1 for x in th]
    sw.simulate(sim)
    sw.switch(SIMULATED)
    for a, b in zip(sw.active(), sim):
        np.testing.assert_array_equal(a, b)
    with pytest.raises(StateError):
        sw.simulate(sim)                     # buffer in use by the model
    with pytest.raises(StateError):
        sw.switch(SIMULATED)                 # double switch
    sw.switch(EXPERT)
    for a, b in zip(sw.active(), th):
        assert a.tobytes() == b.tobytes()
    sw.switch(EXPERT)                        # restoring is idempotent
    with pytest.raises(StateError):
        sw.switch(SIMULATED)                 # stale buffer after restore
    with pytest.raises(ValueError):
        sw.switch(7)


def test_offload_restore_refills_base():
    th, t0 = _lists()
    sw = StorageSwitch(th, t0, offload=True)
    for a, b in zip(sw.buffer, t0):
        np.testing.assert_array_equal(a, b)
    sw.simulate([x * 3 for x in th])
    with pytest.raises(StateError):
        sw.simulate([x * 3 for x in th])     # the buffer holds theta~, not the base, until a restore
    sw.switch(SIMULATED)
    sw.switch(EXPERT)
    for a, b in zip(sw.buffer, t0):
        assert a.tobytes() == b.tobytes()
    sw.simulate([x * 2 for x in th])         # refilled: the next simulate may run
    sw.switch(EXPERT)                        # restoring the expert view without using theta~
    with pytest.raises(StateError):
        sw.simulate([x * 2 for x in th])     # no restore happened (the view was already the expert's)


def test_resident_simulate_may_repeat():
    """Resident mode keeps theta0 apart from the buffer, so simulating again before using theta~
    just replaces it."""
    th, t0 = _lists()
    sw = StorageSwitch(th, t0)
    sw.simulate([x + 1 for x in th])
    sw.simulate([x + 2 for x in th])
    sw.switch(SIMULATED)
    for a, b in zip(sw.active(), th):
        np.testing.assert_array_equal(a, b + 2)


@pytest.mark.parametrize("n", [1, 3, 4, 7, 8, 100, 101])
def test_periodic_schedule_counts(n):
    sims = [k for k in range(n) if oracle.is_simulated_step(k, 4)]
    assert len(sims) == n // 4
    assert all(k % 4 == 3 for k in sims)
    # period 1 simulates every step (lambda = 1)
    assert all(oracle.is_simulated_step(k, 1) for k in range(n))
    with pytest.raises(ValueError):
        oracle.is_simulated_step(0, 0)
