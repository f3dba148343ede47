"""Host logic of the averaged multi-group trainer (stack.AveragedGroups):
every group steps once per step, and the models are averaged, one call per
parameter tensor over the groups' copies, after steps period, 2 period, ...
(sec. 4: averaging every given number of batches).  No GPU: the groups are
stand-ins that count their steps."""
import pytest

from paper_2112_15317_amd.stack import AveragedGroups


class _Group:
    def __init__(self):
        self.steps = 0

    def step(self, stream=None):
        self.steps += 1


@pytest.mark.parametrize("period,steps", [(1, 3), (3, 7), (4, 4)])
def test_average_after_every_period(period, steps):
    ag = object.__new__(AveragedGroups)
    ag.groups = [_Group(), _Group(), _Group()]
    ag.sets = [["w0g0", "w0g1", "w0g2"], ["b0g0", "b0g1", "b0g2"]]
    ag.period, ag.steps_done = period, 0
    log = []
    ag.call = lambda key, fn, *args: log.append((ag.steps_done, key, args[0]))
    for _ in range(steps):
        ag.step()
    assert all(g.steps == steps for g in ag.groups)
    want = []
    for s in range(1, steps + 1):
        if s % period == 0:
            want += [(s, ("avg", 0), ag.sets[0]), (s, ("avg", 1), ag.sets[1])]
    assert log == want


def test_rejects_bad_configuration():
    with pytest.raises(ValueError):
        AveragedGroups(None, 4, 3, 32, [], groups=0, period=1)
    with pytest.raises(ValueError):
        AveragedGroups(None, 4, 3, 32, [], groups=2, period=0)
