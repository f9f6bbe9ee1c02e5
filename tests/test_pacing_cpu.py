"""Host logic of the chunk-walk pacer, with a stand-in for device events."""
import pytest
import torch

from paper_2503_10377_amd import pacing


class FakeEvent:
    log = []
    count = 0

    def __init__(self):
        self.id = FakeEvent.count
        FakeEvent.count += 1
        FakeEvent.log.append(("new", self.id))

    def record(self, stream):
        FakeEvent.log.append(("record", self.id))

    def synchronize(self):
        FakeEvent.log.append(("sync", self.id))


@pytest.fixture
def fake_events(monkeypatch):
    FakeEvent.log = []
    FakeEvent.count = 0
    monkeypatch.setattr(torch.cuda, "Event", FakeEvent)
    return FakeEvent.log


@pytest.mark.parametrize("ahead", [1, 2, 5])
def test_pacer_waits_for_the_boundary_ahead_back(fake_events, ahead):
    p = pacing.HostPacer(ahead)
    for n in range(12):
        p.boundary(None)
        synced = [i for k, i in fake_events if k == "sync"]
        # after boundary n, every boundary up to n - ahead has been waited for, in order
        assert synced == list(range(max(0, n + 1 - ahead)))
    p.drain()
    assert [i for k, i in fake_events if k == "sync"] == list(range(12))


def test_pacer_zero_disables(fake_events):
    p = pacing.HostPacer(0)
    for _ in range(5):
        p.boundary(None)
    assert fake_events == []
    with pytest.raises(ValueError):
        pacing.HostPacer(-1)
