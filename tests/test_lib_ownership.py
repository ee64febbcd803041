"""Host logic of the binding's ownership of spread buffers, on the CPU with a
stand-in library that records the native calls: a context closed while its
buffers live is detached from the API at once and destroyed with the last
buffer; every buffer is freed exactly once, through the context it came from."""
import gc

import pytest

from paper_2609_36662_amd import _lib


class _Recorder:
    def __init__(self):
        self.calls = []

    def autoloco_destroy(self, h):
        self.calls.append(("destroy", h))

    def autoloco_free(self, h, ptr):
        self.calls.append(("free", h, ptr.value))
        return 0


@pytest.fixture()
def rec(monkeypatch):
    r = _Recorder()
    monkeypatch.setattr(_lib, "lib", lambda: r)
    return r


def _ctx(handle):
    c = _lib.Context.__new__(_lib.Context)   # no device: the handle is a token
    c.handle, c.device, c._live, c._held = handle, 0, 0, None
    return c


def test_close_without_buffers_destroys_at_once(rec):
    c = _ctx("H")
    c.close()
    c.close()
    assert rec.calls == [("destroy", "H")] and c.handle is None


def test_context_outlives_close_until_the_last_buffer(rec):
    c = _ctx("H")
    a, b = _lib._DeviceBuffer(c, 0x1000, 64), _lib._DeviceBuffer(c, 0x2000, 64)
    c.close()
    assert c.handle is None and rec.calls == []
    del a
    gc.collect()
    assert rec.calls == [("free", "H", 0x1000)]
    del b
    gc.collect()
    assert rec.calls == [("free", "H", 0x1000), ("free", "H", 0x2000), ("destroy", "H")]
    c.close()
    assert len(rec.calls) == 3


def test_buffers_freed_before_close(rec):
    c = _ctx("H")
    a = _lib._DeviceBuffer(c, 0x1000, 64)
    del a
    gc.collect()
    c.close()
    assert rec.calls == [("free", "H", 0x1000), ("destroy", "H")]


def test_a_failing_free_still_releases_the_context(monkeypatch, rec):
    def boom(h, ptr):
        raise OSError("native free failed")
    c = _ctx("H")
    a = _lib._DeviceBuffer(c, 0x1000, 64)
    c.close()
    monkeypatch.setattr(rec, "autoloco_free", boom)
    a.__del__()
    assert c._live == 0 and rec.calls == [("destroy", "H")]
    a.__del__()   # a second call does nothing
    assert c._live == 0 and rec.calls == [("destroy", "H")]
