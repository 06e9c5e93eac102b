"""Host-side decoding of per-tile traces (no GPU)."""
import json

import numpy as np

from paper_2511_12500_amd import trace as T


def _raw():
    # two tiles, 100 MHz clock (10 ns ticks); tile 1 also has a copy step
    r = np.zeros((2, T.WORDS), dtype=np.uint64)
    r[0, [T.START, T.MAINLOOP, T.STORED, T.RELEASED]] = [1000, 1100, 1150, 1160]
    r[1, [T.START, T.MAINLOOP, T.STORED, T.RELEASED]] = [1010, 1120, 1170, 1180]
    r[1, [T.COPY_WAIT, T.COPY_GO, T.COPY_DONE]] = [1005, 1185, 1300]
    hw = (3 << 8) | (1 << 12) | (2 << 13)          # cu 3, sh 1, se 2
    r[0, T.WHERE] = np.uint64((hw << 32) | (5 << 16) | 17)
    r[1, T.WHERE] = np.uint64((hw << 32) | (0 << 16) | 200)
    return r


def test_decode_times_and_location():
    t = T.decode(_raw(), 100_000)
    assert t["start"].tolist() == [0.0, 0.1]
    assert np.allclose(t["mainloop"], [1.0, 1.2])
    assert np.isnan(t["copy_done"][0]) and np.isclose(t["copy_done"][1], 3.0)
    assert t["wg"].tolist() == [17, 200] and t["xcc"].tolist() == [5, 0]
    assert t["cu"].tolist() == [3, 3] and t["sh"].tolist() == [1, 1] and t["se"].tolist() == [2, 2]


def test_summary_and_chrome_export(tmp_path):
    t = T.decode(_raw(), 100_000)
    s = T.summary(t)
    assert s["tiles"] == 2
    assert np.isclose(s["mainloop_us"]["min"], 1.0) and np.isclose(s["mainloop_us"]["max"], 1.1)
    assert np.isclose(s["copy_wait_us"]["max"], 1.8) and np.isclose(s["span_us"], 3.0)
    path = tmp_path / "tl.json"
    T.write_chrome(t, str(path))
    ev = json.loads(path.read_text())["traceEvents"]
    names = sorted(e["name"] for e in ev)
    assert names == ["copy", "copy wait", "mainloop", "mainloop", "release", "release",
                     "store", "store"]
    assert all(e["dur"] >= 0 for e in ev)


def test_unwritten_tiles_are_skipped():
    r = _raw()
    r[0, :] = 0
    t = T.decode(r, 100_000)
    assert not t["written"][0] and T.summary(t)["tiles"] == 1
    assert len([e for e in T.chrome_events(t) if e["name"] == "mainloop"]) == 1
