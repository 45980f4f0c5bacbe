"""The on-disk profile database of candidate latencies (halt and resume of the
orchestration search): keys, persistence and reuse by the chooser."""

import json

from paper_2406_09465_amd.profile_db import ProfileDB


def test_key_depends_on_source_protocol_and_device():
    k = ProfileDB.key("src", 10, 100, 512 << 20, "gfx950|MI355X")
    assert k == ProfileDB.key("src", 10, 100, 512 << 20, "gfx950|MI355X")
    others = [ProfileDB.key("src2", 10, 100, 512 << 20, "gfx950|MI355X"),
              ProfileDB.key("src", 20, 100, 512 << 20, "gfx950|MI355X"),
              ProfileDB.key("src", 10, 50, 512 << 20, "gfx950|MI355X"),
              ProfileDB.key("src", 10, 100, 256 << 20, "gfx950|MI355X"),
              ProfileDB.key("src", 10, 100, 512 << 20, "gfx942|MI300X")]
    assert len(set(others + [k])) == len(others) + 1


def test_records_persist_and_resume(tmp_path):
    path = str(tmp_path / "db" / "latency.json")
    db = ProfileDB(path, save_every=2)
    db.put("a", 1.5)
    assert not (tmp_path / "db" / "latency.json").exists()
    db.put("b", None)  # unsupported: infinite cost is recorded too
    assert json.load(open(path)) == {"a": 1.5, "b": None}  # saved every 2 records
    db.put("c", 2.25)
    db.save()
    db2 = ProfileDB(path)
    assert db2.get("a") == (True, 1.5)
    assert db2.get("b") == (True, None)
    assert db2.get("c") == (True, 2.25)
    assert db2.get("d") == (False, None)
    assert db2.hits == 3


def test_unreadable_database_starts_empty(tmp_path):
    p = tmp_path / "latency.json"
    p.write_text("{not json")
    assert ProfileDB(str(p)).data == {}


def test_chooser_reuses_recorded_latencies(tmp_path, monkeypatch):
    """profile_candidates takes a recorded latency instead of profiling, and
    records what it profiles (the profiler itself is replaced: no GPU here)."""
    from paper_2406_09465_amd import chooser, graphs
    from paper_2406_09465_amd import profile_db
    monkeypatch.setattr(profile_db, "device_tag", lambda: "gfx950|test")
    w = graphs.mlp(m=64, d=32, h=48)
    g = w.graph
    cands = [tuple(map(tuple, k)) for k in w.kernels("fused")]
    calls = []

    def fake_profile(p, o, warmup, reps, flush_bytes):
        calls.append((p, o))
        return 10.0 + len(p)
    monkeypatch.setattr(g, "profile", fake_profile)
    db = ProfileDB(str(tmp_path / "l.json"))
    c1 = chooser.profile_candidates(g, cands, warmup=2, reps=5, flush_bytes=1 << 20, db=db)
    assert len(calls) == len(cands) and db.new == len(cands)
    db2 = ProfileDB(str(tmp_path / "l.json"))
    c2 = chooser.profile_candidates(g, cands, warmup=2, reps=5, flush_bytes=1 << 20, db=db2)
    assert c2 == c1 and len(calls) == len(cands) and db2.hits == len(cands)
    # another protocol (more reps) profiles again
    db3 = ProfileDB(str(tmp_path / "l.json"))
    chooser.profile_candidates(g, cands, warmup=2, reps=6, flush_bytes=1 << 20, db=db3)
    assert len(calls) == 2 * len(cands)
