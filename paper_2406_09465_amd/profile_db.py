"""On-disk database of measured candidate latencies (the profile cache that
lets the orchestration search halt and resume, as the tuning-time discussion
of Korch's evaluation assumes).

A record is keyed by a hash of the candidate kernel's generated source (which
carries the primitives, shapes, dtypes, layout and the device prelude), the
profiling protocol (warm-up launches, timed repetitions, flush bytes) and the
device (architecture name and marketing name).  A changed code generator,
shape or protocol therefore never reuses a stale latency.  The value is the
median latency in microseconds, or None for a candidate no family implements
(infinite cost).  The file is JSON, written atomically; the database saves
itself every ``save_every`` new records, so an interrupted search resumes
from the last save.
"""

from __future__ import annotations

import hashlib
import json
import os

PKG = os.path.dirname(os.path.abspath(__file__))


def default_path():
    return os.environ.get("KORCH_PROFILE_DB") or os.path.join(PKG, "_profile_db", "latency.json")


def device_tag():
    import torch
    p = torch.cuda.get_device_properties(torch.cuda.current_device())
    return f"{getattr(p, 'gcnArchName', '?')}|{p.name}"


class ProfileDB:
    def __init__(self, path=None, save_every=50):
        self.path = path or default_path()
        self.save_every = save_every
        self.data = {}
        self.new = 0
        self.hits = 0
        if os.path.exists(self.path):
            try:
                self.data = json.load(open(self.path))
            except (OSError, ValueError):
                self.data = {}

    # Version of the measurement protocol (korch_profile_candidate): a change in
    # how a candidate is timed invalidates every record.
    PROTOCOL = "dispatch-timestamps/flush-each-rep/warm-intermediates/median/v3"

    @staticmethod
    def key(source, warmup, reps, flush_bytes, device):
        h = hashlib.sha256()
        cold = os.environ.get("KORCH_PROFILE_COLD", "") == "1"
        wflush = os.environ.get("KORCH_FLUSH_WRITE", "") == "1"
        for part in (ProfileDB.PROTOCOL, "cold" if cold else "warm", "wflush" if wflush else "rflush", source, str(warmup), str(reps),
                     str(flush_bytes), device):
            h.update(part.encode())
            h.update(b"\0")
        return h.hexdigest()[:32]

    def get(self, key):
        """(found, value)."""
        if key in self.data:
            self.hits += 1
            return True, self.data[key]
        return False, None

    def put(self, key, value):
        self.data[key] = value
        self.new += 1
        if self.new % self.save_every == 0:
            self.save()

    def save(self):
        os.makedirs(os.path.dirname(self.path), exist_ok=True)
        tmp = f"{self.path}.tmp{os.getpid()}"
        with open(tmp, "w") as f:
            json.dump(self.data, f)
        os.replace(tmp, self.path)
