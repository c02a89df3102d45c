"""The seed log: generation records survive a JSON round trip exactly (the
binary32 rewards and 64-bit checksums included), and a log of another format
is refused."""
import json

import numpy as np
import pytest

from paper_2608_17310_amd.generation import GenerationRecord, save_log, load_log


def test_seed_log_round_trip(tmp_path):
    rng = np.random.default_rng(0)
    recs = []
    for t in range(5):
        rew = [float(np.float32(x)) for x in rng.standard_normal(6)]
        recs.append(GenerationRecord(seeds=[(1 << 64) - 1 - t, 7, 7, 9, 10, 11],
                                     signs=[1, 1, -1, 1, -1, 1], rewards=rew,
                                     sigma=float(np.float32(1e-3 * (t + 1) / 3)), alpha=5e-4,
                                     flags=4 if t % 2 else 0, zscore_eps=1e-8,
                                     fused_swap=bool(t % 2), round_seed=(1 << 63) + t,
                                     checksum=None if t == 2 else (1 << 64) - 1 - 977 * t))
    path = tmp_path / "log.json"
    save_log(path, recs, meta={"workload": "tiny-1m", "base": "checkpoint-0"})
    back, meta = load_log(path)
    assert back == recs
    assert meta == {"workload": "tiny-1m", "base": "checkpoint-0"}
    for a, b in zip(recs, back):
        assert np.array_equal(np.float32(a.rewards), np.float32(b.rewards))


def test_seed_log_rejects_other_files(tmp_path):
    p = tmp_path / "x.json"
    p.write_text(json.dumps({"format": "something-else", "generations": []}))
    with pytest.raises(ValueError):
        load_log(p)
    p.write_text(json.dumps({"format": "es-generation-log/1", "meta": {},
                             "generations": [{"seeds": [1], "bogus": 2}]}))
    with pytest.raises(ValueError):
        load_log(p)
