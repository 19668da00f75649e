"""Host-side accounting of the benchmark line (CPU): the algorithmic bytes of a
decode step, the lookup of committed HBM counters, and that every leg the
benchmark reports has a counter entry under the name it looks up."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_21042_amd import workload  # noqa: E402


class _Model:
    """Stands in for a device model: only its parameter bytes are read."""

    def __init__(self, n):
        self.n = n

    def weight_bytes(self):
        return self.n


def test_algorithmic_step_bytes_by_hand():
    shape = workload.INDEXTTS2
    d, L, V, n_pos = shape.d_model, shape.n_layer, shape.vocab, shape.n_pos
    params = 1_000_000_000
    ctx = [256, 300]
    got = bench.algorithmic_step_bytes(shape, _Model(params), 2, ctx, 2)
    per_token_kv = L * 2 * d * 2                      # K and V rows of every layer, bf16
    want = (params - (V + n_pos) * d * 2              # embedding tables are read sparsely
            + (257 + 301) * per_token_kv              # cached rows and the new one
            + 2 * per_token_kv                        # the new rows written
            + 2 * 2 * d * 2                           # token + position rows read
            + 2 * V * 4)                              # fp32 logits written
    assert got == want


def test_measured_traffic_needs_workload_and_source_hash(tmp_path, monkeypatch):
    f = tmp_path / "counters.json"
    f.write_text(json.dumps({"entries": [{"workload": "w", "source_sha256": "abc", "hbm_bytes_per_unit": 7}]}))
    monkeypatch.setattr(bench, "COUNTERS", str(f))
    assert bench.measured_traffic("w", "abc") == 7
    assert bench.measured_traffic("w", "abd") is None   # sources changed since the counters were taken
    assert bench.measured_traffic("x", "abc") is None
    assert bench.measured_traffic("w", None) is None    # eager counter runs report none
    monkeypatch.setattr(bench, "COUNTERS", str(tmp_path / "missing.json"))
    assert bench.measured_traffic("w", "abc") is None


def test_every_leg_has_a_counter_entry_under_its_name():
    with open(bench.COUNTERS) as fh:
        names = {e["workload"] for e in json.load(fh)["entries"]}
    fixed = [("bf16", 1, 256), ("w8a16", 1, 256), ("w4a16", 1, 384), ("w8a16", 8, 256)]
    for mode, B, P in fixed:
        assert f"indextts2-gpt {mode} batch={B} prefix={P} greedy decode=512" in names, (mode, B, P)
    paged = ("indextts2-gpt bf16 paged batch=32 prefix~U[128,512] target~U[256,768]+STOP "
             "top-k 30 top-p 0.8 T 0.8")
    assert paged in names
