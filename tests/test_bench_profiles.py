"""The bench's use of the committed rocprofv3 --pmc summaries: a stored
traffic figure is reported only for the kernel source and the workload
definition it was measured on (CPU only: no GPU call is made)."""
import json
import os

import pytest

import bench
from inputs import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TAGS = {"schema": "schema_c3", "pylike": "pylike_c4", "stress": "stress_c5", "gosql": "gosql"}


def _meta(tag):
    for line in open(os.path.join(ROOT, "profiles", f"mask_kernels_{tag}_pmc_traffic.md")):
        if line.startswith("traffic_json: "):
            return json.loads(line[len("traffic_json: "):])
    raise AssertionError(f"no traffic_json line for {tag}")


@pytest.mark.parametrize("name", sorted(TAGS))
def test_stored_traffic_is_read_back_only_for_its_kernel_and_workload(name, monkeypatch):
    wl = configs.get(name)
    meta = _meta(TAGS[name])
    want = meta["kernels"]["fused_fast_kernel"]["hbm_bytes"]
    fresh = meta["source_sha256_16"] == bench.device_code_hash() and \
        meta.get("workload_sha256_16") == bench.workload_fingerprint(wl)
    assert bench.measured_traffic(wl, "fused_fast_kernel") == (want if fresh else None)
    # another kernel source, or another workload definition: no figure
    monkeypatch.setattr(bench, "device_code_hash", lambda: "0" * 16)
    assert bench.measured_traffic(wl, "fused_fast_kernel") is None
    monkeypatch.undo()
    monkeypatch.setattr(bench, "workload_fingerprint", lambda _wl: "0" * 16)
    assert bench.measured_traffic(wl, "fused_fast_kernel") is None


def test_fingerprints_tell_the_workloads_apart():
    fps = {bench.workload_fingerprint(configs.get(n)) for n in ("arithmetic", "json", "schema", "pylike",
                                                                "stress", "gosql")}
    assert len(fps) == 6
