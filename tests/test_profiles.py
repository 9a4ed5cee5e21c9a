"""CPU checks of the committed rocprofv3 summaries under profiles/: one per
workload, each naming the kernel source it was taken on, the commands that
produced it (committed files only) and the figures bench.py reports from it.
A set taken on an earlier kernel source is reported as a skip (bench.py then
leaves its traffic field null), never as a pass."""
import json
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = os.path.join(ROOT, "profiles")


def _bench():
    import sys

    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import bench

    return bench


def _summary(name):
    with open(os.path.join(PROFILES, f"topk_ragged_kernel_{name}.md")) as fh:
        return fh.read()


def _recorded_hash(text):
    m = re.search(r"Kernel source sha256/16: `([0-9a-f]{16})`", text)
    assert m, "summary does not name its kernel source hash"
    return m.group(1)


def test_every_workload_has_a_summary_and_traffic_file():
    bench = _bench()
    for config, name in bench.WORKLOAD_NAMES.items():
        text = _summary(name)
        assert "rocprofv3 --kernel-trace --stats" in text, name
        assert "rocprofv3 --pmc FETCH_SIZE" in text and "rocprofv3 --pmc WRITE_SIZE" in text, name
        assert "SQ_LDS_BANK_CONFLICT" in text, name
        # every command runs committed files only
        for cmd in re.findall(r"^    (rocprofv3 .*|python3 .*)$", text, flags=re.M):
            for path in re.findall(r"python3 (\S+\.py)", cmd):
                assert os.path.exists(os.path.join(ROOT, path)), (name, path)
            assert "_work/" not in cmd, (name, cmd)
        with open(bench.traffic_file(config)) as fh:
            t = json.load(fh)
        assert t["config"] == config, name
        assert t["kernel_source_sha256_16"] == _recorded_hash(text), name
        assert t["hbm_bytes_per_launch"] > 0, name


def test_summaries_share_one_kernel_source():
    bench = _bench()
    hashes = {_recorded_hash(_summary(n)) for n in bench.WORKLOAD_NAMES.values()}
    assert len(hashes) == 1, f"summaries taken on different kernel sources: {sorted(hashes)}"


def test_summaries_match_the_current_kernel_source():
    bench = _bench()
    recorded = _recorded_hash(_summary(bench.WORKLOAD_NAMES[2]))
    current = bench.kernel_source_hash()
    if recorded != current:
        pytest.skip(f"profiles/ was taken on kernel source {recorded}, the source is now "
                    f"{current}: regenerate the summaries (bench.py reports no traffic meanwhile)")
    for config in bench.WORKLOAD_NAMES:
        assert bench.measured_traffic(config) is not None, config
