"""The resolve kernel's phase-timing build on the GPU, through bench.py --resolve-phases in a
process of its own (the variant library replaces the normal one there): every phase's time is
non-negative, the phases add up to the stamped kernel span, and that span lies within the
HIP-event span of the launch."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.gpu
@pytest.mark.parametrize("config", [1, 5])
def test_resolve_phase_stamps(config):
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--resolve-phases",
                        "--config", str(config)], capture_output=True, text=True, timeout=110,
                       cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads([x for x in r.stdout.splitlines() if x.startswith("{")][-1])
    ph = line["phase_us"]
    assert len(ph) == 8 and all(v >= 0 for v in ph.values()), ph
    assert abs(sum(ph.values()) - line["stamped_span_us"]) < 1e-6 * max(1.0, line["stamped_span_us"]) + 1e-3
    assert 0 < line["stamped_span_us"] <= line["stamped_span_max_unit_us"] + 1e-9
    assert line["stamped_span_max_unit_us"] < line["event_span_us"] + 1.0, line
    assert line["misses_per_unit_step"] > 0
