"""bench.py's command-line contract that needs no GPU: more than one GPU is refused with a
message (the benchmark measures one GPU), before anything touches a device."""

import json
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    out = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert out.returncode == 2
    line = json.loads(out.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]


def test_recorded_traffic_needs_matching_mask_and_source():
    """roofline.traffic comes from a committed counter summary only for the mask and kernel
    source it was taken on."""
    sys.path.insert(0, ROOT)
    import bench

    for profile, source in (("routed_attn_fwd_32k-gqa", "attn_fwd.hip"),
                            ("decode_64k-b4-gqa", "decode.hip")):
        path = os.path.join(ROOT, "profiles", f"{profile}_hbm_traffic.md")
        fields = dict(m.groups() for m in (re.match(r"^- (\w+): (`[^`]*`)$", line.strip())
                                           for line in open(path)) if m)
        mask = fields["mask"].strip().strip("`")
        want = int(fields["traffic_bytes_per_launch"].strip().strip("`"))
        digest = fields["kernel_source_sha256"].strip().strip("`")
        got = bench.recorded_traffic(profile, mask, source)
        if digest == bench.kernel_source_digest(source):
            assert got == want
        else:
            assert got is None
        assert bench.recorded_traffic(profile, mask + "-other", source) is None
    assert bench.recorded_traffic("no-such-profile", "bern0.5") is None
