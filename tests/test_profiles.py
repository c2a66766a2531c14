"""The committed rocprofv3 summaries stay in step with the source (CPU only):
bench.py reports the HBM-counter summary as roofline traffic only while it
belongs to the current score kernels (else the traffic is null), and every
summary states the command that made it."""
import hashlib
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROF = os.path.join(ROOT, "profiles")


def test_traffic_summary_matches_score_source():
    with open(os.path.join(PROF, "traffic_score_qwen7b_16k_b4.json")) as f:
        t = json.load(f)
    with open(os.path.join(ROOT, "paper_2607_22586_amd", "csrc", "score.hip"), "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    assert t["workload"] == "qwen7b_16k_b4"
    for k in ("score_lse", "lse_combine", "score_mass"):
        assert t["kernels"][k]["hbm_bytes_per_launch"] > 0, k
    assert 1.5 < t["fetch_factor"] < 2.5 and 0.5 < t["write_factor"] < 1.5
    import sys
    sys.path.insert(0, ROOT)
    import bench
    got = bench.measured_traffic("qwen7b_16k_b4", "score_lse")
    if t["score_hip_sha256"] == sha:
        assert got == t["kernels"]["score_lse"]["hbm_bytes_per_launch"]
    else:
        assert got is None, "bench.py must not report counters taken on another score.hip"


def test_summaries_state_their_command():
    names = [n for n in os.listdir(PROF) if n.endswith(".md")]
    assert names
    for n in names:
        with open(os.path.join(PROF, n)) as f:
            text = f.read()
        assert "bench.py" in text and "```" in text, n
        assert len(text) < 64 * 1024, n
