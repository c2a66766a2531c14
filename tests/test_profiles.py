"""The committed rocprofv3 summaries stay in step with the source (CPU only):
the HBM-counter summary that bench.py reports as roofline traffic belongs to
the current score kernels, and every summary states the command that made it."""
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
    assert t["score_hip_sha256"] == sha, "score.hip changed since the HBM counters were taken"
    for k in ("score_lse", "lse_combine", "score_mass"):
        assert t["kernels"][k]["hbm_bytes_per_launch"] > 0, k
    assert 1.5 < t["fetch_factor"] < 2.5 and 0.5 < t["write_factor"] < 1.5


def test_summaries_state_their_command():
    names = [n for n in os.listdir(PROF) if n.endswith(".md")]
    assert names
    for n in names:
        with open(os.path.join(PROF, n)) as f:
            text = f.read()
        assert "bench.py" in text and "```" in text, n
        assert len(text) < 64 * 1024, n
