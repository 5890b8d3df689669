"""bench.py's host logic on the CPU: one GPU only, the per-unit accounting of
the algorithmic bytes, and the committed figures it reads only while the
kernel sources are the ones they were measured on."""

import json
import os
import subprocess
import sys
import types

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode != 0
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_algorithmic_bytes_per_unit():
    import paper_2603_14002_amd as lbm
    launches = [0] * 6
    launches[lbm.KIND_DECODE] = 2
    s = types.SimpleNamespace(frames=10, expansions=41 * 7, launches=launches, probe_lines=5, lm_lookups=3,
                              word_events=4, fused=6)
    p = types.SimpleNamespace(beam=8, subbeams=3)
    lp = types.SimpleNamespace(max_words_out=16)
    parts = bench.algorithmic_bytes(s, 2, 5, p, lp)
    assert parts["logits"] == 10 * 164                   # a logit row per stream-frame
    assert parts["trie"] == 7 * 16                       # a trie node per 41 expansions
    assert parts["state"] == 2 * 2 * 2 * 8 * (48 + 36)   # in and out, per call, B x K hypotheses
    assert parts["ngram_lines"] == 5 * 64
    assert parts["unigram_lines"] == 3 * 64
    assert parts["history_nodes"] == 4 * 3 * 8           # per completed word and sub-beam
    assert parts["fusion"] == 6 * 3 * 8
    assert parts["output"] == 2 * 2 * 8 * 17 * 4         # per call: B x K rows of W words and a score
    assert parts["total"] == sum(v for k, v in parts.items() if k != "total")
    launches[lbm.KIND_OUTPUT] = 2                         # a separate output launch: not the decode's bytes
    assert "output" not in bench.algorithmic_bytes(s, 2, 5, p, lp)


def _profiles(tmp_path, sha):
    d = tmp_path / "profiles"
    d.mkdir()
    (d / "k_decode_c4.md").write_text(f"# k_decode on c4\n\n- `workload`: `c4`\n"
                                      f"- `traffic_bytes_per_launch`: `1234567`\n"
                                      f"- `kernel_source_sha256`: `{sha}`\n")
    row = dict(config="c4", mode="end", utterances=3, exact=3, near_tie=1, near_tie_excused=0, tie_divergent=0,
               mismatch=0, empty=0, hyps_compared=9)
    (d / "parity_c4.md").write_text(f"# parity\n\n- kernel_source_sha256: `{sha}`\n\n{json.dumps(row)}\n")


def test_committed_figures_only_for_the_same_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    _profiles(tmp_path, bench.kernel_source_hash())
    assert bench.measured_traffic("c4") == 1234567.0
    assert bench.committed_parity("c4")["end"]["exact"] == 3
    assert bench.measured_traffic("c5") is None and bench.committed_parity("c5") is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 64)
    assert bench.measured_traffic("c4") is None
    assert bench.committed_parity("c4") is None
