"""GPU parity at the full workload sizes, in the launch configuration bench.py
times (whole batch in one call, or the c5 streams in 10-frame calls).

The oracle decodes a sample of the utterances one by one; every decoded
output is also checked for properties that hold at any size (ranked scores,
valid word ids, padding).  A sampled utterance decoded alone must equal its
result inside the batch.
"""

import numpy as np
import pytest

from tests.gpu_util import check_parity, gpu_decode, oracle_for, say
from workloads import load_workload
from workloads.gen import WorkloadData

pytestmark = pytest.mark.gpu

SAMPLES = {"c2": [0, 17, 41, 63], "c3": [0, 128, 255], "c4": [0, 311], "c5": [5, 1023]}


def check_properties(d, out):
    W = d.lexicon.n_words
    for b, (words, scores) in enumerate(out):
        assert len(words) == len(scores) <= d.workload.params.beam
        assert np.all(np.isfinite(scores))
        assert np.all(np.diff(scores) <= 0), b
        for ws in words:
            assert all(0 <= w < W for w in ws)


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_size_sampled_parity(name):
    d = load_workload(name)
    B = d.logits.shape[0]
    say(f"[case] full {name}: B={B} T={d.logits.shape[1]} K={d.workload.params.beam} chunk={d.workload.chunk}")
    out = gpu_decode(d, chunk=d.workload.chunk)
    check_properties(d, out)
    orc = oracle_for(d)
    check_parity(d, out, SAMPLES[name], orc=orc, name=f"{name}/end")
    live = gpu_decode(d, chunk=d.workload.chunk, finalize=False)
    check_properties(d, live)
    check_parity(d, live, SAMPLES[name][:1], orc=orc, name=f"{name}/live", finalize=False)
    # an utterance alone equals its result inside the batch
    b = SAMPLES[name][-1]
    sub = WorkloadData(d.workload, d.lexicon, d.lm, d.logits[b:b + 1], d.lengths[b:b + 1],
                       d.targets[b:b + 1], d.words[b:b + 1], d.fusion_seed)
    alone = gpu_decode(sub, chunk=d.workload.chunk)[0]
    assert alone[0] == out[b][0] and np.array_equal(alone[1], out[b][1])
