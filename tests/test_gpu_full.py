"""GPU parity at the full workload sizes, in the launch configuration bench.py
times (the whole batch in one call, or the c5 streams in 10-frame calls), on
every utterance.

The oracle's results for every utterance are stored in
``tests/golden/full_<config>_<mode>.npz`` (written by
``tests/golden/full_parity.py``, which calls only the oracle and the seeded
generators; the files carry digests of the oracle source and of the inputs,
checked here).  ``end`` decodes with LB_END (the final fusion and the
end-of-utterance filter), ``live`` without it (the whole beam ranked).  Every
utterance is classified by tests.parity and the counts are printed, and
written as JSON under $LB_PARITY_DIR when that is set.  Every decoded output
is also checked for properties that hold at any size, and one utterance
decoded alone must equal its result inside the batch.
"""

import json
import os

import numpy as np
import pytest

from tests.golden import full_parity as golden
from tests.gpu_util import gpu_decode, say
from tests.parity import Parity
from workloads import load_workload
from workloads.gen import WorkloadData

pytestmark = pytest.mark.gpu

_DATA = {}


def workload(name):
    if name not in _DATA:
        _DATA.clear()  # one full-size workload in host memory at a time
        _DATA[name] = load_workload(name)
    return _DATA[name]


def check_properties(d, out):
    W = d.lm.vocab_size
    for b, (words, scores) in enumerate(out):
        assert len(words) == len(scores) <= d.workload.params.beam
        assert np.all(np.isfinite(scores))
        assert np.all(np.diff(scores) <= 0), b
        for ws in words:
            assert all(0 <= w < W for w in ws)


@pytest.mark.parametrize("mode", ["end", "live"])
@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_full_batch_parity(name, mode):
    if not os.path.exists(golden.path_of(name, mode)):
        pytest.skip(f"no stored oracle results for {name}/{mode}: run tests/golden/full_parity.py")
    exp, meta = golden.load(name, mode)
    d = workload(name)
    B = d.logits.shape[0]
    K = d.workload.params.beam
    say(f"[case] full {name}/{mode}: B={B} T={d.logits.shape[1]} K={K} chunk={d.workload.chunk}")
    assert meta["oracle_digest"] == golden.oracle_digest(), "oracle changed: regenerate the stored results"
    assert meta["inputs_digest"] == golden.inputs_digest(d), "inputs changed: regenerate the stored results"
    assert len(exp) == B
    out = gpu_decode(d, chunk=d.workload.chunk, finalize=mode == "end")
    check_properties(d, out)
    par = Parity()
    for b in range(B):
        gw, gs = out[b]
        par.add(b, gw, gs, exp[b])
    say(par.report(f"{name}/{mode}"))
    res = dict(config=name, mode=mode, batch=B, beam=K, **par.counts(),
               oracle_seconds=meta["seconds"], oracle_threads=meta["threads"])
    if os.environ.get("LB_PARITY_DIR"):
        os.makedirs(os.environ["LB_PARITY_DIR"], exist_ok=True)
        with open(os.path.join(os.environ["LB_PARITY_DIR"], f"parity_{name}_{mode}.json"), "w") as f:
            json.dump(res, f)
    assert not par.mismatch, "\n".join(par.mismatch[:5])
    # every utterance has an output to compare (the end-of-utterance lists included)
    assert par.empty == 0 and par.n_hyps >= B
    if mode == "end":
        # an utterance decoded alone equals its result inside the batch
        b = B - 1
        sub = WorkloadData(d.workload, d.lexicon, d.lm, d.logits[b:b + 1], d.lengths[b:b + 1],
                           d.targets[b:b + 1], d.words[b:b + 1], d.fusion_seed)
        alone = gpu_decode(sub, chunk=d.workload.chunk)[0]
        assert alone[0] == out[b][0] and np.array_equal(alone[1], out[b][1])
