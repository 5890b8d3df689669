"""Oracle results for every utterance of the full-size workloads.

    python tests/golden/full_parity.py [--configs c2,c3,c4,c5] [--modes end,live] [--threads N]

Decodes each workload's whole batch with the CPU oracle (one utterance per
task over N host threads; at c4 this takes tens of minutes) and writes
``full_<config>_<mode>.npz`` next to this script: per utterance the ranked
hypotheses as (64-bit hash of the words, fp64 total) and the oracle's
decision margins.  ``end`` finalises the utterance (LB_END), ``live`` ranks the
beam after the last frame.  Only the oracle and the seeded input generators
are called.  Each file records a digest of the oracle's source and of the
generated inputs, and the GPU tests refuse a file whose digests differ from
the current tree's.
"""

from __future__ import annotations

import argparse
import hashlib
import os
import re
import sys
import threading
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MODES = ("end", "live")


def path_of(name: str, mode: str) -> str:
    return os.path.join(HERE, f"full_{name}_{mode}.npz")


def oracle_digest() -> str:
    """sha256 of the oracle's source without comments and spacing."""
    with open(os.path.join(ROOT, "oracle", "oracle.cpp")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256(" ".join(text.split()).encode()).hexdigest()


def inputs_digest(d) -> str:
    """sha256 over what the decode reads: the workload's shape and parameters,
    logits, lengths, fusion seed, lexicon, and the LM (counts and the first and
    last 100k entries of every order)."""
    h = hashlib.sha256()
    wl = d.workload
    h.update(repr((wl.name, wl.batch, wl.frames, wl.lm, wl.params, wl.sigma, wl.chunk, wl.ragged)).encode())
    for a in (d.logits, d.lengths, d.lexicon.offsets, d.lexicon.phonemes):
        h.update(np.ascontiguousarray(a).tobytes())
    h.update(str(int(d.fusion_seed)).encode())
    h.update(repr(d.lm.counts).encode())
    for n in range(4):
        for arr in (d.lm.ids[n], d.lm.logp[n], d.lm.bo[n] if n < 3 else None):
            if arr is None or arr.shape[0] == 0:
                continue
            h.update(np.ascontiguousarray(arr[:100_000]).tobytes())
            h.update(np.ascontiguousarray(arr[-100_000:]).tobytes())
    return h.hexdigest()


def load(name: str, mode: str):
    """(list of Expected per utterance, metadata dict) of a stored file."""
    from tests.parity import Expected
    import oracle
    z = np.load(path_of(name, mode), allow_pickle=False)
    off = z["offsets"]
    names = [str(x) for x in z["margin_names"]]
    out = []
    for b in range(off.shape[0] - 1):
        lo, hi = int(off[b]), int(off[b + 1])
        out.append(Expected(z["hashes"][lo:hi].copy(), z["total"][lo:hi].copy(),
                            dict(zip(names, z["margins"][b].tolist()))))
    assert tuple(names) == oracle.MARGIN_NAMES
    meta = dict(oracle_digest=str(z["oracle_digest"]), inputs_digest=str(z["inputs_digest"]),
                seconds=float(z["seconds"]), threads=int(z["threads"]))
    return out, meta


def generate(name: str, modes, threads: int) -> None:
    import oracle
    from tests.parity import Expected
    from workloads import load_workload
    t0 = time.time()
    d = load_workload(name)
    p = d.workload.params
    B = d.logits.shape[0]
    print(f"[golden] {name}: B={B} T={d.logits.shape[1]} K={p.beam} loaded in {time.time() - t0:.0f}s", flush=True)
    orc = oracle.Oracle(d.lexicon, d.lm)
    dig_in, dig_or = inputs_digest(d), oracle_digest()
    for mode in modes:
        op = oracle.params_from(p, fusion_seed=d.fusion_seed, finalize=1 if mode == "end" else 0)
        res = [None] * B
        nxt = [0]
        lock = threading.Lock()

        def work():
            while True:
                with lock:
                    b = nxt[0]
                    nxt[0] += 1
                if b >= B:
                    return
                r = orc.decode(d.logits[b, :d.lengths[b]], op, max_hyps=p.beam)
                res[b] = Expected.from_oracle(r, p.beam)

        t1 = time.time()
        ths = [threading.Thread(target=work) for _ in range(threads)]
        for t in ths:
            t.start()
        for t in ths:
            t.join()
        secs = time.time() - t1
        off = np.zeros(B + 1, np.int64)
        off[1:] = np.cumsum([len(e.total) for e in res])
        np.savez_compressed(
            path_of(name, mode), offsets=off,
            hashes=np.concatenate([e.hashes for e in res]).astype(np.uint64),
            total=np.concatenate([e.total for e in res]).astype(np.float64),
            margins=np.array([[e.margins[k] for k in oracle.MARGIN_NAMES] for e in res], np.float64),
            margin_names=np.array(oracle.MARGIN_NAMES), oracle_digest=np.array(dig_or),
            inputs_digest=np.array(dig_in), seconds=np.array(secs), threads=np.array(threads))
        empty = sum(1 for e in res if len(e.total) == 0)
        print(f"[golden] {name}/{mode}: {int(off[-1])} hypotheses, {empty} empty lists, {secs:.0f}s "
              f"on {threads} threads", flush=True)
    orc.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--configs", default="c2,c3,c4,c5")
    ap.add_argument("--modes", default="end,live")
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    a = ap.parse_args()
    for name in a.configs.split(","):
        generate(name, a.modes.split(","), a.threads)


if __name__ == "__main__":
    main()
