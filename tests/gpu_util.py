"""Helpers for GPU parity tests: run the HIP decoder through the C ABI and
compare its ranked outputs with the oracle's, utterance by utterance."""

from __future__ import annotations

import sys
import time
from typing import Optional

import numpy as np

import oracle
import paper_2603_14002_amd as lbm

from tests.parity import Expected, Parity  # noqa: F401  (the comparison protocol)


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def read_outputs(hyps, scores):
    """The ranked outputs of a decode call (device tensors [B, K, W] and [B, K],
    already synchronised) as (words per rank, fp32 scores) per utterance; the
    rows' padding is checked on the way."""
    H = hyps.cpu().numpy()
    S = scores.cpu().numpy()
    check_padding(H, S)
    B, K, W = H.shape
    out = []
    for b in range(B):
        words, sc = [], []
        for r in range(K):
            if not np.isfinite(S[b, r]):
                break
            row = H[b, r]
            n = int(np.argmax(row < 0)) if (row < 0).any() else W
            words.append([int(x) for x in row[:n]])
            sc.append(S[b, r])
        out.append((words, np.array(sc, dtype=np.float32)))
    return out


def gpu_decode(d, params=None, chunk: int = 0, batch: Optional[int] = None, fusion_source=None,
               profiling=False, max_words: Optional[int] = None, arena_nodes_per_stream: int = 0,
               return_decoder=False, finalize=True, logits: Optional[np.ndarray] = None, lb_overrides=None):
    """Decodes the first `batch` utterances of workload data `d` on cuda:0.

    Returns a list of (words list per rank, scores float32 array) per utterance."""
    import torch
    p = params or d.workload.params
    B = d.logits.shape[0] if batch is None else batch
    T = d.logits.shape[1]
    lp = lbm.make_params(p, max_batch=B, max_frames=T, fusion_seed=d.fusion_seed,
                         fusion_source=fusion_source, arena_nodes_per_stream=arena_nodes_per_stream,
                         **(lb_overrides or {}))
    if max_words is not None:
        lp.max_words_out = max_words
    dec = lbm.Decoder(d.lexicon, d.lm, lp)
    if profiling:
        lbm.lb_set_profiling(dec.handle, lbm.LB_PROFILE_ALL)
    dev = torch.device("cuda:0")
    src = d.logits if logits is None else logits
    logits = torch.from_numpy(np.ascontiguousarray(src[:B])).to(dev)
    lengths = np.ascontiguousarray(d.lengths[:B]).astype(np.int32)
    K, W = lp.beam, lp.max_words_out
    hyps = torch.empty((B, K, W), dtype=torch.int32, device=dev)
    scores = torch.empty((B, K), dtype=torch.float32, device=dev)
    if chunk <= 0:
        st, _, _ = dec.decode(logits, torch.from_numpy(lengths).to(dev),
                              lbm.LB_BEGIN | (lbm.LB_END if finalize else 0),
                              out_hyps=hyps, out_scores=scores)
        assert st == lbm.LB_OK
    else:
        nch = (T + chunk - 1) // chunk
        for c in range(nch):
            lo = c * chunk
            hi = min(T, lo + chunk)
            lg = logits[:, lo:hi].contiguous()
            ln = np.clip(lengths - lo, 0, hi - lo).astype(np.int32)
            fl = (lbm.LB_BEGIN if c == 0 else 0) | (lbm.LB_END if (finalize and c == nch - 1) else 0)
            st, _, _ = dec.decode(lg, torch.from_numpy(ln).to(dev), fl, out_hyps=hyps, out_scores=scores)
            assert st == lbm.LB_OK
    torch.cuda.synchronize()
    st = dec.status()
    assert st == lbm.LB_OK, lbm.lb_last_error()
    out = read_outputs(hyps, scores)
    if return_decoder:
        return out, dec
    dec.close()
    return out


def check_padding(H: np.ndarray, S: np.ndarray) -> None:
    """Every output row holds its words, then -1 to the end; ranks past the
    last hypothesis are all -1 with a score of -inf."""
    neg = H < 0
    first = np.where(neg.any(-1), neg.argmax(-1), H.shape[-1])
    tail = np.arange(H.shape[-1]) >= first[..., None]
    assert np.all(H[tail] == -1), "output rows not -1 padded after their words"
    empty = ~np.isfinite(S)
    assert np.all(H[empty] == -1), "ranks without a hypothesis not all -1"


def oracle_for(d):
    return oracle.Oracle(d.lexicon, d.lm)


def check_parity(d, gpu_out, utts, params=None, orc=None, name="", max_mismatch=0, finalize=True,
                 logits: Optional[np.ndarray] = None, oracle_overrides=None, min_hyps=1):
    """The oracle decodes utterances `utts` one by one and each is classified
    against the decoder's output (tests.parity); no mismatch is allowed and at
    least `min_hyps` hypotheses must have been compared."""
    p = params or d.workload.params
    orc = orc or oracle_for(d)
    op = oracle.params_from(p, fusion_seed=d.fusion_seed, finalize=1 if finalize else 0,
                            **(oracle_overrides or {}))
    src = d.logits if logits is None else logits
    par = Parity()
    t0 = time.time()
    for b in utts:
        res = orc.decode(src[b, :d.lengths[b]], op)
        gw, gs = gpu_out[b]
        par.add(b, gw, gs, Expected.from_oracle(res, p.beam))
    say(par.report(name) + f" oracle {time.time() - t0:.1f}s")
    assert len(par.mismatch) <= max_mismatch, "\n".join(par.mismatch[:5])
    assert par.n_hyps >= min_hyps, f"{name}: only {par.n_hyps} hypotheses compared"
    return par
