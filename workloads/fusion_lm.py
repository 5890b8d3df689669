"""The caller's side of delayed fusion with an external scorer.

In the paper the fusion scores of Eq. (2) come from an LLM that scores the
distinct word sequences of the fused beams in batches (Sec. 3.4.2, App. E.4;
batches of 256).  No trained weights exist here, so ``CausalWordLM`` -- a small
causal Transformer over the n-gram LM's word ids, randomly initialised from a
seed -- stands in for it: it defines a proper distribution over the next word
and returns a sequence's full log-probability in natural log,

    S(w_1..w_n) = sum_i ln p(w_i | <s>, w_1..w_{i-1}).

``score_requests`` turns the decoder's exported request (``lb_fusion_request``:
word ids [B][K][o][W], counts [B][K][o], -1 where no sub-beam is asked for) into
the score array of ``lb_fusion_scores``, scoring each distinct sequence once.
``decode_external`` drives the whole round trip for one call of
``lb_decode_batch``.  All of this is caller code around the decoder's C ABI; the
decoder computes nothing here.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import torch
import torch.nn.functional as F


class CausalWordLM(torch.nn.Module):
    """Pre-norm causal Transformer language model over word ids, fp32, with
    tied input/output embeddings.  Weights are drawn from N(0, std^2) with a
    fixed seed, so every instance with the same arguments is the same model."""

    def __init__(self, vocab: int, bos: int, d_model: int = 256, n_layers: int = 2, n_heads: int = 4,
                 max_len: int = 512, seed: int = 0, std: float = 0.05):
        super().__init__()
        assert d_model % n_heads == 0
        self.vocab, self.bos, self.d, self.h, self.max_len = vocab, bos, d_model, n_heads, max_len
        g = torch.Generator().manual_seed(seed)

        def w(*shape, s=std):
            return torch.nn.Parameter(torch.randn(*shape, generator=g) * s, requires_grad=False)

        self.emb = w(vocab, d_model, s=1.0)
        self.pos = w(max_len, d_model, s=0.1)
        self.layers = torch.nn.ModuleList()
        for _ in range(n_layers):
            m = torch.nn.Module()
            m.qkv = w(3 * d_model, d_model)
            m.proj = w(d_model, d_model)
            m.up = w(4 * d_model, d_model)
            m.down = w(d_model, 4 * d_model)
            self.layers.append(m)
        self.out_scale = 1.0 / math.sqrt(d_model)

    def hidden(self, x: torch.Tensor) -> torch.Tensor:
        """x: int64 [N, L] token ids (position 0 is <s>) -> fp32 [N, L, d]."""
        N, L = x.shape
        hd = self.d // self.h
        z = self.emb[x] + self.pos[:L].unsqueeze(0)
        causal = torch.ones(L, L, dtype=torch.bool, device=x.device).tril()
        for m in self.layers:
            a = F.layer_norm(z, (self.d,))
            q, k, v = F.linear(a, m.qkv).split(self.d, dim=-1)
            q = q.reshape(N, L, self.h, hd).transpose(1, 2).contiguous()
            k = k.reshape(N, L, self.h, hd).transpose(1, 2).contiguous()
            v = v.reshape(N, L, self.h, hd).transpose(1, 2).contiguous()
            kt = k.transpose(-1, -2).contiguous()
            att = torch.matmul(q, kt) / math.sqrt(hd)
            att = att.masked_fill(~causal, float("-inf")).softmax(dim=-1)
            o = torch.matmul(att, v).transpose(1, 2).reshape(N, L, self.d)
            z = z + F.linear(o, m.proj)
            a = F.layer_norm(z, (self.d,))
            z = z + F.linear(F.gelu(F.linear(a, m.up)), m.down)
        return F.layer_norm(z, (self.d,))

    @torch.no_grad()
    def score(self, seqs: torch.Tensor, lengths: torch.Tensor, token_chunk: int = 4096) -> torch.Tensor:
        """Full log-probabilities (fp32, natural log) of the sequences.

        seqs: int [N, Lmax] word ids (entries past lengths[i] are ignored);
        lengths: int [N].  Returns fp32 [N]; an empty sequence scores 0."""
        dev = seqs.device
        N, Lmax = seqs.shape
        assert Lmax + 1 <= self.max_len
        out = torch.zeros(N, dtype=torch.float32, device=dev)
        if N == 0 or Lmax == 0:
            return out
        x = torch.full((N, Lmax + 1), self.bos, dtype=torch.int64, device=dev)
        x[:, 1:] = seqs.to(torch.int64).clamp_min(0)
        h = self.hidden(x[:, :-1])                                  # predicts positions 1..Lmax
        valid = torch.arange(Lmax, device=dev).unsqueeze(0) < lengths.to(dev).unsqueeze(1)
        hv = h[valid]                                               # [tokens, d]
        tgt = x[:, 1:][valid]
        row = torch.arange(N, device=dev).unsqueeze(1).expand(N, Lmax)[valid]
        lp = torch.empty(hv.shape[0], dtype=torch.float32, device=dev)
        for s in range(0, hv.shape[0], token_chunk):
            logits = F.linear(hv[s:s + token_chunk], self.emb) * self.out_scale
            lp[s:s + token_chunk] = (logits.gather(1, tgt[s:s + token_chunk, None]).squeeze(1)
                                     - torch.logsumexp(logits, dim=1))
        return out.index_add_(0, row, lp)


@dataclass
class RoundTripStats:
    events: int = 0
    requested: int = 0      # sub-beam sequences asked for
    scored: int = 0         # distinct sequences scored
    scorer_ms: float = 0.0  # GPU time of the scorer (events on its stream)
    batches: int = 0


def score_requests(words: torch.Tensor, n_words: torch.Tensor, scorer, batch: int = 256,
                   stats: RoundTripStats = None) -> torch.Tensor:
    """Fusion scores [B][K][o] (fp32) for an exported request.

    Distinct sequences are scored once, in batches of `batch` sequences of
    similar length; sub-beams that were not asked for get 0."""
    B, K, O, W = words.shape
    nw = n_words.reshape(-1)
    idx = torch.nonzero(nw >= 0).squeeze(1)
    out = torch.zeros(B * K * O, dtype=torch.float32, device=words.device)
    if idx.numel() == 0:
        return out.reshape(B, K, O)
    lens = nw[idx]
    lmax = int(lens.max())
    rows = words.reshape(-1, W)[idx, :max(lmax, 1)]
    pad = torch.arange(rows.shape[1], device=rows.device).unsqueeze(0) >= lens.unsqueeze(1)
    rows = rows.masked_fill(pad, -1)
    uniq, inv = torch.unique(rows, dim=0, return_inverse=True)
    ulen = (uniq >= 0).sum(dim=1)
    order = torch.argsort(ulen)
    s = torch.empty(uniq.shape[0], dtype=torch.float32, device=words.device)
    for b0 in range(0, uniq.shape[0], batch):
        sel = order[b0:b0 + batch]
        ln = ulen[sel]
        L = int(ln.max())
        s[sel] = scorer(uniq[sel, :L], ln) if L > 0 else torch.zeros(sel.numel(), device=words.device)
        if stats is not None:
            stats.batches += 1
    out[idx] = s[inv]
    if stats is not None:
        stats.requested += int(idx.numel())
        stats.scored += int(uniq.shape[0])
    return out.reshape(B, K, O)


def decode_external(lbm, dec, logits, lengths, flags: int, scorer, out_hyps, out_scores, words, n_words,
                    stream=None, batch: int = 256, stats: RoundTripStats = None) -> int:
    """One lb_decode_batch call with an external fusion scorer: at each
    LB_NEED_FUSION the request is exported, scored and handed back, and the
    call is resumed with the same arguments.  The scorer runs on torch's
    current stream, which must be `stream` (None: the null stream) so that it
    sees the exported request and the decoder sees its scores.  Returns the
    number of events."""
    events = 0
    while True:
        st, _, _ = dec.decode(logits, lengths, flags, stream=stream, out_hyps=out_hyps, out_scores=out_scores)
        if st == lbm.LB_OK:
            break
        assert st == lbm.LB_NEED_FUSION, st
        events += 1
        lbm.lb_fusion_request(dec.handle, words, n_words, stream)
        if stats is not None:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
        fs = score_requests(words, n_words, scorer, batch=batch, stats=stats)
        if stats is not None:
            e1.record()
            e1.synchronize()
            stats.scorer_ms += e0.elapsed_time(e1)
        lbm.lb_fusion_scores(dec.handle, fs, stream)
    if stats is not None:
        stats.events += events
    return events
