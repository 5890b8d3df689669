"""GPU edge cases through the C ABI: the hand-worked pruning cases, capacity
overflows reported by lb_get_status (no write past a buffer), lengths outside
0..frames, and the n-gram tables at load factor 0.9 with probe chains that
wrap past the last bucket."""

import math

import numpy as np
import pytest

import paper_2603_14002_amd as lbm
from tests import test_oracle_pruning_pins as pins
from tests.gpu_util import check_parity, gpu_decode, read_outputs, say
from tests.tinylm import lexicon_from, lm_from_entries, peaked_logits, random_small_lm
from workloads import DecodeParams, load_workload
from workloads.gen import WorkloadData

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm device")
    lbm.lib()


def data_of(lex, lm, lg, params, fusion_seed=0, lengths=None):
    wl = load_workload("t-c1k", batch=1).workload
    wl = wl.__class__(**{**wl.__dict__, "params": params})
    lg = np.asarray(lg, np.float32)
    if lg.ndim == 2:
        lg = lg[None]
    B, T = lg.shape[:2]
    ln = np.full(B, T, np.int32) if lengths is None else np.asarray(lengths, np.int32)
    return WorkloadData(wl, lex, lm, lg, ln, np.zeros((B, T), np.int32), [[]] * B, fusion_seed)


def pin_cases():
    """(name, data, params) of the hand-worked pruning cases."""
    P = pins.BASE
    rep = lambda **kw: P.__class__(**{**P.__dict__, **kw})
    four = lexicon_from([(1,), (2,), (3,), (4,)]), pins.unigram_lm(4, [(-1.0, 0.0)] * 4)
    two = lexicon_from([(1,), (2,)]), pins.unigram_lm(2, [(-0.25, 0.0), (-2.0, 0.0)])
    fuse = lexicon_from([(1,), (1,), (2,), (3,)]), pins.unigram_lm(4, [(-1.0, 0.0)] * 4)
    lam = lexicon_from([(1,), (1,), (1,)]), pins.unigram_lm(3, [(-1.0, 0.0), (-2.5, 0.0), (-2.875, 0.0)])
    ties = (lexicon_from([(1,), (1,), (2,), (2,)]),
            pins.unigram_lm(4, [(-1.0, -0.5), (-1.0, -0.5), (-1.5, 0.0), (-1.5, 0.0)]))
    F = pins.frames
    cases = []
    for K, th in ((2, 30.0), (3, 1.0), (3, 0.75), (5, 1.75)):
        cases.append((f"topk-K{K}-theta{th}", four, pins.ONE_FRAME, rep(beam=K, theta=th), 0))
    cases.append(("key-tie", four, F({0: -4.0, 1: -0.75, 2: -1.0, 3: -0.75}), rep(beam=1), 0))
    cases.append(("key-tie-2", four, F({0: -4.0, 1: -0.75, 2: -1.0, 3: -0.75}), rep(beam=2), 0))
    for th in (4.0, 4.1):
        cases.append((f"theta-word-{th}", two, pins.THETA_FRAMES, rep(omega=1.0, theta=th), 0))
    fl = F({1: -0.5, 2: -1.0, 3: -1.5}, {40: 0.0})
    for f in (1, 2):
        cases.append((f"top-F{f}", fuse, fl, rep(fusion_interval=1, fusion_top_f=f), (4 << 32) | 1))
    for lm_, o in ((4.0, 3), (4.5, 3), (4.5, 2), (0.0, 3)):
        cases.append((f"lambda{lm_}-o{o}", lam, F({1: -0.5}, {40: -0.5}), rep(omega=1.0, subbeams=o, lam=lm_), 0))
    cases.append(("sub-beam-ties", ties, F({1: -0.5}, {40: -0.5}, {2: -0.5}, {40: -0.5}),
                  rep(omega=1.0, subbeams=2, lam=100.0), 0))
    cases.append(("end-no-boundary", four, F({1: -0.5, 2: -1.5, 3: -2.5, 4: -3.0}), rep(beam=5), 0))
    cases.append(("end-inside-second-word", four, F({1: -0.5}, {40: -0.5}, {2: -0.5, 3: -1.0}), rep(beam=5), 0))
    return cases


@pytest.mark.parametrize("case", pin_cases(), ids=lambda c: c[0])
def test_pruning_cases_match_oracle(case):
    name, (lex, lm), lg, p, seed = case
    d = data_of(lex, lm, lg, p, fusion_seed=seed)
    for fin in (False, True):
        say(f"[case] pin {name} finalize={fin}")
        out = gpu_decode(d, params=p, finalize=fin)
        check_parity(d, out, [0], params=p, name=f"pin/{name}/{fin}", finalize=fin)


# ------------------------------------------------------------------ capacity overflows

def decode_guarded(d, p, arena=0, W=None, chunk=0):
    """Decodes with output buffers followed by a guard region of sentinels;
    returns (status of lb_get_status, outputs, guards intact)."""
    import torch
    B, T = d.logits.shape[:2]
    lp = lbm.make_params(p, max_batch=B, max_frames=T, fusion_seed=d.fusion_seed, arena_nodes_per_stream=arena)
    if W is not None:
        lp.max_words_out = W
    dec = lbm.Decoder(d.lexicon, d.lm, lp)
    dev = torch.device("cuda:0")
    K, Wm = lp.beam, lp.max_words_out
    G = 4096
    hyps = torch.full((B * K * Wm + G,), 0x5A5A5A5A, dtype=torch.int32, device=dev)
    scores = torch.full((B * K + G,), 12345.0, dtype=torch.float32, device=dev)
    logits = torch.from_numpy(d.logits).to(dev)
    lengths = torch.from_numpy(d.lengths.astype(np.int32)).to(dev)
    st, _, _ = dec.decode(logits, lengths, lbm.LB_BEGIN | lbm.LB_END, out_hyps=hyps, out_scores=scores)
    assert st == lbm.LB_OK
    torch.cuda.synchronize()
    status = dec.status()
    msg = lbm.lb_last_error()
    guard_ok = bool((hyps[B * K * Wm:] == 0x5A5A5A5A).all()) and bool((scores[B * K:] == 12345.0).all())
    H = hyps[:B * K * Wm].view(B, K, Wm).cpu().numpy()
    S = scores[:B * K].view(B, K).cpu().numpy()
    dec.close()
    return status, msg, H, S, guard_ok


@pytest.mark.parametrize("name", ["t-c20k", "t-k256"])
def test_arena_overflow_is_reported(name):
    """A word-history arena smaller than the words the decode completes: the
    node writes past it are skipped and lb_get_status reports LB_ERR_CAPACITY;
    with the default capacity the same decode is clean."""
    d = load_workload(name, batch=2)
    p = d.workload.params
    say(f"[case] arena overflow {name}")
    st, msg, H, S, guard = decode_guarded(d, p, arena=2 * p.subbeams)
    assert st == lbm.LB_ERR_CAPACITY and "arena" in msg, (st, msg)
    assert guard
    st, msg, H, S, guard = decode_guarded(d, p)
    assert st == lbm.LB_OK and guard


def test_output_words_overflow_is_reported():
    """max_words_out below the decoded word counts: rows hold their first W
    words and no more, nothing is written past the output buffers, and
    lb_get_status reports LB_ERR_CAPACITY exactly when some output row has
    more than W words."""
    d = load_workload("t-c20k", batch=3)
    p = d.workload.params
    st_full, _, Hf, Sf, guard = decode_guarded(d, p, W=256)
    assert st_full == lbm.LB_OK and guard
    most = int((Hf >= 0).sum(-1).max())
    assert most >= 3
    for W in (1, 2, most - 1, most, most + 3):
        say(f"[case] words overflow W={W} (longest row {most})")
        st, msg, H, S, guard = decode_guarded(d, p, W=W)
        assert guard
        if W < most:
            assert st == lbm.LB_ERR_CAPACITY and "max_words_out" in msg, (W, st, msg)
        else:
            assert st == lbm.LB_OK, (W, st, msg)
        # the rows are the full rows cut to W words (-1 padded)
        np.testing.assert_array_equal(S, Sf)
        ref = np.full(H.shape, -1, np.int32)
        k = min(W, Hf.shape[-1])
        ref[:, :, :k] = Hf[:, :, :k]
        np.testing.assert_array_equal(H, ref)


# ------------------------------------------------------------------ lengths outside 0..frames

def test_lengths_outside_range_are_clamped_and_reported():
    """lengths above `frames` or negative: the stream decodes as if clamped to
    0..frames (also its frame counter, which places the fusion frames of the
    next call) and lb_get_status reports LB_ERR_INVALID_ARG."""
    import torch
    d = load_workload("t-c20k", batch=3)
    p = d.workload.params
    B, T = d.logits.shape[:2]
    half = 50
    dev = torch.device("cuda:0")
    logits = torch.from_numpy(d.logits).to(dev)

    def run(first_lengths):
        lp = lbm.make_params(p, max_batch=B, max_frames=T, fusion_seed=d.fusion_seed)
        dec = lbm.Decoder(d.lexicon, d.lm, lp)
        ln1 = torch.tensor(first_lengths, dtype=torch.int32, device=dev)
        dec.decode(logits[:, :half].contiguous(), ln1, lbm.LB_BEGIN)
        ln2 = torch.full((B,), T - half, dtype=torch.int32, device=dev)
        _, H, S = dec.decode(logits[:, half:].contiguous(), ln2, lbm.LB_END)
        torch.cuda.synchronize()
        st = dec.status()
        out = (H.cpu().numpy(), S.cpu().numpy())
        dec.close()
        return st, out

    say("[case] lengths outside 0..frames")
    st_bad, bad = run([half + 7, -3, half])
    st_ok, ok = run([half, 0, half])
    assert st_bad == lbm.LB_ERR_INVALID_ARG and st_ok == lbm.LB_OK
    np.testing.assert_array_equal(bad[0], ok[0])
    np.testing.assert_array_equal(bad[1], ok[1])


def test_rejected_decode_calls_leave_the_decoder_usable():
    """A decode call with no stream (batch 0), more streams than max_batch, a
    negative frame count, an unknown flag or a null device pointer returns
    LB_ERR_INVALID_ARG before anything runs; the streams' state is untouched,
    so a valid call afterwards gives what a fresh decoder gives."""
    import torch
    d = load_workload("t-c1k")
    p = d.workload.params
    B, T = d.logits.shape[:2]
    dev = torch.device("cuda:0")
    logits = torch.from_numpy(d.logits).to(dev)
    lengths = torch.from_numpy(d.lengths.astype(np.int32)).to(dev)
    half = T // 2

    def run(bad_calls):
        lp = lbm.make_params(p, max_batch=B, max_frames=T, fusion_seed=d.fusion_seed)
        dec = lbm.Decoder(d.lexicon, d.lm, lp)
        K, W = lp.beam, lp.max_words_out
        H = torch.empty((B, K, W), dtype=torch.int32, device=dev)
        S = torch.empty((B, K), dtype=torch.float32, device=dev)
        first = torch.clamp(lengths, max=half).contiguous()
        rest = torch.clamp(lengths - half, min=0).contiguous()
        lbm.lb_decode_batch(dec.handle, logits[:, :half].contiguous(), first, B, half, lbm.LB_BEGIN, None, H, S)
        for args in bad_calls:
            with pytest.raises(lbm.LBError) as err:
                lbm.lb_decode_batch(dec.handle, *args(H, S))
            assert err.value.status == lbm.LB_ERR_INVALID_ARG, err.value
        lbm.lb_decode_batch(dec.handle, logits[:, half:].contiguous(), rest, B, T - half, lbm.LB_END, None, H, S)
        torch.cuda.synchronize()
        st = dec.status()
        out = (H.cpu().numpy(), S.cpu().numpy())
        dec.close()
        return st, out

    lg2 = logits[:, half:].contiguous()
    rest = torch.clamp(lengths - half, min=0).contiguous()
    bad = [
        lambda H, S: (lg2, rest, 0, T - half, lbm.LB_END, None, H, S),
        lambda H, S: (lg2, rest, B + 1, T - half, lbm.LB_END, None, H, S),
        lambda H, S: (lg2, rest, B, -1, lbm.LB_END, None, H, S),
        lambda H, S: (lg2, rest, B, T - half, lbm.LB_END | 4, None, H, S),
        lambda H, S: (lg2, None, B, T - half, lbm.LB_END, None, H, S),
        lambda H, S: (None, rest, B, T - half, lbm.LB_END, None, H, S),
    ]
    say("[case] rejected decode calls")
    st_bad, out_bad = run(bad)
    st_ok, out_ok = run([])
    assert st_bad == lbm.LB_OK and st_ok == lbm.LB_OK
    np.testing.assert_array_equal(out_bad[0], out_ok[0])
    np.testing.assert_array_equal(out_bad[1], out_ok[1])


# ------------------------------------------------------------------ load factor 0.9, wrapping probe chains

@pytest.mark.parametrize("name", ["c1", "t-c20k"])
def test_load_factor_09_matches_oracle(name):
    d = load_workload(name)
    B = d.logits.shape[0]
    for fin in (True, False):
        say(f"[case] {name} lm_load_factor=0.9 finalize={fin}")
        out = gpu_decode(d, finalize=fin, lb_overrides=dict(lm_load_factor=0.9))
        check_parity(d, out, range(B), name=f"{name}/lf0.9/{fin}", finalize=fin)


def _bucket(key, nb):
    # the n-gram tables' bucket of a key (multiply-high of a mixed hash), used
    # here only to choose keys that crowd the last bucket
    return (pins.splitmix64(key ^ 0xD6E8FEB86659FD93) * nb) >> 64


def test_probe_chains_wrapping_past_the_last_bucket():
    """10 bigrams at load factor 0.9 fill 3 buckets of 4 slots; six of them
    hash to the last bucket, so at least two are stored past it, in bucket 0,
    and lookups of absent keys there wrap as well.  Trigrams and a 4-gram sit
    in one-bucket tables.  Decoding matches the oracle, with and without the
    explicit-continuation index on every node with two or more words."""
    words = [(1,), (1,), (2,), (3, 1), (2, 2), (3,)]
    W = len(words)
    bos = W
    nb = max(1, math.ceil(math.ceil(10 / 0.9) / 4))
    assert nb == 3
    cand = [(c, w) for c in list(range(W)) + [bos] for w in range(W)]
    last = [k for k in cand if _bucket((k[0] << 32) | k[1], nb) == nb - 1]
    other = [k for k in cand if _bucket((k[0] << 32) | k[1], nb) != nb - 1]
    big = last[:6] + other[:4]
    assert len(big) == 10 and len(last) >= 6
    rng = np.random.default_rng(3)
    uni = [((w,), float(np.round(rng.uniform(-3.0, -0.5), 3)), float(np.round(rng.uniform(-1.0, 0.0), 3)))
           for w in range(W)] + [((bos,), -99.0, -0.4), ((W + 1,), -1.0, 0.0), ((W + 2,), -3.0, 0.0)]
    bigrams = [((c, w), float(np.round(rng.uniform(-2.0, -0.2), 3)), float(np.round(rng.uniform(-0.8, 0.0), 3)))
               for c, w in big]
    tri = [((big[0][0], big[0][1], 1), -0.3, -0.2), ((big[1][0], big[1][1], 2), -0.4, -0.1),
           ((big[2][0], big[2][1], 0), -0.5, 0.0)]
    four = [((big[0][0], big[0][1], 1, 3), -0.1)]
    lm = lm_from_entries(W, [uni, sorted(bigrams), sorted(tri), four])
    lex = lexicon_from(words)
    seqs = [[1, 40, 2, 40, 3, 1, 40, 1, 40, 2, 2, 40, 3, 40], [3, 40, 1, 40, 1, 40, 2, 40, 2, 2, 40, 1, 40]]
    lg = np.stack([peaked_logits([c for c in seqs[s % 2] for _ in range(2)][:26], strong=2.5, seed=s)
                   for s in range(4)])
    p = DecodeParams(beam=16, subbeams=3, fusion_interval=5, fusion_top_f=0, lam=8.0)
    d = data_of(lex, lm, lg, p, fusion_seed=21)
    for heavy in (0, 2):
        for fin in (True, False):
            say(f"[case] wrapping probe chains heavy={heavy} finalize={fin}")
            out = gpu_decode(d, params=p, finalize=fin,
                             lb_overrides=dict(lm_load_factor=0.9, heavy_homophones=heavy))
            check_parity(d, out, range(4), params=p, name=f"wrap/{heavy}/{fin}", finalize=fin)


# ------------------------------------------------------------------ profiling

@pytest.mark.parametrize("name", ["t-c20k", "t-k256"])
def test_profiling_changes_nothing_and_leaves_no_error(name):
    """Event timing of every kernel kind and the decode kernel's phase counters:
    the outputs are bit-identical to an unprofiled decode, every phase counter
    of a decode with frames is positive, and no HIP error is left for the next
    runtime call (torch's here)."""
    import torch
    d = load_workload(name, batch=3)
    say(f"[case] profiling {name}")
    plain = gpu_decode(d)
    prof, dec = gpu_decode(d, profiling=True, return_decoder=True)
    lbm.lb_set_profiling(dec.handle, lbm.LB_PROFILE_ALL | lbm.LB_PROFILE_PHASES)
    lbm.lb_reset_stats(dec.handle)
    dev = torch.device("cuda:0")
    K, W = dec.params.beam, dec.params.max_words_out
    B, T = d.logits.shape[:2]
    st, H, S = dec.decode(torch.from_numpy(d.logits).to(dev), torch.from_numpy(d.lengths.astype(np.int32)).to(dev))
    torch.cuda.synchronize()
    s = lbm.lb_get_stats(dec.handle)
    assert all(int(c) > 0 for c in s.phase_cycles[:3]), list(s.phase_cycles)
    assert s.timed[lbm.KIND_DECODE] == 1 and s.timed[lbm.KIND_BEGIN] == 1
    dec.close()
    x = torch.ones(1 << 20, device=dev).sum()  # raises if a HIP error was left behind
    assert float(x) == float(1 << 20)
    for (w1, s1), (w2, s2) in zip(plain, prof):
        assert w1 == w2 and np.array_equal(s1, s2)
    Hn, Sn = H.cpu().numpy(), S.cpu().numpy()
    for b in range(B):
        n = len(plain[b][0])
        assert np.array_equal(Sn[b, :n], plain[b][1])


# ------------------------------------------------------------------ gather ceiling probe

@pytest.mark.parametrize("theta", [4.0, 1.5])
def test_k256_theta_cut_matches_oracle(theta):
    """A theta small enough to bind inside the beam-256 selection (the cut's
    bin tested exactly against best - theta), in the instance for small
    batches (two lanes per hypothesis) and the one for batches beyond the CU
    count (one lane per hypothesis): the oracle's beams, and every copy of a
    tiled batch decoded like the original."""
    d = load_workload("t-k256")
    p = DecodeParams(**{**d.workload.params.__dict__, "theta": theta})
    n = d.logits.shape[0]
    say(f"[case] k256 theta={theta}: B={n}")
    small = gpu_decode(d, params=p)
    check_parity(d, small, range(n), params=p, name=f"t-k256 theta={theta}")
    big = 300
    reps = (big + n - 1) // n
    tile = lambda a: np.concatenate([a] * reps)[:big]
    db = WorkloadData(d.workload, d.lexicon, d.lm, tile(d.logits), tile(d.lengths), tile(d.targets),
                      (d.words * reps)[:big], d.fusion_seed)
    say(f"[case] k256 theta={theta}: B={big}")
    out = gpu_decode(db, params=p)
    for b in range(big):
        assert out[b][0] == small[b % n][0] and np.array_equal(out[b][1], small[b % n][1]), b


def test_two_decoders_on_two_streams():
    """Two decoders (a 20k-word workload and a beam-256 one) fed 10-frame
    chunks, their calls interleaved, each on a stream of its own: both decode
    exactly as they do alone (decoders share no state)."""
    import torch
    ds = [load_workload("t-c20k"), load_workload("t-k256")]
    chunk = 10
    solo = [gpu_decode(d, chunk=chunk) for d in ds]
    dev = torch.device("cuda:0")
    runs = []
    for d in ds:
        p = d.workload.params
        B, T = d.logits.shape[:2]
        lp = lbm.make_params(p, max_batch=B, max_frames=T, fusion_seed=d.fusion_seed)
        dec = lbm.Decoder(d.lexicon, d.lm, lp)
        lg = torch.from_numpy(np.ascontiguousarray(d.logits)).to(dev)
        nch = (T + chunk - 1) // chunk
        parts = []
        for c in range(nch):
            lo, hi = c * chunk, min(T, (c + 1) * chunk)
            ln = np.clip(d.lengths - lo, 0, hi - lo).astype(np.int32)
            parts.append((lg[:, lo:hi].contiguous(), torch.from_numpy(ln).to(dev)))
        hyps = torch.empty((B, lp.beam, lp.max_words_out), dtype=torch.int32, device=dev)
        scores = torch.empty((B, lp.beam), dtype=torch.float32, device=dev)
        runs.append(dict(dec=dec, parts=parts, hyps=hyps, scores=scores, stream=torch.cuda.Stream()))
    torch.cuda.synchronize()  # the inputs are in place before either stream starts
    say("[case] two decoders on two streams: t-c20k and t-k256, 10-frame chunks")
    for c in range(max(len(r["parts"]) for r in runs)):
        for r in runs:
            n = len(r["parts"])
            if c < n:
                fl = (lbm.LB_BEGIN if c == 0 else 0) | (lbm.LB_END if c == n - 1 else 0)
                st, _, _ = r["dec"].decode(r["parts"][c][0], r["parts"][c][1], fl, stream=r["stream"],
                                           out_hyps=r["hyps"], out_scores=r["scores"])
                assert st == lbm.LB_OK
    torch.cuda.synchronize()
    for r, ref in zip(runs, solo):
        assert r["dec"].status(r["stream"]) == lbm.LB_OK, lbm.lb_last_error()
        out = read_outputs(r["hyps"], r["scores"])
        assert len(out) == len(ref)
        for b, (got, want) in enumerate(zip(out, ref)):
            assert got[0] == want[0] and np.array_equal(got[1], want[1]), b
        r["dec"].close()


@pytest.mark.parametrize("seed", range(8))
def test_random_small_lexicons_match_oracle(seed):
    """Random small lexicons over phonemes 1..5 (one to four phonemes a word,
    so prefix words and doubled phonemes occur, plus two homophones), four
    utterances spelled from them with blank runs, decoded with pruning (beam
    8, 32, 64 or 256, two sub-beams, fusion every 4 frames, of all hypotheses
    for seeds 0..3 and of the best third for seeds 4..7): the oracle's
    outputs, at the end of the utterance and live."""
    rng = np.random.default_rng(500 + seed)
    n = int(rng.integers(6, 12))
    words = []
    while len(words) < n:
        w = tuple(int(x) for x in rng.integers(1, 6, size=int(rng.integers(1, 5))))
        if w not in words:
            words.append(w)
    words += [words[int(rng.integers(0, n))], words[int(rng.integers(0, n))]]
    lex = lexicon_from(words)
    lm = random_small_lm(len(words), 80)
    B, T = 4, 40
    rows = []
    for b in range(B):
        seq = []
        while len(seq) < T:
            for ph in words[int(rng.integers(0, len(words)))]:
                if seq and seq[-1] == ph:
                    seq.append(0)  # a repeated phoneme needs a blank between
                seq += [ph] * int(rng.integers(1, 3))
            seq += [40] + [0] * int(rng.integers(0, 3))
        rows.append(peaked_logits(seq[:T], strong=3.0, seed=seed * 10 + b, sigma=0.8))
    lg = np.stack(rows)
    lengths = np.array([T, T - 7, T, T - 13], np.int32)
    beam = (8, 32, 64, 256)[seed % 4]
    p = DecodeParams(beam=beam, subbeams=2, fusion_interval=4, fusion_top_f=0 if seed < 4 else beam // 3)
    wl = load_workload("t-c1k").workload
    wl = wl.__class__(**{**wl.__dict__, "params": p})
    d = WorkloadData(wl, lex, lm, lg, lengths, np.zeros((B, T), np.int32), [[] for _ in range(B)], 11 + seed)
    for fin in (True, False):
        say(f"[case] random lexicon seed={seed} words={len(words)} K={beam} F={p.fusion_top_f} fin={fin}")
        out = gpu_decode(d, params=p, finalize=fin)
        check_parity(d, out, range(B), params=p, name=f"random-lexicon/{seed}", finalize=fin)


@pytest.mark.parametrize("seed", range(10))
def test_random_parameters_match_oracle(seed):
    """Every decode parameter drawn at random (beam 1..256, sub-beams 1..4,
    alpha, beta, gamma, omega, phi, theta, lambda, fusion interval and top F,
    log-sum-exp or max recombination) over the 1k-, 20k- and 125k-word test
    workloads (the last with ~300-word homophone sets), the first 60 frames:
    the oracle's outputs, at the end of the utterance and live.  Odd seeds
    also decode 300 copies of the batch, which takes the kernels for batches
    beyond the CU count; every copy must equal the small batch's output.
    Decoded in calls of a random number of frames (1..16, the streams' state
    carried from call to call), the output equals the one-shot decode's."""
    rng = np.random.default_rng(900 + seed)
    name = ("t-c1k", "t-c20k", "t-c125k")[seed % 3]
    base = load_workload(name, batch=4)
    beam = int(rng.choice([1, 2, 5, 16, 33, 64, 100, 128, 200, 256]))
    p = DecodeParams(
        beam=beam, subbeams=int(rng.integers(1, 5)),
        alpha=float(rng.choice([0.5, 0.6, 1.0])), beta=float(rng.choice([0.0, 0.75, 1.5])),
        gamma=float(rng.choice([0.0, 1.0, 2.0])), omega=float(rng.choice([0.0, 0.5, 1.25])),
        phi=float(rng.choice([0.5, 1.2])), theta=float(rng.choice([2.0, 8.0, 22.0, 1e30])),
        lam=float(rng.choice([0.5, 4.0, 1e30])), fusion_interval=int(rng.choice([0, 1, 4, 9])),
        fusion_top_f=int(rng.choice([0, 1, max(1, beam // 3)])))
    merge_max = bool(rng.random() < 0.25)
    chunk = int(rng.integers(1, 17))
    T = min(60, base.logits.shape[1])
    B = base.logits.shape[0]
    lengths = np.minimum(base.lengths, T).astype(np.int32)
    wl = base.workload.__class__(**{**base.workload.__dict__, "params": p})
    d = WorkloadData(wl, base.lexicon, base.lm, np.ascontiguousarray(base.logits[:, :T]), lengths,
                     base.targets[:, :T], base.words, base.fusion_seed)
    lb_over = dict(merge=lbm.LB_MERGE_MAX) if merge_max else None
    orc_over = dict(merge_max=1) if merge_max else None
    for fin in (True, False):
        say(f"[case] random parameters seed={seed} {name} {p} merge_max={merge_max} fin={fin}")
        out = gpu_decode(d, params=p, finalize=fin, lb_overrides=lb_over)
        check_parity(d, out, range(B), params=p, name=f"random-params/{seed}", finalize=fin,
                     oracle_overrides=orc_over, min_hyps=0 if fin else 1)
        say(f"[case] random parameters seed={seed} in calls of {chunk} frames fin={fin}")
        outc = gpu_decode(d, params=p, finalize=fin, chunk=chunk, lb_overrides=lb_over)
        for b in range(B):
            assert outc[b][0] == out[b][0] and np.array_equal(outc[b][1], out[b][1]), (b, chunk)
        if seed % 2:
            big = 300
            tile = lambda a: np.concatenate([a] * (big // B))
            db = WorkloadData(wl, base.lexicon, base.lm, tile(d.logits), tile(lengths), tile(d.targets),
                              d.words * (big // B), base.fusion_seed)
            say(f"[case] random parameters seed={seed} B={big} fin={fin}")
            outb = gpu_decode(db, params=p, finalize=fin, lb_overrides=lb_over)
            for b in range(big):
                assert outb[b][0] == out[b % B][0] and np.array_equal(outb[b][1], out[b % B][1]), b


def test_gather_probe_reads_the_lines_it_names():
    """lb_measure_gather reads line mulhi(splitmix64(seed + i), lines) for
    gather i, 8 per thread, and writes each thread's XOR of the 16 words it
    read: the same XOR computed here from the table's contents."""
    import torch
    lines, n, seed = 1000, 8 * 37 + 5, 12345
    rng = np.random.default_rng(4)
    host = rng.integers(0, 2**32, size=(lines, 16), dtype=np.uint64).astype(np.uint32)
    table = torch.from_numpy(host.view(np.int32)).to("cuda:0")
    threads = (n + 7) // 8
    out = torch.full((threads,), -1, dtype=torch.int32, device="cuda:0")
    lbm.lb_measure_gather(table, lines, n, seed, out, threads, None)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32)
    for t in range(threads):
        x = 0
        for g in range(8):
            i = t * 8 + g
            if i < n:
                line = (pins.splitmix64((seed + i) & pins.M64) * lines) >> 64
                for w in host[line]:
                    x ^= int(w)
        assert int(got[t]) == x, t
    with pytest.raises(lbm.LBError):
        lbm.lb_measure_gather(table, lines, n, seed, out, threads - 1, None)
