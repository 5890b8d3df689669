"""Workload definitions: lexicon / LM sizes, batch shapes and decoder parameters.

Class layout: blank = 0, phonemes 1..39, word separator (SEP) = 40.  The
paper lists "39 phonemes, a CTC blank token, and a space token" (Sec. 3.2)
without fixing an order; this order is the one used everywhere here.

Default decoder parameters come from the B2T '24 column of the App. E
hyper-parameter table (alpha=0.6, beta=1.5, gamma=1.0, phi=1.2, theta=22,
o=3, lambda=4), except omega=0.5 which the 125k-word workloads fix and which
is applied to every workload for uniformity.
"""

from dataclasses import dataclass, field, replace

BLANK = 0
SEP = 40
N_PHONEMES = 39
N_CLASSES = 41
FRAME_SECONDS = 0.08  # B2T '25 frame period (Fig. 2 caption)

# Base of every seed sequence (the arXiv identifier).
BASE_SEED = 260314002


@dataclass(frozen=True)
class LexiconSpec:
    name: str
    n_words: int
    max_len: int          # word lengths ~ U{1..max_len} phonemes
    variant_frac: float = 0.0  # share of words given a second pronunciation (one phoneme edited)


@dataclass(frozen=True)
class LMSpec:
    name: str
    lexicon: LexiconSpec
    n_total: int          # total n-grams over all 4 orders (unigrams included)


@dataclass(frozen=True)
class DecodeParams:
    beam: int = 8                 # K
    subbeams: int = 3             # o (homophone / orthographic sub-beams)
    alpha: float = 0.6            # acoustic scale
    beta: float = 1.5             # token insertion bonus
    gamma: float = 1.0            # word boundary bonus
    omega: float = 0.5            # n-gram weight
    phi: float = 1.2              # fusion (LLM) weight
    theta: float = 22.0           # beam prune threshold
    lam: float = 4.0              # homophone prune threshold
    fusion_interval: int = 0      # I, 0 = no fusion
    fusion_top_f: int = 0         # F, 0 = all beams
    fusion_lo: float = -10.0      # synthetic scorer range (natural log)
    fusion_hi: float = -0.5
    max_words_out: int = 256      # W_max of the output word buffer


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    frames: int
    lm: LMSpec
    params: DecodeParams
    sigma: float = 1.0            # logit noise std
    chunk: int = 0                # >0: streaming, fed in chunks of this many frames
    ragged: bool = False          # per-utterance lengths drawn in [frames//2, frames]
    description: str = ""

    @property
    def lexicon(self) -> LexiconSpec:
        return self.lm.lexicon


LEX_1K = LexiconSpec("lex1k", 1_000, 8)
LEX_20K = LexiconSpec("lex20k", 20_000, 8)
LEX_125K = LexiconSpec("lex125k", 125_000, 12)

LM_5K = LMSpec("lm5k", LEX_1K, 5_000)
LM_1M = LMSpec("lm1m", LEX_20K, 1_000_000)
LM_50M = LMSpec("lm50m", LEX_125K, 50_000_000)
LM_200M = LMSpec("lm200m", LEX_125K, 200_000_000)
# Reduced LMs over the same lexicons, for parity tests the oracle finishes quickly.
LM_20K_SMALL = LMSpec("lm20k-200k", LEX_20K, 200_000)
LM_125K_SMALL = LMSpec("lm125k-2m", LEX_125K, 2_000_000)
# 20k words, a fifth of them with a second pronunciation (App. I's word(2) entries)
LEX_20K_VAR = LexiconSpec("lex20k-var", 20_000, 8, variant_frac=0.2)
LM_20K_VAR = LMSpec("lm20kvar-200k", LEX_20K_VAR, 200_000)

_P = DecodeParams()

CONFIGS = {
    "c1": Workload(
        "c1", batch=1, frames=50, lm=LM_5K, sigma=1.0,
        params=replace(_P, beam=8, fusion_interval=0),
        description="tiny: 1 utterance, T=50, 1k words, 5k n-grams, K=8, no fusion"),
    "c2": Workload(
        "c2", batch=64, frames=200, lm=LM_1M, sigma=1.0,
        params=replace(_P, beam=32, fusion_interval=20, fusion_top_f=0),
        description="64 x T=200, 20k words, 1M n-grams, K=32, fusion every 20 frames"),
    "c3": Workload(
        "c3", batch=256, frames=500, lm=LM_50M, sigma=1.5,
        params=replace(_P, beam=64, fusion_interval=16, fusion_top_f=16),
        description="256 x T=500, 125k words, 50M n-grams, K=64, fusion every 16 frames on top 16"),
    "c4": Workload(
        "c4", batch=512, frames=500, lm=LM_200M, sigma=1.5,
        params=replace(_P, beam=256, fusion_interval=16, fusion_top_f=32),
        description="512 x T=500, 125k words, 200M n-grams, K=256, fusion every 16 frames on top 32"),
    "c5": Workload(
        "c5", batch=1024, frames=1000, lm=LM_50M, sigma=1.5, chunk=10,
        params=replace(_P, beam=64, fusion_interval=8, fusion_top_f=0),
        description="1024 streams x T=1000 in 10-frame chunks, 125k words, 50M n-grams, K=64, fusion every 8"),
    # ---- small parity cases (same generators, sizes the oracle finishes in seconds)
    "t-c1k": Workload(
        "t-c1k", batch=7, frames=60, lm=LM_5K, sigma=1.0, ragged=True,
        params=replace(_P, beam=8, fusion_interval=7, fusion_top_f=3)),
    "t-c20k": Workload(
        "t-c20k", batch=5, frames=120, lm=LM_20K_SMALL, sigma=1.0, ragged=True,
        params=replace(_P, beam=32, fusion_interval=20, fusion_top_f=0)),
    "t-c125k": Workload(
        "t-c125k", batch=3, frames=100, lm=LM_125K_SMALL, sigma=1.5, ragged=True,
        params=replace(_P, beam=64, fusion_interval=16, fusion_top_f=16)),
    "t-k256": Workload(
        "t-k256", batch=2, frames=80, lm=LM_125K_SMALL, sigma=1.5,
        params=replace(_P, beam=256, fusion_interval=16, fusion_top_f=32)),
    "t-variants": Workload(
        "t-variants", batch=5, frames=120, lm=LM_20K_VAR, sigma=1.0, ragged=True,
        params=replace(_P, beam=32, fusion_interval=20, fusion_top_f=0)),
    "t-stream": Workload(
        "t-stream", batch=4, frames=90, lm=LM_125K_SMALL, sigma=1.5, chunk=10, ragged=True,
        params=replace(_P, beam=64, fusion_interval=8, fusion_top_f=0)),
}


def get_config(name: str) -> Workload:
    try:
        return CONFIGS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS)}") from None
