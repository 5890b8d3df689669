"""Seeded synthetic workloads for the LightBeam decoding path.

This package only *generates inputs*: a phoneme lexicon, a 4-gram backoff LM,
per-frame CTC log-probabilities and decoder parameters.  It holds none of the
decoder's arithmetic, and both the CPU oracle (``oracle/``) and the HIP
library (``paper_2603_14002_amd``) consume exactly the arrays produced here.

The shapes follow the paper's setting (LightBeam, arXiv 2603.14002):
41 output classes -- blank, 39 phonemes and a word separator (Sec. 3.2);
80 ms encoder frames (Fig. 2 caption, B2T '25); a phoneme lexicon with
homophones (Sec. 3.4.1); a 4-gram backoff LM (Sec. 3.4.1); decoding
hyper-parameters from the App. E table.  The paper's data (Brain-to-Text
'24/'25, the ImagineVille 4-gram, CMUdict) are not reproduced: seeded random
stand-ins of the same structure replace them.
"""

from .configs import (  # noqa: F401
    BLANK, SEP, N_CLASSES, N_PHONEMES, FRAME_SECONDS,
    LexiconSpec, LMSpec, DecodeParams, Workload, CONFIGS, get_config,
)
from .gen import (  # noqa: F401
    Lexicon, NGramLM, make_lexicon, make_lm, make_targets, make_logits,
    load_workload, WorkloadData,
)
