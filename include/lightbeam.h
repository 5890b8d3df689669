/*
 * lightbeam.h -- C ABI of the MI355X (gfx950) LightBeam decoding library.
 *
 * The library decodes batches of per-frame CTC phoneme log-probabilities into
 * word sequences with the method of LightBeam (arXiv 2603.14002):
 * lexicon-constrained CTC prefix beam search (Alg. 1; Sec. 3.4; App. E.1-E.2),
 * homophone ("orthographic") sub-beams scored by a 4-gram backoff LM at word
 * boundaries (Sec. 3.4.1, Eq. (1); App. E.3), and delayed fusion that replaces
 * the sub-beams' word-level scores with a fusion scorer's scores at fixed frame
 * intervals (Sec. 3.4.2, Eq. (2); App. E.4).  The paper's LLM scorer is not part
 * of the library: a seeded synthetic word-bigram scorer stands in for it, or the
 * caller supplies scores (LB_FUSION_EXTERNAL).
 *
 * Class layout of the log-probabilities: 0 = CTC blank, 1..39 = phonemes,
 * 40 = word separator.  All scores are natural-log; LM tables are log10.
 *
 * Conventions:
 *   - every function returns an lb_status and never throws or aborts;
 *   - lb_last_error() gives a thread-local message for the last failure;
 *   - "host" pointers are read during the call only (the library copies what it
 *     keeps); "device" pointers are caller-owned HIP device memory that the
 *     library never frees;
 *   - stream arguments are hipStream_t values passed as void* (NULL = the null
 *     stream); work is enqueued asynchronously on that stream;
 *   - a decoder is not thread-safe: calls on one decoder must be serialised.
 */
#ifndef LIGHTBEAM_H_
#define LIGHTBEAM_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t lb_status;

enum {
  LB_OK = 0,
  LB_ERR_INVALID_ARG = 1,   /* bad pointer, size, id or parameter                  */
  LB_ERR_STATE = 2,         /* call out of order (e.g. fusion scores not requested) */
  LB_ERR_CAPACITY = 3,      /* a fixed-capacity buffer overflowed                   */
  LB_ERR_OUT_OF_MEMORY = 4, /* device or host allocation failed                     */
  LB_ERR_HIP = 5,           /* a HIP runtime call failed                            */
  LB_NEED_FUSION = 6        /* not an error: external fusion scores are required    */
};

enum { LB_BLANK = 0, LB_SEP = 40, LB_NUM_CLASSES = 41, LB_NUM_PHONEMES = 39 };
enum { LB_MAX_BEAM = 256, LB_MAX_SUBBEAMS = 4 };

/* lb_decode_batch flags */
enum { LB_BEGIN = 1u, LB_END = 2u };

/* recombination of the paths that reach one prefix (lb_params.merge) */
enum {
  LB_MERGE_LOGSUMEXP = 0,  /* sum over alignments (classical CTC prefix search)      */
  LB_MERGE_MAX = 1         /* best alignment only (the recombination of App. E.1)    */
};

/* what lb_decode_batch's per-frame scores are (lb_params.input) */
enum {
  LB_INPUT_LOGPROBS = 0,   /* log-probabilities (log-softmax already applied)        */
  LB_INPUT_LOGITS = 1      /* raw scores: log-softmax over the 41 classes per frame  */
};

/* fusion scorer */
enum {
  LB_FUSION_NONE = 0,          /* no delayed fusion                                     */
  LB_FUSION_SYNTH_BIGRAM = 1,  /* seeded synthetic word-bigram scorer (see lb_params)   */
  LB_FUSION_EXTERNAL = 2       /* the caller scores requested word sequences            */
};

/* Lexicon (host memory).  Word w spells phonemes[offsets[w] .. offsets[w+1]),
 * each in 1..39, at least one per word.  Word ids double as LM vocabulary ids.
 * Words with equal spellings are homophones (Sec. 3.4.1). */
typedef struct lb_lexicon_desc {
  int32_t n_entries;         /* pronunciations                                      */
  const int32_t* offsets;    /* [n_entries + 1], increasing, offsets[0] == 0        */
  const int32_t* phonemes;   /* [offsets[n_entries]], values 1..39                  */
  const int32_t* entry_word; /* [n_entries]: LM word id spelled by each entry, so a
                                word may have several pronunciations (App. I);
                                NULL: entry e spells word e                         */
} lb_lexicon_desc;

/* 4-gram backoff LM in ARPA form (host memory), queried per (context, word) as
 * in App. E.3: log10 P(w | u1..um) = p(u1..um w) if present, else
 * bo(u1..um) + log10 P(w | u2..um) (bo = 0 for an absent context), and
 * p(<unk>) for a word without unigram.  Order n (n = 1..4, index n-1) holds
 * count[n-1] entries: ids[n-1] is [count][n] int32 word ids (oldest first),
 * log10p[n-1] and backoff[n-1] float32 (backoff[3] is ignored).  Every entry's
 * context (its first n-1 ids) must itself be an order n-1 entry.  Duplicate
 * entries are rejected. */
typedef struct lb_ngram_desc {
  int32_t vocab_size; /* ids are in [0, vocab_size); the lexicon words come first */
  int32_t bos_id;     /* <s>: the context of a sentence's first word             */
  int32_t unk_id;     /* <unk>                                                   */
  int32_t reserved;
  int64_t count[4];
  const int32_t* ids[4];
  const float* log10p[4];
  const float* backoff[4];
} lb_ngram_desc;

/* Decoder parameters.  Names follow the paper's App. E hyper-parameter table. */
typedef struct lb_params {
  int32_t beam;      /* k: hypotheses kept per stream, 1..LB_MAX_BEAM             */
  int32_t subbeams;  /* o (h): orthographic sub-beams per hypothesis, 1..4        */
  double alpha;      /* acoustic scale: D = alpha * log-probs                    */
  double beta;       /* token insertion bonus, once per new phoneme              */
  double gamma;      /* word boundary bonus, once per new separator              */
  double omega;      /* n-gram weight (Eq. (1)); applied to ln(10) * log10 P      */
  double phi;        /* fusion weight (Eq. (2))                                  */
  double theta;      /* beam prune threshold: drop total < best - theta          */
  double lambda;     /* homophone prune threshold: drop Lw < best Lw - lambda    */
  int32_t fusion_source;   /* LB_FUSION_*                                         */
  int32_t fusion_interval; /* I: fuse after frame t when t % I == 0 and t > 0     */
  int32_t fusion_top_f;    /* F: hypotheses fused per event (0 = all)            */
  int32_t max_batch;       /* streams per decoder                                */
  int32_t max_frames;      /* frames per stream between LB_BEGIN and LB_END      */
  int32_t max_words_out;   /* W_max of out_hyps and of fusion requests           */
  uint64_t fusion_seed;    /* synthetic scorer: Bg(a,b) = lo + (hi-lo) *         */
  double fusion_lo;        /*   (splitmix64(seed ^ (a<<32 | b)) >> 48) / 65536,   */
  double fusion_hi;        /*   S_fus(w1..wn) = sum_i Bg(w_{i-1}, w_i), w0 = <s>  */
  double lm_load_factor;   /* n-gram hash-table load factor (0 = 0.25), <= 0.9    */
  int64_t arena_nodes_per_stream; /* word-history capacity (0 = beam*subbeams*max_frames) */
  int32_t merge;           /* LB_MERGE_*                                          */
  int32_t input;           /* LB_INPUT_*                                          */
  int32_t eos_count;       /* end-of-sentence marks (0..3) tried at LB_END with the
                              synthetic scorer: each sub-beam's sequence is scored
                              with every mark appended, the best counts and is
                              appended to the output words (first of equals wins) */
  int32_t eos_ids[3];      /* the marks' LM word ids                              */
  int32_t heavy_homophones; /* trie nodes with at least this many words are scored
                              through the explicit-continuation index (0 = 3,
                              < 0 = never): per (context, node) only the homophones
                              that have an n-gram entry are looked up, the others
                              back off to their unigrams and are ranked by a walk
                              over the node's words in unigram order.  Results are
                              the same either way (Eq. (1) evaluated exactly)     */
} lb_params;

typedef struct lb_decoder lb_decoder;

/* Counters accumulated since lb_create (or the last lb_reset_stats). */
typedef struct lb_stats {
  int64_t expansions;   /* sum over stream-frames of (live hypotheses x 41)      */
  int64_t word_events;  /* hypotheses that completed a word (n-gram applied)     */
  int64_t lm_queries;   /* (sub-beam, homophone) n-gram queries                   */
  int64_t fused;        /* hypotheses rescored by delayed fusion                  */
  int64_t frames;       /* stream-frames decoded                                  */
  int64_t probe_lines;  /* 64-B hash-table lines read by the LM lookups (n-gram
                           tables and the explicit-continuation index)           */
  int64_t lm_lookups;   /* n-gram lookups done: one per distinct (context, word)
                           among a stream-frame's queries, except homophones of
                           heavy nodes that the continuation index shows to back
                           off to their unigram (scored without a lookup)       */
  int64_t launches[8];  /* kernel launches: [0] decode (all frames of a call), [1]
                           output, [2] external-fusion select, [3] export, [4]
                           apply, [5] stream reset, [6..7] unused                */
  double  kernel_ms[8]; /* summed event-timed durations (when profiling is on)    */
  int64_t timed[8];     /* launches included in kernel_ms                         */
  int64_t index_lines;  /* the part of probe_lines read from the explicit-
                           continuation index                                     */
  int64_t phase_cycles[8]; /* with LB_PROFILE_PHASES: clock cycles of the decode
                           launches' workgroups, summed over streams, by phase:
                           [0] recombination and stay scores, [1] top-K and theta,
                           [2] new beam, [3] grouping of the n-gram queries and
                           the continuation index, [4] n-gram lookups, [5]
                           ranking of the completed words (top-o, lambda) and
                           history nodes, [6] fusion and the rest of the frame,
                           [7] beam load / write-back / output                  */
} lb_stats;

/* Builds a decoder: the lexicon trie (CSR) and the n-gram hash tables are
 * built and uploaded to device memory, and every buffer a decode needs is
 * allocated for max_batch streams.  Synchronous.
 * Errors: LB_ERR_INVALID_ARG (bad ids or parameters, an n-gram whose context is
 * missing, duplicate n-grams), LB_ERR_OUT_OF_MEMORY, LB_ERR_HIP. */
lb_status lb_create(const lb_lexicon_desc* lex, const lb_ngram_desc* lm, const lb_params* params,
                    lb_decoder** out);

/* Frees every device and host resource of the decoder (NULL is ignored). */
void lb_destroy(lb_decoder* dec);

/* Decodes `frames` frames for streams 0..batch-1 (Alg. 1, one loop iteration
 * per frame).
 *   logits      device float32 [batch][frames][41], log-softmax per frame
 *   lengths     device int32 [batch]: frames of this call valid for each stream
 *               (0..frames; the rest of the stream's rows are ignored; a value
 *               outside 0..frames is clamped and reported by lb_get_status)
 *   flags       LB_BEGIN resets streams 0..batch-1 to the empty hypothesis;
 *               LB_END finalises them after the call's frames (final fusion over
 *               every hypothesis; hypotheses inside a word are dropped when some
 *               hypothesis ends at a word boundary, else all are ranked by
 *               their completed words)
 *   out_hyps    device int32 [batch][beam][max_words_out]: word ids of the best
 *               sub-beam of each ranked hypothesis, -1 padded
 *   out_scores  device float32 [batch][beam]: total scores, -inf padded
 * Hypothesis state persists across calls (streaming).  Without LB_END the
 * outputs rank the current hypotheses (completed words only).  With
 * LB_FUSION_EXTERNAL the call may return LB_NEED_FUSION: the caller then calls
 * lb_fusion_request and lb_fusion_scores and repeats this call with the same
 * arguments, which resumes after the fused frame (with LB_END, a last
 * LB_NEED_FUSION precedes the final outputs).  Asynchronous on `stream`, except
 * with LB_FUSION_EXTERNAL, where the call reads `lengths` to the host. */
lb_status lb_decode_batch(lb_decoder* dec, const float* logits, const int32_t* lengths,
                          int32_t batch, int32_t frames, uint32_t flags, void* stream,
                          int32_t* out_hyps, float* out_scores);

/* lb_decode_batch for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, hosts that forbid allocation): the
 * same decode with the same arguments and results, whose n-gram lookup scratch
 * is a fixed array of 64 MiB per device (held until the process ends) instead
 * of memory of the decoder; it calls no allocating routine and creates no
 * events (lb_set_profiling's event timing does not apply; the phase counters
 * do).  The scratch holds batch x (K * subbeams * H * 32 B + K * 256 B), H the
 * largest homophone set of the lexicon, rounded up per region: a batch that
 * needs more returns LB_ERR_CAPACITY (and decodes nothing).  Every such call
 * on a device shares that device's array: calls that overlap in time on one
 * device (other streams, other threads, other decoders) race on it and must be
 * serialised by the caller.  Nothing in the array needs to start at zero (each
 * frame writes what it reads).  Decoders with LB_FUSION_EXTERNAL are refused
 * (LB_ERR_INVALID_ARG): their round trip reads the lengths to the host. */
lb_status lb_decode_batch_noalloc(lb_decoder* dec, const float* logits, const int32_t* lengths, int32_t batch,
                                  int32_t frames, uint32_t flags, void* stream, int32_t* out_hyps,
                                  float* out_scores);

/* Exports the word sequences of a pending fusion event (after LB_NEED_FUSION).
 * Entry [b][r][j] is sub-beam j of the stream's r-th fused hypothesis; the
 * fused hypotheses are the top fusion_top_f (all when 0) by total score at a
 * fusion frame, and all hypotheses at the end of an utterance:
 *   words    device int32 [batch][beam][subbeams][max_words_out], -1 padded
 *   n_words  device int32 [batch][beam][subbeams]: number of words, or -1
 *            where nothing is to be scored (stream not fusing this frame,
 *            fewer hypotheses or sub-beams)
 * LB_ERR_STATE if no fusion is pending. */
lb_status lb_fusion_request(lb_decoder* dec, int32_t* words, int32_t* n_words, void* stream);

/* Applies Eq. (2) with caller-computed fusion scores for the pending event:
 *   fusion_logprobs  device float32 [batch][beam][subbeams], natural-log
 *                    full-sequence scores sum_t log p(w_t | w_<t) of the
 *                    requested sequences (entries with n_words == -1 ignored)
 * Each requested sub-beam's word-level score becomes phi * score and the
 * sub-beams are re-ranked.  LB_ERR_STATE if no fusion is pending. */
lb_status lb_fusion_scores(lb_decoder* dec, const float* fusion_logprobs, void* stream);

/* Synchronises `stream` and reports device-side flags raised since lb_create:
 * LB_ERR_CAPACITY if a word-history arena, an output buffer (words beyond
 * max_words_out) or the top-K selection's boundary buffer overflowed (the
 * writes past them were skipped), LB_ERR_INVALID_ARG if a decode call was
 * given a length outside 0..frames (that stream was decoded, and its frame
 * counter advanced, as if the length were clamped to that range). */
lb_status lb_get_status(lb_decoder* dec, void* stream);

/* Reads the counters (synchronises the device).  With profiling on (see
 * lb_set_profiling), kernel_ms holds event-timed kernel durations. */
lb_status lb_get_stats(lb_decoder* dec, lb_stats* out);
lb_status lb_reset_stats(lb_decoder* dec);

/* Kernel timing with HIP events: bit k of kernel_mask times the kernels of
 * kind k (the index of lb_stats.launches); 0 disables timing and
 * LB_PROFILE_ALL times every launch.  The start / stop events are carried by
 * the kernel's own dispatch (hipExtLaunchKernel), so they time its execution
 * only.  LB_PROFILE_PHASES makes the decode kernel count the clock cycles of
 * each phase of its frames (lb_stats.phase_cycles). */
enum { LB_PROFILE_ALL = 0xFFu, LB_PROFILE_PHASES = 0x100u };
lb_status lb_set_profiling(lb_decoder* dec, uint32_t kernel_mask);

/* Thread-local description of the last error ("" if none). */
const char* lb_last_error(void);

/* Measurement: the random-gather ceiling of the n-gram probes' access
 * pattern (one 64-B bucket line per probe, at random positions of tables far
 * larger than the caches).  Reads n_lines lines of 64 B from the device table
 * `table` (table_lines lines, 16-B aligned) at pseudo-random line indices
 * (the multiply-high of splitmix64(seed + i) and table_lines, for i =
 * 0..n_lines-1), 8 independent lines per thread, and writes each thread's XOR
 * of what it read to out (device uint32, out_len >= ceil(n_lines / 8)).
 * Asynchronous on `stream`; the caller times it.  LB_ERR_INVALID_ARG for
 * null pointers, zero sizes or a short out. */
lb_status lb_measure_gather(const void* table, uint64_t table_lines, uint64_t n_lines, uint64_t seed,
                            uint32_t* out, uint64_t out_len, void* stream);

/* Identity of the build: a hex sha256 over the library's source files
 * (comments and spacing removed) and its compile flags, fixed at build time,
 * so that a caller can check that the library in hand was built from the
 * sources it expects ("unknown" if the build did not define it). */
const char* lb_build_id(void);

#ifdef __cplusplus
}
#endif

#endif /* LIGHTBEAM_H_ */
