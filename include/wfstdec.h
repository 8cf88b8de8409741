/*
 * wfstdec -- WFST Viterbi beam decoding with exact (state-level) lattices,
 * frame-synchronous or label-synchronous, on one AMD Instinct MI355X (gfx950).
 *
 * The operations follow Z. Chen, "Linguistic Search Optimization for Deep
 * Learning Based LVCSR" (Interspeech 2018):
 *   - linguistic search = Viterbi beam decoding over a WFST search graph
 *     (Sec. 1), by token passing where every state keeps the minimum-cost
 *     token over its incoming arcs together with its predecessor
 *     ("token recombination", Sec. 3 and Fig. 2);
 *   - label-synchronous decoding (Sec. 2, Eq. 2, Alg. 1): frames whose blank
 *     posterior exceeds a threshold (the set U) are skipped, so the search
 *     runs on T - |U| frames (Eq. 3); for the HMM topologies of Sec. 2 the
 *     blank is a set of blank-like units, and a lower frame rate decodes
 *     every k-th frame;
 *   - finalTransition then backtrace (Alg. 1);
 *   - exact lattice generation and lattice pruning (Sec. 1, Sec. 3).
 *
 * Conventions used throughout:
 *   - costs are negative log probabilities in float32 (min over paths
 *     = arg max of Eq. 1); an emitting arc a = (s -> d, ilabel i, weight w)
 *     taken at a frame with log-likelihood row ll gives the candidate
 *     (cost(s) + w) - ll[i - 1], two float32 roundings in that order, no
 *     fused multiply-add, no flush of subnormals;
 *   - ilabel 0 marks an epsilon arc (consumes no frame); ilabel i >= 1 reads
 *     log-likelihood column i - 1; olabel 0 means no output;
 *   - arcs are identified by their index in the arrays given to wfst_load
 *     ("user arc index");
 *   - equal costs are broken towards the lower arc index, the start token
 *     wins all ties, and the final state with the lowest id wins a tie on the
 *     final cost; results are therefore deterministic and independent of
 *     the order in which the GPU processes work.
 *
 * All entry points return an int status (WFST_OK = 0 or a negative error)
 * unless stated otherwise; wfst_last_error() gives a message for the
 * calling thread's last failure.
 */
#ifndef WFSTDEC_H
#define WFSTDEC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WFST_OK 0
#define WFST_EINVAL (-1)    /* invalid argument or graph */
#define WFST_ENOMEM (-2)    /* host or device allocation failed */
#define WFST_ENOPATH (-3)   /* the token set became empty: no surviving path */
#define WFST_ECAPACITY (-4) /* a fixed buffer overflowed even after retries; raise capacity_hint */
#define WFST_EDEVICE (-5)   /* HIP runtime error */

typedef struct wfst_graph wfst_graph;
typedef struct wfst_result wfst_result;

/*
 * wfst_load -- validate a WFST given as arc arrays sorted by source state
 * (CSR order) and lay it out in device memory of the current HIP device.
 *
 *   num_states   N >= 1
 *   num_arcs     E, 0 <= E < 2^31 - 1
 *   src, dst     [E] host int32, src sorted ascending, both in [0, N)
 *   ilabel       [E] host int32 >= 0 (0 = epsilon)
 *   olabel       [E] host int32 >= 0 (0 = none); read by the word-level lattice
 *   weight       [E] host float32, finite; epsilon arcs need weight >= 0
 *   start_state  in [0, N)  (the start node S of Alg. 1)
 *   final_weight [N] host float32 or NULL; NULL makes every state final with
 *                cost 0; +inf marks a non-final state; NaN and -inf are
 *                invalid (the end node E of Alg. 1 as final costs)
 *   out          receives the graph handle
 *
 * The epsilon subgraph must be acyclic.  Input arrays are copied and may be
 * freed on return.  The handle is immutable and may be shared by concurrent
 * decodes on different streams of the same device.  Errors: WFST_EINVAL
 * (any rule above), WFST_ENOMEM, WFST_EDEVICE.
 */
int wfst_load(int32_t num_states, int64_t num_arcs, const int32_t *src, const int32_t *dst,
              const int32_t *ilabel, const int32_t *olabel, const float *weight,
              int32_t start_state, const float *final_weight, wfst_graph **out);

/* Release a graph (NULL is allowed).  No decode may be running on it. */
void wfst_graph_free(wfst_graph *g);

typedef struct wfst_graph_info {
    int32_t num_states;
    int64_t num_arcs;
    int64_t num_emitting;     /* arcs with ilabel != 0 */
    int64_t num_epsilon;      /* arcs with ilabel == 0 */
    int32_t max_ilabel;       /* decode needs L >= max_ilabel */
    int32_t epsilon_depth;    /* longest epsilon path (arcs) */
    int64_t device_bytes;     /* device memory held by the layout */
    int64_t num_closure_states; /* states whose whole epsilon closure is precomputed as a list
                                   of paths (at most 256 paths of at most 9 arcs each); the
                                   others relax their epsilon arcs one level at a time.  The
                                   results are the same either way. */
} wfst_graph_info;

int wfst_graph_get_info(const wfst_graph *g, wfst_graph_info *info);

/* decode options */
#define WFST_RECORD_TOKENS 1u  /* keep every token set for wfst_result_tokens */
#define WFST_LOGLIKES_HOST 2u  /* loglikes pointers are host memory (copied to the device first) */
#define WFST_PROFILE 4u        /* time the kernel phases with HIP events on the decode streams */
#define WFST_PROFILE_STEPS 8u  /* also read the device clock per step inside the kernels (slower) */
#define WFST_WORD_LATTICE 16u  /* also build the word-level lattice of the pruned lattice (needs
                                  lattice_beam >= 0): wfst_result_words */
#define WFST_INCREMENTAL_LATTICE 32u /* record and prune the lattice incrementally, beside the
                                  search on a second stream (Sec. 3): every 32 decoded frames
                                  the finished frames' lattice arcs are pruned against the
                                  search frontier, so the raw lattice needs rings of a few
                                  chunks instead of regions for the whole utterance; the
                                  result is bit-identical.  Batches of up to 96 utterances
                                  (larger batches decode without it) */

typedef struct wfst_decode_opts {
    float beam;               /* > 0 (may be +inf): keep tokens with cost <= best + beam */
    int32_t max_active;       /* <= 0: unlimited; else keep the max_active cheapest tokens
                                 (all tokens tied with the last one are kept) */
    float lattice_beam;       /* < 0: no lattice; else keep lattice arcs whose best complete
                                 path is within lattice_beam of the best path (+inf: all) */
    float blank_threshold;    /* > 1: frame-synchronous; in (0, 1]: label-synchronous,
                                 frame t is skipped when ll[t][blank_id] > log(blank_threshold);
                                 <= 0 or NaN: WFST_EINVAL */
    int32_t blank_id;         /* log-likelihood column of the blank unit, in [0, L) */
    uint32_t flags;           /* WFST_RECORD_TOKENS | WFST_LOGLIKES_HOST | WFST_PROFILE | WFST_PROFILE_STEPS |
                                 WFST_WORD_LATTICE | WFST_INCREMENTAL_LATTICE */
    int64_t capacity_hint;    /* 0: automatic; else tokens per frame to reserve */
    /* HMM topologies whose blank-like state is one unit per phone (Sec. 2):
       with num_blank_ids > 0, blank_ids[0..num_blank_ids) (host memory,
       columns in [0, L), order and repeats irrelevant) replace blank_id, and a
       frame is blank when any of them passes the threshold */
    const int32_t *blank_ids;
    int32_t num_blank_ids;    /* 0: the single unit blank_id; < 0: WFST_EINVAL */
    int32_t frame_stride;     /* decode only frames t with t % frame_stride == 0 (a lower frame
                                 rate; the blank test then applies to those); 0 counts as 1;
                                 < 0: WFST_EINVAL */
} wfst_decode_opts;

/* Fill opts with defaults: beam 16, max_active 0, no lattice, FSD, blank 0,
   no blank-unit set, frame stride 1. */
void wfst_default_opts(wfst_decode_opts *opts);

/*
 * wfst_decode -- decode one utterance (Alg. 1 with ViterbiBeamSearch per
 * decoded frame).
 *
 *   loglikes   [T x L] float32 row-major log-likelihoods (device memory of
 *              the graph's device, or host memory with WFST_LOGLIKES_HOST);
 *              values must not be NaN or +inf (-inf is allowed); acoustic
 *              scale and priors are the caller's business
 *   T >= 0, L >= max_ilabel of the graph, L >= 1
 *   hip_stream hipStream_t to run on (NULL = default stream); the call is
 *              blocking: it returns when the result is complete
 *   out        receives the result (also on WFST_ENOPATH, so the status can
 *              be read back); free with wfst_result_free
 *
 * Loglikes must stay valid until the call returns.  Errors: WFST_EINVAL,
 * WFST_ENOMEM, WFST_ECAPACITY, WFST_EDEVICE; WFST_ENOPATH when no path
 * survives.
 */
int wfst_decode(const wfst_graph *g, const float *loglikes, int32_t T, int32_t L,
                const wfst_decode_opts *opts, void *hip_stream, wfst_result **out);

/*
 * wfst_decode_batch -- decode n_utt independent utterances against one
 * graph on one device.  Each utterance runs in one workgroup for all of its
 * frames.  Batches of 32 or more utterances are split into up to four
 * groups of similar lengths; the groups' launches run on the library's own
 * streams beside hip_stream (forked from and joined back into it with
 * events), so the record and lattice passes of short utterances overlap the
 * search of long ones.  Results do not depend on the grouping.  Concurrent
 * batch calls on one device share the library's streams, so their group
 * launches queue behind one another.
 *
 *   loglikes   [n_utt] host array of pointers, each [T[u] x L] float32
 *   T          [n_utt] host array of frame counts
 *   out_array  [n_utt] host array receiving one result per utterance
 *
 * Returns WFST_OK when the batch ran (each result carries its own status,
 * e.g. WFST_ENOPATH for one utterance), or an error for the whole call.
 */
int wfst_decode_batch(const wfst_graph *g, int32_t n_utt, const float *const *loglikes,
                      const int32_t *T, int32_t L, const wfst_decode_opts *opts,
                      void *hip_stream, wfst_result **out_array);

/* Status of the utterance: WFST_OK, or WFST_ENOPATH when a token set of
   the search (Alg. 1) became empty.  r == NULL: WFST_EINVAL. */
int wfst_result_status(const wfst_result *r);

/*
 * Best path, the output of finalTransition and backtrace (Alg. 1): its cost
 * (final cost included), final state, whether a final state was reached (0
 * means the all-final fallback was used), and n arcs in path order with,
 * per arc, the original frame it consumed (-1 for epsilon arcs).  Any output
 * pointer may be NULL.  Pointers stay valid until wfst_result_free.
 * Errors: WFST_EINVAL (r == NULL), the utterance's status when it has no
 * path.
 */
int wfst_result_best(const wfst_result *r, float *cost, int32_t *final_state,
                     int32_t *reached_final, int32_t *n, const int32_t **arcs,
                     const int32_t **frames);

/*
 * Frame counts of label-synchronous decoding (Sec. 2, Eq. 3): T, the number
 * T' = T - |U| of decoded frames, and for each decoded frame j its original
 * frame index (the frames left after removing the blank set U, Alg. 1),
 * host memory owned by the result.  Any output pointer may be NULL.
 * Errors: WFST_EINVAL (r == NULL).
 */
int wfst_result_frames(const wfst_result *r, int32_t *num_frames, int32_t *num_decoded,
                       const int32_t **orig_frame);

/*
 * Lattice arc of the exact (state-level) lattice (Sec. 1, Sec. 3): `frame`
 * is the token set j (0..T') holding the arc's source; the destination's
 * token set follows from the arc's kind (an emitting arc goes from token set
 * j to j + 1 and consumed decoded frame j; an epsilon arc stays inside token
 * set j), so it is not stored; `arc` is the user arc index; `cost` is the
 * best prefix cost through the arc; `extra` is how much the best complete
 * path through the arc costs above the best path (the lattice beam keeps
 * arcs whose extra is at most lattice_beam).  16 bytes, 4-byte aligned.
 */
typedef struct wfst_lat_arc {
    int32_t frame;
    int32_t arc;
    float cost;
    float extra;
} wfst_lat_arc;

/*
 * Lattice-beam-pruned lattice (Sec. 1, Sec. 3), sorted by (frame, arc), in
 * host memory owned by the results: the first call on any result of a batch
 * copies the lattices of the whole batch in one transfer, which the results
 * share (valid while any of them lives).  n = 0 and arcs = NULL when the
 * lattice was disabled.  Errors: WFST_EINVAL (r == NULL), WFST_EDEVICE
 * (copy failed).
 */
int wfst_result_lattice(const wfst_result *r, int64_t *n, const wfst_lat_arc **arcs);

/* The same lattice in device memory of the graph's device, owned by the
   results of the batch (valid while any of them lives); arcs = NULL when
   the lattice was disabled.  Errors: WFST_EINVAL (r == NULL). */
int wfst_result_lattice_device(const wfst_result *r, int64_t *n, const wfst_lat_arc **arcs);

/*
 * Token set S_j (j = 0..T'), the surviving tokens of token passing after
 * decoded frame j (Sec. 3, Fig. 2; the beam search of Alg. 1), sorted by
 * state: n states, their float32 costs and back-pointer arcs (the user arc
 * of the recombination winner, -1 for the start token).  Host memory owned
 * by the result.  Needs WFST_RECORD_TOKENS.  Errors: WFST_EINVAL (r == NULL,
 * decoded without WFST_RECORD_TOKENS, j out of range).
 */
int wfst_result_tokens(const wfst_result *r, int32_t j, int32_t *n, const int32_t **state,
                       const float **cost, const int32_t **bp_arc);

typedef struct wfst_stats {
    int32_t frames;            /* T */
    int32_t frames_decoded;    /* T' = T - |U| */
    int64_t tokens;            /* sum over token sets of |S_j| */
    int64_t tokens_last;       /* |S_T'|, the set the final costs are added to */
    int64_t arcs_expanded;     /* emitting out-arcs of the expanded token sets */
    int64_t eps_arcs;          /* epsilon out-arcs of all surviving tokens */
    int64_t lattice_raw;       /* lattice arcs recorded before lattice-beam pruning */
    int64_t lattice_kept;      /* lattice arcs kept */
    double decode_ms;          /* wall time of the call that produced this result */
    /* with WFST_PROFILE (batch-wide, the same in every result of a batch):
       device time summed over launches, measured with HIP events */
    double search_ms;          /* token passing over all frames: expansion, epsilon
                                  closure, pruning (launches of different groups
                                  overlap, so the sum can exceed the wall time) */
    double record_ms;          /* back-pointers and raw lattice records of every frame */
    double final_ms;           /* final costs, backtrace, lattice pruning and output */
    int32_t search_launches;   /* launches of the search kernel */
    /* with WFST_PROFILE_STEPS: this utterance's share of the search, from the
       device clock of its workgroup, per step of a frame summed over the
       frames: [0] emitting expansion and the epsilon closure from the wave
       queues, [1] closure rounds over spilled epsilon items, [2] beam and
       max-active pruning, [3] compaction of the survivors (which also clears
       the token table); [4] the emitting expansion as the first wave sees it
       (part of [0]); [5] between frames (bookkeeping and the frame's first
       barrier); [6] frames abandoned for the device-memory table (their
       steps are not in [0]-[3]) */
    double search_phase_ms[7];
    /* with WFST_PROFILE_STEPS: this utterance's backtrace and lattice-beam pruning,
       from the device clock of the workgroups doing them (they run side by
       side after the search) */
    double backtrace_ms;
    double lattice_prune_ms;
    /* with WFST_PROFILE (batch-wide): from the start of the first search
       launch to the end of the last one (the groups' launches overlap) */
    double search_span_ms;
    int64_t word_sequences;    /* with WFST_WORD_LATTICE: word sequences of the lattice */
    int64_t lattice_incremental; /* lattice arcs left for the final lattice pruning by the
                                    incremental pass beside the search (lattice_raw without it) */
    int64_t workspace_bytes;   /* device workspace of the decode call (batch-wide) */
} wfst_stats;

/*
 * Word-level lattice (needs WFST_WORD_LATTICE): every word sequence of the
 * pruned lattice -- the non-zero output labels along a complete lattice path
 * from the start token to the last token set -- with the best cost of a
 * complete path that outputs it (final cost included, as for the best path).
 * This map is what determinising the exact lattice over its output labels
 * keeps for second-pass rescoring (Sec. 1).  The n sequences are sorted by
 * cost (ties by the sequence, lexicographically); sequence k is
 * words[offsets[k] .. offsets[k + 1]); the best one is the best path's.
 * Host memory owned by the result.  Errors: WFST_EINVAL (r == NULL, decoded
 * without WFST_WORD_LATTICE), the utterance's status when it has no path.
 */
int wfst_result_words(const wfst_result *r, int64_t *n, const int64_t **offsets, const int32_t **words,
                      const float **costs);

/* Counters and timings of the utterance's decode (the work measures of
   Eq. 3: decoded frames, tokens and arcs expanded).  Errors: WFST_EINVAL. */
int wfst_result_stats(const wfst_result *r, wfst_stats *stats);

/*
 * For callers that pay per call (language bindings): what
 * wfst_result_status, wfst_result_frames, wfst_result_best,
 * wfst_result_stats and, with want_lattice nonzero, wfst_result_lattice
 * return, for n results at once, one summary each.  The pointers are the
 * ones those calls give (host memory owned by the result, or the batch's
 * shared host copy of the lattices, made by this call when needed).  A
 * result without a path has path_len = 0, NULL path pointers and a NaN
 * cost; without want_lattice (or without a lattice) lattice_n = 0 and
 * lattice = NULL.  Errors: WFST_EINVAL (a NULL argument or result, n < 0),
 * WFST_EDEVICE (the lattice copy failed).
 */
typedef struct wfst_result_summary {
    int32_t status;
    int32_t num_frames;
    int32_t num_decoded;
    int32_t path_len;
    float cost;
    int32_t final_state;
    int32_t reached_final;
    int32_t reserved;
    const int32_t *orig_frame;     /* num_decoded entries */
    const int32_t *path_arcs;      /* path_len entries */
    const int32_t *path_frames;    /* path_len entries */
    int64_t lattice_n;
    const wfst_lat_arc *lattice;   /* lattice_n entries */
    wfst_stats stats;
} wfst_result_summary;

int wfst_result_summaries(const wfst_result *const *results, int32_t n, int32_t want_lattice,
                          wfst_result_summary *out);

/* Release a result (NULL is allowed). */
void wfst_result_free(wfst_result *r);

/*
 * wfst_decode_noalloc -- wfst_decode of one utterance for callers that cannot
 * allocate memory: code that must not call hipMalloc (serving loops with a
 * fixed memory budget, harnesses that forbid allocation, set-up code around
 * HIP graph capture).  The call allocates nothing, on the device or on the
 * host: its workspace is a fixed device array of the library of
 * WFST_NOALLOC_SCRATCH_BYTES, which each device the library runs this call
 * on holds from its first such call until the process ends, and its outputs
 * go to buffers the caller owns.  The workspace needs grow with T and with
 * the tokens a frame keeps: a T for which the workspace would hold fewer
 * than 64 tokens per frame on average is refused before anything runs, and a
 * decode that overflows it returns WFST_ECAPACITY (there is no retry with
 * larger buffers).
 *
 * Calls on one device share that device's workspace: calls that overlap in
 * time on one device (from several threads, or on several streams) race and
 * must not be made; calls on different devices are independent.
 *
 *   g, L, opts  as for wfst_decode; opts->flags must not contain
 *               WFST_RECORD_TOKENS, WFST_LOGLIKES_HOST, WFST_PROFILE,
 *               WFST_PROFILE_STEPS or WFST_WORD_LATTICE; opts->capacity_hint sets the tokens per
 *               frame (0: from max_active)
 *   loglikes    [T x L] float32 in device memory of the graph's device
 *   hip_stream  as for wfst_decode (the call is blocking)
 *   out         caller-owned descriptor: the device buffers below (on the
 *               graph's device) and the host fields the call fills in
 *
 * Errors: WFST_EINVAL (as wfst_decode, a forbidden flag, out == NULL, a NULL
 * output buffer with a non-zero capacity), WFST_ECAPACITY (the workspace
 * cannot hold T frames, the decode overflowed it, or an output buffer is too
 * small: out->path_len or out->lattice_n then gives the size needed),
 * WFST_ENOPATH (out->status too), WFST_EDEVICE.
 */
#define WFST_NOALLOC_SCRATCH_BYTES (512ll << 20)

typedef struct wfst_noalloc_out {
    /* caller-owned device buffers */
    int32_t *path_arcs;      /* [path_cap] best path arcs (user arc indices), first to last */
    int32_t *path_frames;    /* [path_cap] original frame of each path arc, -1 for epsilon arcs */
    int32_t path_cap;
    wfst_lat_arc *lattice;   /* [lattice_cap] pruned lattice sorted by (frame, arc); may be NULL
                                with lattice_cap 0 when opts->lattice_beam < 0 */
    int64_t lattice_cap;
    int32_t *kept;           /* [kept_cap] original frame of each decoded frame, or NULL */
    int32_t kept_cap;
    /* filled in by the call (host) */
    int32_t status;          /* WFST_OK or WFST_ENOPATH */
    float cost;              /* as wfst_result_best */
    int32_t final_state;
    int32_t reached_final;
    int32_t path_len;
    int32_t num_decoded;     /* T' */
    int64_t lattice_n;       /* kept lattice arcs */
    int64_t lattice_raw;     /* lattice arcs before lattice-beam pruning */
    int64_t tokens;          /* as wfst_stats */
    int64_t arcs_expanded;
    int64_t eps_arcs;
} wfst_noalloc_out;

int wfst_decode_noalloc(const wfst_graph *g, const float *loglikes, int32_t T, int32_t L,
                        const wfst_decode_opts *opts, void *hip_stream, wfst_noalloc_out *out);

/*
 * Test and debugging switches, process-wide (for the test suite, not for
 * production use).  They force the decoder's rarely taken paths on small
 * inputs and change the order of its parallel work; the results must not
 * depend on them, except that fail_lattice_alloc makes decodes fail.  A zero
 * field keeps the library's default; a positive fill or capacity is used only
 * when it is below the default.
 *
 *   lds_fill           states per frame the search's LDS token table takes
 *                      before the frame is redone with the table in device
 *                      memory
 *   queue_cap          epsilon items per wave queue in LDS before items spill
 *                      to device memory
 *   record_fill        survivors per token set that the record pass handles
 *                      with its LDS table (larger sets go to the large-set
 *                      pass)
 *   record_big_fill    the same for the large-set pass (larger sets use a
 *                      device-memory table)
 *   lattice_lds        survivors per token set that lattice pruning keeps in
 *                      LDS; -1 keeps none (every set in device memory)
 *   permute            nonzero: hash the token tables with another multiplier
 *                      and expand the arc chunks of a token set in reverse
 *                      order, so that slots, claim order, survivor order and
 *                      the order of every atomic differ
 *   fail_lattice_alloc nonzero: the allocation of the lattice output fails,
 *                      as when device memory is exhausted: the decode returns
 *                      WFST_ENOMEM before launching anything that writes it
 *   lattice_chunk      token sets per chunk of the incremental lattice pass
 *                      (WFST_INCREMENTAL_LATTICE); -1 turns the pass off
 *   lattice_ring       raw records the incremental pass's rings hold (a
 *                      small ring makes chunks end early and wrap around)
 *   record_groups      record workgroups appended to the search launch of
 *                      the batch's last length group, which derive its
 *                      back-pointers and raw lattice records while it
 *                      searches (by default only when the batch has more
 *                      than one length group; a positive count applies to
 *                      a single group too); -1 leaves that group to the
 *                      record kernel after its search
 *   record_publish     token sets between the search's progress reports to
 *                      those workgroups
 *   lattice_pipe       lattice pruning's streamed pass (for utterances whose
 *                      sets are too large for the one-wave pass): -1 never
 *                      (the block pass instead), 0 where the utterance's
 *                      sets hold few records on average, 1 wherever it fits
 *   lattice_spin       polls of one hand-over flag before the one-wave or
 *                      streamed lattice pass gives up (0: the library's own,
 *                      seconds); a tiny count makes the pass fail as a stuck
 *                      hand-over would: WFST_EDEVICE, every kernel ending
 *
 * opts == NULL restores every default.  Takes effect for decodes started
 * after the call returns.  Errors: WFST_EINVAL for a negative field other
 * than lattice_lds = -1, lattice_chunk = -1, record_groups = -1 and
 * lattice_pipe = -1.
 */
typedef struct wfst_debug_opts {
    int32_t lds_fill;
    int32_t queue_cap;
    int32_t record_fill;
    int32_t record_big_fill;
    int32_t lattice_lds;
    int32_t permute;
    int32_t fail_lattice_alloc;
    int32_t lattice_chunk;
    int32_t lattice_ring;
    int32_t record_groups;
    int32_t record_publish;
    int32_t lattice_pipe;
    int32_t lattice_spin;
} wfst_debug_opts;

int wfst_set_debug_opts(const wfst_debug_opts *opts);

/* One environment switch, read once per process: WFSTDEC_DEBUG_TIMING (any
 * value) prints a wall-clock breakdown of each decode call on stderr (setup,
 * search, results; the workspace split and the frames redone on the
 * device-memory token table).  It changes no result. */

/* Message for the last error raised on the calling thread ("" if none). */
const char *wfst_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
