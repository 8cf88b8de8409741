/*
 * Serial CPU oracle for WFST Viterbi beam decoding (frame-synchronous and
 * label-synchronous) with state-level lattice generation and lattice-beam
 * pruning.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the GPU decoder.
 * Only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark may load it; the decoder never calls it, and it shares no code,
 * header, table or helper with the GPU path.
 *
 * Written from: Z. Chen, "Linguistic Search Optimization for Deep Learning
 * Based LVCSR" (Interspeech 2018): token passing with per-state min
 * recombination (Sec. 3), Viterbi beam search (Sec. 1), the blank-frame set
 * U and label-synchronous decoding (Sec. 2, Eq. 2, Alg. 1), exact lattices
 * (Sec. 1, Sec. 3).
 */
#ifndef ORACLE_WFST_H
#define ORACLE_WFST_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ORACLE_OK = 0,
    ORACLE_EINVAL = -1,
    ORACLE_ENOMEM = -2,
    ORACLE_ENOPATH = -3,
    ORACLE_EINTERNAL = -9
};

typedef struct oracle_result {
    int32_t status;
    /* best path (Alg. 1: finalTransition then backtrace) */
    float cost;
    int32_t final_state;
    int32_t reached_final;
    int32_t path_len;
    int32_t *path_arcs;     /* user arc indices, first to last */
    int32_t *path_frames;   /* original frame consumed, -1 for epsilon arcs */
    /* decoded frames (label-synchronous compaction) */
    int32_t num_frames;     /* T */
    int32_t num_decoded;    /* T' = T - |U| */
    int32_t *kept;          /* [T'] original frame index of decoded frame j */
    /* surviving tokens of token sets j = 0..T', each sorted by state */
    int64_t *tok_off;       /* [T'+2] */
    int32_t *tok_state;
    uint32_t *tok_cost_bits;/* float32 bit pattern of the token cost */
    int32_t *tok_arc;       /* back-pointer user arc, -1 for the start token */
    uint32_t *cut_key;      /* [T'+1] pruning cutoff of each token set (ordered key) */
    /* lattice after lattice-beam pruning, sorted by (frame, arc) */
    int64_t lat_raw;
    int64_t lat_n;
    int32_t *lat_frame;     /* token set index of the arc's source */
    int32_t *lat_arc;       /* user arc index */
    float *lat_cost;        /* prefix cost through the arc */
    float *lat_extra;       /* extra cost over the best complete path */
    /* counters */
    int64_t arcs_expanded;  /* emitting out-arcs of expanded tokens */
    int64_t eps_arcs;       /* epsilon out-arcs of surviving tokens */
    int64_t tokens;         /* sum of |S_j| */
    double seconds;         /* wall time of the decode proper */
} oracle_result;

/* Validate a graph the way the decoder's loader must (returns ORACLE_OK or
 * ORACLE_EINVAL).  Input arrays are host pointers. */
int oracle_validate_graph(int32_t num_states, int64_t num_arcs, const int32_t *src,
                          const int32_t *dst, const int32_t *ilabel, const int32_t *olabel,
                          const float *weight, int32_t start, const float *final_weight);

/* Decode one utterance.  All pointers are host pointers.  loglikes is
 * [T x L] row-major float32.  final_weight may be NULL (every state final
 * with cost 0).  max_active <= 0 means unlimited; lattice_beam < 0 disables
 * the lattice; blank_threshold > 1 means frame-synchronous decoding.
 * Always returns a result (free with oracle_free); result->status carries
 * the error code. */
oracle_result *oracle_decode(int32_t num_states, int64_t num_arcs, const int32_t *src,
                             const int32_t *dst, const int32_t *ilabel, const int32_t *olabel,
                             const float *weight, int32_t start, const float *final_weight,
                             const float *loglikes, int32_t T, int32_t L, float beam,
                             int32_t max_active, float lattice_beam, float blank_threshold,
                             int32_t blank_id);

/* The same with the label-synchronous test over a set of blank-like units
 * (HMM topologies whose blank-like state is one unit per phone, Sec. 2):
 * frame t is blank when some unit of blank_ids[0..num_blank_ids) has a
 * log-likelihood above log(blank_threshold).  Only frames t with
 * t % frame_stride == 0 are candidates for decoding at all (a lower frame
 * rate; frame_stride >= 1).  oracle_decode is this call with the single unit
 * blank_id and stride 1. */
oracle_result *oracle_decode_ext(int32_t num_states, int64_t num_arcs, const int32_t *src,
                                 const int32_t *dst, const int32_t *ilabel, const int32_t *olabel,
                                 const float *weight, int32_t start, const float *final_weight,
                                 const float *loglikes, int32_t T, int32_t L, float beam,
                                 int32_t max_active, float lattice_beam, float blank_threshold,
                                 const int32_t *blank_ids, int32_t num_blank_ids, int32_t frame_stride);

void oracle_free(oracle_result *r);

#ifdef __cplusplus
}
#endif
#endif
