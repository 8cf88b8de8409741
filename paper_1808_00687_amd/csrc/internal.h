// Internal structures of the wfstdec HIP library (gfx950).
//
// Device layout of a graph (built once by wfst_load):
//   eoff[N+1]  emitting-arc row offsets; earc[] 16-byte records
//              {dst | has_eps << 31, column = ilabel - 1, weight bits, user arc}
//   xoff[N+1]  epsilon-arc row offsets; xarc[] 16-byte records
//              {dst | has_eps << 31, weight bits, user arc, 0}
//   arc_src[E] user arc -> src state | is_epsilon << 31 (cold, back-pointers)
//   final_w[N] final costs or null
//   srec[2N]   32-byte state records: the state's emitting and epsilon row
//              offsets, then a copy of its first epsilon record (zeros if
//              none), so that one load gives a state's rows and, for the
//              common single-epsilon state, its epsilon arc; the copy's last
//              word locates the state's epsilon-closure list
//   ctab[]     epsilon-closure lists: every epsilon path from a state (up to
//              size and length limits) as {last destination, last arc,
//              length, the weights along the path} in three 16-byte words,
//              so the closure from a lowered token needs no chain of
//              dependent loads
// Each state's arcs keep their user order inside the emitting and the
// epsilon partition.  has_eps marks a destination with epsilon out-arcs, so a
// kernel that lowers its token knows without another load whether the
// epsilon closure has to continue from it.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>
#include <vector>

#include "wfstdec.h"

namespace wfd {

constexpr uint64_t kEmptyTok = ~0ull;
// Utterance status of a survivor that the record pass found no back-pointer
// for (never expected: reported as a device error)
constexpr int kStatusNoBackPointer = -9;
// Utterance status: the incremental lattice pass or the record workgroups
// stopped waiting for the search (never expected: reported as a device error)
constexpr int kStatusStreamTimeout = -11;
// Utterance status: the one-wave lattice pass and its loading waves stopped
// waiting for each other (never expected: reported as a device error)
constexpr int kStatusLatticeWait = -12;
// utterances a search launch with record workgroups may hold (their LDS
// keeps a progress count per utterance)
constexpr int kRecMaxUtts = 256;
constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;
constexpr uint32_t kDstMask = 0x7FFFFFFFu;
constexpr int kHistBits = 12;               // radix-select digit width
constexpr int kHistBins = 1 << kHistBits;   // bins per utterance histogram
constexpr int kWave = 64;                   // gfx950 wavefront
// Multipliers of the state hash of the token tables (odd, so the map is a
// bijection); the second one is the debugging permutation.
constexpr uint32_t kHashMul = 0x9E3779B1u;
constexpr uint32_t kHashMulAlt = 0x85EBCA77u;

// The graph on the device.  States are numbered by the position of their
// first record in `node`, an array of 16-byte units where each state's two
// records are followed by its emitting arcs:
//   node[s]     = {first emitting arc, end of its emitting arcs (both unit
//                  indices into node), first and end epsilon record in xarc}
//   node[s + 1] = the state's first epsilon record (destination, weight,
//                  user arc) with the state's closure word as its 4th word
//                  ((first entry + 1) << kClosureSizeBits | size - 1, 0 if
//                  it has no list)
//   node[a]     = an emitting arc: {dst | has-epsilon bit << 31, ilabel - 1,
//                  weight bits, closure word of dst}
// Ids keep the order of the user's state ids; Graph::hdr_pos maps back.
struct DevGraph {
    int32_t n;
    int32_t start;      // device id of the start state
    int64_t e;
    int64_t n_emit, n_eps;
    const int4 *node;
    const int4 *earc;   // = node (arc records by unit index)
    const int4 *srec;   // = node (state records by device id)
    const int32_t *eua; // user arc of each emitting arc record, by unit index
    const int4 *xarc;   // epsilon records by source: {dst | has-epsilon bit, weight, user arc, closure word of dst}
    const int32_t *arc_src;
    const float *final_w;   // by device id (0 elsewhere), or NULL
    const int4 *ctab;   // closure entries, 3 x int4 each: {dst, user arc, path length, w0}, {w1..w4}, {w5..w8}
    const int2 *uarc;   // per user arc: {olabel, index of its record in node or xarc}
};

// Epsilon-closure lists (built by wfst_load): at most kClosureMax paths of at
// most kClosureDepth arcs per state, kClosureEntries entries in all.  The
// state record's closure word holds a list's size - 1 in its low
// kClosureSizeBits bits and its first entry + 1 above them.
constexpr int kClosureSizeBits = 8;
constexpr int kClosureMax = 1 << kClosureSizeBits;
constexpr int kClosureDepth = 9;
constexpr int kClosureStride = 3;   // int4 words per entry
constexpr int64_t kClosureEntries = (int64_t{1} << (32 - kClosureSizeBits)) - 2;

// Host-side graph object behind the opaque wfst_graph handle.
struct Graph {
    DevGraph d;
    int device;
    int32_t max_ilabel;
    int32_t eps_depth;
    int64_t device_bytes;
    int64_t n_closure;   // states with an epsilon-closure list
    std::vector<int32_t> hdr_pos;   // device id of each user state (increasing)
    void *mem;   // single device allocation holding every array
    // lattice-record slots per token that the last decodes on this graph
    // needed (emitting, epsilon), a starting point for the next ones
    mutable std::atomic<int64_t> rec_em{0}, rec_xm{0};
};

// The user's state id of a device state id (-1 stays -1).
inline int32_t user_state(const Graph &g, int32_t dev)
{
    if (dev < 0) return dev;
    const auto it = std::upper_bound(g.hdr_pos.begin(), g.hdr_pos.end(), dev);
    return static_cast<int32_t>(it - g.hdr_pos.begin()) - 1;
}

// Per-utterance decode state in device memory.
struct UttState {
    const float *ll;      // [T x L] log-likelihoods (device)
    int32_t T;
    int32_t Tp;           // decoded frames (set by the classify kernel)
    int32_t status;       // WFST_OK, WFST_ENOPATH or WFST_ECAPACITY
    int32_t gframes;      // frames whose token table overflowed LDS (redone in device memory)
    // written by the search kernel when it ends
    int32_t n_last;       // |S_T'|
    int32_t big_sets;     // some token set is too large for the record kernel's LDS table
    int64_t n_tok;        // survivors of all token sets
    int64_t le_cnt;       // emitting lattice records
    int64_t lx_cnt;       // epsilon lattice records
    int64_t arcs_expanded;
    int64_t eps_arcs;
    // final
    int32_t final_sv;
    int32_t final_state;
    int32_t reached_final;
    float final_cost;
    int32_t path_len;
    int32_t pad1;
    int64_t lat_kept;
    int64_t lat_inc;      // lattice records the incremental pass kept for the final pass
    uint64_t phase_ticks[7];   // device clock ticks per search step (profiling only)
    uint64_t finish_ticks[2];  // device clock ticks of the backtrace and the lattice pruning
};

// Per-utterance regions inside the shared workspace buffers (element offsets).
struct UttLayout {
    int64_t sv0, svcap;       // survivors
    int64_t le0, lecap;       // emitting lattice records
    int64_t lx0, lxcap;       // epsilon lattice records
    int64_t fo0;              // per-frame offset arrays, T + 2 entries each
    int64_t kept0;            // kept-frame list, T entries
    int64_t path0, pathcap;   // best path (arcs and frames)
    int64_t lo0;              // lattice output records
};

// Everything a kernel needs, passed by value.
struct Params {
    DevGraph g;
    int32_t U;
    int32_t L;
    float beam;
    int32_t max_active;
    float lattice_beam;
    int32_t lattice;
    const int32_t *blank_ids;   // the blank-like units (device memory)
    int32_t n_blank;
    int32_t frame_stride;       // >= 1
    float blank_thr;
    int32_t lds_fill;         // states per frame the LDS token table takes (<= its fill limit)
    int32_t gen_lds;          // epsilon pool entries in LDS (<= its capacity)
    int32_t profile;          // count device clock ticks per search step
    int32_t rec_fill;         // survivors per set the record kernel's LDS table takes (<= its fill limit)
    int32_t rec_big_fill;     // the same for the large-set pass's LDS table
    int32_t lat_lds;          // survivors per set the lattice backward pass keeps in LDS (<= its capacity)
    uint32_t hash_mul;        // state hash multiplier of the token tables
    int32_t reverse;          // expand a set's arc chunks last to first (a debugging permutation)
    // Incremental lattice pass beside the search (stream_k > 0): the search
    // publishes in prog[u] how many token sets are complete, every stream_k
    // sets and at the end (-1 when it failed); the lattice pass records the
    // finished sets into a ring of raw records, prunes them against the
    // frontier and keeps the survivors in the lattice regions.
    int32_t stream_k;
    int32_t *prog;            // per utterance
    int4 *rng_e;              // U x rce raw emitting records
    float *rng_ee;            // their extra costs
    int4 *rng_x;              // U x rcx raw epsilon records
    float *rng_xe;
    int64_t rce, rcx;         // ring capacities (records per utterance)
    uint32_t *rkeys;          // U x capG: the lattice pass's own device-memory table (large sets)
    int32_t *rvals;
    UttState *st;
    const UttLayout *lay;
    // survivors (per utterance regions); the search writes state, cost key,
    // first emitting record and emitting prefix, the record pass the
    // back-pointer (source survivor and user arc)
    int32_t *sv_state;
    uint32_t *sv_key;         // ordered key of the token cost
    int32_t *sv_prev;         // survivor the back-pointer arc leaves from (-1 for the start token)
    int32_t *sv_arc;          // back-pointer user arc (-1 for the start token)
    int32_t *sv_ebeg;         // first emitting arc record of the survivor's state
    int32_t *sv_epre;         // exclusive prefix of emitting out-degree within the token set
    unsigned long long *sv_win;   // record pass scratch for sets beyond its LDS table:
                                  // (user arc + 1) << 32 | source survivor of the winning arc
    uint32_t *e_key;          // lattice backward extra cost per survivor (ordered key)
    // lattice raw records {src survivor, dst survivor, user arc, prefix cost bits}
    int4 *lat_e;
    int4 *lat_x;
    float *ex_e;
    float *ex_x;
    int4 *lat_out;            // kept lattice {frame, arc, cost bits, extra bits}
    // per-frame arrays (fo0 region): survivor, lattice-record and output offsets
    int64_t *sv_off;
    int64_t *le_off;          // start of each set's emitting lattice records (what the final pass reads)
    int64_t *lx_off;          // start of each set's epsilon lattice records
    int64_t *rle_off;         // the search's reservation: one emitting-record slot per emitting out-arc
    int64_t *rlx_off;         // of each set and one epsilon slot per epsilon out-arc, prefix over the
                              // sets (the same arrays as le_off / lx_off unless the incremental
                              // lattice pass compacts the records elsewhere)
    int64_t *lo_off;
    int64_t *le_cnt;          // records in each set's regions (the record kernel writes)
    int64_t *lx_cnt;
    uint32_t *cut_arr;        // pruning cutoff key of each token set
    int32_t *kept;
    int32_t *path_arc;
    int32_t *path_frame;
    int2 *path_packed;        // every utterance's path {arc, frame}, one after another
    // search scratch per utterance: token table in device memory (frames that
    // overflow LDS), epsilon item spill lists, emitting candidate lists
    uint32_t *gkeys;          // U x capG
    uint32_t *gvals;
    int32_t *gslots;
    int64_t capG;             // power of two
    uint2 *gspill;            // U x 2 x capO {table slot, cost bits}
    int64_t capO;
    // The search publishes prog[u] every pub_k token sets (0: never): for
    // the incremental pass, or for rec_wg record workgroups appended to the
    // search launch, which take (set, utterance) items from *rec_next (zeroed
    // before the launch) up to set rec_tmax.  (Last: the offsets of the
    // fields above, which the search reads, stay as they were.)
    int32_t pub_k;
    int32_t rec_wg;           // at most kRecMaxUtts utterances in such a launch
    int32_t rec_tmax;
    int32_t *rec_next;
    int32_t lat_pipe;         // the lattice backward pass's streamed form: -1 never, 0 where sets are
                              // small on average, 1 wherever it fits
    int32_t lat_spin;         // > 0: polls of one flag before a lattice pass's wait gives up (else its own)
};

// Workspace of the word-level lattice pass (word_kernel.hip), uniform
// capacities per utterance: capH (node, word prefix) entries, capW word-trie
// nodes (both powers of two).
struct WordWs {
    unsigned long long *hkey;   // U x capH: node << 32 | trie id (~0 = free)
    uint32_t *hval;             // U x capH: cost key of the entry
    int32_t *hnext;             // U x capH: next entry of the same node
    int32_t *ents;              // U x capH: entries in claim order
    int32_t *heads;             // per survivor (utterance survivor regions): first entry of the node
    unsigned long long *tkey;   // U x capW: parent << 32 | word (~0 = free)
    int32_t *tdep;              // U x capW: sequence length of the node
    uint32_t *tbest;            // U x capW: best total cost key of the sequence
    int2 *out_id;               // U x (capW + 1): listed sequences {trie id (-1 = empty), cost key}
    int32_t *out_n;             // U x 4: sequences, words, status
    uint32_t *root_best;        // U: best total of the empty sequence
    int32_t *set_start;         // per token set (utterance frame regions): first entry of the set
    int64_t capH, capW;
};

// The slices of utterance u.
__host__ __device__ inline WordWs word_ws_of(const WordWs &w, int u, const UttLayout &ly)
{
    WordWs r = w;
    r.hkey += u * w.capH;
    r.hval += u * w.capH;
    r.hnext += u * w.capH;
    r.ents += u * w.capH;
    r.tkey += u * w.capW;
    r.tdep += u * w.capW;
    r.tbest += u * w.capW;
    r.out_id += u * (w.capW + 1);
    r.out_n += 4 * u;
    r.root_best += u;
    r.heads += ly.sv0;
    r.set_start += ly.fo0;
    return r;
}

// ---- launchers (search_kernel.hip, search_record_kernel.hip, record_kernel.hip, final_kernels.hip) ----
hipError_t launch_classify(const Params &p, hipStream_t s);
hipError_t launch_search(const Params &p, hipStream_t s);
// the search launch with p.rec_wg record workgroups (launch_search calls it)
hipError_t launch_search_record(const Params &p, hipStream_t s);
hipError_t launch_final(const Params &p, hipStream_t s);
hipError_t launch_record(const Params &p, int max_frames, hipStream_t s);
// only the sets larger than the record kernel's LDS table (after a search
// launch with record workgroups)
hipError_t launch_record_large(const Params &p, hipStream_t s);
hipError_t launch_lattice_stream(const Params &p, hipStream_t s);
hipError_t launch_finish(const Params &p, hipStream_t s);
hipError_t launch_pack_paths(const Params &p, hipStream_t s);
hipError_t launch_lattice_emit(const Params &p, int max_frames, hipStream_t s);
hipError_t launch_zero(void *ptr, size_t bytes, hipStream_t s);   // ptr 16-byte aligned, bytes % 4 == 0
hipError_t launch_word(const Params &p, const WordWs &ws, hipStream_t s);
hipError_t launch_word_flatten(const Params &p, const WordWs &ws, int64_t *off, int32_t *words,
                               const int64_t *base_seq, const int64_t *base_word, hipStream_t s);

// ---- host helpers (graph.cpp) ----
void set_error(const char *fmt, ...);
void clear_error();

}  // namespace wfd

// Opaque handle types of the C ABI.
struct wfst_graph {
    wfd::Graph g;
};
