// The search kernel: one 1024-thread workgroup per utterance loops over every
// decoded frame of its utterance (token passing, Sec. 3; the per-frame
// Viterbi beam search of Alg. 1).
//
// Frame k (token set S_k) in one workgroup:
//   1. expansion of the emitting arcs of S_{k-1}: each wave takes two chunks
//      of 64 consecutive arcs of the set at a time, finds their tokens by a
//      64-ary search over the set's emitting-arc prefix (kept in LDS for sets
//      of up to kSetCache tokens) and issues all their loads together; the
//      frame's log-likelihood row sits in LDS (loaded during the previous
//      frame's compaction).  The frame's tokens live in a hash table in LDS
//      (state -> cost key); recombination is an LDS 32-bit atomicMin on the
//      ordered cost key, the first touch of a state appends its slot to a
//      slot list;
//   2. epsilon closure: every lowered token whose state has epsilon
//      out-arcs goes to its wave's LDS queue, and each wave relaxes its own
//      queue until it is empty, with no barrier between the rounds (a
//      state's first epsilon arc comes with its 32-byte state record).
//      Items beyond a queue's capacity go to a device-memory list that the
//      whole workgroup relaxes after a barrier;
//   3. pruning: beam limit from the frame's best cost key and, when more
//      tokens lie within it than max_active, the exact max_active-th
//      smallest key by radix select over an LDS histogram;
//   4. compaction of the survivors into S_k (device memory, and LDS for the
//      next expansion), with the prefix of their emitting out-degrees, and
//      the set's lattice record regions; the table's slots are cleared as
//      they are read.
// Back-pointers and lattice records need nothing the next frame needs: the
// record kernel derives them afterwards from the stored token sets, every
// frame of every utterance in parallel (a token's back-pointer is the lowest
// arc whose candidate cost equals the token's cost, which is what a minimum
// over (cost, arc) pairs would have kept), so the search keeps costs only
// and writes nothing per candidate.
// A frame that reaches more states than the LDS table holds is redone with
// the same code on a table in device memory.  Every table is private to its
// workgroup and there are no per-frame launches; the only device-scope
// synchronisation is the search's progress count, published every pub_k
// token sets when record workgroups (below) or the incremental lattice pass
// follow it.
//
// This header is compiled twice, once per translation unit:
// search_kernel.hip instantiates the search alone, search_record_kernel.hip
// the search with record workgroups appended to its launch.
#pragma once

#include <type_traits>

#include "device_util.h"
#include "record_set.h"

namespace wfd {

namespace {

constexpr int kT = 1024;                  // threads per workgroup
constexpr int kW = kT / kWave;            // waves per workgroup
constexpr int kSlotBits = 13;
constexpr int kSlots = 1 << kSlotBits;    // LDS hash slots
constexpr int kFill = 6144;               // LDS states per frame before falling back to device memory
constexpr int kQueue = 128;               // LDS epsilon items per wave queue
constexpr int kSetCache = 2944;           // tokens of the previous set kept in LDS for the expansion (a multiple of 64)
constexpr int kCs = 128;                  // 64-arc chunks of the previous set with their first token in LDS
constexpr int kChunks = 2;                // 64-arc chunks a wave has in flight in the expansion
constexpr int kRelChunks = 2;             // 64-path chunks of closure lists a wave has in flight
constexpr int kMaxProbe = 64;             // linear-probe bound (the fill limit keeps probes short)
constexpr int kOverflow = 1;              // frame result: the table filled up
constexpr uint32_t kNoKey = 0xFFFFFFFEu;   // a key no state has (state ids are below 2^31)
constexpr int kRowMax = 6144;             // log-likelihood columns a frame's LDS row holds

static_assert(kHistBins * 4 <= kW * kQueue * 8, "the select histogram aliases the epsilon queues");
static_assert(kRowMax % kT == 0, "every thread loads the same number of a row's columns");
static_assert(kSetCache % 64 == 0, "the token-set arrays keep the offsets of the LDS arrays after them modulo 256 bytes");


// Table loads: plain in LDS; in device memory they bypass the CU's L1, since
// the table's atomics are performed in L2.
template <bool G, typename T>
__device__ __forceinline__ T tld(const T *ptr)
{
    if constexpr (G)
        return __hip_atomic_load(const_cast<T *>(ptr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
        return *ptr;
}

// With the table in device memory its own stores need the full barrier.
template <bool G>
__device__ __forceinline__ void table_barrier()
{
    if constexpr (G) __syncthreads();
    else lds_barrier();
}

// Token table of one frame: keys = state (kEmptyKey if free), vals = the
// ordered cost key of the state's token (kEmptyKey if none).  `slots` lists
// the claimed slots in claim order.
template <bool G>
struct Tab {
    using Slot = typename std::conditional<G, int32_t, uint16_t>::type;
    uint32_t *keys;
    uint32_t *vals;
    Slot *slots;
    uint32_t mask;
    int fill;
    int shift;   // 32 - log2(slots)
    uint32_t mul;   // hash multiplier
};

struct Sh {
    int nslots;          // claimed slots
    int overflow;        // more states than the table's fill limit
    int status;          // sticky error of the utterance
    uint32_t best;       // smallest cost key among the frame's tokens
    int spill_n[2];      // epsilon items in the device-memory lists
    // compaction results of frames of even and odd index: every wave reads
    // its frame's after the frame's last barrier, while thread 0 may already
    // clear the next frame's
    unsigned long long alloc[2];   // emitting degrees << 32 | survivors placed
    int xsum[2];         // epsilon degrees of the survivors
    int bin, before, cnt;
    int scan[52];
};

// Running values of the utterance (in LDS): frame k reads the copy of
// index k & 1 and thread 0 writes the other, so that no wave still reading
// the frame's values after its last barrier sees them change.
struct Run {
    int64_t set0;        // relative survivor index where the next set starts
    int64_t prev0;       // relative start of S_{k-1}
    int n_prev;          // |S_{k-1}|
    int a_prev;          // emitting out-arcs of S_{k-1}
    int64_t le, lx;      // emitting and epsilon regions reserved so far
    int64_t arcs;
    int64_t eps;         // epsilon out-arcs of the survivors
};

// Profiling counters, kept by thread 0 in LDS (in registers they would
// take space in every thread).
struct Prof {
    unsigned long long ph[7];    // device clock ticks per step
    unsigned long long cur[4];   // the current frame's steps
    unsigned long long t_last;
    unsigned long long t_sub;
};

// Profiling: thread 0 adds the device clock since the previous mark to step
// i of the current frame (0-3), or to the time between frames (5).  A frame
// that is completed adds its steps to the totals; one abandoned for the
// device-memory table adds them to slot 6.
__device__ __forceinline__ void phase_mark(const Params &p, Prof &pf, int i)
{
    if (p.profile && threadIdx.x == 0) {
        const unsigned long long t = wall_clock64();
        if (i == 5) pf.ph[5] += t - pf.t_last;
        else pf.cur[i] += t - pf.t_last;
        pf.t_last = t;
    }
}

__device__ __forceinline__ void phase_fold(const Params &p, Prof &pf, bool done)
{
    if (p.profile && threadIdx.x == 0) {
        for (int i = 0; i < 4; i++) {
            pf.ph[done ? i : 6] += pf.cur[i];
            pf.cur[i] = 0;
        }
    }
}

// Profiling of a part of a step as thread 0 sees it: open, then close into
// slot i.
__device__ __forceinline__ void sub_open(const Params &p, Prof &pf)
{
    if (p.profile && threadIdx.x == 0) pf.t_sub = wall_clock64();
}

__device__ __forceinline__ void sub_close(const Params &p, Prof &pf, int i)
{
    if (p.profile && threadIdx.x == 0) pf.ph[i] += wall_clock64() - pf.t_sub;
}

// A wave's epsilon work list: an LDS queue of (table slot, cost bits) items
// with the closure word of each item's state (0 if not known), and the
// device-memory list that takes what does not fit (without closure words).
struct WaveQ {
    uint2 *q;        // this wave's LDS queue
    uint32_t *ql;    // the items' closure words
    int n;           // items in it (the same in every lane)
    int qcap;        // its capacity (<= kQueue)
    uint2 *spill;    // device-memory list of the current round
    int *spill_n;    // its LDS counter
    int scap;        // its capacity
};

// Offer R candidate costs per lane (act[r]) to the table; lowered tokens
// of states with epsilon out-arcs become items of the wave's queue, with the
// closure word cl[r] of the state when the caller knows it (else 0).  The R
// offers go through each step together, so that their LDS atomics are in
// flight at the same time.  With BEST the frame's best key takes the
// smallest offered key (a caller that has already done so passes false):
// every offered key is at least the final token of its state, so the minimum
// is the frame's best token either way.  Called by the whole wave.
template <bool G, int R, bool BEST>
__device__ __forceinline__ void offer(const Tab<G> &t, Sh &sh, WaveQ &wq, const bool *act, const uint32_t *d,
                                      const bool *d_eps, const uint32_t *cl, const float *cand, const uint32_t *key)
{
    int slot[R];
    // slot of each state: a compare-and-swap on the key claims a free slot
    // or finds the state's own, probing linearly on a collision
    uint32_t h[R], k[R];
    bool claimed[R];
#pragma unroll
    for (int r = 0; r < R; r++) h[r] = hash_state(d[r], t.mul) >> t.shift;
    if constexpr (!G) {
        // In LDS every lane issues its compare-and-swap, so that the R
        // atomics of the wave are in flight together instead of one branch
        // (and one wait) each: an inactive lane compares and swaps a key no
        // state has, at a slot of its own, which changes nothing.
#pragma unroll
        for (int r = 0; r < R; r++) {
            const uint32_t at = act[r] ? h[r] : (h[r] + lane_id()) & t.mask;
            k[r] = atomicCAS(t.keys + at, act[r] ? kEmptyKey : kNoKey, act[r] ? d[r] : kNoKey);
        }
    } else {
#pragma unroll
        for (int r = 0; r < R; r++) k[r] = act[r] ? atomicCAS(t.keys + h[r], kEmptyKey, d[r]) : 0u;
    }
    bool over = false;
#pragma unroll
    for (int r = 0; r < R; r++) {
        slot[r] = -1;
        claimed[r] = false;
        if (!act[r]) continue;
        for (int probe = 1; k[r] != kEmptyKey && k[r] != d[r]; probe++) {
            if (probe == kMaxProbe) break;
            h[r] = (h[r] + 1) & t.mask;
            k[r] = atomicCAS(t.keys + h[r], kEmptyKey, d[r]);
        }
        if (k[r] == kEmptyKey || k[r] == d[r]) {
            slot[r] = static_cast<int>(h[r]);
            claimed[r] = k[r] == kEmptyKey;
        } else {
            over = true;
        }
    }
    // recombination: the unsigned minimum of the cost keys; issued before
    // the slot-list add below, so that their LDS round trips overlap (in LDS
    // without a branch: a lane without a slot takes the minimum of a slot of
    // its own and the empty key, which changes nothing)
    uint32_t old[R];
#pragma unroll
    for (int r = 0; r < R; r++) {
        if constexpr (!G) {
            const uint32_t at = slot[r] >= 0 ? static_cast<uint32_t>(slot[r]) : (h[r] + lane_id()) & t.mask;
            old[r] = atomicMin(t.vals + at, slot[r] >= 0 ? key[r] : kEmptyKey);
        } else {
            old[r] = slot[r] >= 0 ? atomicMin(t.vals + slot[r], key[r]) : 0u;
        }
    }
    // newly claimed slots join the slot list, one LDS add per wave
    uint64_t mc[R];
    int pc[R], nc = 0;
#pragma unroll
    for (int r = 0; r < R; r++) {
        mc[r] = __ballot(claimed[r]);
        pc[r] = nc;
        nc += __popcll(mc[r]);
    }
    if (nc) {
        int b = 0;
        if (lane_id() == 0) b = atomicAdd(&sh.nslots, nc);
        b = __builtin_amdgcn_readlane(b, 0);
#pragma unroll
        for (int r = 0; r < R; r++) {
            if (claimed[r]) {
                const int idx = b + pc[r] + rank_in(mc[r]);
                if (idx < t.fill) t.slots[idx] = static_cast<typename Tab<G>::Slot>(slot[r]);
                else over = true;
            }
        }
    }
    if (over) sh.overflow = 1;
    if (BEST) {
        uint32_t mk = kEmptyKey;
#pragma unroll
        for (int r = 0; r < R; r++)
            if (act[r] && key[r] < mk) mk = key[r];
        mk = wave_min_u32(mk);
        if (lane_id() == 0 && mk != kEmptyKey) atomicMin(&sh.best, mk);
    }
    // lowered tokens whose state has epsilon out-arcs
#pragma unroll
    for (int r = 0; r < R; r++) {
        const bool push = slot[r] >= 0 && key[r] < old[r] && d_eps[r];
        const uint64_t m = __ballot(push);
        if (!m) continue;
        if (push) {
            const int idx = wq.n + rank_in(m);
            const uint2 it = make_uint2(static_cast<uint32_t>(slot[r]), __float_as_uint(cand[r]));
            if (idx < wq.qcap) {
                wq.q[idx] = it;
                wq.ql[idx] = cl[r];
            } else {
                const int gi = atomicAdd(wq.spill_n, 1);
                if (gi < wq.scap) wq.spill[gi] = it;
                else sh.status = WFST_ECAPACITY;
            }
        }
        wq.n = min(wq.n + __popcll(m), wq.qcap);
    }
}

// One candidate per lane, the frame's best key included.
template <bool G>
__device__ __forceinline__ void offer1(const Tab<G> &t, Sh &sh, WaveQ &wq, bool act, uint32_t d, bool d_eps,
                                       uint32_t cl, float cand, uint32_t key)
{
    offer<G, 1, true>(t, sh, wq, &act, &d, &d_eps, &cl, &cand, &key);
}

// Bin holding the rank-th smallest (1-based) of a histogram: sets sh.bin and
// sh.before (the count in lower bins).
__device__ __forceinline__ void select_bin(const uint32_t *h, int nbins, int rank, Sh &sh)
{
    const int per = (nbins + kT - 1) / kT;
    const int b0 = threadIdx.x * per;
    int local = 0;
    for (int i = 0; i < per; i++)
        if (b0 + i < nbins) local += static_cast<int>(h[b0 + i]);
    int total;
    const int excl = block_excl_scan(local, sh.scan, &total);
    if (rank > excl && rank <= excl + local) {
        int cum = excl;
        for (int i = 0; i < per && b0 + i < nbins; i++) {
            const int c = static_cast<int>(h[b0 + i]);
            if (rank <= cum + c) {
                sh.bin = b0 + i;
                sh.before = cum;
                break;
            }
            cum += c;
        }
    }
    __syncthreads();
}

// Shift of the first radix digit so that (lim - kb) >> shift fits the histogram.
__device__ __forceinline__ int first_shift(uint32_t kb, uint32_t lim)
{
    const uint32_t span = lim - kb;
    const int nb = span ? 32 - __clz(static_cast<int>(span)) : 0;
    return nb > kHistBits ? nb - kHistBits : 0;
}

// The expansion's view of S_{k-1}: token costs, emitting-arc prefix and
// first emitting record of each token's state, in LDS (sets of at most
// kSetCache tokens) or in the survivor arrays.
template <bool L>
struct SetView;

template <>
struct SetView<true> {
    const float *cost;
    const int32_t *epre;
    const int32_t *ebeg;
    const uint16_t *cs;   // token owning the first arc of each 64-arc chunk (sets of at most kCs chunks)
    __device__ float c(int i) const { return cost[i]; }
};

template <>
struct SetView<false> {
    const uint32_t *key;
    const int32_t *epre;
    const int32_t *ebeg;
    const uint16_t *cs;   // unused
    __device__ float c(int i) const { return okey_val(key[i]); }
};

// Emitting expansion of S_{k-1} into the table (step 1).  The frame's
// log-likelihood row is read from LDS (srow) when it fits there, else from
// device memory (grow).
template <bool G, bool L>
__device__ __forceinline__ void expand(const Params &p, const Tab<G> &t, Sh &sh, const SetView<L> &v, int n_tok,
                                       int A, const float *srow, const float *grow, WaveQ &wq)
{
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    // a set kept in LDS comes with the first token of each chunk
    const bool use_cs = L && A <= kCs * kWave;
    const bool row_lds = p.L <= kRowMax;
    const int nch = (A + kWave - 1) / kWave;
    // wave w takes chunks w, w + kW, w + 2 kW, ... : every wave gets work
    for (int c = wid; c * kWave < A; c += kW * kChunks) {
        if (__builtin_amdgcn_readfirstlane(sh.overflow)) break;   // the frame is redone anyway
        int ob[kChunks], op[kChunks], a[kChunks];
        float oc[kChunks];
        bool ok[kChunks];
#pragma unroll
        for (int r = 0; r < kChunks; r++) {
            // chunk c + r kW, or with the debugging permutation the chunk as
            // far from the end
            const int ch = p.reverse ? nch - 1 - (c + r * kW) : c + r * kW;
            const int a0 = ch < 0 ? A : ch * kWave;
            a[r] = a0 + lane;
            ok[r] = false;
            ob[r] = op[r] = 0;
            oc[r] = 0.0f;
            if (a0 < A) {
                // the 64 tokens from the one owning a0, and each lane's owner among them
                const int t0 = use_cs ? static_cast<int>(v.cs[a0 / kWave]) : search_le(v.epre, n_tok, a0);
                const int tt = t0 + lane;
                int pre = 0x7FFFFFFF, eb = 0, nx = 0x7FFFFFFF;
                float cst = 0.0f;
                if (tt < n_tok) {
                    pre = v.epre[tt];
                    eb = v.ebeg[tt];
                    cst = v.c(tt);
                    nx = tt + 1 < n_tok ? v.epre[tt + 1] : A;
                }
                const int win_end = t0 + kWave < n_tok ? __builtin_amdgcn_readlane(nx, kWave - 1) : A;
                const int o = owner_scan(pre, nx - pre, a0);
                ob[r] = __shfl(eb, o, kWave);
                op[r] = __shfl(pre, o, kWave);
                oc[r] = __shfl(cst, o, kWave);
                ok[r] = a[r] < A;
                if (ok[r] && a[r] >= win_end) {
                    // past the window (tokens without emitting arcs): search the rest
                    int lo = t0 + kWave, hi = n_tok - 1;
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (v.epre[mid] <= a[r]) lo = mid;
                        else hi = mid - 1;
                    }
                    ob[r] = v.ebeg[lo];
                    op[r] = v.epre[lo];
                    oc[r] = v.c(lo);
                }
                ok[r] = ok[r] && op[r] <= a[r];
            }
        }
        int4 rec[kChunks];
#pragma unroll
        for (int r = 0; r < kChunks; r++) rec[r] = ok[r] ? p.g.earc[ob[r] + (a[r] - op[r])] : make_int4(0, 0, 0, 0);
        float lv[kChunks];
#pragma unroll
        for (int r = 0; r < kChunks; r++) lv[r] = !ok[r] ? 0.0f : row_lds ? srow[rec[r].y] : ldg(grow + rec[r].y);
        bool act[kChunks], de[kChunks];
        uint32_t d[kChunks], key[kChunks], cw[kChunks];
        float cnd[kChunks];
        uint32_t km = kEmptyKey;
#pragma unroll
        for (int r = 0; r < kChunks; r++) {
            const float t1 = oc[r] + __int_as_float(rec[r].z);
            cnd[r] = t1 - lv[r];
            key[r] = okey(cnd[r]);
            if (ok[r] && key[r] < km) km = key[r];
            d[r] = static_cast<uint32_t>(rec[r].x) & kDstMask;
            de[r] = rec[r].x < 0;
            cw[r] = static_cast<uint32_t>(rec[r].w);
        }
        // The batch's own cheapest candidate tightens the early-drop bound; it
        // is within that bound itself, so it is offered and the frame's best
        // key may take its value now.
        km = wave_min_u32(km);
        const uint32_t cur = sh.best;
        if (km < cur && lane == 0) atomicMin(&sh.best, km);
        const uint32_t bnd = drop_bound(km < cur ? km : cur, p.beam);
#pragma unroll
        for (int r = 0; r < kChunks; r++) act[r] = ok[r] && key[r] <= bnd;
        offer<G, kChunks, false>(t, sh, wq, act, d, de, cw, cnd, key);
    }
}

// Weight j (1-8) of a closure entry's path from the entry's second and
// third words (j a constant after unrolling).
__device__ __forceinline__ int path_weight(const int4 &c1, const int4 &c2, int j)
{
    switch (j) {
    case 1: return c1.x;
    case 2: return c1.y;
    case 3: return c1.z;
    case 4: return c1.w;
    case 5: return c2.x;
    case 6: return c2.y;
    case 7: return c2.z;
    default: return c2.w;
    }
}

// Relax the epsilon arcs of one item per lane (valid): the item's state
// still holding the item's cost, i.e. no cheaper item of it follows.
//
// A state with an epsilon-closure list offers every epsilon path from it at
// once: the path's cost is the item's cost plus the path's weights, added
// one at a time in path order, which is the arithmetic of relaxing the path
// arc by arc.  The minimum over paths equals the minimum the arc-by-arc
// relaxation reaches (fl(x + w) is monotone in x), so the tokens are the
// same; the list holds every path, so a token it lowers needs no item of its
// own.  A state without a list relaxes its own arcs, and lowered tokens of
// states with epsilon arcs become items.  An item that comes with its
// state's closure word (icl, from the arc that reached the state) goes to
// the list without loading the state record.
template <bool G>
__device__ __forceinline__ void relax(const Params &p, const Tab<G> &t, Sh &sh, WaveQ &wq, bool valid, uint2 it,
                                      uint32_t icl)
{
    const int lane = lane_id();
    int xb = 0, xd = 0, cb = 0, cn = 0;
    bool first = false;
    int4 x0 = make_int4(0, 0, 0, 0);
    const float cst = __uint_as_float(it.y);
    constexpr uint32_t kSizeMask = (1u << kClosureSizeBits) - 1u;
    // Epsilon weights are not negative (the loader rejects such graphs), so
    // every path from the item costs at least the item (fl(x + w) >= x for
    // w >= 0): an item above the early-drop bound offers nothing that could
    // survive, and is dropped before its loads.
    const uint32_t ibnd = drop_bound(sh.best, p.beam);
    if (valid) {
        const uint32_t now = tld<G>(t.vals + it.x);
        if (okey(cst) == now && now <= ibnd) {
            if (icl) {
                cb = static_cast<int>(icl >> kClosureSizeBits) - 1;
                cn = static_cast<int>(icl & kSizeMask) + 1;
            } else {
                const int64_t s = static_cast<int64_t>(tld<G>(t.keys + it.x));
                const int4 lo = p.g.srec[s];
                x0 = p.g.srec[s + 1];
                const uint32_t cl = static_cast<uint32_t>(x0.w);
                // A list of one path is the state's only epsilon arc, into
                // a state without epsilon arcs: the copy of that arc in the
                // state record offers it below without loading the list.
                if (cl && (cl & kSizeMask) != 0u) {
                    cb = static_cast<int>(cl >> kClosureSizeBits) - 1;
                    cn = static_cast<int>(cl & kSizeMask) + 1;
                } else {
                    first = lo.w > lo.z;
                    xb = lo.z + 1;
                    xd = max(lo.w - lo.z - 1, 0);
                }
            }
        }
    }
    // closure lists, spread over the wave, kRelChunks chunks of paths per
    // step so that their loads (all three words of an entry: a load that
    // waited for the path length would add a round trip) are in flight
    // together
    {
        const int incl = wave_incl_scan(cn);
        const int pre = incl - cn;
        const int tot = __builtin_amdgcn_readlane(incl, kWave - 1);
        for (int k0 = 0; k0 < tot; k0 += kWave * kRelChunks) {
            int4 c0[kRelChunks], c1[kRelChunks], c2[kRelChunks];
            float oc[kRelChunks];
            int64_t e[kRelChunks];
#pragma unroll
            for (int r = 0; r < kRelChunks; r++) {
                const int kk = k0 + r * kWave + lane;
                c0[r] = c1[r] = c2[r] = make_int4(0, 0, 0, 0);
                oc[r] = 0.0f;
                e[r] = 0;
                if (k0 + r * kWave < tot) {
                    const int o = owner_scan(pre, cn, k0 + r * kWave);
                    const int ob = __shfl(cb, o, kWave);
                    const int op = __shfl(pre, o, kWave);
                    oc[r] = __shfl(cst, o, kWave);
                    if (kk < tot) {
                        e[r] = kClosureStride * static_cast<int64_t>(ob + (kk - op));
                        c0[r] = p.g.ctab[e[r]];
                        c1[r] = p.g.ctab[e[r] + 1];
                        c2[r] = p.g.ctab[e[r] + 2];
                    }
                }
            }
            const uint32_t bnd = drop_bound(sh.best, p.beam);
            bool act[kRelChunks], de[kRelChunks];
            uint32_t d[kRelChunks], key[kRelChunks], cw[kRelChunks];
            float cnd[kRelChunks];
#pragma unroll
            for (int r = 0; r < kRelChunks; r++) {
                cnd[r] = oc[r] + __int_as_float(c0[r].w);
            }
            // the later weights in path order, while any path of the wave
            // has more (most paths are one or two arcs long)
#pragma unroll
            for (int j = 1; j < kClosureDepth; j++) {
                bool more = false;
#pragma unroll
                for (int r = 0; r < kRelChunks; r++) more = more || c0[r].z > j;
                if (!__ballot(more)) break;
#pragma unroll
                for (int r = 0; r < kRelChunks; r++)
                    if (c0[r].z > j) cnd[r] = cnd[r] + __int_as_float(path_weight(c1[r], c2[r], j));
            }
#pragma unroll
            for (int r = 0; r < kRelChunks; r++) {
                const float c = cnd[r];
                d[r] = static_cast<uint32_t>(c0[r].x);
                de[r] = false;
                cw[r] = 0u;
                key[r] = okey(c);
                act[r] = k0 + r * kWave + lane < tot && key[r] <= bnd;
            }
            offer<G, kRelChunks, true>(t, sh, wq, act, d, de, cw, cnd, key);
        }
    }
    if (__ballot(first)) {
        // the first epsilon arc, from the state record (the closure word of
        // its destination is not at hand there)
        const uint32_t bnd = drop_bound(sh.best, p.beam);
        const float cnd = cst + __int_as_float(x0.y);
        const uint32_t key = okey(cnd);
        offer1<G>(t, sh, wq, first && key <= bnd, static_cast<uint32_t>(x0.x) & kDstMask, x0.x < 0, 0u, cnd, key);
    }
    // the other epsilon arcs, spread over the wave
    const int incl = wave_incl_scan(xd);
    const int pre = incl - xd;
    const int tot = __builtin_amdgcn_readlane(incl, kWave - 1);
    for (int k0 = 0; k0 < tot; k0 += kWave) {
        const int kk = k0 + lane;
        const int o = owner_scan(pre, xd, k0);
        const int ob = __shfl(xb, o, kWave);
        const int op = __shfl(pre, o, kWave);
        const float oc = __shfl(cst, o, kWave);
        const uint32_t bnd = drop_bound(sh.best, p.beam);
        bool act = false, d_eps = false;
        uint32_t d = 0, key = kEmptyKey, cw = 0u;
        float cnd = 0.0f;
        if (kk < tot) {
            const int4 r = p.g.xarc[ob + (kk - op)];
            d = static_cast<uint32_t>(r.x) & kDstMask;
            d_eps = r.x < 0;
            cw = static_cast<uint32_t>(r.w);
            cnd = oc + __int_as_float(r.y);
            key = okey(cnd);
            act = key <= bnd;
        }
        offer1<G>(t, sh, wq, act, d, d_eps, cw, cnd, key);
    }
}

// Relax the wave's queue until it is empty (items pushed meanwhile included).
template <bool G>
__device__ __forceinline__ void drain(const Params &p, const Tab<G> &t, Sh &sh, WaveQ &wq)
{
    const int lane = lane_id();
    while (wq.n > 0) {
        if (__builtin_amdgcn_readfirstlane(sh.overflow)) {   // the frame is redone anyway
            wq.n = 0;
            break;
        }
        const int take = min(wq.n, kWave);
        const int base = wq.n - take;
        // items were stored by other lanes of the wave
        wave_lds_handover();
        const uint2 it = lane < take ? wq.q[base + lane] : make_uint2(0u, 0u);
        const uint32_t icl = lane < take ? wq.ql[base + lane] : 0u;
        wq.n = base;
        relax<G>(p, t, sh, wq, lane < take, it, icl);
    }
}

// One frame: produces S_k from S_{k-1} (or from the start state when k = 0).
// Returns 0, kOverflow (the table filled up; nothing of S_k was written) or
// a negative WFST error.  Every return is taken by the whole workgroup.
template <bool G>
__device__ __forceinline__ int frame(const Params &p, const UttLayout &ly, const float *ll, int Tp, Sh &sh,
                                     const Tab<G> &t, uint2 *aux, uint32_t *auxl, float *s_cost, int32_t *s_epre, int32_t *s_ebeg,
                                     uint16_t *s_cs, float *s_row, uint2 *spill, int gcap, Run *runs, Prof &pf,
                                     int k, int &n_ins)
{
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wid = tid / kWave;
    const Run &run = runs[k & 1];
    WaveQ wq;
    wq.q = aux + wid * kQueue;
    wq.ql = auxl + wid * kQueue;
    wq.n = 0;
    wq.qcap = min(kQueue, p.gen_lds);
    wq.spill = spill;
    wq.spill_n = &sh.spill_n[0];
    wq.scap = gcap;

    phase_mark(p, pf, 5);
    if (tid == 0) {
        sh.nslots = 0;
        sh.overflow = 0;
        sh.best = kEmptyKey;
        sh.spill_n[0] = sh.spill_n[1] = 0;
        sh.alloc[k & 1] = 0ull;
        sh.xsum[k & 1] = 0;
        sh.cnt = 0;
    }
    __syncthreads();
    phase_mark(p, pf, 5);

    // ---- 1. expansion ----
    sub_open(p, pf);
    if (k == 0) {
        if (wid == 0) {
            const int s = p.g.start;
            const int4 lo = p.g.srec[s];
            offer1<G>(t, sh, wq, lane == 0, static_cast<uint32_t>(s), lo.w > lo.z, 0u, 0.0f, okey(0.0f));
        }
    } else {
        const float *row = ll + static_cast<int64_t>(p.kept[ly.kept0 + k - 1]) * p.L;
        if (run.n_prev <= kSetCache) {
            SetView<true> v{s_cost, s_epre, s_ebeg, s_cs};
            expand<G, true>(p, t, sh, v, run.n_prev, run.a_prev, s_row, row, wq);
        } else {
            const int64_t base = ly.sv0 + run.prev0;
            SetView<false> v{p.sv_key + base, p.sv_epre + base, p.sv_ebeg + base, nullptr};
            expand<G, false>(p, t, sh, v, run.n_prev, run.a_prev, s_row, row, wq);
        }
    }
    sub_close(p, pf, 4);
    // ---- 2. epsilon closure: each wave its own queue, then spill rounds ----
    drain<G>(p, t, sh, wq);
    // full barrier: spilled items are read by other waves
    __syncthreads();
    phase_mark(p, pf, 0);
    int sp = 0;
    while (true) {
        const int total = min(sh.spill_n[sp], gcap);
        if (total == 0 || sh.overflow || sh.status) break;
        const uint2 *list = spill + static_cast<int64_t>(sp) * gcap;
        if (tid == 0) sh.spill_n[sp ^ 1] = 0;
        __syncthreads();
        wq.spill = spill + static_cast<int64_t>(sp ^ 1) * gcap;
        wq.spill_n = &sh.spill_n[sp ^ 1];
        for (int c0 = wid * kWave; c0 < total; c0 += kT) {
            const int i = c0 + lane;
            uint2 it = make_uint2(0u, 0u);
            if (i < total) {
                const unsigned long long w = ldg(reinterpret_cast<const unsigned long long *>(list + i));
                it = make_uint2(static_cast<uint32_t>(w), static_cast<uint32_t>(w >> 32));
            }
            relax<G>(p, t, sh, wq, i < total, it, 0u);
            drain<G>(p, t, sh, wq);
        }
        __syncthreads();
        sp ^= 1;
    }
    phase_mark(p, pf, 1);
    if (sh.overflow) {
        phase_fold(p, pf, false);   // the frame is redone on the device-memory table
        return kOverflow;
    }
    if (sh.status) return sh.status;

    // ---- 3. pruning ----
    const int n = sh.nslots;
    n_ins = n;
    const uint32_t kb = sh.best;
    const uint32_t lim = beam_limit(kb, p.beam);
    uint32_t cut = lim;
    if (p.max_active > 0 && n > p.max_active && kb <= lim) {
        uint32_t *hist = reinterpret_cast<uint32_t *>(aux);
        int shf = first_shift(kb, lim);
        for (int i = tid; i < kHistBins; i += kT) hist[i] = 0u;
        __syncthreads();
        int cnt = 0;
        for (int i = tid; i < n; i += kT) {
            const uint32_t key = tld<G>(t.vals + tld<G>(t.slots + i));
            if (key <= lim) {
                cnt++;
                atomicAdd(&hist[(key - kb) >> shf], 1u);
            }
        }
        if (cnt) atomicAdd(&sh.cnt, cnt);
        __syncthreads();
        if (sh.cnt > p.max_active) {
            int rank = p.max_active;
            select_bin(hist, kHistBins, rank, sh);
            uint32_t prefix = static_cast<uint32_t>(sh.bin) << shf;
            rank -= sh.before;
            while (shf > 0) {
                const int nsh = shf > kHistBits ? shf - kHistBits : 0;
                const int nb = 1 << (shf - nsh);
                __syncthreads();
                for (int i = tid; i < nb; i += kT) hist[i] = 0u;
                __syncthreads();
                for (int i = tid; i < n; i += kT) {
                    const uint32_t key = tld<G>(t.vals + tld<G>(t.slots + i));
                    if (key > lim) continue;
                    const uint32_t off = key - kb;
                    if ((off >> shf) == (prefix >> shf)) atomicAdd(&hist[(off >> nsh) & (nb - 1)], 1u);
                }
                __syncthreads();
                select_bin(hist, nb, rank, sh);
                prefix |= static_cast<uint32_t>(sh.bin) << nsh;
                rank -= sh.before;
                shf = nsh;
            }
            const uint32_t theta = kb + prefix;
            cut = theta < lim ? theta : lim;
        }
        __syncthreads();
    }

    phase_mark(p, pf, 2);

    // ---- 4. compaction into S_k ----
    // Each wave takes chunks of the slot list, clears their slots, loads the
    // survivors' state records together and places its survivors with one
    // 64-bit LDS add of (emitting degrees << 32 | count): the returned value
    // gives their positions and the prefix of emitting degrees before them
    // at once.  The order of a token set is internal (sets are reported
    // sorted by state), so no block-wide scan is needed.
    // The next frame's log-likelihood row is loaded meanwhile (the expansion
    // that read this frame's row is over: every wave has passed the barrier
    // after the closure), and stored into LDS at the end.
    const bool next_row = p.L <= kRowMax && k < Tp;
    constexpr int kRowPer = kRowMax / kT;
    float rv[kRowPer];
    if (next_row) {
        const float *nrow = ll + static_cast<int64_t>(p.kept[ly.kept0 + k]) * p.L;
#pragma unroll
        for (int j = 0; j < kRowPer; j++) {
            const int i = tid + j * kT;
            rv[j] = i < p.L ? ldg(nrow + i) : 0.0f;
        }
    }
    using Slot = typename Tab<G>::Slot;
    const int64_t set0 = run.set0;
    int xacc = 0;   // epsilon degrees of this lane's survivors
    // The row goes into LDS in the wave's first chunk, after its state-record
    // loads and before its first survivor stores: vector memory operations
    // complete in issue order, so a wait for the row after any store would
    // also wait for that store.
    bool row_due = next_row;
    for (int c = wid; c * kWave < n; c += kW) {
        const int i = c * kWave + lane;
        bool kp = false;
        uint32_t vv = kEmptyKey;
        int dd = 0;
        if (i < n) {
            const Slot sl = tld<G>(t.slots + i);
            vv = tld<G>(t.vals + sl);
            dd = static_cast<int>(tld<G>(t.keys + sl));
            kp = vv <= cut;
            t.keys[sl] = kEmptyKey;
            t.vals[sl] = kEmptyKey;
        }
        int4 lo = make_int4(0, 0, 0, 0);
        if (kp) lo = p.g.srec[dd];
        if (row_due) {
#pragma unroll
            for (int j = 0; j < kRowPer; j++) {
                const int ri = tid + j * kT;
                if (ri < p.L) s_row[ri] = rv[j];
            }
            row_due = false;
        }
        // (lo is used on every path: a load left pending into the next round
        // would make that round wait before writing its registers)
        const uint64_t km = __ballot(kp);
        const int tc = __popcll(km);
        const int deg = kp ? lo.y - lo.x : 0;
        xacc += kp ? lo.w - lo.z : 0;
        const int id = wave_incl_scan(deg);
        const int td = __builtin_amdgcn_readlane(id, kWave - 1);
        unsigned long long base = 0;
        if (lane == 0 && tc)
            base = atomicAdd(&sh.alloc[k & 1], (static_cast<unsigned long long>(td) << 32) | static_cast<uint32_t>(tc));
        base = (static_cast<unsigned long long>(__builtin_amdgcn_readlane(static_cast<int>(base >> 32), 0)) << 32) |
               static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(base), 0));
        if (!kp) continue;
        const int pos = static_cast<int>(static_cast<uint32_t>(base)) + rank_in(km);
        const int apos = static_cast<int>(base >> 32) + id - deg;
        if (pos < kSetCache) {
            // to the survivor arrays after the barrier below
            s_cost[pos] = okey_val(vv);
            s_epre[pos] = apos;
            s_ebeg[pos] = lo.x;
            // the chunks whose first arc is one of this token's
            for (int ch = (apos + kWave - 1) / kWave; ch * kWave < apos + deg && ch < kCs; ch++)
                s_cs[ch] = static_cast<uint16_t>(pos);
        } else if (set0 + pos < ly.svcap) {
            const int64_t o = ly.sv0 + set0 + pos;
            p.sv_state[o] = dd;
            p.sv_key[o] = vv;
            p.sv_ebeg[o] = lo.x;
            p.sv_epre[o] = apos;
        }
    }
    {
        const int tx = wave_incl_scan(xacc);
        if (lane == kWave - 1 && tx) atomicAdd(&sh.xsum[k & 1], tx);
    }
    if (row_due) {
#pragma unroll
        for (int j = 0; j < kRowPer; j++) {
            const int ri = tid + j * kT;
            if (ri < p.L) s_row[ri] = rv[j];
        }
    }
    // (with the device-memory table, its cleared slots before the next offers)
    table_barrier<G>();
    const unsigned long long alloc = sh.alloc[k & 1];
    const int n_kept = static_cast<int>(static_cast<uint32_t>(alloc));
    // The survivors placed in the LDS copy go to the survivor arrays now, in
    // one batch of stores that overlaps the next frame's start (a state's id
    // is its first emitting unit minus 2).  Stores inside the loop above
    // would make each of its rounds wait for them.
    if (set0 + n_kept > ly.svcap) return WFST_ECAPACITY;
    for (int i = tid; i < min(n_kept, kSetCache); i += kT) {
        const int64_t o = ly.sv0 + set0 + i;
        const int32_t eb = s_ebeg[i];
        p.sv_state[o] = eb - 2;
        p.sv_key[o] = okey(s_cost[i]);
        p.sv_ebeg[o] = eb;
        p.sv_epre[o] = s_epre[i];
    }
    // the next expansion reads S_k from LDS unless it is larger than the LDS
    // copy; then it reads the survivor arrays, which other waves wrote
    if (static_cast<uint32_t>(alloc) > static_cast<uint32_t>(kSetCache)) __syncthreads();
    const int a_kept = static_cast<int>(alloc >> 32);
    const int x_kept = sh.xsum[k & 1];
    const int ns = n_kept;
    phase_mark(p, pf, 3);
    phase_fold(p, pf, true);
    if (ns == 0) return WFST_ENOPATH;
    if (sh.status) return sh.status;
    // Token set k, its cutoff and the lattice record regions of set k: one
    // record per emitting arc of S_k (into S_k+1) at most, one per epsilon
    // arc of S_k at most.  The emitting offsets also give the record pass
    // the emitting arcs of each set.
    const int64_t a_rec = k < Tp ? a_kept : 0;
    // (with the incremental lattice pass the regions only bound the ring use
    // per set; the pass checks its own capacities)
    if (p.lattice && !p.stream_k && (run.le + a_rec > ly.lecap || run.lx + x_kept > ly.lxcap))
        return WFST_ECAPACITY;
    // the next frame's running values: thread 0 writes the other copy,
    // which every thread reads after the next frame's first barrier
    if (tid == 0) {
        p.sv_off[ly.fo0 + k + 1] = set0 + ns;
        p.cut_arr[ly.fo0 + k] = cut;
        p.rle_off[ly.fo0 + k + 1] = run.le + a_rec;
        p.rlx_off[ly.fo0 + k + 1] = run.lx + x_kept;
        Run &nx = runs[(k + 1) & 1];
        nx.le = run.le + a_rec;
        nx.lx = run.lx + x_kept;
        nx.eps = run.eps + x_kept;
        nx.arcs = run.arcs + a_rec;
        nx.prev0 = set0;
        nx.set0 = set0 + ns;
        nx.n_prev = ns;
        nx.a_prev = a_kept;
    }

    return 0;
}

// ---------------------------------------------------------------------------
// Record workgroups beside the search.  A launch may carry rec_wg workgroups
// after its U search workgroups (they are dispatched after them).  They
// derive the back-pointers and raw lattice records of the launch's token
// sets (record_one, the record kernel's work) while the search still runs,
// so that the record pass of the batch's longest utterances ends with their
// search instead of after it.  Items (token set k, utterance u) are taken in
// frame order from a device counter; item (k, u) needs sets k - 1 and k,
// i.e. a published count prog[u] > k (the search publishes every pub_k sets
// and at its end; -1 when it failed).  Thread 0 polls the count with relaxed
// loads; wave 0 then reads every utterance's count into seen[] and takes one
// acquire fence, which makes visible everything those counts cover.  The
// fence invalidates the caches that the searches of the chiplet share, so a
// workgroup takes one only when an item needs a set beyond seen[].
// ---------------------------------------------------------------------------
constexpr long long kRecPolls = 1LL << 22;  // polls of one count (several seconds) before giving up

struct RecLds {
    RSh rsh;
    int item;
    int prog;
    int seen[kRecMaxUtts];
    unsigned long long win[kRFill];
    uint32_t keys[kRSlots];
    int32_t vals[kRSlots];
};

__device__ __forceinline__ void record_role(const Params &p, RecLds &r)
{
    const int U = p.U;
    const int items = (p.rec_tmax + 1) * U;
    const int tid = threadIdx.x;
    for (int i = tid; i < U; i += blockDim.x) r.seen[i] = 0;
    while (true) {
        if (tid == 0) r.item = atomicAdd(p.rec_next, 1);
        __syncthreads();
        const int i = r.item;
        if (i >= items) break;
        const int k = i / U;
        const int u = i - k * U;
        UttState &st = p.st[u];
        // every thread has read the item before thread 0 takes the next
        if (k > st.Tp || r.seen[u] < 0) {
            __syncthreads();
            continue;
        }
        if (r.seen[u] <= k) {
            if (tid == 0) {
                int v = 0;
                for (long long n = 0;; n++) {
                    v = __hip_atomic_load(p.prog + u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (v > k || v < 0) break;
                    // another record workgroup may have given up on it already
                    if (n >= kRecPolls || __hip_atomic_load(&st.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                                              kStatusStreamTimeout) {
                        v = -2;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(32);
                }
                if (v == -2) set_status(st, kStatusStreamTimeout);
                r.prog = v;
            }
            // (seen[] is written only after every thread has read it above)
            __syncthreads();
            if (r.prog > k) {
                if (tid < kWave) {
                    // the counts as they are now; the fence covers them all
                    for (int w = tid; w < U; w += kWave) {
                        const int v = __hip_atomic_load(p.prog + w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        r.seen[w] = v < 0 ? -1 : max(r.seen[w], v);
                    }
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                }
            } else if (tid == 0) {
                // the search failed, or the wait gave up: the utterance's
                // remaining items are skipped
                r.seen[u] = -1;
            }
            __syncthreads();
            if (r.seen[u] <= k) continue;
        }
        record_one(p, u, k, r.keys, r.vals, r.win, r.rsh);
        __syncthreads();
    }
}

template <bool kRec>
__global__ __launch_bounds__(kT) void search_kernel(Params p)
{
    // All LDS in one struct, the small fields first: they then lie below
    // 64 KB, where an LDS instruction reaches them with an immediate offset
    // instead of an address held in a register.
    struct Lds {
        Sh sh;
        Prof pf;
        Run run[2];
        uint16_t cs[kCs];                  // first token of each 64-arc chunk of the last set
        uint2 aux[kW * kQueue];            // per-wave epsilon queues, or the select histogram
        uint32_t auxl[kW * kQueue];        // the queue items' closure words
        float cost[kSetCache];             // the last token set, for the next expansion
        int32_t epre[kSetCache];
        int32_t ebeg[kSetCache];
        uint16_t slots[kFill];
        uint32_t keys[kSlots];
        uint32_t vals[kSlots];
        float row[kRowMax];                // the frame's log-likelihood row (L <= kRowMax)
        // last: the arrays above keep their offsets modulo 256 bytes, which
        // lets paired reads of the hash table use one instruction
        UttLayout ly;                      // the utterance's layout (in LDS: no registers held for it)
    };
    union All {
        Lds s;
        RecLds r;
    };
    static_assert(sizeof(RecLds) <= sizeof(Lds), "the record workgroups fit the search's LDS");
    __shared__ All all;
    Lds &lds = all.s;
    if constexpr (kRec) {
        if (static_cast<int>(blockIdx.x) >= p.U) {
            record_role(p, all.r);
            return;
        }
    }
    Sh &sh = lds.sh;
    Prof &pf = lds.pf;
    uint32_t *s_keys = lds.keys;
    uint32_t *s_vals = lds.vals;
    float *s_row = lds.row;
    uint16_t *s_slots = lds.slots;
    uint2 *s_aux = lds.aux;
    uint32_t *s_auxl = lds.auxl;
    float *s_cost = lds.cost;
    int32_t *s_epre = lds.epre;
    int32_t *s_ebeg = lds.ebeg;
    uint16_t *s_cs = lds.cs;

    const int u = blockIdx.x;
    const int tid = threadIdx.x;
    UttState &st = p.st[u];
    if (st.status != 0) {
        if (p.pub_k && tid == 0) __hip_atomic_store(p.prog + u, -1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    // the layout is copied into LDS: a reference into device memory would be
    // reloaded after every barrier, and a copy in registers would hold a
    // dozen of them for the whole kernel
    if (tid == 0) lds.ly = p.lay[u];
    __syncthreads();
    const UttLayout &ly = lds.ly;
    const int Tp = st.Tp;
    const float *ll = st.ll;

    Tab<false> lt;
    lt.keys = s_keys;
    lt.vals = s_vals;
    lt.slots = s_slots;
    lt.mask = kSlots - 1;
    lt.fill = min(kFill, p.lds_fill);
    lt.shift = 32 - kSlotBits;
    lt.mul = p.hash_mul;
    Tab<true> gt;
    const int64_t gbase = static_cast<int64_t>(u) * p.capG;
    gt.keys = p.gkeys + gbase;
    gt.vals = p.gvals + gbase;
    gt.slots = p.gslots + gbase;
    gt.mask = static_cast<uint32_t>(p.capG - 1);
    gt.fill = static_cast<int>(p.capG / 4 * 3);
    gt.shift = 32 - (31 - __clz(static_cast<int>(p.capG)));
    gt.mul = p.hash_mul;
    const int gcap = static_cast<int>(p.capO);
    uint2 *spill = p.gspill + static_cast<int64_t>(u) * 2 * p.capO;

    for (int i = tid; i < kSlots; i += kT) {
        s_keys[i] = kEmptyKey;
        s_vals[i] = kEmptyKey;
    }
    if (tid == 0) {
        sh.status = 0;
    }
    __syncthreads();

    Run *runs = lds.run;   // running values of the utterance, written by thread 0
    if (tid == 0) runs[0] = Run{};
    int gframes = 0;       // frames redone on the device-memory table (thread 0's count)
    int kd = 0;            // frames completed
    if (tid == 0) {
        for (int i = 0; i < 7; i++) pf.ph[i] = 0;
        for (int i = 0; i < 4; i++) pf.cur[i] = 0;
        pf.t_last = wall_clock64();
        pf.t_sub = 0;
    }
    bool gclean = false;
    // After a frame that needed the device-memory table, the next frames go
    // there directly while their tables stay close to the LDS limit: a frame
    // started in LDS would most likely be abandoned half-way.
    bool in_g = false;
    const int g_stay = lt.fill - lt.fill / 8;
    int rc = 0;
    for (int k = 0; k <= Tp; k++) {
        int n_ins = 0;
        if (!in_g)
            rc = frame<false>(p, ly, ll, Tp, sh, lt, s_aux, s_auxl, s_cost, s_epre, s_ebeg, s_cs, s_row, spill, gcap, runs,
                              pf, k, n_ins);
        if (in_g || rc == kOverflow) {
            if (!in_g) {
                // the abandoned attempt left states in the LDS table
                for (int i = tid; i < kSlots; i += kT) {
                    s_keys[i] = kEmptyKey;
                    s_vals[i] = kEmptyKey;
                }
            }
            if (!gclean) {
                for (int64_t i = tid; i < p.capG; i += kT) {
                    gt.keys[i] = kEmptyKey;
                    gt.vals[i] = kEmptyKey;
                }
                gclean = true;
            }
            __syncthreads();
            rc = frame<true>(p, ly, ll, Tp, sh, gt, s_aux, s_auxl, s_cost, s_epre, s_ebeg, s_cs, s_row, spill, gcap, runs,
                             pf, k, n_ins);
            if (rc == kOverflow) rc = WFST_ECAPACITY;
            gframes++;
            in_g = n_ins > g_stay;
        }
        if (rc != 0) break;
        kd = k + 1;
        // publish every pub_k finished token sets to the record workgroups
        // or the incremental lattice pass: every wave's stores of the sets
        // complete in L2 first (the last barrier of a frame orders LDS only),
        // then one release store of the count (which writes the cache back
        // for readers possibly on another chiplet)
        if (p.pub_k && (k + 1) % p.pub_k == 0 && k < Tp) {
            block_sync_vm();
            if (tid == 0) __hip_atomic_store(p.prog + u, k + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if (tid == 0) {
        const Run &run = runs[kd & 1];
        st.n_tok = run.set0;
        st.n_last = run.n_prev;
        st.arcs_expanded = run.arcs;
        st.eps_arcs = run.eps;
        st.gframes = gframes;
        for (int i = 0; i < 7; i++) st.phase_ticks[i] = pf.ph[i];
        if (rc != 0) st.status = rc;
    }
    if (p.pub_k) {
        block_sync_vm();
        if (tid == 0) __hip_atomic_store(p.prog + u, rc == 0 ? Tp + 1 : -1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
}

}  // namespace

}  // namespace wfd
