// Decode driver and result objects of the C ABI.
//
// One call decodes a batch of utterances: classify frames (label-synchronous
// compaction), one search launch in which a workgroup per utterance produces
// every token set with its back-pointers and lattice records, then final
// costs, backtrace, lattice-beam pruning and the sorted lattice.  Buffers
// are carved from a per-device arena kept between calls; a buffer that
// overflows makes the call decode again with larger ones.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <memory>
#include <mutex>
#include <new>
#include <numeric>
#include <vector>

#include "internal.h"

using namespace wfd;

namespace {

struct DevBuf {
    void *p = nullptr;
    int device = 0;
    DevBuf() = default;
    DevBuf(const DevBuf &) = delete;
    DevBuf &operator=(const DevBuf &) = delete;
    ~DevBuf()
    {
        if (!p) return;
        int cur = 0;
        (void)hipGetDevice(&cur);
        if (cur != device) (void)hipSetDevice(device);
        (void)hipFree(p);
        if (cur != device) (void)hipSetDevice(cur);
    }
};

// The lattices of one batch in host memory: copied from the device buffer in
// one transfer when the first result asks for its lattice, then shared.
struct LatHost {
    std::mutex mu;
    bool loaded = false;
    int64_t total = 0;
    std::vector<wfst_lat_arc> arcs;
};

// Lattice output buffers.  The results of a batch share one buffer; when the
// last of them is freed the buffer returns to a small per-device pool, so a
// steady sequence of decodes allocates no lattice memory.
constexpr int kLatPoolKeep = 4;

struct LatPool {
    std::mutex mu;
    std::vector<std::pair<size_t, void *>> free_bufs[64];
};

LatPool &lat_pool()
{
    static LatPool *p = new LatPool();
    return *p;
}

struct LatBuf {
    void *p = nullptr;
    size_t bytes = 0;
    int device = 0;
    LatBuf() = default;
    LatBuf(const LatBuf &) = delete;
    LatBuf &operator=(const LatBuf &) = delete;
    ~LatBuf()
    {
        if (!p) return;
        void *drop = nullptr;
        if (device >= 0 && device < 64) {
            LatPool &pool = lat_pool();
            std::lock_guard<std::mutex> lk(pool.mu);
            auto &fl = pool.free_bufs[device];
            fl.emplace_back(bytes, p);
            if (static_cast<int>(fl.size()) > kLatPoolKeep) {
                // keep the largest buffers
                auto it = std::min_element(fl.begin(), fl.end());
                drop = it->second;
                fl.erase(it);
            }
        } else {
            drop = p;
        }
        if (drop) {
            int cur = 0;
            (void)hipGetDevice(&cur);
            if (cur != device) (void)hipSetDevice(device);
            (void)hipFree(drop);
            if (cur != device) (void)hipSetDevice(cur);
        }
    }
};

// A lattice output buffer of at least `need` bytes on the current device:
// the smallest pooled one that fits, else a new allocation.
hipError_t lat_take(int device, size_t need, bool fail, std::shared_ptr<LatBuf> &out)
{
    if (fail) return hipErrorOutOfMemory;
    auto b = std::make_shared<LatBuf>();
    b->device = device;
    if (device >= 0 && device < 64) {
        LatPool &pool = lat_pool();
        std::lock_guard<std::mutex> lk(pool.mu);
        auto &fl = pool.free_bufs[device];
        int best = -1;
        for (int i = 0; i < static_cast<int>(fl.size()); i++)
            if (fl[i].first >= need && (best < 0 || fl[i].first < fl[best].first)) best = i;
        if (best >= 0) {
            b->bytes = fl[best].first;
            b->p = fl[best].second;
            fl.erase(fl.begin() + best);
            out = b;
            return hipSuccess;
        }
    }
    const size_t want = std::max<size_t>(need + need / 4, size_t{1} << 20);
    hipError_t e = hipMalloc(&b->p, want);
    if (e != hipSuccess) {
        b->p = nullptr;
        e = hipMalloc(&b->p, need);
        if (e != hipSuccess) {
            b->p = nullptr;
            return e;
        }
        b->bytes = need;
    } else {
        b->bytes = want;
    }
    out = b;
    return hipSuccess;
}

}  // namespace

struct wfst_result {
    int status = WFST_OK;
    float cost = std::numeric_limits<float>::quiet_NaN();
    int32_t final_state = -1;
    int32_t reached_final = 0;
    std::vector<int32_t> path_arcs, path_frames, kept;
    int32_t T = 0, Tp = 0;
    std::shared_ptr<LatBuf> lat_dev;
    int64_t lat_off = 0, lat_n = 0;
    std::shared_ptr<LatHost> lat_host;   // the batch's lattice in host memory, copied on first use
    bool has_words = false;
    std::vector<int64_t> w_off;        // word sequences: offsets into w_words
    std::vector<int32_t> w_words;
    std::vector<float> w_cost;
    bool has_tokens = false;
    std::vector<int64_t> tok_off;
    std::vector<int32_t> tok_state, tok_arc;
    std::vector<float> tok_cost;
    wfst_stats stats{};
};

namespace {

int fail(int code, const char *msg)
{
    set_error("%s", msg);
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    set_error("%s: %s", what, hipGetErrorString(e));
    return e == hipErrorOutOfMemory ? WFST_ENOMEM : WFST_EDEVICE;
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev)
    {
        (void)hipGetDevice(&prev);
        if (prev != dev) (void)hipSetDevice(dev);
        else prev = -1;
    }
    ~DeviceGuard()
    {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

// Device workspace of one decode call: every buffer is carved from one
// arena.  A first pass over the same carving code only measures the size.
struct Arena {
    char *base = nullptr;
    size_t off = 0;
    template <typename T>
    T *get(int64_t count)
    {
        const size_t bytes = (static_cast<size_t>(std::max<int64_t>(count, 1)) * sizeof(T) + 255) &
                             ~static_cast<size_t>(255);
        T *ptr = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += bytes;
        return ptr;
    }
};

// One arena per device is kept between calls and only ever grows, so that
// steady-state decoding allocates nothing.  A call that finds it in use by a
// concurrent call takes a private allocation instead.
struct ArenaCache {
    std::mutex mu;
    bool busy = false;
    void *ptr = nullptr;
    size_t cap = 0;
};

ArenaCache &arena_cache(int dev, int kind = 0)
{
    // kind 0: the decode workspace; kind 1: the word-lattice pass
    static ArenaCache *c = new ArenaCache[2 * 64];
    return c[kind * 64 + dev];
}

struct ArenaLease {
    int dev = -1;
    void *ptr = nullptr;
    bool cached = false;
    ArenaLease() = default;
    ArenaLease(const ArenaLease &) = delete;
    ArenaLease &operator=(const ArenaLease &) = delete;
    int kind = 0;
    hipError_t acquire(int device, size_t need, int which = 0)
    {
        dev = device;
        kind = which;
        if (dev >= 0 && dev < 64) {
            ArenaCache &c = arena_cache(dev, kind);
            std::lock_guard<std::mutex> lk(c.mu);
            if (!c.busy) {
                if (c.cap < need) {
                    if (c.ptr) (void)hipFree(c.ptr);
                    c.ptr = nullptr;
                    c.cap = 0;
                    size_t want = need + need / 4;
                    hipError_t e = hipMalloc(&c.ptr, want);
                    if (e != hipSuccess) {
                        want = need;
                        e = hipMalloc(&c.ptr, want);
                    }
                    if (e != hipSuccess) {
                        c.ptr = nullptr;
                        return e;
                    }
                    c.cap = want;
                }
                c.busy = true;
                cached = true;
                ptr = c.ptr;
                return hipSuccess;
            }
        }
        return hipMalloc(&ptr, need);
    }
    ~ArenaLease()
    {
        if (cached) {
            ArenaCache &c = arena_cache(dev, kind);
            std::lock_guard<std::mutex> lk(c.mu);
            c.busy = false;
        } else if (ptr) {
            (void)hipFree(ptr);
        }
    }
};

// Page-locked host memory for the transfers of one call (utterance states
// and layouts in, states, kept frames, paths and set offsets out): one
// buffer per device, kept between calls and only ever grown, so that each
// transfer is a single DMA into memory the runtime need not pin on the fly
// and steady-state decoding allocates nothing.  A call that finds it in use
// by a concurrent call takes a private one; if pinning fails, pageable
// memory serves (slower transfers, same results).
struct PinnedCache {
    std::mutex mu;
    bool busy = false;
    void *ptr = nullptr;
    size_t cap = 0;
};

PinnedCache &pinned_cache(int dev)
{
    static PinnedCache *c = new PinnedCache[64];
    return c[dev];
}

struct PinnedLease {
    int dev = -1;
    char *ptr = nullptr;
    bool cached = false;
    bool pinned = false;
    std::vector<char> fallback;
    PinnedLease() = default;
    PinnedLease(const PinnedLease &) = delete;
    PinnedLease &operator=(const PinnedLease &) = delete;
    void acquire(int device, size_t need)
    {
        dev = device;
        if (dev >= 0 && dev < 64) {
            PinnedCache &c = pinned_cache(dev);
            std::lock_guard<std::mutex> lk(c.mu);
            if (!c.busy) {
                if (c.cap < need) {
                    if (c.ptr) (void)hipHostFree(c.ptr);
                    c.ptr = nullptr;
                    c.cap = 0;
                    const size_t want = need + need / 4;
                    if (hipHostMalloc(&c.ptr, want, hipHostMallocDefault) == hipSuccess) c.cap = want;
                    else c.ptr = nullptr;
                }
                if (c.ptr) {
                    c.busy = true;
                    cached = pinned = true;
                    ptr = static_cast<char *>(c.ptr);
                    return;
                }
            }
        }
        void *q = nullptr;
        if (hipHostMalloc(&q, need, hipHostMallocDefault) == hipSuccess) {
            pinned = true;
            ptr = static_cast<char *>(q);
            return;
        }
        fallback.resize(need);
        ptr = fallback.data();
    }
    ~PinnedLease()
    {
        if (cached) {
            PinnedCache &c = pinned_cache(dev);
            std::lock_guard<std::mutex> lk(c.mu);
            c.busy = false;
        } else if (pinned) {
            (void)hipHostFree(ptr);
        }
    }
};

// Launches whose workgroups wait on other workgroups (the record
// workgroups beside a search, the incremental lattice pass) need the waited-on
// workgroups to find CUs: one call per device at a time uses them, and only
// when the batch's search workgroups and the waiting ones fit the device's
// CUs together.  A call that cannot take the device's flag decodes without
// them (the same results).
std::atomic<bool> &wait_flag(int dev)
{
    static std::atomic<bool> *f = new std::atomic<bool>[64]();
    return f[dev];
}

int device_cus(int dev)
{
    static std::atomic<int> *n = new std::atomic<int>[64]();
    int v = n[dev].load();
    if (v == 0) {
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) v = -1;
        n[dev].store(v);
    }
    return v;
}

struct WaitGuard {
    int dev = -1;
    bool held = false;
    bool take(int device)
    {
        if (device < 0 || device >= 64) return false;
        bool expect = false;
        held = wait_flag(device).compare_exchange_strong(expect, true);
        if (held) dev = device;
        return held;
    }
    ~WaitGuard()
    {
        if (held) wait_flag(dev).store(false);
    }
};

// Test and debugging switches (wfst_set_debug_opts), process-wide.
struct DebugState {
    std::mutex mu;
    wfst_debug_opts o{};
};

DebugState &debug_state()
{
    static DebugState d;   // no heap allocation, also on first use
    return d;
}

wfst_debug_opts debug_snapshot()
{
    DebugState &d = debug_state();
    std::lock_guard<std::mutex> lk(d.mu);
    return d.o;
}

// A positive override below the default replaces it.
int limit_or(int32_t v, int dflt) { return v >= 1 && v < dflt ? v : dflt; }

struct Sizes {
    int64_t capA;      // tokens per frame on average over an utterance
    int64_t capF;      // tokens per frame
    int64_t capT;      // reached states per frame
    int64_t capO;      // overflow epsilon items per frame (per generation)
    int64_t em;        // emitting lattice-record slots per token (emitting out-degree)
    int64_t xm;        // epsilon lattice-record slots per token (epsilon out-degree)
};

// Events for phase timing, kept for reuse across calls: creating thousands
// of events per decode would stall the launch loop.
struct EventPool {
    std::mutex mu;
    std::vector<hipEvent_t> free_ev[64];
    hipEvent_t get(int dev)
    {
        {
            std::lock_guard<std::mutex> lk(mu);
            if (!free_ev[dev].empty()) {
                hipEvent_t e = free_ev[dev].back();
                free_ev[dev].pop_back();
                return e;
            }
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
    void put(int dev, hipEvent_t e)
    {
        std::lock_guard<std::mutex> lk(mu);
        free_ev[dev].push_back(e);
    }
};

EventPool &event_pool()
{
    static EventPool *pool = new EventPool();
    return *pool;
}

// Phase timing with HIP events (WFST_PROFILE): a start/stop pair per phase
// launch, recorded on the stream the phase runs on.
struct Timer {
    bool on = false;
    int dev = 0;
    struct Span {
        hipEvent_t a, b;
        int kind;
    };
    std::vector<Span> spans;
    hipEvent_t open_ev = nullptr;
    void start(hipStream_t s)
    {
        if (!on) return;
        open_ev = event_pool().get(dev);
        if (open_ev) (void)hipEventRecord(open_ev, s);
    }
    void stop(int kind, hipStream_t s)
    {
        if (!on || !open_ev) return;
        hipEvent_t e = event_pool().get(dev);
        if (!e) return;
        (void)hipEventRecord(e, s);
        spans.push_back({open_ev, e, kind});
        open_ev = nullptr;
    }
    ~Timer()
    {
        for (auto &x : spans) {
            event_pool().put(dev, x.a);
            event_pool().put(dev, x.b);
        }
        if (open_ev) event_pool().put(dev, open_ev);
    }
};

// Wall-clock breakdown of each decode call on stderr when the environment
// variable WFSTDEC_DEBUG_TIMING is set (read once per process).
bool debug_timing()
{
    static const bool on = getenv("WFSTDEC_DEBUG_TIMING") != nullptr;
    return on;
}

struct WallTrace {
    bool on = debug_timing();
    double t = now();
    static double now()
    {
        return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now().time_since_epoch()).count();
    }
    void mark(const char *what)
    {
        if (!on) return;
        double x = now();
        fprintf(stderr, "[wfstdec] %-22s %9.3f ms\n", what, x - t);
        t = x;
    }
};

enum { PH_SEARCH = 0, PH_RECORD = 1, PH_FINAL = 2, PH_COUNT = 3 };

// Streams of the library's own (default priority, per device, created once)
// on which groups of a batch run beside the caller's stream.
// (up to three search groups beside the caller's stream, or one stream for
// the incremental lattice pass)
constexpr int kGroupStreams = 3;
constexpr int kAuxStreams = kGroupStreams + 1;
// Token sets between the search's progress reports to the incremental
// lattice pass, and the largest batch that uses it (its blocks and the
// search's must be resident together: two per utterance, one per CU).
constexpr int kStreamK = 32;
constexpr int kStreamMaxUtts = 96;
// Record workgroups appended to the search launch of the last (longest)
// length group, and the token sets between the search's progress reports to
// them: the record pass of those utterances then ends with their search.
constexpr int kRecGroups = 96;
constexpr int kRecPublish = 16;
// The lattice regions with the incremental pass: this fraction of the
// one-shot regions (the pass keeps a few percent of the raw arcs; an
// overflow grows every buffer and decodes again)
constexpr int64_t kCompactDiv = 8;

hipStream_t aux_stream(int dev, int i)
{
    static std::mutex mu;
    static hipStream_t tab[64][kAuxStreams] = {};
    if (dev < 0 || dev >= 64 || i < 0 || i >= kAuxStreams) return nullptr;
    std::lock_guard<std::mutex> lk(mu);
    if (!tab[dev][i] && hipStreamCreateWithFlags(&tab[dev][i], hipStreamNonBlocking) != hipSuccess)
        tab[dev][i] = nullptr;
    return tab[dev][i];
}

// run_batch result: the word-lattice tables overflowed (final, not retried)
constexpr int kWordCapacity = -10;

// Per-frame offset arrays of an utterance: survivors, emitting and epsilon
// record regions, lattice output, emitting and epsilon record counts, and the
// the search's reservations (arrays of their own with the incremental
// lattice pass).
constexpr int kOffsetArrays = 8;

// Element counts of the workspace regions summed over a batch.
struct Totals {
    int64_t sv = 0, le = 0, lx = 0, fo = 0, kp = 0, pa = 0;
};

// Regions of one utterance of Tu frames, appended after those in `tot`.
void layout_utt(int64_t Tu, const Sizes &z, bool lattice, int depth, Totals &tot, UttLayout &l, int64_t cdiv = 1)
{
    l.sv0 = tot.sv;
    // survivor indices are 32-bit; one frame may reach capF tokens
    l.svcap = std::min<int64_t>((Tu + 1) * z.capA + z.capF, std::numeric_limits<int32_t>::max());
    tot.sv += l.svcap;
    // with a lattice, a set's emitting region holds one lattice record per
    // emitting out-arc of its tokens, its epsilon region one per epsilon
    // out-arc
    l.le0 = tot.le;
    l.lecap = lattice ? std::max<int64_t>((Tu * z.capA + z.capF) * z.em / cdiv, z.capF * z.em) : 0;
    tot.le += l.lecap;
    l.lx0 = tot.lx;
    l.lxcap = lattice ? std::max<int64_t>(((Tu + 1) * z.capA + z.capF) * z.xm / cdiv, z.capF * z.xm) : 0;
    tot.lx += l.lxcap;
    l.fo0 = tot.fo;
    tot.fo += Tu + 2;
    l.kept0 = tot.kp;
    tot.kp += std::max<int64_t>(Tu, 1);
    l.path0 = tot.pa;
    l.pathcap = (Tu + 1) * (depth + 1) + 1;
    tot.pa += l.pathcap;
    l.lo0 = 0;
}

// Option-derived kernel parameters shared by every decode entry point.
void set_params(Params &p, const Graph &G, int U, int L, const wfst_decode_opts &o, float thr,
                const wfst_debug_opts &dbg, const Sizes &z, int n_blank, bool stream)
{
    p.g = G.d;
    p.U = U;
    p.L = L;
    p.beam = o.beam;
    p.max_active = o.max_active;
    p.lattice_beam = o.lattice_beam;
    p.lattice = o.lattice_beam >= 0.0f ? 1 : 0;
    p.n_blank = n_blank;
    p.frame_stride = std::max(1, o.frame_stride);
    p.blank_thr = thr;
    p.lds_fill = limit_or(dbg.lds_fill, 1 << 30);
    p.gen_lds = limit_or(dbg.queue_cap, 1 << 30);
    p.profile = (o.flags & WFST_PROFILE_STEPS) ? 1 : 0;
    p.rec_fill = limit_or(dbg.record_fill, 1 << 30);
    p.rec_big_fill = limit_or(dbg.record_big_fill, 1 << 30);
    p.lat_lds = dbg.lattice_lds < 0 ? 0 : limit_or(dbg.lattice_lds, 1 << 30);
    p.lat_pipe = dbg.lattice_pipe < 0 ? -1 : (dbg.lattice_pipe > 0 ? 1 : 0);
    p.lat_spin = dbg.lattice_spin;
    p.hash_mul = dbg.permute ? kHashMulAlt : kHashMul;
    p.reverse = dbg.permute ? 1 : 0;
    p.capG = 8192;
    while (p.capG < z.capT) p.capG *= 2;
    p.capO = z.capO;
    // the incremental lattice pass: chunks of stream_k token sets, rings
    // for two chunks' raw records
    p.stream_k = 0;
    p.rce = p.rcx = 0;
    if (stream && p.lattice && (o.flags & WFST_INCREMENTAL_LATTICE) && dbg.lattice_chunk >= 0) {
        p.stream_k = dbg.lattice_chunk > 0 ? dbg.lattice_chunk : kStreamK;
        const int64_t per = 2 * p.stream_k * z.capA + 2 * z.capF;
        p.rce = per * z.em;
        p.rcx = per * z.xm;
        if (dbg.lattice_ring > 0) {
            p.rce = std::min<int64_t>(p.rce, dbg.lattice_ring);
            p.rcx = std::min<int64_t>(p.rcx, dbg.lattice_ring);
        }
    }
}

// Carve every workspace buffer of U utterances with the region totals
// `tot` from the arena (a measuring arena only adds up the size).  The
// per-frame offset arrays come from *fo_all (kOffsetArrays arrays of tot.fo
// entries).
void carve_ws(Arena &a, Params &p, int U, const Totals &tot, UttLayout **d_lay, int64_t **fo_all)
{
    const bool lattice = p.lattice != 0;
    p.st = a.get<UttState>(U);
    *d_lay = a.get<UttLayout>(U);
    p.lay = *d_lay;
    p.gkeys = a.get<uint32_t>(U * p.capG);
    p.gvals = a.get<uint32_t>(U * p.capG);
    p.gslots = a.get<int32_t>(U * p.capG);
    p.gspill = a.get<uint2>(U * 2 * p.capO);
    p.sv_state = a.get<int32_t>(tot.sv);
    p.sv_key = a.get<uint32_t>(tot.sv);
    p.sv_prev = a.get<int32_t>(tot.sv);
    p.sv_arc = a.get<int32_t>(tot.sv);
    p.sv_ebeg = a.get<int32_t>(tot.sv);
    p.sv_epre = a.get<int32_t>(tot.sv);
    p.sv_win = a.get<unsigned long long>(tot.sv);
    p.e_key = lattice ? a.get<uint32_t>(tot.sv) : nullptr;
    p.lat_e = lattice ? a.get<int4>(tot.le) : nullptr;
    p.lat_x = lattice ? a.get<int4>(tot.lx) : nullptr;
    p.ex_e = lattice ? a.get<float>(tot.le) : nullptr;
    p.ex_x = lattice ? a.get<float>(tot.lx) : nullptr;
    *fo_all = a.get<int64_t>(kOffsetArrays * tot.fo);
    p.blank_ids = a.get<int32_t>(p.n_blank);
    p.cut_arr = a.get<uint32_t>(tot.fo);
    p.kept = a.get<int32_t>(tot.kp);
    p.path_arc = a.get<int32_t>(tot.pa);
    p.path_frame = a.get<int32_t>(tot.pa);
    p.path_packed = a.get<int2>(tot.pa);
    const int64_t fo = tot.fo;
    int64_t *f = *fo_all;
    p.sv_off = f;
    p.le_off = f ? f + fo : nullptr;
    p.lx_off = f ? f + 2 * fo : nullptr;
    p.lo_off = f ? f + 3 * fo : nullptr;
    p.le_cnt = f ? f + 4 * fo : nullptr;
    p.lx_cnt = f ? f + 5 * fo : nullptr;
    // the reservations: separate arrays when the incremental lattice pass
    // writes compact offsets into le_off / lx_off while the search still
    // reserves (possibly on another chiplet), else the same arrays
    p.rle_off = p.stream_k && f ? f + 6 * fo : p.le_off;
    p.rlx_off = p.stream_k && f ? f + 7 * fo : p.lx_off;
    if (p.stream_k || p.rec_wg) {
        // progress counts, then the record workgroups' item counter
        p.prog = a.get<int32_t>(U + 1);
        p.rec_next = p.prog + U;
    }
    if (p.stream_k) {
        p.rng_e = a.get<int4>(U * p.rce);
        p.rng_ee = a.get<float>(U * p.rce);
        p.rng_x = a.get<int4>(U * p.rcx);
        p.rng_xe = a.get<float>(U * p.rcx);
        p.rkeys = a.get<uint32_t>(U * p.capG);
        p.rvals = a.get<int32_t>(U * p.capG);
    }
}

// The word-level lattice of every utterance with a path (after lattice
// pruning, on stream s, with the decode's workspace still in place): the
// forward pass over (node, word prefix) in word_kernel.hip, then the listed
// sequences written out and copied to the results, sorted by cost and
// sequence.  Capacities start from the lattice sizes and grow on overflow.
int run_words(const Graph &G, Params &p, int U, const std::vector<UttLayout> &lay, const std::vector<UttState> &st,
              const Totals &tot, hipStream_t s, std::vector<wfst_result *> &out)
{
    int64_t maxk = 1;
    for (int u = 0; u < U; u++)
        if (st[u].status == WFST_OK) maxk = std::max<int64_t>(maxk, st[u].lat_kept);
    int64_t capH = 4096;
    while (capH < 32 * maxk) capH *= 2;
    std::vector<int32_t> on(static_cast<size_t>(4) * U);
    for (int attempt = 0; attempt < 4; attempt++) {
        const int64_t capW = capH;
        WordWs ws{};
        ws.capH = capH;
        ws.capW = capW;
        auto carve = [&](Arena &a) {
            ws.hkey = a.get<unsigned long long>(U * capH);
            ws.hval = a.get<uint32_t>(U * capH);
            ws.hnext = a.get<int32_t>(U * capH);
            ws.ents = a.get<int32_t>(U * capH);
            ws.heads = a.get<int32_t>(tot.sv);
            ws.tkey = a.get<unsigned long long>(U * capW);
            ws.tdep = a.get<int32_t>(U * capW);
            ws.tbest = a.get<uint32_t>(U * capW);
            ws.out_id = a.get<int2>(U * (capW + 1));
            ws.out_n = a.get<int32_t>(4 * U);
            ws.root_best = a.get<uint32_t>(U);
            ws.set_start = a.get<int32_t>(tot.fo);
        };
        Arena measure;
        carve(measure);
        ArenaLease lease;
        hipError_t e = lease.acquire(G.device, measure.off, 1);
        if (e != hipSuccess) return hip_fail(e, "decode: word-lattice workspace");
        Arena arena;
        arena.base = static_cast<char *>(lease.ptr);
        carve(arena);
        auto chk = [&](hipError_t r) {
            if (e == hipSuccess && r != hipSuccess) e = r;
        };
        chk(launch_word(p, ws, s));
        chk(hipMemcpyAsync(on.data(), ws.out_n, on.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s));
        chk(hipStreamSynchronize(s));
        if (e != hipSuccess) return hip_fail(e, "decode: word lattice");
        bool over = false;
        for (int u = 0; u < U; u++)
            if (st[u].status == WFST_OK && on[4 * u + 2] != 0) over = true;
        if (over) {
            capH *= 8;
            continue;
        }
        // listed sequences: offsets (n + 1 per utterance) and words
        std::vector<int64_t> bseq(static_cast<size_t>(U)), bword(static_cast<size_t>(U));
        int64_t ns = 0, nw = 0;
        for (int u = 0; u < U; u++) {
            bseq[u] = ns;
            bword[u] = nw;
            if (st[u].status != WFST_OK) continue;
            ns += on[4 * u];
            nw += on[4 * u + 1];
        }
        const size_t b_off = ((static_cast<size_t>(ns + U) * 8) + 255) & ~static_cast<size_t>(255);
        const size_t b_words = ((static_cast<size_t>(std::max<int64_t>(nw, 1)) * 4) + 255) & ~static_cast<size_t>(255);
        const size_t b_base = static_cast<size_t>(U) * 8;
        std::shared_ptr<LatBuf> obuf;
        e = lat_take(G.device, b_off + b_words + 2 * b_base, false, obuf);
        if (e != hipSuccess) return hip_fail(e, "decode: word-lattice output");
        char *ob = static_cast<char *>(obuf->p);
        int64_t *d_off = reinterpret_cast<int64_t *>(ob);
        int32_t *d_words = reinterpret_cast<int32_t *>(ob + b_off);
        int64_t *d_bseq = reinterpret_cast<int64_t *>(ob + b_off + b_words);
        int64_t *d_bword = d_bseq + U;
        chk(hipMemcpyAsync(d_bseq, bseq.data(), b_base, hipMemcpyHostToDevice, s));
        chk(hipMemcpyAsync(d_bword, bword.data(), b_base, hipMemcpyHostToDevice, s));
        chk(launch_word_flatten(p, ws, d_off, d_words, d_bseq, d_bword, s));
        std::vector<int64_t> h_off(static_cast<size_t>(ns + U));
        std::vector<int32_t> h_words(static_cast<size_t>(std::max<int64_t>(nw, 1)));
        std::vector<int2> h_id;
        if (ns + U > 0) chk(hipMemcpyAsync(h_off.data(), d_off, (ns + U) * 8, hipMemcpyDeviceToHost, s));
        if (nw > 0) chk(hipMemcpyAsync(h_words.data(), d_words, nw * 4, hipMemcpyDeviceToHost, s));
        std::vector<std::vector<int2>> ids(static_cast<size_t>(U));
        for (int u = 0; u < U; u++) {
            if (st[u].status != WFST_OK || on[4 * u] == 0) continue;
            ids[u].resize(static_cast<size_t>(on[4 * u]));
            chk(hipMemcpyAsync(ids[u].data(), ws.out_id + u * (capW + 1), on[4 * u] * sizeof(int2),
                               hipMemcpyDeviceToHost, s));
        }
        chk(hipStreamSynchronize(s));
        if (e != hipSuccess) return hip_fail(e, "decode: word-lattice results");
        for (int u = 0; u < U; u++) {
            wfst_result *r = out[u];
            r->has_words = true;
            r->w_off.assign(1, 0);
            r->w_words.clear();
            r->w_cost.clear();
            if (st[u].status != WFST_OK) continue;
            const int n = on[4 * u];
            const int64_t *of = h_off.data() + bseq[u] + u;
            const int32_t *wd = h_words.data() + bword[u];
            // sort by (cost key, sequence)
            std::vector<int> idx(static_cast<size_t>(n));
            std::iota(idx.begin(), idx.end(), 0);
            std::sort(idx.begin(), idx.end(), [&](int a, int b) {
                const uint32_t ka = static_cast<uint32_t>(ids[u][a].y), kb = static_cast<uint32_t>(ids[u][b].y);
                if (ka != kb) return ka < kb;
                return std::lexicographical_compare(wd + of[a], wd + of[a + 1], wd + of[b], wd + of[b + 1]);
            });
            r->w_off.reserve(static_cast<size_t>(n) + 1);
            r->w_cost.reserve(static_cast<size_t>(n));
            for (int q : idx) {
                r->w_words.insert(r->w_words.end(), wd + of[q], wd + of[q + 1]);
                r->w_off.push_back(static_cast<int64_t>(r->w_words.size()));
                const uint32_t k = static_cast<uint32_t>(ids[u][q].y);
                const uint32_t bits = (k >> 31) ? (k & 0x7FFFFFFFu) : ~k;
                float c;
                std::memcpy(&c, &bits, 4);
                r->w_cost.push_back(c);
            }
            r->stats.word_sequences = n;
        }
        return WFST_OK;
    }
    set_error("decode: the word-lattice tables overflowed (more than %lld entries per utterance)",
              static_cast<long long>(capH / 8));
    return WFST_ECAPACITY;
}

// One attempt at decoding the batch with the given buffer sizes.  Returns
// WFST_OK, an error, or WFST_ECAPACITY when a buffer overflowed.
int run_batch(const Graph &G, int U, const float *const *ll_in, const int32_t *T_in, int L,
              const wfst_decode_opts &o, float thr, hipStream_t s, const Sizes &z,
              std::vector<wfst_result *> &out_in, double t_start, const wfst_debug_opts &dbg)
{
    // Utterances in order of length: a group of similar lengths runs its
    // search, record and final passes on a stream of its own, so a group of
    // short utterances does its record and lattice passes while the longer
    // ones still search.  Results do not depend on the grouping.
    std::vector<int> perm(static_cast<size_t>(U));
    std::iota(perm.begin(), perm.end(), 0);
    std::stable_sort(perm.begin(), perm.end(), [&](int a, int b) { return T_in[a] < T_in[b]; });
    std::vector<const float *> ll_v(static_cast<size_t>(U));
    std::vector<int32_t> T_v(static_cast<size_t>(U));
    std::vector<wfst_result *> out(static_cast<size_t>(U));
    for (int i = 0; i < U; i++) {
        ll_v[i] = ll_in[perm[i]];
        T_v[i] = T_in[perm[i]];
        out[i] = out_in[perm[i]];
    }
    const float *const *ll = ll_v.data();
    const int32_t *T = T_v.data();
    const bool lattice = o.lattice_beam >= 0.0f;
    const int depth = G.eps_depth;
    Timer tm;
    tm.on = (o.flags & WFST_PROFILE) != 0 && G.device >= 0 && G.device < 64;
    tm.dev = G.device;

    std::vector<UttLayout> lay(U);
    Totals tot;
    // with the incremental lattice pass the lattice regions only take the
    // arcs that pass its pruning, a small part of the raw lattice
    // launches that wait on others (see WaitGuard)
    const bool want_inc = lattice && (o.flags & WFST_INCREMENTAL_LATTICE) && U <= kStreamMaxUtts &&
                          dbg.lattice_chunk >= 0;
    const int rec_want = dbg.record_groups < 0 ? 0 : (dbg.record_groups > 0 ? dbg.record_groups : kRecGroups);
    const int ng_est = std::max(1, std::min(1 + kGroupStreams, U / 16));
    const bool want_rec = !want_inc && rec_want > 0 && (ng_est > 1 || dbg.record_groups > 0) &&
                          U + rec_want <= device_cus(G.device);
    WaitGuard wguard;
    const bool waits = (want_inc || want_rec) && wguard.take(G.device);
    const bool incremental = want_inc && waits;
    for (int u = 0; u < U; u++) layout_utt(T[u], z, lattice, depth, tot, lay[u], incremental ? kCompactDiv : 1);
    const int64_t fo = tot.fo, kp = tot.kp;

    // the blank-like units: the set when given, else the single blank unit
    std::vector<int32_t> blank_h;
    if (o.num_blank_ids > 0) blank_h.assign(o.blank_ids, o.blank_ids + o.num_blank_ids);
    else blank_h.push_back(o.blank_id);
    Params p{};
    set_params(p, G, U, L, o, thr, dbg, z, static_cast<int32_t>(blank_h.size()), incremental);
    // record workgroups beside the last length group's search (the
    // incremental pass records beside the search itself)
    const int rec_wg = want_rec && waits ? rec_want : 0;
    const int rec_pub = dbg.record_publish > 0 ? dbg.record_publish : kRecPublish;
    p.rec_wg = rec_wg;
    WallTrace wt;
    UttLayout *d_lay = nullptr;
    int64_t *fo_all = nullptr;
    Arena measure;
    carve_ws(measure, p, U, tot, &d_lay, &fo_all);
    ArenaLease lease;
    {
        const hipError_t ae = lease.acquire(G.device, measure.off);
        if (ae != hipSuccess) {
            set_error("decode: workspace allocation of %zu bytes: %s", measure.off, hipGetErrorString(ae));
            return ae == hipErrorOutOfMemory ? WFST_ENOMEM : WFST_EDEVICE;
        }
    }
    Arena arena;
    arena.base = static_cast<char *>(lease.ptr);
    carve_ws(arena, p, U, tot, &d_lay, &fo_all);
    wt.mark("allocate");
    if (wt.on) {
        const double gib = 1.0 / (1024.0 * 1024.0 * 1024.0);
        fprintf(stderr, "[wfstdec] workspace %.2f GiB: survivors %.2f, emitting regions %.2f, epsilon regions %.2f\n",
                measure.off * gib, tot.sv * (lattice ? 36.0 : 32.0) * gib, tot.le * 20.0 * gib, tot.lx * 20.0 * gib);
    }

    std::vector<UttState> st(U);
    for (int u = 0; u < U; u++) {
        std::memset(&st[u], 0, sizeof(UttState));
        st[u].ll = ll[u];
        st[u].T = T[u];
    }
    hipError_t e = hipSuccess;
    auto chk = [&](hipError_t r) {
        if (e == hipSuccess && r != hipSuccess) e = r;
    };
    // host staging of the call's transfers: states, layouts and blank ids
    // in; states, kept frames, packed paths and (with token sets) the set
    // offsets out
    const bool want_tokens = (o.flags & WFST_RECORD_TOKENS) != 0;
    const bool all_frames = !(thr < std::numeric_limits<float>::infinity()) && p.frame_stride == 1;
    auto rnd = [](size_t b) { return (b + 255) & ~static_cast<size_t>(255); };
    const size_t g_lay = rnd(U * sizeof(UttState));
    const size_t g_blank = g_lay + rnd(U * sizeof(UttLayout));
    const size_t g_kept = g_blank + rnd(blank_h.size() * sizeof(int32_t));
    const size_t g_path = g_kept + (all_frames ? 0 : rnd(static_cast<size_t>(kp) * sizeof(int32_t)));
    const size_t g_fo = g_path + rnd(static_cast<size_t>(std::max<int64_t>(tot.pa, 1)) * sizeof(int2));
    const size_t g_end = g_fo + (want_tokens ? rnd(static_cast<size_t>(fo) * sizeof(int64_t)) : 0);
    PinnedLease stage;
    stage.acquire(G.device, g_end);
    UttState *h_st = reinterpret_cast<UttState *>(stage.ptr);
    UttLayout *h_lay = reinterpret_cast<UttLayout *>(stage.ptr + g_lay);
    int32_t *h_blank = reinterpret_cast<int32_t *>(stage.ptr + g_blank);
    const int32_t *kept_h = reinterpret_cast<const int32_t *>(stage.ptr + g_kept);
    const int2 *paths_h = reinterpret_cast<const int2 *>(stage.ptr + g_path);
    const int64_t *fo_h = reinterpret_cast<const int64_t *>(stage.ptr + g_fo);
    std::memcpy(h_st, st.data(), U * sizeof(UttState));
    std::memcpy(h_lay, lay.data(), U * sizeof(UttLayout));
    std::memcpy(h_blank, blank_h.data(), blank_h.size() * sizeof(int32_t));
    chk(hipMemcpyAsync(p.st, h_st, U * sizeof(UttState), hipMemcpyHostToDevice, s));
    chk(hipMemcpyAsync(d_lay, h_lay, U * sizeof(UttLayout), hipMemcpyHostToDevice, s));
    chk(launch_zero(fo_all, kOffsetArrays * fo * sizeof(int64_t), s));
    // the progress counts start at 0: a stale count from an earlier decode
    // would let the lattice pass read token sets before they exist
    if (p.prog) chk(launch_zero(p.prog, (U + 1) * sizeof(int32_t), s));
    chk(hipMemcpyAsync(const_cast<int32_t *>(p.blank_ids), h_blank, blank_h.size() * sizeof(int32_t),
                       hipMemcpyHostToDevice, s));
    chk(launch_classify(p, s));
    // decoded frames are at most the frames: size the per-frame launches by T
    int Tmax = 0;
    for (int u = 0; u < U; u++) Tmax = std::max(Tmax, T[u]);
    wt.mark("setup");

    // one group per 16 utterances, at most one per stream
    // With the incremental lattice pass the whole batch is one search
    // launch on the caller's stream and one lattice launch beside it on a
    // stream of the library's (the records are made during the search, so
    // length groups gain nothing, and every stream more may share a hardware
    // queue with a waiting lattice launch).  Otherwise one group per 16
    // utterances, at most one per stream.
    const bool streaming = p.stream_k > 0;
    const int ng = streaming ? 1 : std::max(1, std::min(1 + kGroupStreams, U / 16));
    std::vector<hipStream_t> gs(static_cast<size_t>(ng), s), ls(static_cast<size_t>(ng), nullptr);
    std::vector<hipEvent_t> evs;
    for (int g = 1; g < ng; g++) {
        gs[g] = aux_stream(G.device, g - 1);
        if (!gs[g]) chk(hipErrorOutOfMemory);
    }
    if (streaming) {
        ls[0] = aux_stream(G.device, kGroupStreams);
        if (!ls[0]) chk(hipErrorOutOfMemory);
    }
    if ((ng > 1 || streaming) && e == hipSuccess) {
        hipEvent_t fork = event_pool().get(G.device);
        if (!fork) chk(hipErrorOutOfMemory);
        else {
            evs.push_back(fork);
            chk(hipEventRecord(fork, s));
            for (int g = 1; g < ng; g++) chk(hipStreamWaitEvent(gs[g], fork, 0));
            if (streaming) chk(hipStreamWaitEvent(ls[0], fork, 0));
        }
    }
    // Group bounds: equal groups, except that with four groups the last
    // (longest) one is half as large and the first takes the rest: after the
    // last search ends only that group's record and lattice passes remain.
    std::vector<int> gb(static_cast<size_t>(ng) + 1);
    for (int g = 0; g <= ng; g++) gb[g] = static_cast<int>(static_cast<int64_t>(U) * g / ng);
    if (ng == 4) {
        static const int kEighths[5] = {0, 3, 5, 7, 8};
        for (int g = 0; g <= ng; g++) gb[g] = static_cast<int>(static_cast<int64_t>(U) * kEighths[g] / 8);
    }
    for (int g = 0; g < ng && e == hipSuccess; g++) {
        const int u0 = gb[g];
        const int u1 = gb[g + 1];
        Params pg = p;
        pg.U = u1 - u0;
        pg.st = p.st + u0;
        pg.lay = p.lay + u0;
        pg.gkeys = p.gkeys + u0 * p.capG;
        pg.gvals = p.gvals + u0 * p.capG;
        pg.gslots = p.gslots + u0 * p.capG;
        pg.gspill = p.gspill + static_cast<int64_t>(u0) * 2 * p.capO;
        if (streaming) {
            pg.prog = p.prog + u0;
            pg.rng_e = p.rng_e + u0 * p.rce;
            pg.rng_ee = p.rng_ee + u0 * p.rce;
            pg.rng_x = p.rng_x + u0 * p.rcx;
            pg.rng_xe = p.rng_xe + u0 * p.rcx;
            pg.rkeys = p.rkeys + u0 * p.capG;
            pg.rvals = p.rvals + u0 * p.capG;
        }
        int Tg = 0;
        for (int u = u0; u < u1; u++) Tg = std::max(Tg, T[u]);
        pg.pub_k = p.stream_k;
        pg.rec_wg = 0;
        // (by default only when the batch has several groups: alone, a
        // group's record pass after its search is short and all parallel,
        // and the progress reports would slow its search for nothing)
        const bool fused = rec_wg > 0 && g == ng - 1 && pg.U <= kRecMaxUtts && (ng > 1 || dbg.record_groups > 0);
        if (fused) {
            pg.prog = p.prog + u0;
            pg.pub_k = rec_pub;
            pg.rec_wg = rec_wg;
            pg.rec_tmax = Tg;
        }
        const hipStream_t q = gs[g];
        tm.start(q);
        chk(launch_search(pg, q));
        tm.stop(PH_SEARCH, q);
        if (streaming) {
            // the incremental lattice pass follows the search on its own
            // stream; the final passes wait for it
            tm.start(ls[g]);
            chk(launch_lattice_stream(pg, ls[g]));
            tm.stop(PH_RECORD, ls[g]);
            hipEvent_t done = event_pool().get(G.device);
            if (!done) {
                chk(hipErrorOutOfMemory);
                break;
            }
            evs.push_back(done);
            chk(hipEventRecord(done, ls[g]));
            chk(hipStreamWaitEvent(q, done, 0));
        } else {
            // with record workgroups in the search launch only the sets
            // beyond their LDS table are left
            tm.start(q);
            chk(fused ? launch_record_large(pg, q) : launch_record(pg, Tg, q));
            tm.stop(PH_RECORD, q);
        }
        tm.start(q);
        chk(launch_final(pg, q));
        chk(launch_finish(pg, q));
        tm.stop(PH_FINAL, q);
        if (g > 0) {
            hipEvent_t join = event_pool().get(G.device);
            if (!join) {
                chk(hipErrorOutOfMemory);
                break;
            }
            evs.push_back(join);
            chk(hipEventRecord(join, q));
            chk(hipStreamWaitEvent(s, join, 0));
        }
    }
    tm.start(s);
    chk(launch_pack_paths(p, s));
    tm.stop(PH_FINAL, s);
    wt.mark("enqueue frames");
    chk(hipMemcpyAsync(h_st, p.st, U * sizeof(UttState), hipMemcpyDeviceToHost, s));
    chk(hipStreamSynchronize(s));
    // the groups' streams are done once s is (after an error too, before the
    // workspace is given back)
    for (int g = 1; g < ng; g++) chk(hipStreamSynchronize(gs[g]));
    for (int g = 0; streaming && g < ng; g++) chk(hipStreamSynchronize(ls[g]));
    for (hipEvent_t x : evs) event_pool().put(G.device, x);
    std::memcpy(st.data(), h_st, U * sizeof(UttState));
    wt.mark("wait search");
    if (wt.on) {
        int64_t gf = 0;
        for (int u = 0; u < U; u++) gf += st[u].gframes;
        fprintf(stderr, "[wfstdec] frames redone with the device-memory table: %lld\n", static_cast<long long>(gf));
    }
    if (e != hipSuccess) return hip_fail(e, "decode: search");
    for (int u = 0; u < U; u++)
        if (st[u].status == WFST_ECAPACITY) return WFST_ECAPACITY;
    for (int u = 0; u < U; u++) {
        if (st[u].status == kStatusNoBackPointer)
            return fail(WFST_EDEVICE, "decode: internal error, a surviving token without a back-pointer");
        if (st[u].status == kStatusStreamTimeout)
            return fail(WFST_EDEVICE, "decode: internal error, a pass beside the search stopped waiting for it");
        if (st[u].status == kStatusLatticeWait)
            return fail(WFST_EDEVICE, "decode: internal error, a lattice pass stopped waiting for its other waves");
    }

    std::shared_ptr<LatBuf> lat_buf;
    std::shared_ptr<LatHost> lat_host;
    if (lattice) {
        int64_t tot = 0;
        for (int u = 0; u < U; u++) {
            lay[u].lo0 = tot;
            if (st[u].status == WFST_OK) tot += st[u].lat_kept;
        }
        lat_host = std::make_shared<LatHost>();
        lat_host->total = tot;
        // every stream is idle here: on failure nothing is left running
        const hipError_t le = lat_take(G.device, static_cast<size_t>(std::max<int64_t>(tot, 1)) * sizeof(int4),
                                       dbg.fail_lattice_alloc != 0, lat_buf);
        if (le != hipSuccess) return hip_fail(le, "decode: lattice output allocation");
        p.lat_out = static_cast<int4 *>(lat_buf->p);
        // (the stream has drained: the staged layouts were consumed)
        std::memcpy(h_lay, lay.data(), U * sizeof(UttLayout));
        chk(hipMemcpyAsync(d_lay, h_lay, U * sizeof(UttLayout), hipMemcpyHostToDevice, s));
        tm.start(s);
        chk(launch_lattice_emit(p, Tmax, s));
        tm.stop(PH_FINAL, s);
    }

    wt.mark("lattice output");
    if (lattice && (o.flags & WFST_WORD_LATTICE)) {
        const int wr = run_words(G, p, U, lay, st, tot, s, out);
        // the decode itself fit: more attempts with larger decode buffers
        // would not help the word tables
        if (wr == WFST_ECAPACITY) return kWordCapacity;
        if (wr != WFST_OK) return wr;
        wt.mark("word lattice");
    }
    // gather results
    // the set offsets serve only the token sets; the kept frames are every
    // frame when no frame can be skipped
    if (want_tokens)
        chk(hipMemcpyAsync(const_cast<int64_t *>(fo_h), p.sv_off, fo * sizeof(int64_t), hipMemcpyDeviceToHost, s));
    if (!all_frames)
        chk(hipMemcpyAsync(const_cast<int32_t *>(kept_h), p.kept, kp * sizeof(int32_t), hipMemcpyDeviceToHost, s));
    // the packed best paths, in utterance order
    int64_t path_total = 0;
    std::vector<int64_t> path_off(static_cast<size_t>(U), 0);
    for (int u = 0; u < U; u++) {
        path_off[u] = path_total;
        if (st[u].status == WFST_OK) path_total += st[u].path_len;
    }
    if (path_total > std::max<int64_t>(tot.pa, 1)) return fail(WFST_EDEVICE, "decode: internal error, path overflow");
    if (path_total)
        chk(hipMemcpyAsync(const_cast<int2 *>(paths_h), p.path_packed, path_total * sizeof(int2),
                           hipMemcpyDeviceToHost, s));
    for (int u = 0; u < U; u++) {
        wfst_result *r = out[u];
        const UttState &x = st[u];
        r->status = x.status;
        r->T = T[u];
        r->Tp = x.Tp;
        r->stats.frames = T[u];
        r->stats.frames_decoded = x.Tp;
        if (x.status != WFST_OK) continue;
        r->cost = x.final_cost;
        r->final_state = user_state(G, x.final_state);
        r->reached_final = x.reached_final;
        r->path_arcs.resize(x.path_len);
        r->path_frames.resize(x.path_len);
        r->stats.tokens = x.n_tok;
        r->stats.tokens_last = x.n_last;
        r->stats.arcs_expanded = x.arcs_expanded;
        r->stats.eps_arcs = x.eps_arcs;
        r->stats.lattice_raw = x.le_cnt + x.lx_cnt;
        r->stats.lattice_kept = lattice ? x.lat_kept : 0;
        r->stats.lattice_incremental = p.stream_k ? x.lat_inc : r->stats.lattice_raw;
        r->stats.workspace_bytes = static_cast<int64_t>(measure.off);
        if (lattice) {
            r->lat_dev = lat_buf;
            r->lat_host = lat_host;
            r->lat_off = lay[u].lo0;
            r->lat_n = x.lat_kept;
        }
    }
    std::vector<std::vector<int32_t>> tst(U), tarc(U);
    std::vector<std::vector<uint32_t>> tkey(U);
    if (o.flags & WFST_RECORD_TOKENS) {
        chk(hipStreamSynchronize(s));
        for (int u = 0; u < U; u++) {
            if (st[u].status != WFST_OK) continue;
            const int64_t ntok = fo_h[lay[u].fo0 + st[u].Tp + 1];
            tst[u].resize(static_cast<size_t>(ntok));
            tkey[u].resize(static_cast<size_t>(ntok));
            tarc[u].resize(static_cast<size_t>(ntok));
            chk(hipMemcpyAsync(tst[u].data(), p.sv_state + lay[u].sv0, ntok * 4, hipMemcpyDeviceToHost, s));
            chk(hipMemcpyAsync(tkey[u].data(), p.sv_key + lay[u].sv0, ntok * 4, hipMemcpyDeviceToHost, s));
            chk(hipMemcpyAsync(tarc[u].data(), p.sv_arc + lay[u].sv0, ntok * 4, hipMemcpyDeviceToHost, s));
        }
    }
    chk(hipStreamSynchronize(s));
    wt.mark("copy results");
    if (e != hipSuccess) return hip_fail(e, "decode: results");

    double ph[PH_COUNT] = {0, 0, 0};
    int nexp = 0;
    // the search launches' span, on the clock of the first one's start event
    hipEvent_t s_ref = nullptr;
    double s_lo = 0.0, s_hi = 0.0;
    for (const auto &x : tm.spans) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, x.a, x.b) == hipSuccess) ph[x.kind] += ms;
        if (x.kind != PH_SEARCH) continue;
        nexp++;
        if (!s_ref) s_ref = x.a;
        float a = 0.0f, b = 0.0f;
        if (hipEventElapsedTime(&a, s_ref, x.a) == hipSuccess && hipEventElapsedTime(&b, s_ref, x.b) == hipSuccess) {
            s_lo = std::min(s_lo, static_cast<double>(a));
            s_hi = std::max(s_hi, static_cast<double>(b));
        }
    }
    const double wall = std::chrono::duration<double, std::milli>(
                            std::chrono::steady_clock::now().time_since_epoch()).count() - t_start;
    for (int u = 0; u < U; u++) {
        wfst_result *r = out[u];
        for (size_t i = 0; i < r->path_arcs.size(); i++) {
            r->path_arcs[i] = paths_h[path_off[u] + i].x;
            r->path_frames[i] = paths_h[path_off[u] + i].y;
        }
        if (all_frames) {
            r->kept.resize(static_cast<size_t>(std::max(st[u].Tp, 0)));
            std::iota(r->kept.begin(), r->kept.end(), 0);
        } else {
            r->kept.assign(kept_h + lay[u].kept0, kept_h + lay[u].kept0 + st[u].Tp);
        }
        r->stats.decode_ms = wall;
        r->stats.search_ms = ph[PH_SEARCH];
        r->stats.record_ms = ph[PH_RECORD];
        r->stats.final_ms = ph[PH_FINAL];
        r->stats.search_launches = nexp;
        r->stats.search_span_ms = s_hi - s_lo;
        if (p.profile) {
            int khz = 0;
            if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, G.device) == hipSuccess && khz > 0)
            {
                for (int i = 0; i < 7; i++)
                    r->stats.search_phase_ms[i] = static_cast<double>(st[u].phase_ticks[i]) / khz;
                r->stats.backtrace_ms = static_cast<double>(st[u].finish_ticks[0]) / khz;
                r->stats.lattice_prune_ms = static_cast<double>(st[u].finish_ticks[1]) / khz;
            }
        }
        if ((o.flags & WFST_RECORD_TOKENS) && r->status == WFST_OK) {
            // token sets sorted by state for the caller
            const int Tp = st[u].Tp;
            r->has_tokens = true;
            r->tok_off.assign(fo_h + lay[u].fo0, fo_h + lay[u].fo0 + Tp + 2);
            const int64_t ntok = r->tok_off.back();
            r->tok_state.resize(static_cast<size_t>(ntok));
            r->tok_cost.resize(static_cast<size_t>(ntok));
            r->tok_arc.resize(static_cast<size_t>(ntok));
            std::vector<int64_t> idx;
            for (int j = 0; j <= Tp; j++) {
                const int64_t a = r->tok_off[j], b = r->tok_off[j + 1];
                idx.resize(static_cast<size_t>(b - a));
                std::iota(idx.begin(), idx.end(), a);
                std::sort(idx.begin(), idx.end(), [&](int64_t x, int64_t y) { return tst[u][x] < tst[u][y]; });
                for (int64_t i = a; i < b; i++) {
                    const int64_t q = idx[i - a];
                    const uint32_t k = tkey[u][q];
                    const uint32_t bits = (k >> 31) ? (k & 0x7FFFFFFFu) : ~k;
                    float c;
                    std::memcpy(&c, &bits, 4);
                    r->tok_state[i] = user_state(G, tst[u][q]);
                    r->tok_cost[i] = c;
                    r->tok_arc[i] = tarc[u][q];
                }
            }
        }
    }
    wt.mark("finish");
    return WFST_OK;
}

std::atomic<int64_t> &learned_capA()
{
    static std::atomic<int64_t> a{2048};
    return a;
}

// Buffer sizes before anything is learned from earlier decodes (capA, the
// average tokens per frame, is left to the caller).
Sizes initial_sizes(const Graph &G, const wfst_decode_opts &o)
{
    const int64_t N = G.d.n;
    Sizes z{};
    if (o.capacity_hint > 0) z.capF = std::min<int64_t>(o.capacity_hint, N);
    else if (o.max_active > 0) z.capF = std::min<int64_t>(N, o.max_active + o.max_active / 4 + 256);
    else z.capF = std::min<int64_t>(N, 65536);
    z.capT = std::min<int64_t>(N, std::max<int64_t>(16 * z.capF, 4096));
    // epsilon items of one generation are bounded by the candidates that
    // produce them
    const int64_t E = G.d.e;
    z.capO = std::min<int64_t>(E + 1, std::max<int64_t>(2 * z.capT, 65536));
    // lattice-record slots per token: what the last decodes on this graph
    // needed, else twice the graph's mean out-degrees
    z.em = G.rec_em.load();
    z.xm = G.rec_xm.load();
    if (z.em <= 0) z.em = std::max<int64_t>(2, 2 * G.d.n_emit / std::max<int64_t>(N, 1) + 1);
    if (z.xm <= 0) z.xm = std::max<int64_t>(1, 2 * G.d.n_eps / std::max<int64_t>(N, 1) + 1);
    z.capA = 0;
    return z;
}

// Checks of the decode options shared by every entry point; on success *thr
// is the log-domain blank threshold.
int check_opts(const Graph &G, const wfst_decode_opts &o, int32_t L, float *thr)
{
    if (!(o.beam > 0.0f)) return fail(WFST_EINVAL, "decode: beam must be > 0");
    if (std::isnan(o.lattice_beam)) return fail(WFST_EINVAL, "decode: lattice_beam is NaN");
    if (!(o.blank_threshold > 0.0f)) return fail(WFST_EINVAL, "decode: blank_threshold must be > 0");
    if (L < 1 || L < G.max_ilabel) return fail(WFST_EINVAL, "decode: L smaller than the largest ilabel");
    if (o.blank_id < 0 || o.blank_id >= L) return fail(WFST_EINVAL, "decode: blank_id out of range");
    if (o.num_blank_ids < 0 || (o.num_blank_ids > 0 && !o.blank_ids))
        return fail(WFST_EINVAL, "decode: bad blank-unit set");
    for (int i = 0; i < o.num_blank_ids; i++)
        if (o.blank_ids[i] < 0 || o.blank_ids[i] >= L) return fail(WFST_EINVAL, "decode: blank unit out of range");
    if (o.frame_stride < 0) return fail(WFST_EINVAL, "decode: negative frame_stride");
    if (o.capacity_hint < 0) return fail(WFST_EINVAL, "decode: negative capacity_hint");
    if ((o.flags & WFST_WORD_LATTICE) && !(o.lattice_beam >= 0.0f))
        return fail(WFST_EINVAL, "decode: the word-level lattice needs lattice_beam >= 0");
    *thr = o.blank_threshold > 1.0f ? std::numeric_limits<float>::infinity()
                                    : static_cast<float>(std::log(static_cast<double>(o.blank_threshold)));
    return WFST_OK;
}

int decode_impl(const wfst_graph *gh, int32_t n_utt, const float *const *loglikes, const int32_t *T,
                int32_t L, const wfst_decode_opts *opts, void *hip_stream, wfst_result **out_array)
{
    clear_error();
    const double t0 = std::chrono::duration<double, std::milli>(
                          std::chrono::steady_clock::now().time_since_epoch()).count();
    if (!gh || !opts || !out_array || !T || !loglikes) return fail(WFST_EINVAL, "decode: NULL argument");
    if (n_utt < 1) return fail(WFST_EINVAL, "decode: n_utt must be >= 1");
    for (int u = 0; u < n_utt; u++) out_array[u] = nullptr;
    const Graph &G = gh->g;
    const wfst_decode_opts o = *opts;
    const wfst_debug_opts dbg = debug_snapshot();
    float thr = 0.0f;
    {
        const int rc0 = check_opts(G, o, L, &thr);
        if (rc0 != WFST_OK) return rc0;
    }
    for (int u = 0; u < n_utt; u++) {
        if (T[u] < 0) return fail(WFST_EINVAL, "decode: negative T");
        if (T[u] > 0 && !loglikes[u]) return fail(WFST_EINVAL, "decode: NULL loglikes");
    }

    DeviceGuard dg(G.device);
    hipStream_t s = static_cast<hipStream_t>(hip_stream);

    std::vector<const float *> ll(loglikes, loglikes + n_utt);
    std::vector<std::unique_ptr<DevBuf>> host_copies;
    if (o.flags & WFST_LOGLIKES_HOST) {
        for (int u = 0; u < n_utt; u++) {
            auto b = std::make_unique<DevBuf>();
            b->device = G.device;
            size_t bytes = static_cast<size_t>(std::max(T[u], 1)) * L * sizeof(float);
            hipError_t e = hipMalloc(&b->p, bytes);
            if (e != hipSuccess) return hip_fail(e, "decode: loglikes copy");
            if (T[u]) {
                e = hipMemcpy(b->p, loglikes[u], static_cast<size_t>(T[u]) * L * sizeof(float), hipMemcpyHostToDevice);
                if (e != hipSuccess) return hip_fail(e, "decode: loglikes copy");
            }
            ll[u] = static_cast<const float *>(b->p);
            host_copies.push_back(std::move(b));
        }
    }

    std::vector<wfst_result *> res(n_utt);
    for (int u = 0; u < n_utt; u++) {
        res[u] = new (std::nothrow) wfst_result();
        if (!res[u]) {
            for (int v = 0; v < u; v++) delete res[v];
            return fail(WFST_ENOMEM, "decode: host allocation");
        }
    }
    const int64_t N = G.d.n;
    const int64_t E = G.d.e;
    Sizes z = initial_sizes(G, o);
    // average tokens per frame: start from what the last calls needed
    z.capA = std::min<int64_t>(z.capF, learned_capA().load());
    int rc = WFST_ECAPACITY;
    for (int attempt = 0; attempt < 8 && rc == WFST_ECAPACITY; attempt++) {
        if (attempt) {
            for (int u = 0; u < n_utt; u++) {
                delete res[u];
                res[u] = new (std::nothrow) wfst_result();
            }
            z.capF = std::min<int64_t>(N, z.capF * 4);
            z.capA = std::min<int64_t>(z.capF, z.capA * 4);
            z.capT = std::min<int64_t>(N, z.capT * 4);
            z.capO = std::min<int64_t>(E + 1, z.capO * 2);
            z.em *= 2;
            z.xm *= 2;
        }
        rc = run_batch(G, n_utt, ll.data(), T, L, o, thr, s, z, res, t0, dbg);
    }
    if (rc == WFST_OK) {
        int64_t cur = learned_capA().load();
        while (z.capA > cur && !learned_capA().compare_exchange_weak(cur, z.capA)) {
        }
        // the slots per token this batch needed, with a margin
        int64_t em = 1, xm = 1;
        for (int u = 0; u < n_utt; u++) {
            const wfst_stats &x = res[u]->stats;
            const int64_t tok = std::max<int64_t>(x.tokens, 1);
            em = std::max<int64_t>(em, (5 * x.arcs_expanded / tok) / 4 + 1);
            xm = std::max<int64_t>(xm, (5 * x.eps_arcs / tok) / 4 + 1);
        }
        G.rec_em.store(std::min(em, z.em));
        G.rec_xm.store(std::min(xm, z.xm));
    }
    if (rc == kWordCapacity) rc = WFST_ECAPACITY;   // message set by the word pass
    else if (rc == WFST_ECAPACITY) set_error("decode: buffers overflowed; raise capacity_hint");
    if (rc != WFST_OK) {
        for (int u = 0; u < n_utt; u++) delete res[u];
        return rc;
    }
    for (int u = 0; u < n_utt; u++) out_array[u] = res[u];
    return WFST_OK;
}

}  // namespace

extern "C" void wfst_default_opts(wfst_decode_opts *o)
{
    if (!o) return;
    o->beam = 16.0f;
    o->max_active = 0;
    o->lattice_beam = -1.0f;
    o->blank_threshold = 2.0f;
    o->blank_id = 0;
    o->flags = 0;
    o->capacity_hint = 0;
    o->blank_ids = nullptr;
    o->num_blank_ids = 0;
    o->frame_stride = 1;
}

extern "C" int wfst_decode(const wfst_graph *g, const float *loglikes, int32_t T, int32_t L,
                           const wfst_decode_opts *opts, void *hip_stream, wfst_result **out)
{
    if (!out) {
        set_error("wfst_decode: out is NULL");
        return WFST_EINVAL;
    }
    *out = nullptr;
    int rc = decode_impl(g, 1, &loglikes, &T, L, opts, hip_stream, out);
    if (rc != WFST_OK) return rc;
    if ((*out)->status == WFST_ENOPATH) set_error("wfst_decode: no surviving path");
    return (*out)->status;
}

extern "C" int wfst_decode_batch(const wfst_graph *g, int32_t n_utt, const float *const *loglikes,
                                 const int32_t *T, int32_t L, const wfst_decode_opts *opts,
                                 void *hip_stream, wfst_result **out_array)
{
    return decode_impl(g, n_utt, loglikes, T, L, opts, hip_stream, out_array);
}

extern "C" int wfst_result_status(const wfst_result *r)
{
    if (!r) return fail(WFST_EINVAL, "wfst_result_status: NULL result");
    return r->status;
}

extern "C" int wfst_result_best(const wfst_result *r, float *cost, int32_t *final_state,
                                int32_t *reached_final, int32_t *n, const int32_t **arcs,
                                const int32_t **frames)
{
    clear_error();
    if (!r) return fail(WFST_EINVAL, "wfst_result_best: NULL result");
    if (r->status != WFST_OK) return fail(r->status, "wfst_result_best: utterance has no path");
    if (cost) *cost = r->cost;
    if (final_state) *final_state = r->final_state;
    if (reached_final) *reached_final = r->reached_final;
    if (n) *n = static_cast<int32_t>(r->path_arcs.size());
    if (arcs) *arcs = r->path_arcs.data();
    if (frames) *frames = r->path_frames.data();
    return WFST_OK;
}

extern "C" int wfst_result_frames(const wfst_result *r, int32_t *num_frames, int32_t *num_decoded,
                                  const int32_t **orig_frame)
{
    clear_error();
    if (!r) return fail(WFST_EINVAL, "wfst_result_frames: NULL result");
    if (num_frames) *num_frames = r->T;
    if (num_decoded) *num_decoded = r->Tp;
    if (orig_frame) *orig_frame = r->kept.data();
    return WFST_OK;
}

namespace {

// The result's lattice in the batch's host copy, made on first use.
int lattice_host(const wfst_result *r, int64_t *n, const wfst_lat_arc **arcs, const char *who)
{
    if (!r->lat_host) {
        if (n) *n = 0;
        if (arcs) *arcs = nullptr;
        return WFST_OK;
    }
    LatHost &h = *r->lat_host;
    {
        std::lock_guard<std::mutex> lk(h.mu);
        if (!h.loaded) {
            h.arcs.resize(static_cast<size_t>(std::max<int64_t>(h.total, 1)));
            if (h.total) {
                DeviceGuard dg(r->lat_dev->device);
                hipError_t e = hipMemcpy(h.arcs.data(), r->lat_dev->p, h.total * sizeof(wfst_lat_arc),
                                         hipMemcpyDeviceToHost);
                if (e != hipSuccess) return hip_fail(e, who);
            }
            h.loaded = true;
        }
    }
    if (n) *n = r->lat_n;
    if (arcs) *arcs = h.arcs.data() + r->lat_off;
    return WFST_OK;
}

}  // namespace

extern "C" int wfst_result_lattice(const wfst_result *r, int64_t *n, const wfst_lat_arc **arcs)
{
    clear_error();
    if (!r) return fail(WFST_EINVAL, "wfst_result_lattice: NULL result");
    return lattice_host(r, n, arcs, "wfst_result_lattice: copy");
}

extern "C" int wfst_result_lattice_device(const wfst_result *r, int64_t *n, const wfst_lat_arc **arcs)
{
    clear_error();
    if (!r) return fail(WFST_EINVAL, "wfst_result_lattice_device: NULL result");
    if (n) *n = r->lat_n;
    if (arcs)
        *arcs = r->lat_dev ? reinterpret_cast<const wfst_lat_arc *>(static_cast<int4 *>(r->lat_dev->p) + r->lat_off)
                           : nullptr;
    return WFST_OK;
}

extern "C" int wfst_result_tokens(const wfst_result *r, int32_t j, int32_t *n, const int32_t **state,
                                  const float **cost, const int32_t **bp_arc)
{
    clear_error();
    if (!r) return fail(WFST_EINVAL, "wfst_result_tokens: NULL result");
    if (!r->has_tokens) return fail(WFST_EINVAL, "wfst_result_tokens: decoded without WFST_RECORD_TOKENS");
    if (j < 0 || j > r->Tp) return fail(WFST_EINVAL, "wfst_result_tokens: token set out of range");
    const int64_t a = r->tok_off[j], b = r->tok_off[j + 1];
    if (n) *n = static_cast<int32_t>(b - a);
    if (state) *state = r->tok_state.data() + a;
    if (cost) *cost = r->tok_cost.data() + a;
    if (bp_arc) *bp_arc = r->tok_arc.data() + a;
    return WFST_OK;
}

extern "C" int wfst_result_words(const wfst_result *r, int64_t *n, const int64_t **offsets, const int32_t **words,
                                 const float **costs)
{
    clear_error();
    if (!r) return fail(WFST_EINVAL, "wfst_result_words: NULL result");
    if (!r->has_words) return fail(WFST_EINVAL, "wfst_result_words: decoded without WFST_WORD_LATTICE");
    if (r->status != WFST_OK) return fail(r->status, "wfst_result_words: utterance has no path");
    if (n) *n = static_cast<int64_t>(r->w_cost.size());
    if (offsets) *offsets = r->w_off.data();
    if (words) *words = r->w_words.data();
    if (costs) *costs = r->w_cost.data();
    return WFST_OK;
}

extern "C" int wfst_result_stats(const wfst_result *r, wfst_stats *stats)
{
    clear_error();
    if (!r || !stats) return fail(WFST_EINVAL, "wfst_result_stats: NULL argument");
    *stats = r->stats;
    return WFST_OK;
}

extern "C" int wfst_result_summaries(const wfst_result *const *results, int32_t n, int32_t want_lattice,
                                     wfst_result_summary *out)
{
    clear_error();
    if (n < 0 || (n > 0 && (!results || !out))) return fail(WFST_EINVAL, "wfst_result_summaries: bad arguments");
    for (int32_t i = 0; i < n; i++)
        if (!results[i]) return fail(WFST_EINVAL, "wfst_result_summaries: NULL result");
    for (int32_t i = 0; i < n; i++) {
        const wfst_result *r = results[i];
        wfst_result_summary &s = out[i];
        s = wfst_result_summary{};
        s.status = r->status;
        s.num_frames = r->T;
        s.num_decoded = r->Tp;
        s.orig_frame = r->kept.data();
        s.cost = std::numeric_limits<float>::quiet_NaN();
        if (r->status == WFST_OK) {
            s.cost = r->cost;
            s.final_state = r->final_state;
            s.reached_final = r->reached_final;
            s.path_len = static_cast<int32_t>(r->path_arcs.size());
            s.path_arcs = r->path_arcs.data();
            s.path_frames = r->path_frames.data();
        }
        s.stats = r->stats;
        if (want_lattice) {
            const int rc = lattice_host(r, &s.lattice_n, &s.lattice, "wfst_result_summaries: lattice copy");
            if (rc != WFST_OK) return rc;
        }
    }
    return WFST_OK;
}

extern "C" void wfst_result_free(wfst_result *r) { delete r; }

extern "C" int wfst_set_debug_opts(const wfst_debug_opts *opts)
{
    clear_error();
    wfst_debug_opts o{};
    if (opts) {
        o = *opts;
        if (o.lds_fill < 0 || o.queue_cap < 0 || o.record_fill < 0 || o.record_big_fill < 0 ||
            o.lattice_lds < -1 || o.permute < 0 || o.fail_lattice_alloc < 0 || o.lattice_chunk < -1 ||
            o.lattice_ring < 0 || o.record_groups < -1 || o.record_publish < 0 || o.lattice_pipe < -1 ||
            o.lattice_spin < 0)
            return fail(WFST_EINVAL, "wfst_set_debug_opts: negative field");
    }
    DebugState &d = debug_state();
    std::lock_guard<std::mutex> lk(d.mu);
    d.o = o;
    return WFST_OK;
}

// ---------------------------------------------------------------------------
// wfst_decode_noalloc: one utterance with a fixed workspace and caller-owned
// outputs, for callers that cannot allocate.
// ---------------------------------------------------------------------------

namespace {

// The fixed workspace.  In host code `scratch` names a host-side stand-in,
// not device memory: its device address is taken once per device with
// hipGetSymbolAddress and only that address is used.
static __device__ __align__(256) char scratch[WFST_NOALLOC_SCRATCH_BYTES];

struct ScratchAddr {
    std::mutex mu;
    void *ptr[64] = {};
};

ScratchAddr &scratch_addr()
{
    static ScratchAddr a;   // no heap allocation, also on first use
    return a;
}

// Device address of the workspace on `device` (the current device).
hipError_t scratch_ptr(int device, void **out)
{
    if (device < 0 || device >= 64) return hipErrorInvalidDevice;
    ScratchAddr &a = scratch_addr();
    std::lock_guard<std::mutex> lk(a.mu);
    if (!a.ptr[device]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        a.ptr[device] = ptr;
    }
    *out = a.ptr[device];
    return hipSuccess;
}

// Workspace bytes of one utterance of T frames with sizes z.
size_t noalloc_bytes(const Graph &G, int U, int L, const wfst_decode_opts &o, float thr, const wfst_debug_opts &dbg,
                     const Sizes &z, int n_blank, int64_t T, Totals *tot_out, UttLayout *lay_out)
{
    Totals tot;
    UttLayout lay{};
    layout_utt(T, z, o.lattice_beam >= 0.0f, G.eps_depth, tot, lay);
    Params p{};
    set_params(p, G, U, L, o, thr, dbg, z, n_blank, false);
    Arena measure;
    UttLayout *d_lay = nullptr;
    int64_t *fo_all = nullptr;
    carve_ws(measure, p, U, tot, &d_lay, &fo_all);
    if (tot_out) *tot_out = tot;
    if (lay_out) *lay_out = lay;
    return measure.off;
}

int noalloc_impl(const wfst_graph *gh, const float *ll, int32_t T, int32_t L, const wfst_decode_opts *opts,
                 void *hip_stream, wfst_noalloc_out *out)
{
    clear_error();
    if (!gh || !opts || !out) return fail(WFST_EINVAL, "wfst_decode_noalloc: NULL argument");
    const Graph &G = gh->g;
    const wfst_decode_opts o = *opts;
    const bool lattice = o.lattice_beam >= 0.0f;
    out->status = WFST_EINVAL;
    out->path_len = 0;
    out->lattice_n = 0;
    out->num_decoded = 0;
    if (o.flags & (WFST_RECORD_TOKENS | WFST_LOGLIKES_HOST | WFST_PROFILE | WFST_PROFILE_STEPS | WFST_WORD_LATTICE))
        return fail(WFST_EINVAL, "wfst_decode_noalloc: token recording, host log-likelihoods and profiling "
                                 "are not available");
    if (T < 0) return fail(WFST_EINVAL, "wfst_decode_noalloc: negative T");
    if (T > 0 && !ll) return fail(WFST_EINVAL, "wfst_decode_noalloc: NULL loglikes");
    if ((out->path_cap > 0 && (!out->path_arcs || !out->path_frames)) || out->path_cap < 0 ||
        (out->lattice_cap > 0 && !out->lattice) || out->lattice_cap < 0 || (out->kept_cap > 0 && !out->kept) ||
        out->kept_cap < 0)
        return fail(WFST_EINVAL, "wfst_decode_noalloc: bad output buffer");
    float thr = 0.0f;
    {
        const int rc = check_opts(G, o, L, &thr);
        if (rc != WFST_OK) return rc;
    }
    // at most this many blank-like units (their copy sits in the workspace)
    constexpr int kMaxBlank = 1024;
    const int n_blank = o.num_blank_ids > 0 ? o.num_blank_ids : 1;
    if (n_blank > kMaxBlank) return fail(WFST_EINVAL, "wfst_decode_noalloc: more than 1024 blank-like units");
    const wfst_debug_opts dbg = debug_snapshot();

    // Sizes: as wfst_decode's first attempt, with the average tokens per
    // frame as large as the fixed workspace allows (sizes grow linearly in
    // it).
    Sizes z = initial_sizes(G, o);
    const size_t cap = static_cast<size_t>(WFST_NOALLOC_SCRATCH_BYTES);
    z.capA = 0;
    const size_t base = noalloc_bytes(G, 1, L, o, thr, dbg, z, n_blank, T, nullptr, nullptr);
    z.capA = 1024;
    const size_t at1k = noalloc_bytes(G, 1, L, o, thr, dbg, z, n_blank, T, nullptr, nullptr);
    const double per = static_cast<double>(at1k - base) / 1024.0;
    if (base >= cap || per <= 0.0) {
        set_error("wfst_decode_noalloc: %d frames need more than the fixed workspace of %lld bytes", T,
                  static_cast<long long>(WFST_NOALLOC_SCRATCH_BYTES));
        return WFST_ECAPACITY;
    }
    z.capA = std::min<int64_t>(z.capF, static_cast<int64_t>(static_cast<double>(cap - base) / per));
    Totals tot;
    UttLayout lay{};
    size_t need = noalloc_bytes(G, 1, L, o, thr, dbg, z, n_blank, T, &tot, &lay);
    while (need > cap && z.capA > 0) {   // rounding of the carve
        z.capA -= std::max<int64_t>(1, z.capA / 64);
        need = noalloc_bytes(G, 1, L, o, thr, dbg, z, n_blank, T, &tot, &lay);
    }
    // refuse up front a T for which the workspace would hold fewer than
    // kMinAvgTokens tokens per frame on average: such a decode would almost
    // surely overflow
    constexpr int64_t kMinAvgTokens = 64;
    if (z.capA < std::min<int64_t>(kMinAvgTokens, z.capF) || need > cap) {
        set_error("wfst_decode_noalloc: %d frames need more than the fixed workspace of %lld bytes", T,
                  static_cast<long long>(WFST_NOALLOC_SCRATCH_BYTES));
        return WFST_ECAPACITY;
    }

    DeviceGuard dg(G.device);
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    void *ws = nullptr;
    {
        const hipError_t e = scratch_ptr(G.device, &ws);
        if (e != hipSuccess) return hip_fail(e, "wfst_decode_noalloc: workspace address");
    }
    Params p{};
    set_params(p, G, 1, L, o, thr, dbg, z, n_blank, false);
    Arena arena;
    arena.base = static_cast<char *>(ws);
    UttLayout *d_lay = nullptr;
    int64_t *fo_all = nullptr;
    carve_ws(arena, p, 1, tot, &d_lay, &fo_all);

    UttState st;
    std::memset(&st, 0, sizeof(st));
    st.ll = ll;
    st.T = T;
    hipError_t e = hipSuccess;
    auto chk = [&](hipError_t r) {
        if (e == hipSuccess && r != hipSuccess) e = r;
    };
    chk(hipMemcpyAsync(p.st, &st, sizeof(UttState), hipMemcpyHostToDevice, s));
    chk(hipMemcpyAsync(d_lay, &lay, sizeof(UttLayout), hipMemcpyHostToDevice, s));
    chk(launch_zero(fo_all, kOffsetArrays * tot.fo * sizeof(int64_t), s));
    if (o.num_blank_ids > 0)
        chk(hipMemcpyAsync(const_cast<int32_t *>(p.blank_ids), o.blank_ids, n_blank * sizeof(int32_t),
                           hipMemcpyHostToDevice, s));
    else
        chk(hipMemcpyAsync(const_cast<int32_t *>(p.blank_ids), &o.blank_id, sizeof(int32_t), hipMemcpyHostToDevice,
                           s));
    chk(launch_classify(p, s));
    chk(launch_search(p, s));
    chk(launch_record(p, T, s));
    chk(launch_final(p, s));
    chk(launch_finish(p, s));
    chk(hipMemcpyAsync(&st, p.st, sizeof(UttState), hipMemcpyDeviceToHost, s));
    chk(hipStreamSynchronize(s));
    if (e != hipSuccess) return hip_fail(e, "wfst_decode_noalloc: search");
    if (st.status == kStatusNoBackPointer)
        return fail(WFST_EDEVICE, "wfst_decode_noalloc: internal error, a surviving token without a back-pointer");
    if (st.status == kStatusLatticeWait)
        return fail(WFST_EDEVICE, "wfst_decode_noalloc: internal error, a lattice pass stopped waiting for its other waves");
    if (st.status == WFST_ECAPACITY) {
        set_error("wfst_decode_noalloc: the decode overflowed the fixed workspace");
        return WFST_ECAPACITY;
    }
    out->status = st.status;
    out->num_decoded = st.Tp;
    if (st.status != WFST_OK) {
        if (st.status == WFST_ENOPATH) set_error("wfst_decode_noalloc: no surviving path");
        return st.status;
    }
    out->cost = st.final_cost;
    out->final_state = user_state(G, st.final_state);
    out->reached_final = st.reached_final;
    out->path_len = st.path_len;
    out->tokens = st.n_tok;
    out->arcs_expanded = st.arcs_expanded;
    out->eps_arcs = st.eps_arcs;
    out->lattice_raw = lattice ? st.le_cnt + st.lx_cnt : 0;
    out->lattice_n = lattice ? st.lat_kept : 0;
    if (st.path_len > out->path_cap || (lattice && st.lat_kept > out->lattice_cap) ||
        (out->kept && st.Tp > out->kept_cap)) {
        set_error("wfst_decode_noalloc: output buffer too small (path %d, lattice %lld, decoded frames %d)",
                  st.path_len, static_cast<long long>(lattice ? st.lat_kept : 0), st.Tp);
        return WFST_ECAPACITY;
    }
    // the path lies at the end of the utterance's path region
    const int64_t p0 = lay.path0 + lay.pathcap - st.path_len;
    if (st.path_len > 0) {
        chk(hipMemcpyAsync(out->path_arcs, p.path_arc + p0, st.path_len * sizeof(int32_t), hipMemcpyDeviceToDevice,
                           s));
        chk(hipMemcpyAsync(out->path_frames, p.path_frame + p0, st.path_len * sizeof(int32_t),
                           hipMemcpyDeviceToDevice, s));
    }
    if (out->kept && st.Tp > 0)
        chk(hipMemcpyAsync(out->kept, p.kept + lay.kept0, st.Tp * sizeof(int32_t), hipMemcpyDeviceToDevice, s));
    if (lattice && st.lat_kept > 0) {
        p.lat_out = reinterpret_cast<int4 *>(out->lattice);
        chk(launch_lattice_emit(p, T, s));
    }
    chk(hipStreamSynchronize(s));
    if (e != hipSuccess) return hip_fail(e, "wfst_decode_noalloc: results");
    return WFST_OK;
}

}  // namespace

extern "C" int wfst_decode_noalloc(const wfst_graph *g, const float *loglikes, int32_t T, int32_t L,
                                   const wfst_decode_opts *opts, void *hip_stream, wfst_noalloc_out *out)
{
    return noalloc_impl(g, loglikes, T, L, opts, hip_stream, out);
}
