// Per-frame search kernels: one pass of token passing (Sec. 3 of the paper)
// for every utterance of a batch.  Producing token set k takes six launches:
//
//   expand         emitting arcs of S_{k-1} with loglike row kept[k-1], token
//                  recombination by 64-bit atomicMin on packed (cost key,
//                  arc + 1), and the epsilon closure by eager propagation
//                  (every lowered token pushes its epsilon arcs, handled by
//                  the same wave); k = 0 seeds the start token instead
//   prune_gather   reads the reached tokens, counts those within the beam and
//                  builds the first radix-select histogram
//   prune_select   one block per utterance: the max_active-th smallest cost
//                  key (exact radix select) and the cutoff
//   prune_compact  survivors -> S_k, token table reset, state -> survivor map
//   record         back-pointer survivor indices; lattice arcs of token set k
//   advance        per-utterance bookkeeping, k += 1
//
// Every result is order-independent: recombination is a min over packed keys,
// the closure's fixed point is unique on the acyclic epsilon graph, and
// pruning is a pure function of the final token values.
#include "device_util.h"

namespace wfd {

namespace {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;

struct EpsQ {
    uint2 *q;
    int head, tail, mask;
};

struct Ctx {
    int u;
    UttState *st;
    uint64_t *tok;
    int32_t *touched;
    uint64_t *ovf;
    uint32_t wbest;   // the wave's smallest candidate key so far
    uint32_t bnd;     // early-drop bound derived from it
};

__device__ __forceinline__ Ctx make_ctx(const Params &p, int u)
{
    Ctx c;
    c.u = u;
    c.st = p.st + u;
    c.tok = p.tok + static_cast<int64_t>(u) * p.g.n;
    c.touched = p.touched + static_cast<int64_t>(u) * p.capT;
    c.ovf = p.ovf + static_cast<int64_t>(u) * p.capO;
    c.wbest = ld_relaxed(&c.st->best);
    c.bnd = drop_bound(c.wbest, p.beam);
    return c;
}

__device__ __forceinline__ void refresh_bound(const Params &p, Ctx &c)
{
    uint32_t gb = ld_relaxed(&c.st->best);
    if (gb < c.wbest) {
        c.wbest = gb;
        c.bnd = drop_bound(gb, p.beam);
    }
}

// After a batch of atomicMin: record first touches, lower the utterance's
// best key, and queue lowered states that have epsilon out-arcs.
__device__ __forceinline__ void post(const Params &p, Ctx &c, EpsQ &q, bool first, bool impr,
                                     bool push, int d, float cand, uint32_t key, bool spill_only)
{
    const int lane = lane_id();
    uint64_t mf = __ballot(first);
    if (mf) {
        int cnt = __popcll(mf);
        int base = 0;
        if (lane == 0) base = atomicAdd(&c.st->ntouched, cnt);
        base = __shfl(base, 0, kWave);
        if (first) {
            int idx = base + rank_in(mf);
            if (idx < p.capT) c.touched[idx] = d;
            else set_status(*c.st, WFST_ECAPACITY);
        }
    }
    uint64_t mi = __ballot(impr);
    if (mi) {
        uint32_t mk = wave_min_u32(impr ? key : kEmptyKey);
        if (mk < c.wbest) {
            c.wbest = mk;
            c.bnd = drop_bound(mk, p.beam);
            if (lane == 0) atomicMin(&c.st->best, mk);
        }
    }
    uint64_t mp = __ballot(push);
    if (mp) {
        int cnt = __popcll(mp);
        if (!spill_only && q.tail - q.head + cnt <= q.mask + 1) {
            if (push) q.q[(q.tail + rank_in(mp)) & q.mask] = make_uint2(static_cast<uint32_t>(d), __float_as_uint(cand));
            q.tail += cnt;
        } else {
            int base = 0;
            if (lane == 0) base = atomicAdd(&c.st->ovf, cnt);
            base = __shfl(base, 0, kWave);
            if (push) {
                int idx = base + rank_in(mp);
                if (idx < p.capO)
                    c.ovf[idx] = (static_cast<uint64_t>(d) << 32) | __float_as_uint(cand);
                else
                    set_status(*c.st, WFST_ECAPACITY);
            }
        }
    }
}

// Relax the epsilon arcs of up to 64 states (one per lane), load-balanced
// over the wave by a prefix scan of their epsilon out-degrees.
__device__ void eps_round(const Params &p, Ctx &c, EpsQ &q, bool valid, int s, float cst,
                          bool spill_only)
{
    const int lane = lane_id();
    int xb = 0, xd = 0;
    if (valid) {
        xb = p.g.xoff[s];
        xd = p.g.xoff[s + 1] - xb;
    }
    int incl = wave_incl_scan(xd);
    int pre = incl - xd;
    int total = __shfl(incl, kWave - 1, kWave);
    for (int k0 = 0; k0 < total; k0 += kWave) {
        refresh_bound(p, c);
        int kk = k0 + lane;
        int o = owner_lane(pre, kk);
        int ob = __shfl(xb, o, kWave);
        int op = __shfl(pre, o, kWave);
        float oc = __shfl(cst, o, kWave);
        bool first = false, impr = false, push = false;
        int d = 0;
        float cand = 0.0f;
        uint32_t key = kEmptyKey;
        if (kk < total) {
            int4 r = p.g.xarc[ob + (kk - op)];
            d = r.x & static_cast<int>(kDstMask);
            cand = oc + __int_as_float(r.y);
            key = okey(cand);
            if (key <= c.bnd) {
                uint64_t v = make_tok(key, r.z);
                uint64_t old = atomicMin(reinterpret_cast<unsigned long long *>(c.tok + d),
                                         static_cast<unsigned long long>(v));
                first = old == kEmptyTok;
                impr = v < old;
                push = impr && (r.x < 0);
            }
        }
        post(p, c, q, first, impr, push, d, cand, key, spill_only);
    }
}

__device__ void drain(const Params &p, Ctx &c, EpsQ &q)
{
    const int lane = lane_id();
    while (q.tail != q.head) {
        int m = min(kWave, q.tail - q.head);
        bool valid = lane < m;
        int s = 0;
        float cst = 0.0f;
        if (valid) {
            uint2 it = q.q[(q.head + lane) & q.mask];
            s = static_cast<int>(it.x);
            cst = __uint_as_float(it.y);
        }
        q.head += m;
        eps_round(p, c, q, valid, s, cst, false);
    }
}

// Token set 0: the start token (cost +0, no arc) and its epsilon closure.
__device__ void init_chunk(const Params &p, Ctx &c, EpsQ &q)
{
    const int lane = lane_id();
    const int s = p.g.start;
    const uint32_t key = okey(0.0f);
    bool first = false, impr = false, push = false;
    if (lane == 0) {
        uint64_t v = make_tok(key, -1);
        uint64_t old = atomicMin(reinterpret_cast<unsigned long long *>(c.tok + s),
                                 static_cast<unsigned long long>(v));
        first = old == kEmptyTok;
        impr = v < old;
        push = impr && (p.g.xoff[s + 1] > p.g.xoff[s]);
    }
    post(p, c, q, first, impr, push, s, 0.0f, key, false);
    drain(p, c, q);
}

// Emitting expansion of 64 tokens of S_{k-1} (chunk ci of utterance c.u).
__device__ void expand_chunk(const Params &p, Ctx &c, EpsQ &q, int k, int ci)
{
    const int lane = lane_id();
    const UttLayout &ly = p.lay[c.u];
    const int n = c.st->n_cur;
    const int64_t base = ly.sv0 + p.sv_off[ly.fo0 + k - 1] + static_cast<int64_t>(ci) * kWave;
    const bool valid = ci * kWave + lane < n;
    int eb = 0, ed = 0;
    float cst = 0.0f;
    if (valid) {
        int s = p.sv_state[base + lane];
        cst = tok_cost(p.sv_tok[base + lane]);
        eb = p.g.eoff[s];
        ed = p.g.eoff[s + 1] - eb;
    }
    int incl = wave_incl_scan(ed);
    int pre = incl - ed;
    int total = __shfl(incl, kWave - 1, kWave);
    if (lane == 0 && total)
        atomicAdd(reinterpret_cast<unsigned long long *>(&c.st->arcs_expanded),
                  static_cast<unsigned long long>(total));
    const float *row = c.st->ll + static_cast<int64_t>(p.kept[ly.kept0 + k - 1]) * p.L;
    for (int k0 = 0; k0 < total; k0 += kWave) {
        refresh_bound(p, c);
        int kk = k0 + lane;
        int o = owner_lane(pre, kk);
        int ob = __shfl(eb, o, kWave);
        int op = __shfl(pre, o, kWave);
        float oc = __shfl(cst, o, kWave);
        bool first = false, impr = false, push = false;
        int d = 0;
        float cand = 0.0f;
        uint32_t key = kEmptyKey;
        if (kk < total) {
            int4 r = p.g.earc[ob + (kk - op)];
            d = r.x & static_cast<int>(kDstMask);
            float t1 = oc + __int_as_float(r.z);
            cand = t1 - row[r.y];
            key = okey(cand);
            if (key <= c.bnd) {
                uint64_t v = make_tok(key, r.w);
                uint64_t old = atomicMin(reinterpret_cast<unsigned long long *>(c.tok + d),
                                         static_cast<unsigned long long>(v));
                first = old == kEmptyTok;
                impr = v < old;
                push = impr && (r.x < 0);
            }
        }
        post(p, c, q, first, impr, push, d, cand, key, false);
        drain(p, c, q);
    }
}

__global__ __launch_bounds__(kBlock) void expand_kernel(Params p)
{
    __shared__ uint2 qmem[kWavesPerBlock * kQueueCap];
    __shared__ int sh_last;
    __shared__ int sh_tail;
    const int k = *p.cur;
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    EpsQ q{qmem + wid * kQueueCap, 0, 0, p.qcap - 1};
    const int gw = blockIdx.x * kWavesPerBlock + wid;
    const int nw = gridDim.x * kWavesPerBlock;
    for (int grp = 0; grp < p.U; grp += kWave) {
        int u = grp + lane;
        int n_u = 0;
        if (u < p.U && live(p.st[u], k)) n_u = (k == 0) ? 1 : p.st[u].n_cur;
        ChunkGroup cg = chunk_group(n_u, kWave);
        for (int c = gw; c < cg.total; c += nw) {
            int ul, ci;
            chunk_locate(cg, c, ul, ci);
            Ctx cx = make_ctx(p, grp + ul);
            if (k == 0) init_chunk(p, cx, q);
            else expand_chunk(p, cx, q, k, ci);
        }
    }

    // Epsilon items that did not fit a wave's queue: the last block to
    // finish closes them, round by round, until no token changes.
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned t = atomicAdd(p.done, 1u);
        sh_last = (t == gridDim.x - 1);
    }
    __syncthreads();
    if (!sh_last) return;
    __threadfence();
    for (int u = 0; u < p.U; u++) {
        UttState &st = p.st[u];
        if (ld_relaxed(&st.status) != 0 || k > st.Tp) continue;
        if (ld_relaxed(&st.ovf) == 0) continue;
        Ctx cx = make_ctx(p, u);
        int head = 0;
        while (true) {
            __syncthreads();
            if (threadIdx.x == 0) {
                int t = ld_relaxed(&st.ovf);
                sh_tail = t < p.capO ? t : static_cast<int>(p.capO);
            }
            __syncthreads();
            const int tail = sh_tail;
            if (head >= tail) break;
            for (int c0 = head + wid * kWave; c0 < tail; c0 += kWavesPerBlock * kWave) {
                int i = c0 + lane;
                bool valid = i < tail;
                int s = 0;
                float cst = 0.0f;
                if (valid) {
                    uint64_t it = ld_relaxed(cx.ovf + i);
                    s = static_cast<int>(it >> 32);
                    cst = __uint_as_float(static_cast<uint32_t>(it));
                }
                eps_round(p, cx, q, valid, s, cst, true);
            }
            __threadfence();
            head = tail;
        }
    }
    if (threadIdx.x == 0) *p.done = 0u;
}

// Shift of the first radix-select level: the span [best, limit] split into
// 12-bit digits from the top.
__device__ __forceinline__ int first_shift(uint32_t kb, uint32_t lim)
{
    if (kb > lim) return 0;
    uint32_t span = lim - kb;
    int nb = span ? 32 - __clz(static_cast<int>(span)) : 0;
    return nb > kHistBits ? nb - kHistBits : 0;
}

__global__ __launch_bounds__(kBlock) void prune_gather_kernel(Params p)
{
    const int k = *p.cur;
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    const int gw = blockIdx.x * kWavesPerBlock + wid;
    const int nw = gridDim.x * kWavesPerBlock;
    for (int grp = 0; grp < p.U; grp += kWave) {
        int u = grp + lane;
        int n_u = 0;
        if (u < p.U && live(p.st[u], k)) n_u = min(p.st[u].ntouched, static_cast<int>(p.capT));
        ChunkGroup cg = chunk_group(n_u, kWave);
        for (int c = gw; c < cg.total; c += nw) {
            int ul, ci;
            chunk_locate(cg, c, ul, ci);
            const int uu = grp + ul;
            UttState &st = p.st[uu];
            const int n = min(st.ntouched, static_cast<int>(p.capT));
            const uint32_t kb = st.best;
            const uint32_t lim = beam_limit(kb, p.beam);
            const int sh1 = first_shift(kb, lim);
            const int i = ci * kWave + lane;
            bool inb = false;
            if (i < n) {
                const int64_t o = static_cast<int64_t>(uu) * p.capT + i;
                int d = p.touched[o];
                uint64_t v = p.tok[static_cast<int64_t>(uu) * p.g.n + d];
                p.pk[o] = v;
                uint32_t key = static_cast<uint32_t>(v >> 32);
                inb = key <= lim;
                if (inb) atomicAdd(p.hist + static_cast<int64_t>(uu) * kHistBins + ((key - kb) >> sh1), 1u);
            }
            uint64_t m = __ballot(inb);
            if (lane == 0 && m) atomicAdd(&st.n_in_beam, __popcll(m));
        }
    }
}

// Find the bin holding the rank-th smallest element (1-based) of an LDS
// histogram of nbins bins; returns the bin and the count before it.
__device__ void select_bin(const uint32_t *h, int nbins, int rank, int *sh_scan, int *out_bin,
                           int *out_before)
{
    const int per = (nbins + blockDim.x - 1) / blockDim.x;
    const int b0 = threadIdx.x * per;
    int local = 0;
    for (int i = 0; i < per; i++)
        if (b0 + i < nbins) local += static_cast<int>(h[b0 + i]);
    int total;
    int excl = block_excl_scan(local, sh_scan, &total);
    if (rank > excl && rank <= excl + local) {
        int cum = excl;
        for (int i = 0; i < per && b0 + i < nbins; i++) {
            int c = static_cast<int>(h[b0 + i]);
            if (rank <= cum + c) {
                *out_bin = b0 + i;
                *out_before = cum;
                break;
            }
            cum += c;
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(1024) void prune_select_kernel(Params p)
{
    __shared__ uint32_t h[kHistBins];
    __shared__ int sh_scan[17];
    __shared__ int sh_bin, sh_before;
    const int k = *p.cur;
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    uint32_t *gh = p.hist + static_cast<int64_t>(u) * kHistBins;
    if (!live(st, k)) return;
    const uint32_t kb = st.best;
    const uint32_t lim = beam_limit(kb, p.beam);
    const int cnt = st.n_in_beam;
    const bool limit = p.max_active > 0 && cnt > p.max_active && kb <= lim;
    for (int i = threadIdx.x; i < kHistBins; i += blockDim.x) {
        h[i] = limit ? gh[i] : 0u;
        gh[i] = 0u;
    }
    __syncthreads();
    uint32_t cut = lim;
    if (limit) {
        int rank = p.max_active;
        int sh = first_shift(kb, lim);
        select_bin(h, kHistBins, rank, sh_scan, &sh_bin, &sh_before);
        uint32_t prefix = static_cast<uint32_t>(sh_bin) << sh;
        rank -= sh_before;
        const int n = min(st.ntouched, static_cast<int>(p.capT));
        const uint64_t *pk = p.pk + static_cast<int64_t>(u) * p.capT;
        while (sh > 0) {
            const int nsh = sh > kHistBits ? sh - kHistBits : 0;
            const int width = sh - nsh;
            const int nb = 1 << width;
            for (int i = threadIdx.x; i < nb; i += blockDim.x) h[i] = 0u;
            __syncthreads();
            for (int i = threadIdx.x; i < n; i += blockDim.x) {
                uint32_t key = static_cast<uint32_t>(pk[i] >> 32);
                if (key > lim) continue;
                uint32_t off = key - kb;
                if ((off >> sh) == (prefix >> sh)) atomicAdd(&h[(off >> nsh) & (nb - 1)], 1u);
            }
            __syncthreads();
            select_bin(h, nb, rank, sh_scan, &sh_bin, &sh_before);
            prefix |= static_cast<uint32_t>(sh_bin) << nsh;
            rank -= sh_before;
            sh = nsh;
        }
        uint32_t theta = kb + prefix;
        cut = theta < lim ? theta : lim;
    }
    if (threadIdx.x == 0) st.cut = cut;
}

__global__ __launch_bounds__(kBlock) void prune_compact_kernel(Params p)
{
    const int k = *p.cur;
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    const int gw = blockIdx.x * kWavesPerBlock + wid;
    const int nw = gridDim.x * kWavesPerBlock;
    const int par = k & 1;
    for (int grp = 0; grp < p.U; grp += kWave) {
        int u = grp + lane;
        int n_u = 0;
        if (u < p.U && live(p.st[u], k)) n_u = min(p.st[u].ntouched, static_cast<int>(p.capT));
        ChunkGroup cg = chunk_group(n_u, kWave);
        for (int c = gw; c < cg.total; c += nw) {
            int ul, ci;
            chunk_locate(cg, c, ul, ci);
            const int uu = grp + ul;
            UttState &st = p.st[uu];
            const UttLayout &ly = p.lay[uu];
            const int n = min(st.ntouched, static_cast<int>(p.capT));
            const uint32_t cut = st.cut;
            const uint32_t kb = st.best;
            const int i = ci * kWave + lane;
            bool keep = false;
            int d = 0;
            uint64_t v = 0;
            if (i < n) {
                const int64_t o = static_cast<int64_t>(uu) * p.capT + i;
                d = p.touched[o];
                v = p.pk[o];
                p.tok[static_cast<int64_t>(uu) * p.g.n + d] = kEmptyTok;
                keep = static_cast<uint32_t>(v >> 32) <= cut;
            }
            uint64_t m = __ballot(keep);
            if (!m) continue;
            int base = 0;
            if (lane == 0) base = atomicAdd(&st.n_new, __popcll(m));
            base = __shfl(base, 0, kWave);
            if (keep) {
                int64_t rel = st.sv_base + base + rank_in(m);
                if (rel < ly.svcap) {
                    p.sv_state[ly.sv0 + rel] = d;
                    p.sv_tok[ly.sv0 + rel] = v;
                    p.pos[(static_cast<int64_t>(uu) * 2 + par) * p.g.n + d] = static_cast<int32_t>(rel);
                    if (static_cast<uint32_t>(v >> 32) == kb) st.best_sv = static_cast<int32_t>(rel);
                } else {
                    set_status(st, WFST_ECAPACITY);
                }
            }
        }
    }
}

// Lattice record: append up to one record per lane.
__device__ __forceinline__ void put_records(int4 *buf, int64_t base0, int64_t cap, int64_t *cnt,
                                            UttState &st, bool rec, int4 r)
{
    const int lane = lane_id();
    uint64_t m = __ballot(rec);
    if (!m) return;
    long long b = 0;
    if (lane == 0) b = atomicAdd(reinterpret_cast<unsigned long long *>(cnt), static_cast<unsigned long long>(__popcll(m)));
    b = __shfl(b, 0, kWave);
    if (rec) {
        int64_t idx = b + rank_in(m);
        if (idx < cap) buf[base0 + idx] = r;
        else set_status(st, WFST_ECAPACITY);
    }
}

__global__ __launch_bounds__(kBlock) void record_kernel(Params p)
{
    const int k = *p.cur;
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    const int gw = blockIdx.x * kWavesPerBlock + wid;
    const int nw = gridDim.x * kWavesPerBlock;
    const int par = k & 1;
    // part A: the new token set S_k (back-pointer indices, epsilon lattice arcs)
    // part B: S_{k-1} (emitting lattice arcs into S_k), only with a lattice
    for (int part = 0; part < 2; part++) {
        if (part == 1 && (!p.lattice || k == 0)) break;
        for (int grp = 0; grp < p.U; grp += kWave) {
            int u = grp + lane;
            int n_u = 0;
            if (u < p.U && live(p.st[u], k)) n_u = part == 0 ? p.st[u].n_new : p.st[u].n_cur;
            ChunkGroup cg = chunk_group(n_u, kWave);
            for (int c = gw; c < cg.total; c += nw) {
                int ul, ci;
                chunk_locate(cg, c, ul, ci);
                const int uu = grp + ul;
                UttState &st = p.st[uu];
                const UttLayout &ly = p.lay[uu];
                const uint32_t cut = st.cut;
                const int32_t *pos_cur = p.pos + (static_cast<int64_t>(uu) * 2 + par) * p.g.n;
                const int32_t *pos_prev = p.pos + (static_cast<int64_t>(uu) * 2 + (par ^ 1)) * p.g.n;
                const int n = part == 0 ? st.n_new : st.n_cur;
                const int64_t set0 = part == 0 ? st.sv_base : p.sv_off[ly.fo0 + k - 1];
                const int idx = ci * kWave + lane;
                const bool valid = idx < n;
                const int64_t rel = set0 + static_cast<int64_t>(ci) * kWave + lane;
                int s = 0;
                float cst = 0.0f;
                int ab = 0, ad = 0;
                if (valid) {
                    s = p.sv_state[ly.sv0 + rel];
                    uint64_t v = p.sv_tok[ly.sv0 + rel];
                    cst = tok_cost(v);
                    if (part == 0) {
                        int a = tok_arc(v);
                        int prev = -1;
                        if (a >= 0) {
                            int info = p.g.arc_src[a];
                            int src = info & static_cast<int>(kDstMask);
                            prev = info < 0 ? pos_cur[src] : pos_prev[src];
                        }
                        p.sv_prev[ly.sv0 + rel] = prev;
                        ab = p.g.xoff[s];
                        ad = p.g.xoff[s + 1] - ab;
                    } else {
                        ab = p.g.eoff[s];
                        ad = p.g.eoff[s + 1] - ab;
                    }
                }
                int incl = wave_incl_scan(ad);
                int pre = incl - ad;
                int total = __shfl(incl, kWave - 1, kWave);
                if (part == 0) {
                    uint64_t mv = __ballot(valid);
                    if (lane == 0) {
                        atomicAdd(reinterpret_cast<unsigned long long *>(&st.eps_arcs),
                                  static_cast<unsigned long long>(total));
                        atomicAdd(reinterpret_cast<unsigned long long *>(&st.tokens),
                                  static_cast<unsigned long long>(__popcll(mv)));
                    }
                }
                if (!p.lattice) continue;
                const float *row = part == 1
                    ? st.ll + static_cast<int64_t>(p.kept[ly.kept0 + k - 1]) * p.L
                    : nullptr;
                for (int k0 = 0; k0 < total; k0 += kWave) {
                    int kk = k0 + lane;
                    int o = owner_lane(pre, kk);
                    int ob = __shfl(ab, o, kWave);
                    int op = __shfl(pre, o, kWave);
                    float oc = __shfl(cst, o, kWave);
                    int orel = static_cast<int>(__shfl(static_cast<int>(rel), o, kWave));
                    bool rec = false;
                    int4 r = make_int4(0, 0, 0, 0);
                    if (kk < total) {
                        float pc;
                        int d, arc;
                        if (part == 0) {
                            int4 x = p.g.xarc[ob + (kk - op)];
                            d = x.x & static_cast<int>(kDstMask);
                            pc = oc + __int_as_float(x.y);
                            arc = x.z;
                        } else {
                            int4 x = p.g.earc[ob + (kk - op)];
                            d = x.x & static_cast<int>(kDstMask);
                            float t1 = oc + __int_as_float(x.z);
                            pc = t1 - row[x.y];
                            arc = x.w;
                        }
                        if (okey(pc) <= cut) {
                            rec = true;
                            r = make_int4(orel, pos_cur[d], arc, __float_as_int(pc));
                        }
                    }
                    if (part == 0) put_records(p.lat_x, ly.lx0, ly.lxcap, &st.lx_cnt, st, rec, r);
                    else put_records(p.lat_e, ly.le0, ly.lecap, &st.le_cnt, st, rec, r);
                }
            }
        }
    }
}

__global__ void advance_kernel(Params p)
{
    const int k = *p.cur;
    for (int u = threadIdx.x; u < p.U; u += blockDim.x) {
        UttState &st = p.st[u];
        if (!live(st, k)) continue;
        const UttLayout &ly = p.lay[u];
        const int n = st.n_new;
        if (n == 0) {
            st.status = WFST_ENOPATH;
            continue;
        }
        p.sv_off[ly.fo0 + k + 1] = st.sv_base + n;
        p.le_off[ly.fo0 + k] = st.le_cnt;
        p.lx_off[ly.fo0 + k + 1] = st.lx_cnt;
        st.sv_base += n;
        st.n_cur = n;
        st.ntouched = 0;
        st.n_in_beam = 0;
        st.best = kEmptyKey;
        st.n_new = 0;
        st.ovf = 0;
    }
    __syncthreads();
    if (threadIdx.x == 0) *p.cur = k + 1;
}

__global__ void fill_u64_kernel(uint64_t *ptr, int64_t n, uint64_t v)
{
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        ptr[i] = v;
}

__global__ void fill_u32_kernel(uint32_t *ptr, int64_t n, uint32_t v)
{
    for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        ptr[i] = v;
}

// isBlankFrame (Sec. 2, Alg. 1): frame t is blank when ll[t][blank] exceeds
// the threshold (log domain); the kept frames are compacted in order.
__global__ __launch_bounds__(kBlock) void classify_kernel(Params p)
{
    __shared__ int sh_scan[17];
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    const UttLayout &ly = p.lay[u];
    const int T = st.T;
    int base = 0;
    for (int t0 = 0; t0 < T; t0 += blockDim.x) {
        int t = t0 + threadIdx.x;
        int keep = 0;
        if (t < T) keep = !(st.ll[static_cast<int64_t>(t) * p.L + p.blank_id] > p.blank_thr);
        int total;
        int ex = block_excl_scan(keep, sh_scan, &total);
        if (keep) p.kept[ly.kept0 + base + ex] = t;
        base += total;
    }
    if (threadIdx.x == 0) st.Tp = base;
}

int grid_for(int64_t n, int block)
{
    int64_t g = (n + block - 1) / block;
    if (g < 1) g = 1;
    if (g > 4096) g = 4096;
    return static_cast<int>(g);
}

}  // namespace

hipError_t launch_fill_u64(uint64_t *ptr, int64_t n, uint64_t v, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u64_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, ptr, n, v);
    return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t *ptr, int64_t n, uint32_t v, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, ptr, n, v);
    return hipGetLastError();
}

hipError_t launch_classify(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(classify_kernel, dim3(p.U), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_expand(const Params &p, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(expand_kernel, dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_init(const Params &p, hipStream_t s)
{
    return launch_expand(p, (p.U + kWavesPerBlock - 1) / kWavesPerBlock, s);
}

hipError_t launch_prune_gather(const Params &p, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(prune_gather_kernel, dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_prune_select(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(prune_select_kernel, dim3(p.U), dim3(1024), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_prune_compact(const Params &p, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(prune_compact_kernel, dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_record(const Params &p, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(record_kernel, dim3(grid), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_advance(const Params &p, hipStream_t s)
{
    hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace wfd
