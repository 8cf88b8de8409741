// Per-frame search kernels: one pass of token passing (Sec. 3 of the paper)
// for every utterance of a batch.  Producing token set k takes three kernels:
//
//   expand   (main stream) emitting arcs of S_{k-1} with loglike row
//            kept[k-1]; token recombination by 64-bit atomicMin on packed
//            (cost key, arc + 1); the epsilon closure by eager propagation:
//            every lowered token pushes its epsilon arcs into the same wave's
//            LDS queue.  k = 0 seeds the start token instead.
//   prune    (main stream) one block per utterance: closes epsilon items that
//            overflowed a wave queue, gathers the reached tokens, finds the
//            beam limit and, when more than max_active tokens are within it,
//            the max_active-th smallest cost key by exact radix select, then
//            compacts the survivors into S_k and resets the token table.
//   record   (second stream, overlapping the next frame) back-pointer
//            survivor indices of S_k and the lattice arcs into S_k.
//
// Every result is order-independent: recombination is a min over packed keys,
// the closure's fixed point is unique on the acyclic epsilon graph, and
// pruning is a pure function of the final token values.
#include "device_util.h"

namespace wfd {

namespace {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kStageCap = 256;       // first-touched states staged per wave
constexpr int kPruneThreads = 1024;
constexpr int kPruneWaves = kPruneThreads / kWave;
constexpr int kSpillQueue = 64;      // LDS queue per wave inside the prune block

struct EpsQ {
    uint2 *q;
    int head, tail, mask;
};

// Per-wave LDS staging of first touches, flushed to the utterance's touched
// list with one atomic per flush instead of one per batch.
struct Stage {
    int *buf;
    int n;
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
    c.wbest = c.st->hint;
    c.bnd = drop_bound(c.wbest, p.beam);
    return c;
}

__device__ void flush_stage(const Params &p, Ctx &c, Stage &sg)
{
    if (sg.n == 0) return;
    const int lane = lane_id();
    int base = 0;
    if (lane == 0) base = atomicAdd(&c.st->ntouched, sg.n);
    base = __shfl(base, 0, kWave);
    for (int i = lane; i < sg.n; i += kWave) {
        int idx = base + i;
        if (idx < p.capT) c.touched[idx] = sg.buf[i];
        else set_status(*c.st, WFST_ECAPACITY);
    }
    sg.n = 0;
}

// After a batch of atomicMin: stage first touches, tighten the wave's
// early-drop bound, and queue lowered states that have epsilon out-arcs.
__device__ __forceinline__ void post(const Params &p, Ctx &c, EpsQ &q, Stage &sg, bool first,
                                     bool impr, bool push, int d, float cand, uint32_t key,
                                     bool spill_only)
{
    const int lane = lane_id();
    uint64_t mf = __ballot(first);
    if (mf) {
        int cnt = __popcll(mf);
        if (sg.n + cnt > kStageCap) flush_stage(p, c, sg);
        if (first) sg.buf[sg.n + rank_in(mf)] = d;
        sg.n += cnt;
    }
    uint64_t mi = __ballot(impr);
    if (mi) {
        uint32_t mk = wave_min_u32(impr ? key : kEmptyKey);
        if (mk < c.wbest) {
            c.wbest = mk;
            c.bnd = drop_bound(mk, p.beam);
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
__device__ void eps_round(const Params &p, Ctx &c, EpsQ &q, Stage &sg, bool valid, int s, float cst,
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
        post(p, c, q, sg, first, impr, push, d, cand, key, spill_only);
    }
}

__device__ void drain(const Params &p, Ctx &c, EpsQ &q, Stage &sg)
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
        eps_round(p, c, q, sg, valid, s, cst, false);
    }
}

// Token set 0: the start token (cost +0, no arc) and its epsilon closure.
__device__ void init_chunk(const Params &p, Ctx &c, EpsQ &q, Stage &sg)
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
    post(p, c, q, sg, first, impr, push, s, 0.0f, key, false);
    drain(p, c, q, sg);
}

// Largest index t in [0, n) with epre[t] <= a, where epre is non-decreasing
// and epre[0] <= a: a 64-ary search by the whole wave, one load per level.
__device__ int wave_search_le(const int32_t *epre, int n, int a)
{
    const int lane = lane_id();
    int lo = 0, end = n;
    while (end - lo > 1) {
        const int step = (end - lo + kWave - 1) / kWave;
        const int idx = lo + lane * step;
        const int v = idx < end ? epre[idx] : 0x7FFFFFFF;
        const uint64_t m = __ballot(v <= a);
        const int l = 63 - __clzll(static_cast<long long>(m));
        lo += l * step;
        end = min(lo + step, end);
    }
    return lo;
}

// Emitting expansion of arcs [64 ci, 64 ci + 64) of S_{k-1}'s emitting arcs
// (chunk ci of utterance c.u): every wave gets exactly 64 arcs, whatever the
// out-degrees of the tokens they come from.
__device__ void expand_chunk(const Params &p, Ctx &c, EpsQ &q, Stage &sg, int k, int ci)
{
    const int lane = lane_id();
    const UttLayout &ly = p.lay[c.u];
    const int n_tok = c.st->n_cur;
    const int A = c.st->n_arcs;
    const int64_t base = ly.sv0 + p.sv_off[ly.fo0 + k - 1];
    const int32_t *epre = p.sv_epre + base;
    const int a0 = ci * kWave;
    const int a_end = min(a0 + kWave, A);
    const float *row = c.st->ll + static_cast<int64_t>(p.kept[ly.kept0 + k - 1]) * p.L;
    int t0 = wave_search_le(epre, n_tok, a0);
    int done = a0;
    while (done < a_end) {
        const int t = t0 + lane;
        const bool valid = t < n_tok;
        int pre = 0x7FFFFFFF, eb = 0;
        float cst = 0.0f;
        if (valid) {
            pre = epre[t];
            eb = p.sv_ebeg[base + t];
            cst = tok_cost(p.sv_tok[base + t]);
        }
        const int win_end = t0 + kWave < n_tok ? epre[t0 + kWave] : A;
        const int hi = min(a_end, win_end);
        const int a = done + lane;
        const int o = owner_lane(pre, a);
        const int ob = __shfl(eb, o, kWave);
        const int op = __shfl(pre, o, kWave);
        const float oc = __shfl(cst, o, kWave);
        bool first = false, impr = false, push = false;
        int d = 0;
        float cand = 0.0f;
        uint32_t key = kEmptyKey;
        if (a < hi && op <= a) {
            int4 r = p.g.earc[ob + (a - op)];
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
        post(p, c, q, sg, first, impr, push, d, cand, key, false);
        drain(p, c, q, sg);
        done = hi;
        t0 += kWave;
    }
}

__global__ __launch_bounds__(kBlock) void expand_kernel(Params p, int k)
{
    __shared__ uint2 qmem[kWavesPerBlock * kQueueCap];
    __shared__ int smem[kWavesPerBlock * kStageCap];
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    EpsQ q{qmem + wid * kQueueCap, 0, 0, p.qcap - 1};
    Stage sg{smem + wid * kStageCap, 0};
    const int gw = blockIdx.x * kWavesPerBlock + wid;
    const int nw = gridDim.x * kWavesPerBlock;
    for (int grp = 0; grp < p.U; grp += kWave) {
        int u = grp + lane;
        int n_u = 0;
        if (u < p.U && live(p.st[u], k)) n_u = (k == 0) ? 1 : p.st[u].n_arcs;
        ChunkGroup cg = chunk_group(n_u, kWave);
        for (int c = gw; c < cg.total; c += nw) {
            int ul, ci;
            chunk_locate(cg, c, ul, ci);
            Ctx cx = make_ctx(p, grp + ul);
            if (k == 0) init_chunk(p, cx, q, sg);
            else expand_chunk(p, cx, q, sg, k, ci);
            flush_stage(p, cx, sg);
        }
    }
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

// Two block-wide exclusive scans at once (counts and arc degrees).
__device__ __forceinline__ int2 block_excl_scan2(int x, int y, int *sh, int2 *total)
{
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int nw = blockDim.x / kWave;
    int ix = wave_incl_scan(x), iy = wave_incl_scan(y);
    if (lane == kWave - 1) {
        sh[w] = ix;
        sh[16 + w] = iy;
    }
    __syncthreads();
    if (threadIdx.x < kWave) {
        int vx = threadIdx.x < nw ? sh[threadIdx.x] : 0;
        int vy = threadIdx.x < nw ? sh[16 + threadIdx.x] : 0;
        int sx = wave_incl_scan(vx), sy = wave_incl_scan(vy);
        if (threadIdx.x < nw) {
            sh[threadIdx.x] = sx - vx;
            sh[16 + threadIdx.x] = sy - vy;
        }
        if (threadIdx.x == kWave - 1) {
            sh[32] = sx;
            sh[33] = sy;
        }
    }
    __syncthreads();
    int2 r = make_int2(ix - x + sh[w], iy - y + sh[16 + w]);
    *total = make_int2(sh[32], sh[33]);
    __syncthreads();
    return r;
}

constexpr int kPruneRegs = 8;   // reached tokens held in registers per thread (n <= 8192)

// Viterbi beam pruning of one utterance's reached tokens (one block).
__global__ __launch_bounds__(kPruneThreads) void prune_kernel(Params p, int k)
{
    __shared__ uint2 qmem[kPruneWaves * kSpillQueue];
    __shared__ int smem[kPruneWaves * kStageCap];
    __shared__ uint32_t h[kHistBins];
    __shared__ int sh_scan[34];
    __shared__ int sh_tail, sh_bin, sh_before, sh_cnt;
    __shared__ int sh_best_pos, sh_best_eb, sh_best_ed;
    __shared__ float sh_best_cost;
    __shared__ uint32_t sh_min;
    const int u = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = lane_id();
    const int wid = tid / kWave;
    UttState &st = p.st[u];
    if (!live(st, k)) return;
    const UttLayout &ly = p.lay[u];

    // 1. epsilon items spilled by the expansion (rare): close them here
    if (st.ovf > 0) {
        Ctx cx = make_ctx(p, u);
        EpsQ q{qmem + wid * kSpillQueue, 0, 0, min(p.qcap, kSpillQueue) - 1};
        Stage sg{smem + wid * kStageCap, 0};
        int head = 0;
        while (true) {
            __syncthreads();
            if (tid == 0) {
                int t = ld_relaxed(&st.ovf);
                sh_tail = t < p.capO ? t : static_cast<int>(p.capO);
            }
            __syncthreads();
            const int tail = sh_tail;
            if (head >= tail) break;
            for (int c0 = head + wid * kWave; c0 < tail; c0 += kPruneWaves * kWave) {
                int i = c0 + lane;
                bool valid = i < tail;
                int s = 0;
                float cst = 0.0f;
                if (valid) {
                    uint64_t it = ld_relaxed(cx.ovf + i);
                    s = static_cast<int>(it >> 32);
                    cst = __uint_as_float(static_cast<uint32_t>(it));
                }
                eps_round(p, cx, q, sg, valid, s, cst, true);
            }
            flush_stage(p, cx, sg);
            __threadfence();
            head = tail;
        }
        __syncthreads();
    }

    // 2. gather the reached tokens (registers for the first 8 x 1024, the
    // rest through pk) and their minimum cost key
    const int n = min(ld_relaxed(&st.ntouched), static_cast<int>(p.capT));
    const int32_t *touched = p.touched + static_cast<int64_t>(u) * p.capT;
    uint64_t *pk = p.pk + static_cast<int64_t>(u) * p.capT;
    uint64_t *tok = p.tok + static_cast<int64_t>(u) * p.g.n;
    if (tid == 0) {
        sh_min = kEmptyKey;
        sh_cnt = 0;
        sh_best_pos = -1;
    }
    int dR[kPruneRegs];
    uint64_t vR[kPruneRegs];
#pragma unroll
    for (int r = 0; r < kPruneRegs; r++) {
        const int i = r * kPruneThreads + tid;
        dR[r] = i < n ? touched[i] : -1;
    }
#pragma unroll
    for (int r = 0; r < kPruneRegs; r++) vR[r] = dR[r] >= 0 ? tok[dR[r]] : kEmptyTok;
    uint32_t m = kEmptyKey;
#pragma unroll
    for (int r = 0; r < kPruneRegs; r++) {
        const uint32_t key = static_cast<uint32_t>(vR[r] >> 32);
        m = key < m ? key : m;
    }
    for (int i = kPruneRegs * kPruneThreads + tid; i < n; i += kPruneThreads) {
        const uint64_t v = tok[touched[i]];
        pk[i] = v;
        const uint32_t key = static_cast<uint32_t>(v >> 32);
        m = key < m ? key : m;
    }
    m = wave_min_u32(m);
    __syncthreads();
    if (lane == 0 && m != kEmptyKey) atomicMin(&sh_min, m);
    __syncthreads();
    const uint32_t kb = sh_min;
    const uint32_t lim = beam_limit(kb, p.beam);
    auto key_at = [&](int r, int i) -> uint32_t {
        return static_cast<uint32_t>((r < kPruneRegs ? vR[r] : pk[i]) >> 32);
    };

    // 3. max-active: exact radix select of the max_active-th smallest key
    uint32_t cut = lim;
    if (p.max_active > 0 && kb <= lim && n > p.max_active) {
        int sh = first_shift(kb, lim);
        for (int i = tid; i < kHistBins; i += kPruneThreads) h[i] = 0u;
        __syncthreads();
        int cnt = 0;
#pragma unroll
        for (int r = 0; r < kPruneRegs; r++) {
            const uint32_t key = key_at(r, 0);
            if (dR[r] >= 0 && key <= lim) {
                cnt++;
                atomicAdd(&h[(key - kb) >> sh], 1u);
            }
        }
        for (int i = kPruneRegs * kPruneThreads + tid; i < n; i += kPruneThreads) {
            const uint32_t key = static_cast<uint32_t>(pk[i] >> 32);
            if (key <= lim) {
                cnt++;
                atomicAdd(&h[(key - kb) >> sh], 1u);
            }
        }
        if (cnt) atomicAdd(&sh_cnt, cnt);
        __syncthreads();
        if (sh_cnt > p.max_active) {
            int rank = p.max_active;
            select_bin(h, kHistBins, rank, sh_scan, &sh_bin, &sh_before);
            uint32_t prefix = static_cast<uint32_t>(sh_bin) << sh;
            rank -= sh_before;
            while (sh > 0) {
                const int nsh = sh > kHistBits ? sh - kHistBits : 0;
                const int width = sh - nsh;
                const int nb = 1 << width;
                for (int i = tid; i < nb; i += kPruneThreads) h[i] = 0u;
                __syncthreads();
                auto count = [&](uint32_t key) {
                    if (key > lim) return;
                    const uint32_t off = key - kb;
                    if ((off >> sh) == (prefix >> sh)) atomicAdd(&h[(off >> nsh) & (nb - 1)], 1u);
                };
#pragma unroll
                for (int r = 0; r < kPruneRegs; r++)
                    if (dR[r] >= 0) count(key_at(r, 0));
                for (int i = kPruneRegs * kPruneThreads + tid; i < n; i += kPruneThreads)
                    count(static_cast<uint32_t>(pk[i] >> 32));
                __syncthreads();
                select_bin(h, nb, rank, sh_scan, &sh_bin, &sh_before);
                prefix |= static_cast<uint32_t>(sh_bin) << nsh;
                rank -= sh_before;
                sh = nsh;
            }
            const uint32_t theta = kb + prefix;
            cut = theta < lim ? theta : lim;
        }
    }

    // 4. compact the survivors into S_k in reached order, with the exclusive
    // prefix of their emitting out-degrees (the next expansion's arc space),
    // and reset the token table
    int32_t *pos = p.pos + (static_cast<int64_t>(u) * 3 + k % 3) * p.g.n;
    const int64_t base = st.sv_base;
    int ebR[kPruneRegs], edR[kPruneRegs];
#pragma unroll
    for (int r = 0; r < kPruneRegs; r++) {
        ebR[r] = 0;
        edR[r] = -1;
        if (dR[r] >= 0 && key_at(r, 0) <= cut) {
            ebR[r] = p.g.eoff[dR[r]];
            edR[r] = p.g.eoff[dR[r] + 1];
        }
    }
    int run_n = 0, run_a = 0;
    auto emit = [&](int d, uint64_t v, bool keep, int eb, int ed) {
        int2 tot;
        const int2 ex = block_excl_scan2(keep ? 1 : 0, keep ? ed - eb : 0, sh_scan, &tot);
        if (d >= 0) tok[d] = kEmptyTok;
        if (keep) {
            const int64_t rel = base + run_n + ex.x;
            if (rel < ly.svcap) {
                const int64_t o = ly.sv0 + rel;
                p.sv_state[o] = d;
                p.sv_tok[o] = v;
                p.sv_ebeg[o] = eb;
                p.sv_epre[o] = run_a + ex.y;
                pos[d] = static_cast<int32_t>(rel);
                if (static_cast<uint32_t>(v >> 32) == kb &&
                    atomicCAS(&sh_best_pos, -1, static_cast<int32_t>(rel)) == -1) {
                    sh_best_eb = eb;
                    sh_best_ed = ed;
                    sh_best_cost = tok_cost(v);
                }
            } else {
                set_status(st, WFST_ECAPACITY);
            }
        }
        run_n += tot.x;
        run_a += tot.y;
    };
    const int nchunks = (n + kPruneThreads - 1) / kPruneThreads;
#pragma unroll
    for (int r = 0; r < kPruneRegs; r++) {
        if (r >= nchunks) break;
        emit(dR[r], vR[r], edR[r] >= 0, ebR[r], edR[r]);
    }
    for (int c = kPruneRegs; c < nchunks; c++) {
        const int i = c * kPruneThreads + tid;
        int d = -1, eb = 0, ed = -1;
        uint64_t v = kEmptyTok;
        if (i < n) {
            d = touched[i];
            v = pk[i];
            if (static_cast<uint32_t>(v >> 32) <= cut) {
                eb = p.g.eoff[d];
                ed = p.g.eoff[d + 1];
            }
        }
        emit(d, v, ed >= 0, eb, ed);
    }
    __syncthreads();

    // 5. bookkeeping for S_k
    const int ns = run_n;
    const int64_t end = base + ns;
    const bool ok = ns > 0 && end <= ly.svcap;
    if (tid == 0) {
        if (ns == 0) {
            st.status = WFST_ENOPATH;
        } else if (ok) {
            p.sv_off[ly.fo0 + k + 1] = end;
            p.cut_arr[ly.fo0 + k] = cut;
            st.sv_base = end;
            st.n_cur = ns;
            st.n_arcs = run_a;
            if (k < st.Tp) st.arcs_expanded += run_a;
        }
        st.ntouched = 0;
        st.ovf = 0;
    }
    // 6. seed of the next expansion's early-drop bound: the cheapest
    // candidate of one cheapest token of S_k, itself a real candidate
    if (wid == 0 && ok && k < st.Tp) {
        const float c = sh_best_cost;
        const float *row = st.ll + static_cast<int64_t>(p.kept[ly.kept0 + k]) * p.L;
        uint32_t hint = kEmptyKey;
        for (int a = sh_best_eb + lane; a < sh_best_ed; a += kWave) {
            const int4 r = p.g.earc[a];
            const float t1 = c + __int_as_float(r.z);
            const uint32_t key = okey(t1 - row[r.y]);
            hint = key < hint ? key : hint;
        }
        hint = wave_min_u32(hint);
        if (lane == 0) st.hint = hint;
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

// Back-pointer survivor indices of S_k and the lattice arcs into S_k: part A
// walks S_k (epsilon arcs inside S_k), part B walks S_{k-1} (emitting arcs
// into S_k).  An arc is recorded when its own prefix cost is within S_k's
// cutoff; its destination then survives.
__global__ __launch_bounds__(kBlock) void record_kernel(Params p, int k)
{
    const int lane = lane_id();
    const int wid = threadIdx.x / kWave;
    const int gw = blockIdx.x * kWavesPerBlock + wid;
    const int nw = gridDim.x * kWavesPerBlock;
    for (int part = 0; part < 2; part++) {
        if (part == 1 && (!p.lattice || k == 0)) break;
        for (int grp = 0; grp < p.U; grp += kWave) {
            int u = grp + lane;
            int n_u = 0;
            if (u < p.U && live(p.st[u], k)) {
                const int64_t *so = p.sv_off + p.lay[u].fo0;
                n_u = static_cast<int>(part == 0 ? so[k + 1] - so[k] : so[k] - so[k - 1]);
            }
            ChunkGroup cg = chunk_group(n_u, kWave);
            for (int c = gw; c < cg.total; c += nw) {
                int ul, ci;
                chunk_locate(cg, c, ul, ci);
                const int uu = grp + ul;
                UttState &st = p.st[uu];
                const UttLayout &ly = p.lay[uu];
                const int64_t *so = p.sv_off + ly.fo0;
                const uint32_t cut = p.cut_arr[ly.fo0 + k];
                const int32_t *pos_cur = p.pos + (static_cast<int64_t>(uu) * 3 + k % 3) * p.g.n;
                const int32_t *pos_prev = p.pos + (static_cast<int64_t>(uu) * 3 + (k + 2) % 3) * p.g.n;
                const int64_t set0 = part == 0 ? so[k] : so[k - 1];
                const int n = static_cast<int>(part == 0 ? so[k + 1] - so[k] : so[k] - so[k - 1]);
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
                    int orel = __shfl(static_cast<int>(rel), o, kWave);
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

hipError_t launch_expand(const Params &p, int k, int grid, hipStream_t s)
{
    if (k == 0) grid = (p.U + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(expand_kernel, dim3(grid), dim3(kBlock), 0, s, p, k);
    return hipGetLastError();
}

hipError_t launch_prune(const Params &p, int k, hipStream_t s)
{
    hipLaunchKernelGGL(prune_kernel, dim3(p.U), dim3(kPruneThreads), 0, s, p, k);
    return hipGetLastError();
}

hipError_t launch_record(const Params &p, int k, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(record_kernel, dim3(grid), dim3(kBlock), 0, s, p, k);
    return hipGetLastError();
}

}  // namespace wfd
