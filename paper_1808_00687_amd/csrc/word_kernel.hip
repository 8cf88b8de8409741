// Word-level lattice: every word sequence of the pruned state-level lattice
// with the best cost of a complete lattice path that outputs it.  Exact
// lattices serve second-pass rescoring (Sec. 1, after the exact-lattice
// work the paper cites); determinising the lattice over its output labels
// keeps exactly this map from word sequences to best costs.
//
// It is computed by a forward pass over the token sets, one block per
// utterance.  A state of the pass is (lattice node, word prefix): the node is
// a surviving token (j, s), the prefix a node of a trie of word sequences
// (parent, word), the value the smallest forward cost of a lattice path from
// (0, start) to the node that outputs the prefix.  An arc of the pruned
// lattice from a node with prefix t and cost c gives its destination the
// prefix t extended by the arc's output label (if any) and the cost
// fl(c + w) (epsilon arc) or fl(fl(c + w) - ll[kept[j]][i - 1]) (emitting arc
// of set j), the decoder's arithmetic; fl(x + w) and fl(x - l) are monotone
// in x, so the minimum over paths equals this minimum over predecessors.
// Epsilon arcs inside a set are relaxed in rounds until nothing changes (the
// epsilon graph is acyclic), emitting arcs then lead to the next set.  At the
// last set the final cost is added (Alg. 1's final transition) and each
// prefix keeps its smallest total.
#include "device_util.h"

namespace wfd {

namespace {

constexpr int kWT = 1024;                        // threads of a word block
constexpr unsigned long long kNoEntry = ~0ull;   // empty hash key
constexpr uint32_t kRootTrie = 0xFFFFFFFFu;      // the empty word sequence

// The tables are changed by atomics (performed in L2) while the block runs:
// their loads bypass the CU cache, and a barrier that publishes changes
// first waits for the block's device-memory operations.
template <typename T>
__device__ __forceinline__ T ld_l2(const T *ptr)
{
    return __hip_atomic_load(const_cast<T *>(ptr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void block_sync_mem()
{
    __threadfence();
    __syncthreads();
}

__device__ __forceinline__ uint32_t hash64(unsigned long long k)
{
    const uint32_t a = static_cast<uint32_t>(k), b = static_cast<uint32_t>(k >> 32);
    return (a * 0x9E3779B1u) ^ (b * 0x85EBCA77u) ^ ((a ^ b) >> 15);
}

struct WSh {
    int changed;
    int status;
    int nent;        // entries claimed so far (WordState copy kept in LDS)
    int linked;      // entries linked into their node's list
    int scan[17];
};

// The child of trie node t by word w (claimed if new); returns its slot or
// -1 when the trie is full.  A node's slot is its id.
__device__ __forceinline__ int trie_child(const WordWs &ws, uint32_t t, int32_t w)
{
    const unsigned long long key = (static_cast<unsigned long long>(t) << 32) | static_cast<uint32_t>(w);
    const uint32_t mask = static_cast<uint32_t>(ws.capW - 1);
    uint32_t h = hash64(key) & mask;
    for (int64_t probe = 0; probe < ws.capW; probe++) {
        const unsigned long long old = atomicCAS(ws.tkey + h, kNoEntry, key);
        if (old == kNoEntry) {
            // depth of the new node, read only after the pass
            const int pd = t == kRootTrie ? 0 : ld_l2(ws.tdep + t);
            __hip_atomic_store(ws.tdep + h, pd + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return static_cast<int>(h);
        }
        if (old == key) return static_cast<int>(h);
        h = (h + 1) & mask;
    }
    return -1;
}

// Offer cost key c to (node, trie prefix t): returns 1 when the entry is new
// or its cost went down, 0 if not, -1 when the table is full.  New entries
// are appended to the entry list (linked into their node's list later).
__device__ __forceinline__ int offer_entry(const WordWs &ws, WSh &sh, int32_t node, uint32_t t, uint32_t c)
{
    const unsigned long long key = (static_cast<unsigned long long>(static_cast<uint32_t>(node)) << 32) | t;
    const uint32_t mask = static_cast<uint32_t>(ws.capH - 1);
    uint32_t h = hash64(key) & mask;
    for (int64_t probe = 0; probe < ws.capH; probe++) {
        const unsigned long long old = atomicCAS(ws.hkey + h, kNoEntry, key);
        if (old == kNoEntry || old == key) {
            const uint32_t prev = atomicMin(ws.hval + h, c);
            if (old == kNoEntry) {
                const int e = atomicAdd(&sh.nent, 1);
                if (e >= ws.capH) return -1;
                __hip_atomic_store(ws.ents + e, static_cast<int32_t>(h), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            return (old == kNoEntry || c < prev) ? 1 : 0;
        }
        h = (h + 1) & mask;
    }
    return -1;
}

// Link the entries claimed since the last call into their nodes' lists.
// Called by the whole block between barriers (nobody walks a list meanwhile).
__device__ __forceinline__ void link_new(const WordWs &ws, WSh &sh)
{
    block_sync_mem();
    const int a = sh.linked, b = min(sh.nent, static_cast<int>(ws.capH));
    for (int i = a + static_cast<int>(threadIdx.x); i < b; i += blockDim.x) {
        const int slot = ld_l2(ws.ents + i);
        const int32_t node = static_cast<int32_t>(ld_l2(ws.hkey + slot) >> 32);
        const int32_t old = atomicExch(ws.heads + node, slot);
        __hip_atomic_store(ws.hnext + slot, old, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    block_sync_mem();
    if (threadIdx.x == 0) sh.linked = b;
    __syncthreads();
}

// Pass the entries of one lattice arc's source along it (one arc per
// thread): the source node's entry list, each entry's prefix extended by the
// arc's output label, the cost by the arc's weight (and log-likelihood).
__device__ __forceinline__ void pass_arc(const Params &p, const WordWs &ws, WSh &sh, const int4 &r, const float *row,
                                         bool emitting, int &changed)
{
    const int32_t src = r.x, dst = r.y, arc = r.z;
    const int2 ua = p.g.uarc[arc];
    float w, lv = 0.0f;
    if (emitting) {
        const int4 rec = p.g.earc[ua.y];
        w = __int_as_float(rec.z);
        lv = ldg(row + rec.y);
    } else {
        w = __int_as_float(p.g.xarc[ua.y].y);
    }
    const int32_t ol = ua.x;
    for (int slot = ld_l2(ws.heads + src); slot >= 0; slot = ld_l2(ws.hnext + slot)) {
        const uint32_t t = static_cast<uint32_t>(ld_l2(ws.hkey + slot));
        const float c = okey_val(ld_l2(ws.hval + slot));
        uint32_t tn = t;
        if (ol != 0) {
            const int ch = trie_child(ws, t, ol);
            if (ch < 0) {
                sh.status = WFST_ECAPACITY;
                return;
            }
            tn = static_cast<uint32_t>(ch);
        }
        const float t1 = c + w;
        const float cn = emitting ? t1 - lv : t1;
        const int rc = offer_entry(ws, sh, dst, tn, okey(cn));
        if (rc < 0) {
            sh.status = WFST_ECAPACITY;
            return;
        }
        changed |= rc;
    }
}

__global__ __launch_bounds__(kWT) void word_kernel(Params p, WordWs wsb)
{
    __shared__ WSh sh;
    const int u = blockIdx.x;
    UttState &st = p.st[u];
    if (st.status != 0) return;
    const UttLayout ly = p.lay[u];
    WordWs ws = word_ws_of(wsb, u, ly);
    const int tid = threadIdx.x;
    const int Tp = st.Tp;
    const float lb = p.lattice_beam;
    const int64_t *so = p.sv_off + ly.fo0;

    // clear the tables
    for (int64_t i = tid; i < ws.capH; i += kWT) {
        ws.hkey[i] = kNoEntry;
        ws.hval[i] = kEmptyKey;
    }
    for (int64_t i = tid; i < ws.capW; i += kWT) {
        ws.tkey[i] = kNoEntry;
        ws.tbest[i] = kEmptyKey;
    }
    for (int64_t i = so[0] + tid; i < so[1]; i += kWT) ws.heads[i] = -1;
    if (tid == 0) {
        sh.status = 0;
        sh.nent = 0;
        sh.linked = 0;
        ws.out_n[0] = 0;
        ws.out_n[1] = 0;
        ws.out_n[2] = 0;
        ws.root_best[0] = kEmptyKey;
    }
    block_sync_mem();
    // the start entry: the start state's token of S_0, the empty prefix
    for (int64_t i = so[0] + tid; i < so[1]; i += kWT)
        if (p.sv_state[ly.sv0 + i] == p.g.start) (void)offer_entry(ws, sh, static_cast<int32_t>(i), kRootTrie, okey(0.0f));
    __syncthreads();
    link_new(ws, sh);

    for (int j = 0; j <= Tp; j++) {
        // ---- epsilon arcs of set j, in rounds until nothing changes ----
        const int64_t x0 = ly.lx0 + p.lx_off[ly.fo0 + j];
        const int64_t nx = p.lx_cnt[ly.fo0 + j];
        while (nx > 0) {
            if (tid == 0) sh.changed = 0;
            __syncthreads();
            int changed = 0;
            for (int64_t r = tid; r < nx && sh.status == 0; r += kWT) {
                if (!(p.ex_x[x0 + r] <= lb)) continue;
                pass_arc(p, ws, sh, p.lat_x[x0 + r], nullptr, false, changed);
            }
            if (changed) sh.changed = 1;
            __syncthreads();
            const int again = sh.changed && sh.status == 0;
            link_new(ws, sh);
            if (!again) break;
        }
        if (sh.status) break;
        if (j == Tp) break;
        // ---- emitting arcs of set j into set j + 1 ----
        for (int64_t i = so[j + 1] + tid; i < so[j + 2]; i += kWT) ws.heads[i] = -1;
        if (tid == 0) ws.set_start[j + 1] = sh.nent;
        block_sync_mem();
        const int64_t e0 = ly.le0 + p.le_off[ly.fo0 + j];
        const int64_t ne = p.le_cnt[ly.fo0 + j];
        const float *row = st.ll + static_cast<int64_t>(p.kept[ly.kept0 + j]) * p.L;
        int dummy = 0;
        for (int64_t r = tid; r < ne && sh.status == 0; r += kWT) {
            if (!(p.ex_e[e0 + r] <= lb)) continue;
            pass_arc(p, ws, sh, p.lat_e[e0 + r], row, true, dummy);
        }
        link_new(ws, sh);
        if (sh.status) break;
    }
    if (sh.status) {
        if (tid == 0) ws.out_n[2] = sh.status;
        return;
    }
    // ---- final costs: the smallest total per word sequence ----
    const bool use_final = p.g.final_w != nullptr && st.reached_final;
    const int last0 = Tp == 0 ? 0 : ws.set_start[Tp];
    const int nent = min(sh.nent, static_cast<int>(ws.capH));
    for (int i = last0 + tid; i < nent; i += kWT) {
        const int slot = ld_l2(ws.ents + i);
        const unsigned long long key = ld_l2(ws.hkey + slot);
        const int32_t node = static_cast<int32_t>(key >> 32);
        const uint32_t t = static_cast<uint32_t>(key);
        const float c = okey_val(ld_l2(ws.hval + slot));
        const float f = use_final ? p.g.final_w[p.sv_state[ly.sv0 + node]] : 0.0f;
        const float tot = c + f;
        if (!(okey(tot) < okey(__int_as_float(0x7F800000)))) continue;   // +inf: no complete path
        if (t == kRootTrie) atomicMin(ws.root_best, okey(tot));
        else atomicMin(ws.tbest + t, okey(tot));
    }
    block_sync_mem();
    // ---- the word sequences that reached the end, listed ----
    for (int64_t t = tid; t <= ws.capW; t += kWT) {
        uint32_t b;
        int dep;
        int32_t id;
        if (t == ws.capW) {
            b = ld_l2(ws.root_best);
            dep = 0;
            id = -1;
        } else {
            b = ld_l2(ws.tbest + t);
            dep = b != kEmptyKey ? ld_l2(ws.tdep + t) : 0;
            id = static_cast<int32_t>(t);
        }
        if (b == kEmptyKey) continue;
        const int k = atomicAdd(ws.out_n, 1);
        atomicAdd(ws.out_n + 1, dep);
        if (k < ws.capW + 1) ws.out_id[k] = make_int2(id, static_cast<int32_t>(b));
    }
}

// The listed word sequences written out, one block per utterance: the
// sequence of trie node id (-1 = empty) is found by walking its parents, last
// word first.  off[k] gives where sequence k starts in words (an exclusive
// scan over the sequence lengths).
__global__ __launch_bounds__(256) void word_flatten_kernel(Params p, WordWs wsb, int64_t *off_all, int32_t *words_all,
                                                           const int64_t *base_seq, const int64_t *base_word)
{
    __shared__ int scan[17];
    const int u = blockIdx.x;
    const UttLayout ly = p.lay[u];
    WordWs ws = word_ws_of(wsb, u, ly);
    if (p.st[u].status != 0 || ws.out_n[2] != 0) return;
    const int n = ws.out_n[0];
    int64_t *off = off_all + base_seq[u] + u;   // n + 1 offsets per utterance
    int32_t *words = words_all + base_word[u];
    int64_t carry = 0;
    for (int k0 = 0; k0 < n; k0 += blockDim.x) {
        const int k = k0 + threadIdx.x;
        int dep = 0;
        int32_t id = -1;
        if (k < n) {
            id = ws.out_id[k].x;
            dep = id < 0 ? 0 : ws.tdep[id];
        }
        int total;
        const int ex = block_excl_scan(dep, scan, &total);
        if (k < n) {
            const int64_t o = carry + ex;
            off[k] = o;
            uint32_t t = static_cast<uint32_t>(id);
            for (int d = dep - 1; d >= 0; d--) {
                const unsigned long long key = ws.tkey[t];
                words[o + d] = static_cast<int32_t>(static_cast<uint32_t>(key));
                t = static_cast<uint32_t>(key >> 32);
            }
        }
        carry += total;
    }
    if (threadIdx.x == 0) off[n] = carry;
}

}  // namespace

hipError_t launch_word(const Params &p, const WordWs &ws, hipStream_t s)
{
    hipLaunchKernelGGL(word_kernel, dim3(p.U), dim3(kWT), 0, s, p, ws);
    return hipGetLastError();
}

hipError_t launch_word_flatten(const Params &p, const WordWs &ws, int64_t *off, int32_t *words,
                               const int64_t *base_seq, const int64_t *base_word, hipStream_t s)
{
    hipLaunchKernelGGL(word_flatten_kernel, dim3(p.U), dim3(256), 0, s, p, ws, off, words, base_seq, base_word);
    return hipGetLastError();
}

}  // namespace wfd
