// wfst_load: validation and device layout of the search graph.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "internal.h"

namespace wfd {

// The calling thread's last error message, in a fixed buffer (setting it
// allocates nothing).
static thread_local char g_err[512];

void set_error(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
}

void clear_error() { g_err[0] = '\0'; }

const char *last_error() { return g_err; }

}  // namespace wfd

using namespace wfd;

extern "C" const char *wfst_last_error(void) { return wfd::last_error(); }

namespace {

int fail(int code, const char *msg)
{
    set_error("%s", msg);
    return code;
}

}  // namespace

extern "C" int wfst_load(int32_t n, int64_t e, const int32_t *src, const int32_t *dst,
                         const int32_t *ilabel, const int32_t *olabel, const float *weight,
                         int32_t start, const float *final_weight, wfst_graph **out)
{
    clear_error();
    if (!out) return fail(WFST_EINVAL, "wfst_load: out is NULL");
    *out = nullptr;
    if (n < 1) return fail(WFST_EINVAL, "wfst_load: num_states must be >= 1");
    if (e < 0 || e >= 2147483647LL) return fail(WFST_EINVAL, "wfst_load: num_arcs out of range");
    if (start < 0 || start >= n) return fail(WFST_EINVAL, "wfst_load: start_state out of range");
    if (e > 0 && (!src || !dst || !ilabel || !olabel || !weight))
        return fail(WFST_EINVAL, "wfst_load: NULL arc array");

    int32_t max_il = 0;
    int64_t n_eps = 0;
    for (int64_t a = 0; a < e; a++) {
        if (src[a] < 0 || src[a] >= n) return fail(WFST_EINVAL, "wfst_load: src out of range");
        if (a && src[a] < src[a - 1]) return fail(WFST_EINVAL, "wfst_load: src not sorted");
        if (dst[a] < 0 || dst[a] >= n) return fail(WFST_EINVAL, "wfst_load: dst out of range");
        if (ilabel[a] < 0 || olabel[a] < 0) return fail(WFST_EINVAL, "wfst_load: negative label");
        if (!std::isfinite(weight[a])) return fail(WFST_EINVAL, "wfst_load: non-finite weight");
        if (ilabel[a] == 0) {
            if (weight[a] < 0.0f) return fail(WFST_EINVAL, "wfst_load: negative epsilon weight");
            n_eps++;
        }
        if (ilabel[a] > max_il) max_il = ilabel[a];
    }
    if (final_weight) {
        for (int32_t s = 0; s < n; s++) {
            float f = final_weight[s];
            if (std::isnan(f) || (std::isinf(f) && f < 0))
                return fail(WFST_EINVAL, "wfst_load: final weight NaN or -inf");
        }
    }
    const int64_t n_emit = e - n_eps;

    std::vector<int32_t> eoff, xoff, arc_src, eua;
    std::vector<int4> earc, xarc, srec, ctab;
    std::vector<int2> uarc;
    // the node layout (see below)
    std::vector<int32_t> hdr_pos, node_eua;
    std::vector<int4> node;
    std::vector<float> node_fin;
    int64_t n_units = 0;
    int64_t n_closure = 0;
    std::vector<uint8_t> has_eps;
    int32_t depth = 0;
    try {
        eoff.assign(static_cast<size_t>(n) + 1, 0);
        xoff.assign(static_cast<size_t>(n) + 1, 0);
        for (int64_t a = 0; a < e; a++) {
            if (ilabel[a]) eoff[src[a] + 1]++;
            else xoff[src[a] + 1]++;
        }
        for (int32_t s = 0; s < n; s++) {
            eoff[s + 1] += eoff[s];
            xoff[s + 1] += xoff[s];
        }
        has_eps.assign(static_cast<size_t>(n), 0);
        for (int32_t s = 0; s < n; s++) has_eps[s] = xoff[s + 1] > xoff[s];

        // epsilon subgraph: acyclic (Kahn) and its longest path
        std::vector<int32_t> indeg(static_cast<size_t>(n), 0), lvl(static_cast<size_t>(n), 0), q;
        q.reserve(static_cast<size_t>(n));
        std::vector<int64_t> row(static_cast<size_t>(n) + 1, 0);
        for (int64_t a = 0; a < e; a++) row[src[a] + 1]++;
        for (int32_t s = 0; s < n; s++) row[s + 1] += row[s];
        for (int64_t a = 0; a < e; a++)
            if (!ilabel[a]) indeg[dst[a]]++;
        for (int32_t s = 0; s < n; s++)
            if (!indeg[s]) q.push_back(s);
        for (size_t h = 0; h < q.size(); h++) {
            int32_t s = q[h];
            for (int64_t a = row[s]; a < row[s + 1]; a++) {
                if (ilabel[a]) continue;
                int32_t d = dst[a];
                if (lvl[s] + 1 > lvl[d]) lvl[d] = lvl[s] + 1;
                if (lvl[d] > depth) depth = lvl[d];
                if (--indeg[d] == 0) q.push_back(d);
            }
        }
        if (static_cast<int64_t>(q.size()) != n) return fail(WFST_EINVAL, "wfst_load: epsilon cycle");

        earc.resize(static_cast<size_t>(n_emit));
        eua.resize(static_cast<size_t>(n_emit));
        xarc.resize(static_cast<size_t>(n_eps));
        arc_src.resize(static_cast<size_t>(e));
        uarc.resize(static_cast<size_t>(e));
        std::vector<int32_t> ef(eoff.begin(), eoff.end() - 1), xf(xoff.begin(), xoff.end() - 1);
        for (int64_t a = 0; a < e; a++) {
            int32_t s = src[a], d = dst[a];
            int32_t dflag = d | (has_eps[d] ? static_cast<int32_t>(0x80000000u) : 0);
            int32_t wb;
            std::memcpy(&wb, &weight[a], 4);
            if (ilabel[a]) {
                uarc[a] = make_int2(olabel[a], ef[s]);
                eua[ef[s]] = static_cast<int32_t>(a);
                earc[ef[s]++] = make_int4(dflag, ilabel[a] - 1, wb, 0);
                arc_src[a] = s;
            } else {
                uarc[a] = make_int2(olabel[a], xf[s]);
                xarc[xf[s]++] = make_int4(dflag, wb, static_cast<int32_t>(a), 0);
                arc_src[a] = s | static_cast<int32_t>(0x80000000u);
            }
        }
        srec.assign(2 * static_cast<size_t>(n), make_int4(0, 0, 0, 0));
        for (int32_t s = 0; s < n; s++) {
            srec[2 * static_cast<size_t>(s)] = make_int4(eoff[s], eoff[s + 1], xoff[s], xoff[s + 1]);
            if (xoff[s + 1] > xoff[s]) srec[2 * static_cast<size_t>(s) + 1] = xarc[xoff[s]];
        }
        // Epsilon-closure lists: for a state whose epsilon paths number at
        // most kClosureMax and are at most kClosureDepth arcs long, every
        // such path as one entry {last destination, last arc, length, the
        // path's weights in order}.  Children come before parents in reverse
        // topological order, so a state's list is its arcs followed by each
        // child's list behind the arc to it.
        std::vector<int32_t> cl_size(static_cast<size_t>(n), 0), cl_depth(static_cast<size_t>(n), 0);
        std::vector<int64_t> cl_off(static_cast<size_t>(n), -1);
        for (size_t h = q.size(); h-- > 0;) {
            const int32_t s = q[h];
            if (xoff[s + 1] == xoff[s]) continue;
            int64_t size = 0;
            int32_t dep = 0;
            bool child_listed = true;
            for (int32_t x = xoff[s]; x < xoff[s + 1]; x++) {
                const int32_t d = xarc[x].x & 0x7FFFFFFF;
                size += 1 + cl_size[d];
                dep = std::max(dep, 1 + cl_depth[d]);
                if (cl_size[d] > 0 && cl_off[d] < 0) child_listed = false;
            }
            cl_size[s] = static_cast<int32_t>(std::min<int64_t>(size, kClosureMax + 1));
            cl_depth[s] = std::min(dep, kClosureDepth + 1);
            if (size > kClosureMax || dep > kClosureDepth || !child_listed) continue;
            const int64_t off = static_cast<int64_t>(ctab.size() / kClosureStride);
            if (off + size >= kClosureEntries) continue;
            for (int32_t x = xoff[s]; x < xoff[s + 1]; x++) {
                const int4 r = xarc[x];
                const int32_t d = r.x & 0x7FFFFFFF;
                ctab.push_back(make_int4(d, r.z, 1, r.y));
                ctab.push_back(make_int4(0, 0, 0, 0));
                ctab.push_back(make_int4(0, 0, 0, 0));
                if (cl_size[d] == 0) continue;
                for (int32_t i = 0; i < cl_size[d]; i++) {
                    const size_t ci = kClosureStride * static_cast<size_t>(cl_off[d] + i);
                    const int4 c0 = ctab[ci], c1 = ctab[ci + 1], c2 = ctab[ci + 2];
                    // the arc to d, then the child's path (at most
                    // kClosureDepth - 1 arcs, so its last weight slot is free)
                    ctab.push_back(make_int4(c0.x, c0.y, c0.z + 1, r.y));
                    ctab.push_back(make_int4(c0.w, c1.x, c1.y, c1.z));
                    ctab.push_back(make_int4(c1.w, c2.x, c2.y, c2.z));
                }
            }
            cl_off[s] = off;
            srec[2 * static_cast<size_t>(s) + 1].w = static_cast<int32_t>(
                (static_cast<uint32_t>(off + 1) << kClosureSizeBits) | static_cast<uint32_t>(size - 1));
            n_closure++;
        }
        // every arc record carries its destination's closure word: an
        // epsilon work item then reaches the list without the state record
        for (auto &r : earc) r.w = srec[2 * static_cast<size_t>(r.x & 0x7FFFFFFF) + 1].w;
        for (auto &r : xarc) r.w = srec[2 * static_cast<size_t>(r.x & 0x7FFFFFFF) + 1].w;

        // Node layout: each state's two records (its rows, then its first
        // epsilon record with its closure word) followed by its emitting
        // arcs, in one array of 16-byte units.  A state's id on the device is
        // the unit index of its first record, so the record that tells the
        // compaction a survivor's rows shares a cache line with the first
        // arcs the next expansion reads.  Ids keep the states' order (ties
        // broken by the lowest id stay the same).
        hdr_pos.resize(static_cast<size_t>(n));
        for (int32_t s = 0; s < n; s++) {
            hdr_pos[s] = static_cast<int32_t>(n_units);
            n_units += 2 + (eoff[s + 1] - eoff[s]);
            if (n_units >= 0x7FFFFFFFLL) return fail(WFST_EINVAL, "wfst_load: graph too large (2^31 16-byte units)");
        }
        auto remap = [&](int32_t x) {   // keeps the has-epsilon flag
            return hdr_pos[x & 0x7FFFFFFF] | (x & static_cast<int32_t>(0x80000000u));
        };
        node.assign(static_cast<size_t>(n_units), make_int4(0, 0, 0, 0));
        node_eua.assign(static_cast<size_t>(n_units), 0);
        if (final_weight) node_fin.assign(static_cast<size_t>(n_units), 0.0f);
        for (int32_t s = 0; s < n; s++) {
            const int64_t h = hdr_pos[s];
            const int32_t deg = eoff[s + 1] - eoff[s];
            node[h] = make_int4(static_cast<int32_t>(h + 2), static_cast<int32_t>(h + 2 + deg), xoff[s], xoff[s + 1]);
            int4 x0 = srec[2 * static_cast<size_t>(s) + 1];
            if (xoff[s + 1] > xoff[s]) x0.x = remap(x0.x);
            node[h + 1] = x0;
            for (int32_t j = 0; j < deg; j++) {
                int4 r = earc[eoff[s] + j];
                r.x = remap(r.x);
                node[h + 2 + j] = r;
                node_eua[h + 2 + j] = eua[eoff[s] + j];
            }
            if (final_weight) node_fin[h] = final_weight[s];
        }
        for (auto &r : xarc) r.x = remap(r.x);
        for (size_t i = 0; i < ctab.size(); i += kClosureStride) ctab[i].x = hdr_pos[ctab[i].x];
        for (int64_t a = 0; a < e; a++)
            if (ilabel[a]) uarc[a].y = hdr_pos[src[a]] + 2 + (uarc[a].y - eoff[src[a]]);
        std::vector<int4>().swap(earc);
        std::vector<int4>().swap(srec);
        std::vector<int32_t>().swap(eua);
    } catch (const std::bad_alloc &) {
        return fail(WFST_ENOMEM, "wfst_load: host allocation failed");
    }

    auto align = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
    const size_t units = static_cast<size_t>(n_units);
    const size_t b_node = align(units * 16 + 16);
    const size_t b_eua = align(units * 4 + 4);
    const size_t b_xarc = align(static_cast<size_t>(n_eps) * 16 + 16);
    const size_t b_src = align(static_cast<size_t>(e) * 4 + 4);
    const size_t b_fin = final_weight ? align(units * 4) : 0;
    const size_t b_ctab = align(ctab.size() * 16 + 16);
    const size_t b_uarc = align(static_cast<size_t>(e) * 8 + 8);
    const size_t total = b_node + b_eua + b_xarc + b_src + b_fin + b_ctab + b_uarc;

    wfst_graph *h = new (std::nothrow) wfst_graph();
    if (!h) return fail(WFST_ENOMEM, "wfst_load: host allocation failed");
    Graph &g = h->g;
    if (hipGetDevice(&g.device) != hipSuccess) {
        delete h;
        return fail(WFST_EDEVICE, "wfst_load: no HIP device");
    }
    char *mem = nullptr;
    hipError_t err = hipMalloc(reinterpret_cast<void **>(&mem), total);
    if (err != hipSuccess) {
        delete h;
        set_error("wfst_load: hipMalloc(%zu) failed: %s", total, hipGetErrorString(err));
        return err == hipErrorOutOfMemory ? WFST_ENOMEM : WFST_EDEVICE;
    }
    size_t off = 0;
    auto put = [&](const void *hostp, size_t bytes, size_t span) -> void * {
        void *d = mem + off;
        off += span;
        if (bytes && err == hipSuccess) err = hipMemcpy(d, hostp, bytes, hipMemcpyHostToDevice);
        return d;
    };
    g.d.n = n;
    g.d.e = e;
    g.d.start = hdr_pos[start];
    g.d.n_emit = n_emit;
    g.d.n_eps = n_eps;
    g.d.node = static_cast<const int4 *>(put(node.data(), node.size() * 16, b_node));
    g.d.earc = g.d.node;
    g.d.srec = g.d.node;
    g.d.eua = static_cast<const int32_t *>(put(node_eua.data(), node_eua.size() * 4, b_eua));
    g.d.xarc = static_cast<const int4 *>(put(xarc.data(), xarc.size() * 16, b_xarc));
    g.d.arc_src = static_cast<const int32_t *>(put(arc_src.data(), arc_src.size() * 4, b_src));
    g.d.final_w = final_weight ? static_cast<const float *>(put(node_fin.data(), units * 4, b_fin)) : nullptr;
    g.d.ctab = static_cast<const int4 *>(put(ctab.data(), ctab.size() * 16, b_ctab));
    g.d.uarc = static_cast<const int2 *>(put(uarc.data(), uarc.size() * 8, b_uarc));
    if (err != hipSuccess) {
        (void)hipFree(mem);
        delete h;
        set_error("wfst_load: hipMemcpy failed: %s", hipGetErrorString(err));
        return WFST_EDEVICE;
    }
    g.mem = mem;
    g.max_ilabel = max_il;
    g.eps_depth = depth;
    g.device_bytes = static_cast<int64_t>(total);
    g.n_closure = n_closure;
    g.hdr_pos = std::move(hdr_pos);
    *out = h;
    return WFST_OK;
}

extern "C" void wfst_graph_free(wfst_graph *h)
{
    if (!h) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    if (cur != h->g.device) (void)hipSetDevice(h->g.device);
    (void)hipFree(h->g.mem);
    if (cur != h->g.device) (void)hipSetDevice(cur);
    delete h;
}

extern "C" int wfst_graph_get_info(const wfst_graph *h, wfst_graph_info *info)
{
    clear_error();
    if (!h || !info) return fail(WFST_EINVAL, "wfst_graph_get_info: NULL argument");
    info->num_states = h->g.d.n;
    info->num_arcs = h->g.d.e;
    info->num_emitting = h->g.d.n_emit;
    info->num_epsilon = h->g.d.n_eps;
    info->max_ilabel = h->g.max_ilabel;
    info->epsilon_depth = h->g.eps_depth;
    info->device_bytes = h->g.device_bytes;
    info->num_closure_states = h->g.n_closure;
    return WFST_OK;
}
