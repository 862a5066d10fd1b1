// Graph handles of the gnnk library: the in-CSR, the reverse graph's CSR with
// the original edge ids (Appendix A, definition of the reverse graph), the
// degree arrays, rows sorted by degree, and the segment tables of hub rows.
//
// The structures are built on the host from one copy of the index arrays
// (stable counting sorts, so the edges of a node keep ascending edge id) and
// uploaded into the caller's workspace.
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <numeric>

#include "host.h"

namespace gnnk {

// ---------------------------------------------------------------------------
// errors and options

static thread_local std::string g_err;

gnnk_status fail(gnnk_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return st;
}

gnnk_status hip_fail(hipError_t e, const char* what) {
    return fail(GNNK_EHIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

void clear_error() { g_err.clear(); }

Options& options() {
    static Options o;
    return o;
}

int64_t Dir::count_above(int64_t t) const {
    // sorted_deg is descending: the first position whose degree is <= t is the
    // first x with t >= x
    auto it = std::upper_bound(sorted_deg.begin(), sorted_deg.end(), (int32_t)std::min<int64_t>(t, INT32_MAX),
                               [](int32_t v, int32_t x) { return v >= x; });
    return (int64_t)(it - sorted_deg.begin());
}

void* graph_scratch(gnnk_graph* g, size_t bytes, int slot) {
    std::lock_guard<std::mutex> lk(g->scratch_mu);
    void*& buf = slot ? g->scratch2 : g->scratch;
    size_t& have = slot ? g->scratch2_bytes : g->scratch_bytes;
    if (bytes <= have) return buf;
    if (buf) {
        (void)hipDeviceSynchronize();  // in-flight kernels may still read the old buffer
        (void)hipFree(buf);
        buf = nullptr;
        have = 0;
    }
    size_t want = bytes + bytes / 4;
    if (hipMalloc(&buf, want) != hipSuccess) {
        buf = nullptr;
        return nullptr;
    }
    have = want;
    return buf;
}

// ---------------------------------------------------------------------------
// workspace layout

namespace {

constexpr size_t ALIGN = 256;

struct Layout {
    size_t in_ptr = 0, in_idx = 0, in_eid = 0, out_ptr = 0, out_idx = 0, out_eid = 0;
    size_t in_deg = 0, out_deg = 0, in_perm = 0, out_perm = 0;
    size_t in_seg = 0, out_seg = 0, in_hub = 0, out_hub = 0, in_row = 0, out_row = 0, out_pos = 0, flag = 0,
           total = 0;
};

struct Bump {
    size_t off = 0;
    size_t take(size_t bytes) {
        size_t o = off;
        off += (bytes + ALIGN - 1) / ALIGN * ALIGN;
        return o;
    }
};

Layout make_layout(int64_t n_src, int64_t n_dst, int64_t E, size_t ps, bool own_in, bool in_eid, int64_t seg_in,
                   int64_t seg_out, int64_t hub_in, int64_t hub_out) {
    Layout L;
    Bump b;
    if (own_in) {
        L.in_ptr = b.take((size_t)(n_dst + 1) * ps);
        L.in_idx = b.take((size_t)E * 4);
    }
    if (in_eid) L.in_eid = b.take((size_t)E * 4);
    L.out_ptr = b.take((size_t)(n_src + 1) * ps);
    L.out_idx = b.take((size_t)E * 4);
    L.out_eid = b.take((size_t)E * 4);
    L.in_deg = b.take((size_t)n_dst * 4);
    L.out_deg = b.take((size_t)n_src * 4);
    L.in_perm = b.take((size_t)n_dst * 4);
    L.out_perm = b.take((size_t)n_src * 4);
    L.in_seg = b.take((size_t)seg_in * 16);
    L.out_seg = b.take((size_t)seg_out * 16);
    L.in_hub = b.take((size_t)(hub_in + 1) * 4);
    L.out_hub = b.take((size_t)(hub_out + 1) * 4);
    L.in_row = b.take((size_t)E * 4);
    L.out_row = b.take((size_t)E * 4);
    L.out_pos = b.take((size_t)E * 4);
    L.flag = b.take(ALIGN);
    L.total = b.off;
    return L;
}

bool sizes_ok(int64_t n_src, int64_t n_dst, int64_t E) {
    return n_src >= 0 && n_dst >= 0 && E >= 0 && n_src < INT32_MAX && n_dst < INT32_MAX && E < INT32_MAX;
}

// edges of each row in ascending edge id (stable counting sort by key)
void counting_csr(int64_t n_rows, int64_t E, const int32_t* key, const int32_t* other, std::vector<int64_t>& ptr,
                  std::vector<int32_t>& idx, std::vector<int32_t>& eid) {
    ptr.assign((size_t)n_rows + 1, 0);
    for (int64_t e = 0; e < E; ++e) ptr[(size_t)key[e] + 1]++;
    for (int64_t r = 0; r < n_rows; ++r) ptr[r + 1] += ptr[r];
    std::vector<int64_t> fill(ptr.begin(), ptr.end() - 1);
    idx.resize((size_t)E);
    eid.resize((size_t)E);
    for (int64_t e = 0; e < E; ++e) {
        int64_t p = fill[(size_t)key[e]]++;
        idx[(size_t)p] = other[e];
        eid[(size_t)p] = (int32_t)e;
    }
}

struct HostDir {
    std::vector<int32_t> deg, perm, hub_off;
    std::vector<int4> seg;
    int64_t n_nz = 0, n_hub = 0, max_deg = 0;
};

void schedule_dir(const std::vector<int64_t>& ptr, int64_t n_rows, int64_t S, HostDir& h, Dir& d) {
    h.deg.resize((size_t)n_rows);
    for (int64_t r = 0; r < n_rows; ++r) h.deg[(size_t)r] = (int32_t)(ptr[r + 1] - ptr[r]);
    h.perm.resize((size_t)n_rows);
    std::iota(h.perm.begin(), h.perm.end(), 0);
    std::stable_sort(h.perm.begin(), h.perm.end(),
                     [&](int32_t a, int32_t b) { return h.deg[(size_t)a] > h.deg[(size_t)b]; });
    d.sorted_deg.resize((size_t)n_rows);
    for (int64_t k = 0; k < n_rows; ++k) d.sorted_deg[(size_t)k] = h.deg[(size_t)h.perm[(size_t)k]];
    h.max_deg = n_rows ? d.sorted_deg[0] : 0;
    h.n_nz = d.count_above(0);
    h.n_hub = d.count_above(S);
    h.hub_off.assign((size_t)h.n_hub + 1, 0);
    h.seg.clear();
    for (int64_t k = 0; k < h.n_hub; ++k) {
        int32_t r = h.perm[(size_t)k];
        int64_t b = ptr[r], e = ptr[r + 1];
        h.hub_off[(size_t)k] = (int32_t)h.seg.size();
        for (int64_t s = b; s < e; s += S)
            h.seg.push_back(make_int4(r, (int32_t)s, (int32_t)std::min(e, s + S), (int32_t)k));
    }
    h.hub_off[(size_t)h.n_hub] = (int32_t)h.seg.size();
    d.n_rows = n_rows;
    d.n_nz = h.n_nz;
    d.n_hub = h.n_hub;
    d.n_seg = (int64_t)h.seg.size();
    d.max_deg = h.max_deg;
}

template <typename T>
hipError_t upload(void* dst, const T* src, size_t n, hipStream_t s) {
    if (n == 0) return hipSuccess;
    return hipMemcpyAsync(dst, src, n * sizeof(T), hipMemcpyHostToDevice, s);
}

hipError_t upload_ptr(void* dst, const std::vector<int64_t>& p, int ptr64, hipStream_t s) {
    if (ptr64) return upload(dst, p.data(), p.size(), s);
    std::vector<int32_t> q(p.begin(), p.end());
    hipError_t e = upload(dst, q.data(), q.size(), s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // q is about to go away
    return e;
}

template <typename T>
hipError_t download(std::vector<T>& dst, const void* src, size_t n, hipStream_t s) {
    dst.resize(n);
    if (n == 0) return hipSuccess;
    hipError_t e = hipMemcpyAsync(dst.data(), src, n * sizeof(T), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    return e;
}

// Build everything from edges given by id (src_of_e, dst_of_e) and upload.
// in_ptr/in_idx/in_eid_h describe the in-CSR to traverse (own == true: built
// here and uploaded; false: the caller's arrays, device pointers given).
gnnk_status finish_build(gnnk_graph* g, const std::vector<int32_t>& src_of_e, const std::vector<int32_t>& dst_of_e,
                         const std::vector<int64_t>& in_ptr, bool own_in, const std::vector<int32_t>* in_idx_h,
                         const std::vector<int32_t>* in_eid_h, bool in_eid_needed, const void* user_ptr,
                         const int32_t* user_idx, const int32_t* user_eid, void* ws, size_t ws_bytes,
                         hipStream_t s) {
    const int64_t E = g->n_edges;
    const size_t ps = g->ptr64 ? 8 : 4;
    std::vector<int64_t> out_ptr;
    std::vector<int32_t> out_idx, out_eid;
    counting_csr(g->n_src, E, src_of_e.data(), dst_of_e.data(), out_ptr, out_idx, out_eid);

    HostDir hin, hout;
    schedule_dir(in_ptr, g->n_dst, g->seg_edges, hin, g->in);
    schedule_dir(out_ptr, g->n_src, g->seg_edges, hout, g->out);

    Layout L = make_layout(g->n_src, g->n_dst, E, ps, own_in, own_in && in_eid_needed, g->in.n_seg, g->out.n_seg,
                           g->in.n_hub, g->out.n_hub);
    if (!ws || ws_bytes < L.total)
        return fail(GNNK_ENOMEM, "workspace of %zu bytes is smaller than the %zu bytes this graph needs", ws_bytes,
                    L.total);
    char* W = reinterpret_cast<char*>(ws);
    if ((uintptr_t)W % ALIGN) return fail(GNNK_EINVAL, "workspace must be 256-byte aligned");
    hipError_t e = hipSuccess;
    auto chk = [&](hipError_t x) {
        if (e == hipSuccess) e = x;
    };
    if (own_in) {
        chk(upload_ptr(W + L.in_ptr, in_ptr, g->ptr64, s));
        chk(upload(W + L.in_idx, in_idx_h->data(), (size_t)E, s));
        g->in.ptr = W + L.in_ptr;
        g->in.idx = reinterpret_cast<int32_t*>(W + L.in_idx);
        if (in_eid_needed) {
            chk(upload(W + L.in_eid, in_eid_h->data(), (size_t)E, s));
            g->in.eid = reinterpret_cast<int32_t*>(W + L.in_eid);
        } else {
            g->in.eid = nullptr;
        }
    } else {
        g->in.ptr = user_ptr;
        g->in.idx = user_idx;
        g->in.eid = user_eid;
    }
    chk(upload_ptr(W + L.out_ptr, out_ptr, g->ptr64, s));
    chk(upload(W + L.out_idx, out_idx.data(), (size_t)E, s));
    chk(upload(W + L.out_eid, out_eid.data(), (size_t)E, s));
    g->out.ptr = W + L.out_ptr;
    g->out.idx = reinterpret_cast<int32_t*>(W + L.out_idx);
    g->out.eid = reinterpret_cast<int32_t*>(W + L.out_eid);

    g->in.deg = reinterpret_cast<int32_t*>(W + L.in_deg);
    g->out.deg = reinterpret_cast<int32_t*>(W + L.out_deg);
    g->in.perm = reinterpret_cast<int32_t*>(W + L.in_perm);
    g->out.perm = reinterpret_cast<int32_t*>(W + L.out_perm);
    g->in.seg = reinterpret_cast<int4*>(W + L.in_seg);
    g->out.seg = reinterpret_cast<int4*>(W + L.out_seg);
    g->in.hub_off = reinterpret_cast<int32_t*>(W + L.in_hub);
    g->out.hub_off = reinterpret_cast<int32_t*>(W + L.out_hub);
    g->in.row = reinterpret_cast<int32_t*>(W + L.in_row);
    g->out.row = reinterpret_cast<int32_t*>(W + L.out_row);
    g->out.pos = reinterpret_cast<int32_t*>(W + L.out_pos);
    g->flag = reinterpret_cast<int32_t*>(W + L.flag);
    chk(launch_fill_rows(g->in.ptr, g->ptr64, g->n_dst, E, g->in.row, s));
    chk(launch_fill_rows(g->out.ptr, g->ptr64, g->n_src, E, g->out.row, s));
    chk(launch_inverse(g->out.eid, E, g->out.pos, s));
    chk(upload(g->in.deg, hin.deg.data(), hin.deg.size(), s));
    chk(upload(g->out.deg, hout.deg.data(), hout.deg.size(), s));
    chk(upload(g->in.perm, hin.perm.data(), hin.perm.size(), s));
    chk(upload(g->out.perm, hout.perm.data(), hout.perm.size(), s));
    chk(upload(g->in.seg, hin.seg.data(), hin.seg.size(), s));
    chk(upload(g->out.seg, hout.seg.data(), hout.seg.size(), s));
    chk(upload(g->in.hub_off, hin.hub_off.data(), hin.hub_off.size(), s));
    chk(upload(g->out.hub_off, hout.hub_off.data(), hout.hub_off.size(), s));
    chk(hipMemsetAsync(g->flag, 0, 4, s));
    chk(hipStreamSynchronize(s));
    if (e != hipSuccess) return hip_fail(e, "graph upload");
    g->ws_used = L.total;
    return GNNK_OK;
}

}  // namespace
}  // namespace gnnk

using namespace gnnk;

extern "C" {

gnnk_status graph_workspace_bytes(int64_t num_src, int64_t num_dst, int64_t num_edges, gnnk_itype ptr_t,
                                  size_t* bytes) {
    clear_error();
    if (!bytes) return fail(GNNK_EINVAL, "bytes is NULL");
    if (!sizes_ok(num_src, num_dst, num_edges)) return fail(GNNK_EINVAL, "sizes out of range (int32 ids)");
    if (ptr_t != GNNK_I32 && ptr_t != GNNK_I64) return fail(GNNK_EINVAL, "bad ptr type");
    int64_t S = options().seg_edges;
    int64_t seg = 2 * num_edges / S + 2, hub = num_edges / S + 1;
    Layout L = make_layout(num_src, num_dst, num_edges, ptr_t == GNNK_I64 ? 8 : 4, true, true, seg, seg, hub, hub);
    *bytes = L.total;
    return GNNK_OK;
}

gnnk_status graph_create_coo(int64_t num_src, int64_t num_dst, int64_t num_edges, const int32_t* src,
                             const int32_t* dst, gnnk_itype ptr_t, void* workspace, size_t ws_bytes,
                             hipStream_t stream, gnnk_graph_t* out) {
    clear_error();
    if (!out) return fail(GNNK_EINVAL, "out is NULL");
    *out = nullptr;
    if (!sizes_ok(num_src, num_dst, num_edges)) return fail(GNNK_EINVAL, "sizes out of range (int32 ids)");
    if (ptr_t != GNNK_I32 && ptr_t != GNNK_I64) return fail(GNNK_EINVAL, "bad ptr type");
    if (num_edges > 0 && (!src || !dst)) return fail(GNNK_EINVAL, "src/dst is NULL");
    std::vector<int32_t> hs, hd;
    hipError_t e = download(hs, src, (size_t)num_edges, stream);
    if (e == hipSuccess) e = download(hd, dst, (size_t)num_edges, stream);
    if (e != hipSuccess) return hip_fail(e, "reading the edge list");
    for (int64_t i = 0; i < num_edges; ++i) {
        if (hs[(size_t)i] < 0 || hs[(size_t)i] >= num_src || hd[(size_t)i] < 0 || hd[(size_t)i] >= num_dst)
            return fail(GNNK_EINVAL, "edge %lld has an endpoint out of range", (long long)i);
    }
    gnnk_graph* g = new gnnk_graph();
    g->n_src = num_src;
    g->n_dst = num_dst;
    g->n_edges = num_edges;
    g->ptr64 = ptr_t == GNNK_I64;
    g->seg_edges = options().seg_edges;
    std::vector<int64_t> in_ptr;
    std::vector<int32_t> in_idx, in_eid;
    counting_csr(num_dst, num_edges, hd.data(), hs.data(), in_ptr, in_idx, in_eid);
    bool identity = true;
    for (int64_t p = 0; p < num_edges && identity; ++p) identity = in_eid[(size_t)p] == (int32_t)p;
    g->identity_eids = identity;
    gnnk_status st = finish_build(g, hs, hd, in_ptr, true, &in_idx, &in_eid, !identity, nullptr, nullptr, nullptr,
                                  workspace, ws_bytes, stream);
    if (st != GNNK_OK) {
        delete g;
        return st;
    }
    *out = g;
    return GNNK_OK;
}

gnnk_status graph_create_csr(int64_t num_src, int64_t num_dst, int64_t num_edges, const void* indptr,
                             gnnk_itype ptr_t, const int32_t* indices, const int32_t* eids, void* workspace,
                             size_t ws_bytes, hipStream_t stream, gnnk_graph_t* out) {
    clear_error();
    if (!out) return fail(GNNK_EINVAL, "out is NULL");
    *out = nullptr;
    if (!sizes_ok(num_src, num_dst, num_edges)) return fail(GNNK_EINVAL, "sizes out of range (int32 ids)");
    if (ptr_t != GNNK_I32 && ptr_t != GNNK_I64) return fail(GNNK_EINVAL, "bad ptr type");
    if (!indptr || (num_edges > 0 && !indices)) return fail(GNNK_EINVAL, "indptr/indices is NULL");
    std::vector<int64_t> hp;
    std::vector<int32_t> hi, he;
    hipError_t e;
    if (ptr_t == GNNK_I64) {
        e = download(hp, indptr, (size_t)num_dst + 1, stream);
    } else {
        std::vector<int32_t> t;
        e = download(t, indptr, (size_t)num_dst + 1, stream);
        hp.assign(t.begin(), t.end());
    }
    if (e == hipSuccess) e = download(hi, indices, (size_t)num_edges, stream);
    if (e == hipSuccess && eids) e = download(he, eids, (size_t)num_edges, stream);
    if (e != hipSuccess) return hip_fail(e, "reading the CSR");
    if (hp[0] != 0 || hp[(size_t)num_dst] != num_edges)
        return fail(GNNK_EINVAL, "indptr must start at 0 and end at num_edges");
    for (int64_t r = 0; r < num_dst; ++r)
        if (hp[(size_t)r + 1] < hp[(size_t)r]) return fail(GNNK_EINVAL, "indptr decreases at row %lld", (long long)r);
    std::vector<int32_t> src_of_e((size_t)num_edges), dst_of_e((size_t)num_edges);
    std::vector<uint8_t> seen(eids ? (size_t)num_edges : 0, 0);
    bool identity = true;
    for (int64_t r = 0; r < num_dst; ++r) {
        for (int64_t p = hp[(size_t)r]; p < hp[(size_t)r + 1]; ++p) {
            int32_t u = hi[(size_t)p];
            if (u < 0 || u >= num_src) return fail(GNNK_EINVAL, "index %lld out of range", (long long)p);
            int64_t eid = p;
            if (eids) {
                eid = he[(size_t)p];
                if (eid < 0 || eid >= num_edges || seen[(size_t)eid])
                    return fail(GNNK_EINVAL, "eids is not a permutation of 0..num_edges-1");
                seen[(size_t)eid] = 1;
                identity = identity && eid == p;
            }
            src_of_e[(size_t)eid] = u;
            dst_of_e[(size_t)eid] = (int32_t)r;
        }
    }
    gnnk_graph* g = new gnnk_graph();
    g->n_src = num_src;
    g->n_dst = num_dst;
    g->n_edges = num_edges;
    g->ptr64 = ptr_t == GNNK_I64;
    g->seg_edges = options().seg_edges;
    g->identity_eids = identity;
    gnnk_status st = finish_build(g, src_of_e, dst_of_e, hp, false, nullptr, nullptr, false, indptr, indices,
                                  identity ? nullptr : eids, workspace, ws_bytes, stream);
    if (st != GNNK_OK) {
        delete g;
        return st;
    }
    *out = g;
    return GNNK_OK;
}

gnnk_status graph_info(gnnk_graph_t g, gnnk_graph_info* info) {
    clear_error();
    if (!g || !info) return fail(GNNK_EINVAL, "NULL argument");
    info->num_src = g->n_src;
    info->num_dst = g->n_dst;
    info->num_edges = g->n_edges;
    info->ptr_type = g->ptr64 ? GNNK_I64 : GNNK_I32;
    info->identity_eids = g->identity_eids;
    info->max_in_degree = g->in.max_deg;
    info->max_out_degree = g->out.max_deg;
    info->empty_dst_rows = g->n_dst - g->in.n_nz;
    info->empty_src_rows = g->n_src - g->out.n_nz;
    info->seg_edges = g->seg_edges;
    info->hub_dst_rows = g->in.n_hub;
    info->hub_src_rows = g->out.n_hub;
    info->segments_in = g->in.n_seg;
    info->segments_out = g->out.n_seg;
    info->workspace_bytes = g->ws_used;
    return GNNK_OK;
}

gnnk_status graph_in_degrees(gnnk_graph_t g, int32_t* out, hipStream_t stream) {
    clear_error();
    if (!g || (!out && g->n_dst > 0)) return fail(GNNK_EINVAL, "NULL argument");
    if (g->n_dst == 0) return GNNK_OK;
    hipError_t e = hipMemcpyAsync(out, g->in.deg, (size_t)g->n_dst * 4, hipMemcpyDeviceToDevice, stream);
    return e == hipSuccess ? GNNK_OK : hip_fail(e, "graph_in_degrees");
}

gnnk_status graph_out_degrees(gnnk_graph_t g, int32_t* out, hipStream_t stream) {
    clear_error();
    if (!g || (!out && g->n_src > 0)) return fail(GNNK_EINVAL, "NULL argument");
    if (g->n_src == 0) return GNNK_OK;
    hipError_t e = hipMemcpyAsync(out, g->out.deg, (size_t)g->n_src * 4, hipMemcpyDeviceToDevice, stream);
    return e == hipSuccess ? GNNK_OK : hip_fail(e, "graph_out_degrees");
}

gnnk_status graph_csr_export(gnnk_graph_t g, int reverse, void* indptr, int32_t* indices, int32_t* eids,
                             hipStream_t stream) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    const Dir& d = reverse ? g->out : g->in;
    const int64_t E = g->n_edges;
    hipError_t e = hipSuccess;
    if (indptr) e = launch_copy_ptr(d.ptr, g->ptr64, indptr, g->ptr64, d.n_rows + 1, stream);
    if (e == hipSuccess && indices && E > 0)
        e = hipMemcpyAsync(indices, d.idx, (size_t)E * 4, hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess && eids && E > 0) {
        if (d.eid) e = hipMemcpyAsync(eids, d.eid, (size_t)E * 4, hipMemcpyDeviceToDevice, stream);
        else e = launch_iota(eids, E, stream);
    }
    return e == hipSuccess ? GNNK_OK : hip_fail(e, "graph_csr_export");
}

gnnk_status graph_validate(gnnk_graph_t g, hipStream_t stream) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    hipError_t e = hipMemsetAsync(g->flag, 0, 4, stream);
    const int64_t E = g->n_edges;
    if (e == hipSuccess) e = launch_validate_ptr(g->in.ptr, g->ptr64, g->n_dst, E, g->flag, stream);
    if (e == hipSuccess) e = launch_validate_ptr(g->out.ptr, g->ptr64, g->n_src, E, g->flag, stream);
    if (e == hipSuccess) e = launch_validate(g->in.idx, E, g->n_src, g->flag, stream);
    if (e == hipSuccess) e = launch_validate(g->out.idx, E, g->n_dst, g->flag, stream);
    if (e == hipSuccess && g->in.eid) e = launch_validate(g->in.eid, E, E, g->flag, stream);
    if (e == hipSuccess) e = launch_validate(g->out.eid, E, E, g->flag, stream);
    int32_t h = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&h, g->flag, 4, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return hip_fail(e, "graph_validate");
    if (h) return fail(GNNK_ERANGE, "graph has out-of-range entries (flags %d)", h);
    return GNNK_OK;
}

gnnk_status graph_destroy(gnnk_graph_t g) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (g->scratch2) {
        (void)hipDeviceSynchronize();
        (void)hipFree(g->scratch2);
    }
    if (g->scratch) {
        (void)hipDeviceSynchronize();
        (void)hipFree(g->scratch);
    }
    delete g;
    return GNNK_OK;
}

gnnk_status gnnk_set_option(const char* key, int64_t value) {
    clear_error();
    if (!key) return fail(GNNK_EINVAL, "NULL key");
    std::string k(key);
    if (k == "seg_edges") {
        if (value < 32 || value > (1 << 30)) return fail(GNNK_EINVAL, "seg_edges must be in [32, 2^30]");
        options().seg_edges = value;
    } else if (k == "no_split") {
        if (value != 0 && value != 1) return fail(GNNK_EINVAL, "no_split is 0 or 1");
        options().no_split = value;
    } else if (k == "small_deg") {
        if (value < -1 || value > 4096) return fail(GNNK_EINVAL, "small_deg must be in [-1, 4096]");
        options().small_deg = value;
    } else if (k == "schedule") {
        if (value < 0 || value > 3) return fail(GNNK_EINVAL, "schedule is 0 (auto), 1 (row), 2 (edge) or 3 (edge, atomic)");
        options().schedule = value;
    } else if (k == "edge_chunk") {
        if (value != 0 && (value < 4 || value > (1 << 20) || value % 4))
            return fail(GNNK_EINVAL, "edge_chunk is 0 (auto) or a multiple of 4 in [4, 2^20]");
        options().edge_chunk = value;
    } else if (k == "no_fast") {
        if (value != 0 && value != 1) return fail(GNNK_EINVAL, "no_fast is 0 or 1");
        options().no_fast = value;
    } else {
        return fail(GNNK_EINVAL, "unknown option '%s'", key);
    }
    return GNNK_OK;
}

const char* gnnk_last_error(void) { return g_err.c_str(); }

}  // extern "C"
