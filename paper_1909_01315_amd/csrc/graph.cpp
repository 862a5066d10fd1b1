// Graph handles of the gnnk library: the in-CSR, the reverse graph's CSR with
// the original edge ids (Appendix B, definition of the reverse graph), the
// degree arrays, rows sorted by degree, and the segment tables of hub rows.
//
// Every structure is built on the device (build.hip: stable radix sorts, so
// the edges of a node keep ascending edge id) into the caller's workspace.
// The host reads back only a flag word and the sorted degrees, from which it
// derives the role boundaries of the schedule and the hub segment offsets.
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <numeric>

#include "host.h"

namespace gnnk {

// ---------------------------------------------------------------------------
// errors and options

static thread_local char g_err[512];
// bytes of scratch the last call on this thread that ran short asked for
static thread_local size_t g_need = 0;
static thread_local bool g_plan = false;
static thread_local size_t g_plan_peak = 0;

gnnk_status fail(gnnk_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

gnnk_status hip_fail(hipError_t e, const char* what) {
    return fail(GNNK_EHIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

void clear_error() {
    g_err[0] = 0;
    g_need = 0;
}

Options& options() {
    static Options o;
    return o;
}

int64_t seg_edges_for(int64_t E, bool reverse) {
    if (options().seg_edges > 0) return options().seg_edges;
    // in-CSR segments of 512 edges: on the 114.6M-edge graph the gathers of
    // the in-CSR passes take 0.15-0.37 ms less each than with 2048 (more of
    // every hub row runs in narrow, source-ordered pieces); the reverse
    // passes gain nothing from it (copy_e sums and the argmax scatter lose)
    const int64_t cap = reverse ? 2048 : 512, div = reverse ? 2048 : 8192;
    int64_t S = 64;
    while (S < cap && S * div < E) S <<= 1;
    return S;
}

int64_t seg_edges_fine_for(int64_t E) {
    if (options().seg_edges > 0) return options().seg_edges;
    // the reverse passes that gather node rows (dX of the sums, the fused
    // attention's source pass) run faster on 256-edge pieces of the hub rows
    // (c3 dX of u_mul_e/sum 5.53 -> 5.06 ms); the copy_e sums and the argmax
    // scatter keep the coarser table
    int64_t S = 64;
    while (S < 256 && S * 16384 < E) S <<= 1;
    return S;
}

int64_t Dir::count_above(int64_t t) const {
    // sorted_deg is descending: the first position whose degree is <= t is the
    // first x with t >= x
    auto it = std::upper_bound(sorted_deg.begin(), sorted_deg.end(), (int32_t)std::min<int64_t>(t, INT32_MAX),
                               [](int32_t v, int32_t x) { return v >= x; });
    return (int64_t)(it - sorted_deg.begin());
}

void* Scratch::take(size_t n) {
    const size_t at = used;
    used += (n + 255) / 256 * 256;
    if (g_plan) {
        if (used > g_plan_peak) g_plan_peak = used;
        return base + at;
    }
    if (used > bytes) {
        g_need = used;
        return nullptr;
    }
    return base + at;
}

Scratch scratch_of(gnnk_graph* g, hipStream_t s) {
    Scratch sc;
    if (g_plan) {
        // a stand-in that no kernel sees: nothing is launched while planning
        sc.base = reinterpret_cast<char*>((uintptr_t)1 << 20);
        sc.bytes = SIZE_MAX;
        return sc;
    }
    std::lock_guard<std::mutex> lk(g->lent_mu);
    for (int k = 0; k < g->n_lent; ++k)
        if (g->lent[k].stream == s) {
            sc.base = g->lent[k].buf;
            sc.bytes = g->lent[k].bytes;
        }
    return sc;
}

bool planning() { return g_plan; }

gnnk_status planned(gnnk_graph* g, hipStream_t s, const std::function<gnnk_status()>& run) {
    if (g_plan) return run();
    g_plan = true;
    g_plan_peak = 0;
    const gnnk_status st = run();
    g_plan = false;
    if (st != GNNK_OK) return st;
    Scratch have = g ? scratch_of(g, s) : Scratch{};
    if (g_plan_peak > have.bytes) {
        g_need = g_plan_peak;
        return scratch_fail(have);
    }
    return run();
}

gnnk_status scratch_fail(const Scratch& sc) {
    return fail(GNNK_ENOMEM,
                "the call needs at least %zu bytes of scratch on its stream and has %zu: lend a larger buffer with "
                "graph_attach_scratch (graph_scratch_bytes gives a bound, gnnk_scratch_needed this call's need)",
                g_need, sc.bytes);
}

// ---------------------------------------------------------------------------
// workspace layout

namespace {

constexpr size_t ALIGN = 256;

// flag bits of the validation and build kernels
constexpr int32_t FLAG_INDEX = 1;     // an endpoint or index out of range
constexpr int32_t FLAG_PTR = 2;       // row offsets not a valid CSR
constexpr int32_t FLAG_PERM = 4;      // edge ids not a permutation
constexpr int32_t FLAG_NOT_IDENT = 8; // edge ids differ from in-CSR positions

// Fixed-size regions first, then the hub tables whose sizes are known only
// once the degrees are sorted.
struct Layout {
    size_t in_ptr = 0, in_idx = 0, in_eid = 0, out_ptr = 0, out_idx = 0, out_eid = 0;
    size_t in_deg = 0, out_deg = 0, in_perm = 0, out_perm = 0, in_row = 0, out_row = 0, out_pos = 0, flag = 0;
    size_t tmp = 0, tmp_words = 0;  // the build's temporaries (radix-sort counts, degree and segment sort keys)
    size_t in_hub = 0, out_hub = 0, in_seg = 0, out_seg = 0, in_sego = 0, out_sego = 0, total = 0;
    size_t fine_hub = 0, fine_seg = 0, fine_sego = 0;  // the reverse CSR's finer hub tables
    size_t in_rowt = 0, out_rowt = 0, in_segw = 0, out_segw = 0, fine_segw = 0;  // per-wavefront lookup tables
    size_t ifine_hub = 0, ifine_seg = 0, ifine_sego = 0, ifine_segw = 0;  // the in-CSR's finer hub tables
};

struct Bump {
    size_t off = 0;
    size_t take(size_t bytes) {
        size_t o = off;
        off += (bytes + ALIGN - 1) / ALIGN * ALIGN;
        return o;
    }
};

// segments a graph can have at most: hub rows have more than S edges, so at
// most E / S of them, and at most E / S + (hub rows) <= 2 E / S + 2 segments
int64_t max_segments(int64_t E, int64_t S) { return 2 * E / S + 2; }

// the smallest segment size of a graph's tables (the most segments)
int64_t min_seg_edges(const gnnk_graph* g) {
    return std::min({g->seg_edges, g->seg_edges_out, g->seg_edges_fine, g->seg_edges_in_fine});
}

// uint32 words of build temporaries: the radix sort of the edges, or four
// row-sized arrays plus the sort of the degree keys, or the same for the
// segment keys
size_t build_tmp_words(int64_t n_src, int64_t n_dst, int64_t E, int64_t S) {
    const int64_t n = std::max(n_src, n_dst);
    const int64_t m = max_segments(E, S);
    auto pad = [](int64_t x) { return (size_t)((x + 63) / 64 * 64); };
    return std::max({radix_scratch_words(E), 4 * pad(n + 64) + radix_scratch_words(n),
                     4 * pad(m) + radix_scratch_words(m)});
}

Layout make_layout(int64_t n_src, int64_t n_dst, int64_t E, size_t ps, int64_t S, int64_t hub_in, int64_t hub_out,
                   int64_t seg_in, int64_t seg_out, int64_t hub_fine = 0, int64_t seg_fine = 0,
                   int64_t hub_ifine = 0, int64_t seg_ifine = 0) {
    Layout L;
    Bump b;
    L.in_ptr = b.take((size_t)(n_dst + 1) * ps);
    L.in_idx = b.take((size_t)E * 4);
    L.in_eid = b.take((size_t)E * 4);
    L.out_ptr = b.take((size_t)(n_src + 1) * ps);
    L.out_idx = b.take((size_t)E * 4);
    L.out_eid = b.take((size_t)E * 4);
    L.in_deg = b.take((size_t)n_dst * 4);
    L.out_deg = b.take((size_t)n_src * 4);
    L.in_perm = b.take((size_t)n_dst * 4);
    L.out_perm = b.take((size_t)n_src * 4);
    L.in_row = b.take((size_t)E * 4);
    L.out_row = b.take((size_t)E * 4);
    L.out_pos = b.take((size_t)E * 4);
    L.flag = b.take(ALIGN);
    L.in_rowt = b.take((size_t)n_dst * 16);
    L.out_rowt = b.take((size_t)n_src * 16);
    L.tmp_words = build_tmp_words(n_src, n_dst, E, S);
    L.tmp = b.take(L.tmp_words * 4);
    L.in_hub = b.take((size_t)(hub_in + 1) * 4);
    L.out_hub = b.take((size_t)(hub_out + 1) * 4);
    L.in_seg = b.take((size_t)seg_in * 16);
    L.out_seg = b.take((size_t)seg_out * 16);
    L.in_sego = b.take((size_t)seg_in * 4);
    L.out_sego = b.take((size_t)seg_out * 4);
    L.fine_hub = b.take((size_t)(hub_fine + 1) * 4);
    L.fine_seg = b.take((size_t)seg_fine * 16);
    L.fine_sego = b.take((size_t)seg_fine * 4);
    L.in_segw = b.take((size_t)seg_in * 16);
    L.out_segw = b.take((size_t)seg_out * 16);
    L.fine_segw = b.take((size_t)seg_fine * 16);
    L.ifine_hub = b.take((size_t)(hub_ifine + 1) * 4);
    L.ifine_seg = b.take((size_t)seg_ifine * 16);
    L.ifine_sego = b.take((size_t)seg_ifine * 4);
    L.ifine_segw = b.take((size_t)seg_ifine * 16);
    L.total = b.off;
    return L;
}

// Edge ids and CSR positions are int32.  The walks advance a position past a
// row's end by at most 64 lane groups x 4 slots before testing it, so edge
// counts stay 2^16 below the int32 limit and no position arithmetic wraps.
constexpr int64_t MAX_EDGES = (int64_t)INT32_MAX - 65536;

bool sizes_ok(int64_t n_src, int64_t n_dst, int64_t E) {
    return n_src >= 0 && n_dst >= 0 && E >= 0 && n_src < INT32_MAX && n_dst < INT32_MAX && E <= MAX_EDGES;
}

// bits of a row id below n_rows
int row_bits(int64_t n_rows) { return key_bits(n_rows > 1 ? (uint64_t)(n_rows - 1) : 0); }

// one traversal direction's derived host state from its sorted degrees
void schedule_host(Dir& d, int64_t S, std::vector<int32_t>& hub_off) {
    d.max_deg = d.n_rows ? d.sorted_deg[0] : 0;
    d.n_nz = d.count_above(0);
    d.n_hub = d.count_above(S);
    hub_off.assign((size_t)d.n_hub + 1, 0);
    for (int64_t k = 0; k < d.n_hub; ++k)
        hub_off[(size_t)k + 1] = hub_off[(size_t)k] + (int32_t)((d.sorted_deg[(size_t)k] + S - 1) / S);
    d.n_seg = hub_off[(size_t)d.n_hub];
}

struct Builder {
    gnnk_graph* g;
    char* W;
    Layout L;
    uint32_t* scratch = nullptr;
    hipStream_t s;
    hipError_t err = hipSuccess;
    size_t scratch_words = 0;  // uint32 words of `scratch`

    void chk(hipError_t x) {
        if (err == hipSuccess) err = x;
    }
    template <typename T>
    T* at(size_t off) {
        return reinterpret_cast<T*>(W + off);
    }
    int32_t read_flag() {
        int32_t h = 0;
        chk(hipMemcpyAsync(&h, g->flag, 4, hipMemcpyDeviceToHost, s));
        chk(hipStreamSynchronize(s));
        return h;
    }

    // the build's temporaries, a region of the workspace
    void get_scratch() {
        scratch = at<uint32_t>(L.tmp);
        scratch_words = L.tmp_words;
    }

    // the reverse graph's CSR from the source and destination of every edge id
    void build_reverse(const int32_t* src_of_e, const int32_t* dst_of_e) {
        const int64_t E = g->n_edges;
        Dir& d = g->out;
        d.ptr = W + L.out_ptr;
        d.idx = at<int32_t>(L.out_idx);
        d.eid = at<int32_t>(L.out_eid);
        d.row = at<int32_t>(L.out_row);
        d.pos = at<int32_t>(L.out_pos);
        chk(radix_sort_pairs(reinterpret_cast<const uint32_t*>(src_of_e), nullptr, E, row_bits(g->n_src),
                             at<uint32_t>(L.out_row), at<uint32_t>(L.out_eid), at<uint32_t>(L.out_idx),
                             at<uint32_t>(L.out_pos), scratch, s));
        chk(launch_ptr_from_keys(at<uint32_t>(L.out_row), E, g->n_src, W + L.out_ptr, g->ptr64, s));
        chk(launch_gather(dst_of_e, at<uint32_t>(L.out_eid), E, at<int32_t>(L.out_idx), s));
        chk(launch_inverse(at<int32_t>(L.out_eid), E, at<int32_t>(L.out_pos), s));
    }

    // degrees and rows by descending degree (ties by row id) on the device;
    // the sorted degrees are copied into d.sorted_deg (complete after the
    // next synchronisation of s)
    void order_rows(Dir& d, std::vector<uint32_t>& keys_h) {
        const int64_t n = d.n_rows, E = g->n_edges;
        const int64_t pad = (n + 63) / 64 * 64;
        uint32_t* key = scratch;
        uint32_t* sorted = key + pad;
        uint32_t* tk = sorted + pad;
        uint32_t* tv = tk + pad;
        uint32_t* rs = tv + pad;
        chk(launch_degrees(d.ptr, g->ptr64, n, d.deg, key, (uint32_t)E, s));
        chk(radix_sort_pairs(key, nullptr, n, key_bits((uint64_t)E), sorted, reinterpret_cast<uint32_t*>(d.perm), tk,
                             tv, rs, s));
        keys_h.resize((size_t)n);
        if (n > 0) chk(hipMemcpyAsync(keys_h.data(), sorted, (size_t)n * 4, hipMemcpyDeviceToHost, s));
    }

    // The order in which wavefronts take the hub segments of a direction:
    // by the neighbour ids a segment covers (its key, the halves of its
    // first and last neighbour id summed), a stable sort, so equal keys keep
    // table order.  Where rows list their neighbours in ascending order, the
    // segments that run at the same time then gather from one slice of the
    // neighbour table; elsewhere the order changes nothing.  Results do not
    // depend on it (partials are combined in table order).
    void order_segments(Dir& d, int64_t n_cols) {
        const int64_t n = d.n_seg;
        if (n <= 0) return;
        const int64_t pad = (n + 63) / 64 * 64;
        // the temporaries are sized for the largest segment count a graph of
        // this size can have
        if (4 * (size_t)pad + radix_scratch_words(n) > scratch_words) {
            if (err == hipSuccess) err = hipErrorInvalidValue;
            return;
        }
        uint32_t* key = scratch;
        uint32_t* sorted = key + pad;
        uint32_t* tk = sorted + pad;
        uint32_t* tv = tk + pad;
        uint32_t* rs = tv + pad;
        chk(launch_seg_keys(d.seg, n, d.idx, key, s));
        chk(radix_sort_pairs(key, nullptr, n, key_bits(n_cols > 1 ? (uint64_t)(n_cols - 1) : 0), sorted,
                             reinterpret_cast<uint32_t*>(d.seg_order), tk, tv, rs, s));
    }

    // common tail: degree order, identity flag, hub tables
    gnnk_status finish(size_t ws_bytes, bool check_identity) {
        const int64_t E = g->n_edges;
        Dir& in = g->in;
        Dir& out = g->out;
        in.n_rows = g->n_dst;
        out.n_rows = g->n_src;
        in.deg = at<int32_t>(L.in_deg);
        out.deg = at<int32_t>(L.out_deg);
        in.perm = at<int32_t>(L.in_perm);
        out.perm = at<int32_t>(L.out_perm);
        std::vector<uint32_t> kin, kout;
        order_rows(in, kin);
        order_rows(out, kout);
        const int32_t h = read_flag();  // also completes the two copies above
        if (err != hipSuccess) return hip_fail(err, "graph build");
        if (check_identity) {
            g->identity_eids = !(h & FLAG_NOT_IDENT);
            if (g->identity_eids) in.eid = nullptr;
        }
        in.sorted_deg.resize(kin.size());
        for (size_t k = 0; k < kin.size(); ++k) in.sorted_deg[k] = (int32_t)((uint32_t)E - kin[k]);
        out.sorted_deg.resize(kout.size());
        for (size_t k = 0; k < kout.size(); ++k) out.sorted_deg[k] = (int32_t)((uint32_t)E - kout[k]);
        std::vector<int32_t>& hin = in.hub_host;
        std::vector<int32_t>& hout = out.hub_host;
        schedule_host(in, g->seg_edges, hin);
        schedule_host(out, g->seg_edges_out, hout);
        Dir& fine = g->out_fine;
        const bool finer = g->seg_edges_fine < g->seg_edges_out;
        fine = out;
        if (finer) schedule_host(fine, g->seg_edges_fine, fine.hub_host);
        Dir& ifine = g->in_fine;
        const bool ifiner = g->seg_edges_in_fine < g->seg_edges;
        ifine = in;
        if (ifiner) schedule_host(ifine, g->seg_edges_in_fine, ifine.hub_host);
        L = make_layout(g->n_src, g->n_dst, E, g->ptr64 ? 8 : 4, min_seg_edges(g), in.n_hub, out.n_hub, in.n_seg,
                        out.n_seg, finer ? fine.n_hub : 0, finer ? fine.n_seg : 0, ifiner ? ifine.n_hub : 0,
                        ifiner ? ifine.n_seg : 0);
        if (ws_bytes < L.total)
            return fail(GNNK_ENOMEM, "workspace of %zu bytes is smaller than the %zu bytes this graph needs",
                        ws_bytes, L.total);
        in.hub_off = at<int32_t>(L.in_hub);
        out.hub_off = at<int32_t>(L.out_hub);
        in.seg = at<int4>(L.in_seg);
        out.seg = at<int4>(L.out_seg);
        in.seg_order = at<int32_t>(L.in_sego);
        out.seg_order = at<int32_t>(L.out_sego);
        in.segw = at<int4>(L.in_segw);
        out.segw = at<int4>(L.out_segw);
        in.rowt = at<int4>(L.in_rowt);
        out.rowt = at<int4>(L.out_rowt);
        chk(launch_row_table(in.ptr, g->ptr64, in.perm, in.n_rows, in.rowt, s));
        chk(launch_row_table(out.ptr, g->ptr64, out.perm, out.n_rows, out.rowt, s));
        chk(hipMemcpyAsync(in.hub_off, hin.data(), hin.size() * 4, hipMemcpyHostToDevice, s));
        chk(hipMemcpyAsync(out.hub_off, hout.data(), hout.size() * 4, hipMemcpyHostToDevice, s));
        chk(launch_hub_segments(in.ptr, g->ptr64, in.perm, in.hub_off, in.n_hub, g->seg_edges, in.seg, s));
        chk(launch_hub_segments(out.ptr, g->ptr64, out.perm, out.hub_off, out.n_hub, g->seg_edges_out, out.seg, s));
        order_segments(in, g->n_src);
        order_segments(out, g->n_dst);
        chk(launch_seg_wave(in.seg, in.seg_order, in.n_seg, in.segw, s));
        chk(launch_seg_wave(out.seg, out.seg_order, out.n_seg, out.segw, s));
        if (finer) {
            fine.hub_off = at<int32_t>(L.fine_hub);
            fine.seg = at<int4>(L.fine_seg);
            fine.seg_order = at<int32_t>(L.fine_sego);
            fine.segw = at<int4>(L.fine_segw);
            fine.rowt = out.rowt;
            chk(hipMemcpyAsync(fine.hub_off, fine.hub_host.data(), fine.hub_host.size() * 4, hipMemcpyHostToDevice,
                               s));
            chk(launch_hub_segments(fine.ptr, g->ptr64, fine.perm, fine.hub_off, fine.n_hub, g->seg_edges_fine,
                                    fine.seg, s));
            order_segments(fine, g->n_dst);
            chk(launch_seg_wave(fine.seg, fine.seg_order, fine.n_seg, fine.segw, s));
        } else {
            fine = out;
        }
        if (ifiner) {
            ifine.hub_off = at<int32_t>(L.ifine_hub);
            ifine.seg = at<int4>(L.ifine_seg);
            ifine.seg_order = at<int32_t>(L.ifine_sego);
            ifine.segw = at<int4>(L.ifine_segw);
            ifine.rowt = in.rowt;
            chk(hipMemcpyAsync(ifine.hub_off, ifine.hub_host.data(), ifine.hub_host.size() * 4,
                               hipMemcpyHostToDevice, s));
            chk(launch_hub_segments(ifine.ptr, g->ptr64, ifine.perm, ifine.hub_off, ifine.n_hub,
                                    g->seg_edges_in_fine, ifine.seg, s));
            order_segments(ifine, g->n_src);
            chk(launch_seg_wave(ifine.seg, ifine.seg_order, ifine.n_seg, ifine.segw, s));
        } else {
            ifine = in;
        }
        chk(hipMemsetAsync(g->flag, 0, 4, s));
        // the host copies of the hub offsets stay with the handle, so the
        // copies above may still be in flight when the call returns
        if (err != hipSuccess) return hip_fail(err, "graph build");
        g->ws_used = L.total;
        return GNNK_OK;
    }
};

// The handle owns no device memory (its arrays live in the caller's
// workspace, its scratch is lent by the caller), so destroying it is a host
// operation; kernels still in flight keep reading the caller's buffers.
void free_graph(gnnk_graph* g) { delete g; }

gnnk_graph* new_graph(int64_t num_src, int64_t num_dst, int64_t num_edges, gnnk_itype ptr_t) {
    gnnk_graph* g = new gnnk_graph();
    g->n_src = num_src;
    g->n_dst = num_dst;
    g->n_edges = num_edges;
    g->ptr64 = ptr_t == GNNK_I64;
    g->seg_edges = seg_edges_for(num_edges, false);
    g->seg_edges_out = seg_edges_for(num_edges, true);
    g->seg_edges_fine = seg_edges_fine_for(num_edges);
    g->seg_edges_in_fine = seg_edges_fine_for(num_edges);
    return g;
}

// workspace checks shared by both constructors; fills b.W, b.L, g->flag
gnnk_status begin_build(Builder& b, void* ws, size_t ws_bytes) {
    gnnk_graph* g = b.g;
    b.L = make_layout(g->n_src, g->n_dst, g->n_edges, g->ptr64 ? 8 : 4, min_seg_edges(g), 0, 0, 0, 0);
    if (!ws || ws_bytes < b.L.total)
        return fail(GNNK_ENOMEM, "workspace of %zu bytes is smaller than the %zu bytes this graph needs", ws_bytes,
                    b.L.total);
    b.W = reinterpret_cast<char*>(ws);
    if ((uintptr_t)b.W % ALIGN) return fail(GNNK_EINVAL, "workspace must be 256-byte aligned");
    g->flag = b.at<int32_t>(b.L.flag);
    b.chk(hipMemsetAsync(g->flag, 0, 4, b.s));
    return GNNK_OK;
}

gnnk_status create_coo(Builder& b, const int32_t* src, const int32_t* dst, void* ws, size_t ws_bytes) {
    gnnk_graph* g = b.g;
    const int64_t E = g->n_edges;
    gnnk_status st = begin_build(b, ws, ws_bytes);
    if (st != GNNK_OK) return st;
    b.chk(launch_validate(src, E, g->n_src, g->flag, b.s));
    b.chk(launch_validate(dst, E, g->n_dst, g->flag, b.s));
    const int32_t h = b.read_flag();
    if (b.err != hipSuccess) return hip_fail(b.err, "checking the edge list");
    if (h & FLAG_INDEX) return fail(GNNK_EINVAL, "an edge has an endpoint out of range");
    b.get_scratch();
    const Layout& L = b.L;
    Dir& in = g->in;
    in.ptr = b.W + L.in_ptr;
    in.idx = b.at<int32_t>(L.in_idx);
    in.eid = b.at<int32_t>(L.in_eid);
    in.row = b.at<int32_t>(L.in_row);
    // in-CSR: edges sorted by destination, ties in edge-id order
    b.chk(radix_sort_pairs(reinterpret_cast<const uint32_t*>(dst), nullptr, E, row_bits(g->n_dst),
                           b.at<uint32_t>(L.in_row), b.at<uint32_t>(L.in_eid), b.at<uint32_t>(L.out_row),
                           b.at<uint32_t>(L.out_pos), b.scratch, b.s));
    b.chk(launch_ptr_from_keys(b.at<uint32_t>(L.in_row), E, g->n_dst, b.W + L.in_ptr, g->ptr64, b.s));
    b.chk(launch_gather(src, b.at<uint32_t>(L.in_eid), E, b.at<int32_t>(L.in_idx), b.s));
    b.chk(launch_check_identity(b.at<int32_t>(L.in_eid), E, g->flag, FLAG_NOT_IDENT, b.s));
    b.build_reverse(src, dst);
    return b.finish(ws_bytes, true);
}

gnnk_status create_csr(Builder& b, const void* indptr, const int32_t* indices, const int32_t* eids, void* ws,
                       size_t ws_bytes) {
    gnnk_graph* g = b.g;
    const int64_t E = g->n_edges;
    gnnk_status st = begin_build(b, ws, ws_bytes);
    if (st != GNNK_OK) return st;
    const Layout& L = b.L;
    b.chk(launch_validate_ptr(indptr, g->ptr64, g->n_dst, E, g->flag, b.s));
    b.chk(launch_validate(indices, E, g->n_src, g->flag, b.s));
    if (eids) {
        b.chk(launch_check_permutation(eids, E, b.at<uint32_t>(L.out_pos), g->flag, FLAG_PERM, b.s));
        b.chk(launch_check_identity(eids, E, g->flag, FLAG_NOT_IDENT, b.s));
    }
    const int32_t h = b.read_flag();
    if (b.err != hipSuccess) return hip_fail(b.err, "checking the CSR");
    if (h & FLAG_PTR)
        return fail(GNNK_EINVAL, "indptr must start at 0, end at num_edges and never decrease");
    if (h & FLAG_INDEX) return fail(GNNK_EINVAL, "an index is out of range");
    if (h & FLAG_PERM) return fail(GNNK_EINVAL, "eids is not a permutation of 0..num_edges-1");
    b.get_scratch();
    const bool identity = !eids || !(h & FLAG_NOT_IDENT);
    g->identity_eids = identity;
    Dir& in = g->in;
    in.ptr = indptr;
    in.idx = indices;
    in.eid = identity ? nullptr : eids;
    in.row = b.at<int32_t>(L.in_row);
    b.chk(launch_fill_rows(indptr, g->ptr64, g->n_dst, E, in.row, b.s));
    if (identity) {
        b.build_reverse(indices, in.row);
    } else {
        int32_t* src_of_e = b.at<int32_t>(L.in_idx);
        int32_t* dst_of_e = b.at<int32_t>(L.in_eid);
        b.chk(launch_edge_ends(indices, eids, in.row, E, src_of_e, dst_of_e, b.s));
        b.build_reverse(src_of_e, dst_of_e);
    }
    return b.finish(ws_bytes, false);
}

}  // namespace
}  // namespace gnnk

using namespace gnnk;

extern "C" {

gnnk_status graph_workspace_bytes(int64_t num_src, int64_t num_dst, int64_t num_edges, gnnk_itype ptr_t,
                                  size_t* bytes) {
    clear_error();
    if (!bytes) return fail(GNNK_EINVAL, "bytes is NULL");
    if (!sizes_ok(num_src, num_dst, num_edges)) return fail(GNNK_EINVAL, "sizes out of range (node counts < 2^31 - 1, edges <= 2^31 - 2^16 - 1)");
    if (ptr_t != GNNK_I32 && ptr_t != GNNK_I64) return fail(GNNK_EINVAL, "bad ptr type");
    // hub rows have more than S edges: at most E / S of them, and at most
    // E / S + (hub rows) <= 2 E / S segments
    const int64_t Si = seg_edges_for(num_edges, false), So = seg_edges_for(num_edges, true);
    const int64_t Sf = seg_edges_fine_for(num_edges);  // both CSRs' finer tables
    Layout L = make_layout(num_src, num_dst, num_edges, ptr_t == GNNK_I64 ? 8 : 4, std::min({Si, So, Sf}),
                           num_edges / Si + 1, num_edges / So + 1, max_segments(num_edges, Si),
                           max_segments(num_edges, So), Sf < So ? num_edges / Sf + 1 : 0,
                           Sf < So ? max_segments(num_edges, Sf) : 0, Sf < Si ? num_edges / Sf + 1 : 0,
                           Sf < Si ? max_segments(num_edges, Sf) : 0);
    *bytes = L.total;
    return GNNK_OK;
}

gnnk_status graph_create_coo(int64_t num_src, int64_t num_dst, int64_t num_edges, const int32_t* src,
                             const int32_t* dst, gnnk_itype ptr_t, void* workspace, size_t ws_bytes,
                             hipStream_t stream, gnnk_graph_t* out) {
    clear_error();
    if (!out) return fail(GNNK_EINVAL, "out is NULL");
    *out = nullptr;
    if (!sizes_ok(num_src, num_dst, num_edges)) return fail(GNNK_EINVAL, "sizes out of range (node counts < 2^31 - 1, edges <= 2^31 - 2^16 - 1)");
    if (ptr_t != GNNK_I32 && ptr_t != GNNK_I64) return fail(GNNK_EINVAL, "bad ptr type");
    if (num_edges > 0 && (!src || !dst)) return fail(GNNK_EINVAL, "src/dst is NULL");
    Builder b{new_graph(num_src, num_dst, num_edges, ptr_t), nullptr, {}, nullptr, stream};
    gnnk_status st = create_coo(b, src, dst, workspace, ws_bytes);
    if (st != GNNK_OK) {
        free_graph(b.g);
        return st;
    }
    *out = b.g;
    return GNNK_OK;
}

gnnk_status graph_create_csr(int64_t num_src, int64_t num_dst, int64_t num_edges, const void* indptr,
                             gnnk_itype ptr_t, const int32_t* indices, const int32_t* eids, void* workspace,
                             size_t ws_bytes, hipStream_t stream, gnnk_graph_t* out) {
    clear_error();
    if (!out) return fail(GNNK_EINVAL, "out is NULL");
    *out = nullptr;
    if (!sizes_ok(num_src, num_dst, num_edges)) return fail(GNNK_EINVAL, "sizes out of range (node counts < 2^31 - 1, edges <= 2^31 - 2^16 - 1)");
    if (ptr_t != GNNK_I32 && ptr_t != GNNK_I64) return fail(GNNK_EINVAL, "bad ptr type");
    if (!indptr || (num_edges > 0 && !indices)) return fail(GNNK_EINVAL, "indptr/indices is NULL");
    Builder b{new_graph(num_src, num_dst, num_edges, ptr_t), nullptr, {}, nullptr, stream};
    gnnk_status st = create_csr(b, indptr, indices, eids, workspace, ws_bytes);
    if (st != GNNK_OK) {
        free_graph(b.g);
        return st;
    }
    *out = b.g;
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
    info->seg_edges_out = g->seg_edges_out;
    info->seg_edges_gather = g->seg_edges_fine;
    info->segments_gather = g->out_fine.n_seg;
    info->seg_edges_in_gather = g->seg_edges_in_fine;
    info->segments_in_gather = g->in_fine.n_seg;
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
    free_graph(g);
    return GNNK_OK;
}

gnnk_status graph_attach_scratch(gnnk_graph_t g, hipStream_t stream, void* buf, size_t bytes) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (bytes > 0 && !buf) return fail(GNNK_EINVAL, "buf is NULL");
    if ((uintptr_t)buf % ALIGN) return fail(GNNK_EINVAL, "scratch must be 256-byte aligned");
    std::lock_guard<std::mutex> lk(g->lent_mu);
    int k = 0;
    while (k < g->n_lent && g->lent[k].stream != stream) ++k;
    if (!buf || bytes == 0) {
        if (k < g->n_lent) g->lent[k] = g->lent[--g->n_lent];
        return GNNK_OK;
    }
    if (k == g->n_lent) {
        if (g->n_lent == gnnk_graph::MAX_STREAMS)
            return fail(GNNK_EINVAL, "a handle takes scratch for at most %d streams", gnnk_graph::MAX_STREAMS);
        ++g->n_lent;
    }
    g->lent[k] = {stream, reinterpret_cast<char*>(buf), bytes};
    return GNNK_OK;
}

gnnk_status gnnk_scratch_needed(size_t* bytes) {
    // not clear_error(): this reports on the previous call
    if (!bytes) return GNNK_EINVAL;
    *bytes = g_need;
    return GNNK_OK;
}

gnnk_status gnnk_set_option(const char* key, int64_t value) {
    clear_error();
    if (!key) return fail(GNNK_EINVAL, "NULL key");
    std::string k(key);
    if (k == "seg_edges") {
        if (value != 0 && (value < 32 || value > (1 << 30)))
            return fail(GNNK_EINVAL, "seg_edges is 0 (per graph, from its edge count) or in [32, 2^30]");
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
    } else if (k == "fused_dw") {
        if (value < -1 || value > 1) return fail(GNNK_EINVAL, "fused_dw is -1 (auto), 0 or 1");
        options().fused_dw = value;
    } else if (k == "sddmm_split") {
        if (value < 0 || value > 8) return fail(GNNK_EINVAL, "sddmm_split is 0 (auto) or in [1, 8]");
        options().sddmm_split = value;
    } else if (k == "no_fast") {
        if (value != 0 && value != 1) return fail(GNNK_EINVAL, "no_fast is 0 or 1");
        options().no_fast = value;
    } else {
        return fail(GNNK_EINVAL, "unknown option '%s'", key);
    }
    return GNNK_OK;
}

const char* gnnk_last_error(void) { return g_err; }

}  // extern "C"
