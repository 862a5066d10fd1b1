// Host-side state of the gnnk library: graph handles, options, errors.
#pragma once

#include <stdarg.h>
#include <stdint.h>

#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/gnnk.h"
#include "internal.h"

namespace gnnk {

// One traversal direction: the in-CSR (rows = destinations) or the reverse
// graph's CSR (rows = sources).
struct Dir {
    int64_t n_rows = 0;
    const void* ptr = nullptr;     // device row offsets (graph ptr type)
    const int32_t* idx = nullptr;  // device neighbour ids
    const int32_t* eid = nullptr;  // device edge ids, nullptr = identity
    int32_t* deg = nullptr;        // device degree per row
    int32_t* perm = nullptr;       // device rows by descending degree
    int4* seg = nullptr;           // device segments of hub rows
    int32_t* seg_order = nullptr;  // device segment of each hub-segment wavefront
    int4* segw = nullptr;          // device seg[seg_order[w]] with the table index in .w
    int4* rowt = nullptr;          // device {perm[k], begin, end, 0} per degree-order position
    int32_t* hub_off = nullptr;    // device first segment per hub row (n_hub + 1)
    int32_t* row = nullptr;        // device row of each position (COO form)
    int32_t* pos = nullptr;        // device position of each edge id in this CSR
    int64_t n_seg = 0, n_hub = 0, n_nz = 0, max_deg = 0;
    std::vector<int32_t> sorted_deg;  // host, descending (bin boundaries by binary search)
    std::vector<int32_t> hub_host;    // host copy of hub_off (the source of its upload)
    int64_t count_above(int64_t t) const;  // rows with degree > t
};

}  // namespace gnnk

struct gnnk_graph {
    int64_t n_src = 0, n_dst = 0, n_edges = 0;
    int ptr64 = 0;
    int identity_eids = 1;
    int64_t seg_edges = 512;       // edges per segment of a hub row of the in-CSR
    int64_t seg_edges_out = 2048;  // the same for the reverse graph's CSR
    int64_t seg_edges_fine = 256;  // the reverse graph's CSR for passes that gather node rows
    int64_t seg_edges_in_fine = 256;  // the in-CSR for passes that gather node rows
    gnnk::Dir in, out;
    // the in-CSR with segments of seg_edges_in_fine edges (its own hub tables
    // and segment order, every other array shared with `in`)
    gnnk::Dir in_fine;
    // the reverse graph's CSR with segments of seg_edges_fine edges (its own
    // hub tables and segment order, every other array shared with `out`)
    gnnk::Dir out_fine;
    int32_t* flag = nullptr;  // device word for graph_validate
    size_t ws_used = 0;
    // scratch buffers the caller lent to the handle, one per stream
    static constexpr int MAX_STREAMS = 16;
    struct Lent {
        hipStream_t stream;
        char* buf;
        size_t bytes;
    };
    Lent lent[MAX_STREAMS];
    int n_lent = 0;
    std::mutex lent_mu;
};

namespace gnnk {

struct Options {
    int64_t seg_edges = 0;  // 0: chosen per graph from its edge count (seg_edges_for)
    int64_t no_split = 0;
    int64_t small_deg = -1;
    int64_t no_fast = 0;  // 1: every call uses the runtime-layout kernels
    int64_t schedule = 0; // 0 auto, 1 row engine, 2 edge-parallel, 3 edge-parallel with atomics
    int64_t edge_chunk = 0; // positions per lane group of edge-parallel walks, 0 = auto
    int64_t fused_dw = -1;  // u_mul_e/sum's weight gradient inside the reverse dX pass: 1 always, 0 never, -1 one-column weights
    int64_t sddmm_split = 0;  // wavefronts per hub segment of a g-SDDMM, 0 = auto
};
Options& options();

// edges per hub-row segment for a graph of E edges: the option when set, else
// for the in-CSR the next power of two of E / 8192 within [64, 512], for the
// reverse graph's CSR the next power of two of E / 2048 within [64, 2048] --
// small graphs split their long rows so that enough wavefronts share the work
int64_t seg_edges_for(int64_t E, bool reverse);
// the finer segment size of the reverse graph's CSR (passes that gather node
// rows): the option when set, else the next power of two of E / 16384 within
// [64, 256]
int64_t seg_edges_fine_for(int64_t E);

gnnk_status fail(gnnk_status st, const char* fmt, ...);
gnnk_status hip_fail(hipError_t e, const char* what);
void clear_error();

// Device scratch of one compute call: the buffer lent to the handle for the
// call's stream (or the library's static buffer of the no-allocation entry
// point), handed out front to back in 256-byte steps.  take() returns
// nullptr when the buffer is too small, after recording how many bytes the
// call asked for up to that point (gnnk_scratch_needed).
struct Scratch {
    char* base = nullptr;
    size_t bytes = 0;
    size_t used = 0;
    void* take(size_t n);
};

// the buffer lent to g for stream s (empty when none)
Scratch scratch_of(gnnk_graph* g, hipStream_t s);

// status and message of a call that did not get the scratch it needs
gnnk_status scratch_fail(const Scratch& sc);

// A call made of several passes (a gradient pair, the max/min backward's
// masks and the walk that reads them, slices of heads) runs twice: first as a
// plan, with every launch skipped and its scratch only counted, so that an
// argument error or a scratch shortfall (its whole need) comes back before
// anything runs on the GPU; then for real.  While planning, scratch_of()
// hands out an unbounded buffer whose addresses are never used.
bool planning();
gnnk_status planned(gnnk_graph* g, hipStream_t s, const std::function<gnnk_status()>& run);

// gspmm with its scratch from sc (api.cpp)
gnnk_status gspmm_impl(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                       const gnnk_tensor* rhs, gnnk_tensor* out, int32_t* arg_lhs, int32_t* arg_rhs,
                       hipStream_t stream, Scratch& sc);

// size of the fixed scratch buffer of gspmm_noalloc (one per GPU)
constexpr size_t STATIC_SCRATCH_BYTES = (size_t)64 << 20;

// the fixed buffer of the GPU that `stream` runs on (noalloc.hip)
gnnk_status static_scratch(hipStream_t stream, Scratch& sc);

}  // namespace gnnk
