// C ABI of the gnnk operators: argument checks, the geometry of a call
// (broadcast pattern, vector width, lanes per edge), the schedule over the
// degree-sorted rows, and the kernel launches.
//
// Theorem 1 of the paper drives the backward entry points: every gradient is
// one more pass of the same row engine, a g-SpMM over the in-CSR or the
// reverse graph's CSR, or a g-SDDMM over the in-CSR, with the message of the
// corresponding lemma.
#include <algorithm>
#include <vector>

#include "host.h"

namespace gnnk {
namespace {

enum Kind { K_FULL = 0, K_HEADS = 1, K_SCALAR = 2, K_BAD = 3 };

bool tensor_ok(const gnnk_tensor* t) {
    return t && t->heads >= 1 && t->feat >= 1 && (t->dtype == GNNK_F32 || t->dtype == GNNK_BF16) &&
           t->row_stride >= (int64_t)t->heads * t->feat && t->row_stride < ((int64_t)1 << 31) && t->rows >= 0 &&
           (t->data || t->rows == 0);
}

// shape of a tensor against an (H, F) message
Kind kind_of(const gnnk_tensor* t, int H, int F) {
    if (t->heads == H && t->feat == F) return K_FULL;
    if (H == 1 && t->heads == 1 && t->feat == F) return K_FULL;
    if (t->heads == H && t->feat == 1) return K_HEADS;
    if (t->heads == 1 && t->feat == 1) return K_SCALAR;
    return K_BAD;
}

struct Member {
    const gnnk_tensor* t;
    Kind kind;
};

struct Geo {
    int H = 1, F = 1, vec = 1, NV = 1, L = 1, log2L = 0, G = 64, nchunk = 1;
    bool merged = false;
    int64_t D = 1;
};

int pow2ceil(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

// Choose the canonical geometry of an (Hm, Fm) message read and written by
// `ms`.  When no tensor broadcasts over features only, heads and features
// merge into one row of Hm * Fm columns, unless keep_heads (a kernel that
// needs each lane's head, as the fused attention does; with Fm = 1 its
// per-head scores have the shape of a full operand).
gnnk_status choose_geo(int Hm, int Fm, std::vector<Member>& ms, const std::vector<const void*>& int_arrays, Geo& g,
                       bool keep_heads = false) {
    for (auto& m : ms) {
        m.kind = kind_of(m.t, Hm, Fm);
        if (m.kind == K_BAD)
            return fail(GNNK_EINVAL, "tensor (%d, %d) does not broadcast against the (%d, %d) message", m.t->heads,
                        m.t->feat, Hm, Fm);
    }
    bool any_heads = false;
    for (auto& m : ms) any_heads = any_heads || (m.kind == K_HEADS);
    g.merged = !any_heads && !keep_heads;
    g.H = g.merged ? 1 : Hm;
    g.F = g.merged ? Hm * Fm : Fm;
    g.D = (int64_t)Hm * Fm;
    const int es = ms.empty() ? 4 : (ms[0].t->dtype == GNNK_BF16 ? 2 : 4);
    int cand[4] = {8, 4, 2, 1};
    g.vec = 1;
    for (int v : cand) {
        if (v == 8 && es == 4) continue;
        if (g.F % v) continue;
        bool ok = true;
        for (auto& m : ms) {
            if (m.kind != K_FULL) continue;
            if ((uintptr_t)m.t->data % (size_t)(v * es) || m.t->row_stride % v) ok = false;
        }
        for (const void* p : int_arrays)
            if (p && (uintptr_t)p % (size_t)std::min(16, v * 4)) ok = false;
        if (ok) {
            g.vec = v;
            break;
        }
    }
    g.NV = (int)(g.D / g.vec);
    if (g.NV > 64) {
        g.L = 64;
        g.nchunk = (g.NV + 63) / 64;
    } else {
        g.L = pow2ceil(g.NV);
        g.nchunk = 1;
    }
    g.log2L = 0;
    while ((1 << g.log2L) < g.L) ++g.log2L;
    g.G = 64 / g.L;
    return GNNK_OK;
}

OperandDev operand(const gnnk_tensor* t, Kind k, int32_t target) {
    OperandDev o{};
    if (!t) return o;
    o.data = t->data;
    o.stride = t->row_stride;
    o.target = target;
    o.full = k == K_FULL;
    o.hmul = k == K_HEADS ? 1 : 0;
    return o;
}

// output reduction over broadcast positions
gnnk_status out_desc(const gnnk_tensor* t, Kind k, const Geo& g, OutDev& o) {
    o.data = t->data;
    o.stride = t->row_stride;
    if (k == K_FULL) {
        o.reduce = 0;
        o.red = 1;
        o.per_head = 0;
        return GNNK_OK;
    }
    o.reduce = 1;
    if (k == K_HEADS && g.F != g.D) {
        // the entry points split the heads into slices of at most one pass
        if (g.nchunk > 1) return fail(GNNK_EUNSUPPORTED, "per-head sums wider than one pass of the wavefront");
        o.red = g.F / g.vec;
        o.per_head = 1;
    } else {
        // the whole row: lanes past NV hold zeros, so a run of L lanes (a
        // power of two) gives the same sum
        o.red = g.L;
        o.per_head = 0;
    }
    return GNNK_OK;
}

CsrDev csr_of(const gnnk_graph* g, const Dir& d) {
    CsrDev c{};
    c.ptr = d.ptr;
    c.idx = d.idx;
    c.eid = d.eid;
    c.perm = d.perm;
    c.seg = d.seg;
    c.seg_order = d.seg_order;
    c.hub_off = d.hub_off;
    c.row = d.row;
    c.segw = d.segw;
    c.rowt = d.rowt;
    c.ptr64 = g->ptr64;
    return c;
}

// hub_above >= 0: the hub rows are the rows longer than hub_above, taken
// whole (a kernel that gives each one a workgroup, with no segments)
SchedDev schedule(const Dir& d, const Geo& geo, bool fill_empty, int64_t hub_above = -1) {
    SchedDev s{};
    const Options& o = options();
    const bool split = o.no_split == 0;
    const int64_t n_hub = hub_above >= 0 ? (split ? d.count_above(hub_above) : 0) : (split ? d.n_hub : 0);
    const int64_t n_seg = hub_above >= 0 ? 0 : (split ? d.n_seg : 0);
    // rows of at most T edges take one lane group each; automatic: 32 (at
    // least the lane groups of a wavefront), none when a wavefront is one group
    int64_t T = o.small_deg >= 0 ? o.small_deg : (geo.G > 1 ? std::max<int64_t>(geo.G, 32) : 0);
    int64_t n_big = std::max(d.count_above(T), n_hub);
    n_big = std::min(n_big, d.n_nz);
    const int fr = 4;
    s.n_seg = (int32_t)n_seg;
    s.n_hub = (int32_t)n_hub;
    s.n_big = (int32_t)n_big;
    s.n_nz = (int32_t)d.n_nz;
    s.n_rows = (int32_t)d.n_rows;
    s.w_big_end = (int32_t)(n_seg + (n_big - n_hub));
    s.w_small_end = (int32_t)(s.w_big_end + (d.n_nz - n_big + geo.G - 1) / geo.G);
    s.fill_rows_per_group = fr;
    int64_t fill_waves = fill_empty ? (d.n_rows - d.n_nz + (int64_t)geo.G * fr - 1) / ((int64_t)geo.G * fr) : 0;
    s.w_total = (int32_t)(s.w_small_end + fill_waves);
    return s;
}

void set_geo(EngineArgs& A, const Geo& g) {
    A.geo.F = g.F;
    A.geo.NV = g.NV;
    A.geo.L = g.L;
    A.geo.log2L = g.log2L;
    A.geo.G = g.G;
    A.geo.nchunk = g.nchunk;
}

int dtype_code(const gnnk_tensor* t) { return t->dtype == GNNK_BF16 ? 1 : 0; }

bool same_dtype(std::initializer_list<const gnnk_tensor*> ts) {
    int d = -1;
    for (auto t : ts) {
        if (!t) continue;
        if (d < 0) d = t->dtype;
        else if (t->dtype != d) return false;
    }
    return true;
}

int64_t rows_of_target(const gnnk_graph* g, int t) {
    return t == GNNK_SRC ? g->n_src : (t == GNNK_DST ? g->n_dst : g->n_edges);
}

gnnk_status launch_status(hipError_t e, const char* what) { return e == hipSuccess ? GNNK_OK : hip_fail(e, what); }

// a kernel launch, skipped (and not evaluated) while a call is being planned
#define GNNK_LAUNCH(call, what) (planning() ? GNNK_OK : launch_status((call), (what)))

// A node table addressed with 32-bit byte offsets by the fast kernels.
bool fits32(const OperandDev& o, int64_t rows, int es) {
    if (!o.data) return false;
    const uint64_t rb = (uint64_t)o.stride * (uint64_t)es;
    return rows < (1 << 24) && rb < (1u << 24) && (uint64_t)rows * rb <= 0xFFFFFFFFull;
}

// rows of the table an operand reads during a walk over `d`
int64_t table_rows(const gnnk_graph* g, const Dir& d, int32_t target) {
    const bool in = &d == &g->in || &d == &g->in_fine;
    if (target == T_EDGE) return g->n_edges;
    if (target == T_NBR) return in ? g->n_src : g->n_dst;
    return in ? g->n_dst : g->n_src;
}

struct Pick {
    int spec = SP_DYN;
    int gc = 0;
};

bool fast_geo(const Geo& geo, int dtype) {
    return geo.G >= 1 && geo.G <= 32 && fast_vec(dtype, geo.vec);
}

// the compile-time layout of a g-SpMM call, when one matches
Pick pick_spmm(const gnnk_graph* g, const Dir& d, EngineArgs& A, const Geo& geo, int dtype, int opk, bool maxmin) {
    Pick p;
    // outputs summed over broadcast positions keep the runtime-layout kernels
    if (options().no_fast || !fast_geo(geo, dtype) || A.out.reduce) return p;
    const int es = dtype == 1 ? 2 : 4;
    const int64_t nrows = table_rows(g, d, T_NBR);
    if (A.a.target != T_NBR || !A.a.full || !fits32(A.a, nrows, es)) return p;
    const int ext = ext_of(A.flags);
    if (ext == EXT_MASK) {
        OperandDev m{};
        m.data = A.mask_arg;
        m.stride = A.mask_ld;
        if (!fits32(m, nrows, 4)) return p;
    }
    if (opk == 0) {
        p.spec = SP_CU;
        p.gc = geo.G;
        return p;
    }
    if (maxmin || opk != 1 || A.op != M_MUL || ext != EXT_NONE || A.b.target != T_EDGE || A.b.full) return p;
    const bool head = A.b.hmul != 0;
    const int hb = head ? geo.H : 1;
    const bool cb = d.eid == nullptr && (hb & (hb - 1)) == 0 && geo.G * ENGINE_UNR * hb <= 64;
    int lg = 0;
    while ((1 << lg) < hb) ++lg;
    A.log2hb = lg;
    p.spec = head ? (cb ? SP_UE_H_CB : SP_UE_H) : (cb ? SP_UE_R_CB : SP_UE_R);
    p.gc = geo.G;
    return p;
}

// the compile-time layout of a g-SDDMM call (walks the in-CSR)
Pick pick_sddmm(const gnnk_graph* g, const EngineArgs& A, const Geo& geo, int dtype, int opk) {
    Pick p;
    if (options().no_fast || !fast_geo(geo, dtype) || ext_of(A.flags) != EXT_NONE || opk == 0) return p;
    if (!A.a.full || !A.b.full) return p;
    // reduced outputs need power-of-two runs of lanes (DPP sums) within one
    // pass of the wavefront
    if (A.out.reduce && ((A.out.red & (A.out.red - 1)) != 0 || geo.nchunk > 1)) return p;
    const int es = dtype == 1 ? 2 : 4;
    if (A.a.target == T_NBR && A.b.target == T_SELF && fits32(A.a, g->n_src, es) && fits32(A.b, g->n_dst, es) &&
        (opk == 1 || A.op != M_NEGDIV2)) {
        p.spec = SP_UV;
        p.gc = geo.G;
    } else if (A.a.target == T_SELF && A.b.target == T_NBR && opk == 1 && fits32(A.a, g->n_dst, es) &&
               fits32(A.b, g->n_src, es)) {
        p.spec = SP_VU;
        p.gc = geo.G;
    }
    return p;
}

// Walk chosen for a pass: 0 the row engine, else the edge-parallel (COO)
// walk, 2 deterministic or 3 with atomics (g-SpMM; g-SDDMM has no
// reduction).  The automatic choice is the row engine: with compile-time
// layouts for 1-32 lane groups it is faster than the edge walk for g-SpMM
// and g-SDDMM at every feature width from 1 to 128 on a constant-degree
// graph and on both power-law graphs of the benchmark set (the sensitivity
// sweep, python -m paper_1909_01315_amd.sweep); the edge walk stays
// available as an explicit schedule.
int pick_walk(const Dir& d, bool reduced_out) {
    const int64_t o = options().schedule;
    if (o == 1 || reduced_out || d.n_rows == 0) return 0;
    return o >= 2 ? (int)o : 0;
}

// positions per lane group of an edge-parallel walk: enough lane groups to
// fill the chip several times, a bounded partial buffer
void set_edge_chunks(EngineArgs& A, int64_t E, const Geo& geo) {
    int64_t target = E / ((int64_t)65536 * geo.G);
    int64_t sub = 64;
    while (sub < target && sub < 2048) sub <<= 1;
    if (options().edge_chunk > 0) sub = options().edge_chunk;
    A.sub_edges = (int32_t)sub;
    A.n_sub = (int32_t)((E + sub - 1) / sub);
}

// A row-reduction (g-SpMM) pass: sums, with hub partials and their combine.
// fused_dw (nullable): the caller set A.x2 / A.out2 / A.red2 / A.per_head2
// for a u_mul_e/sum backward and asks for the edge gradient in this pass;
// *fused_dw tells whether it was written (else the caller runs its g-SDDMM)
gnnk_status run_spmm_sum(gnnk_graph* g, const Dir& d, EngineArgs& A, const Geo& geo, int dtype, int opk,
                         hipStream_t s, Scratch& sc, bool* fused_dw = nullptr) {
    A.csr = csr_of(g, d);
    set_geo(A, geo);
    A.sch = schedule(d, geo, true);
    A.partial_stride = geo.D;
    const Pick pk = pick_spmm(g, d, A, geo, dtype, opk, false);
    const int walk = pick_walk(d, A.out.reduce != 0);
    if (fused_dw) {
        const int r2 = A.red2;
        *fused_dw = walk == 0 && (pk.spec == SP_UE_H || pk.spec == SP_UE_R) &&
                    (pk.gc == 1 || pk.gc == 2 || pk.gc == 4) && geo.nchunk == 1 && r2 >= 1 &&
                    (r2 & (r2 - 1)) == 0 && r2 <= geo.L;
    }
    if (walk) {
        set_edge_chunks(A, g->n_edges, geo);
        const size_t need = walk == 3 ? (size_t)d.n_rows * geo.D * 8 : (size_t)2 * A.n_sub * geo.D * 8;
        if (need > 0) {
            A.partial = sc.take(need);
            if (!A.partial) return scratch_fail(sc);
        }
        gnnk_status st = GNNK_LAUNCH(launch_spmm_edge(A, g->n_edges, d.n_rows, dtype, geo.vec, opk, pk.spec, pk.gc,
                                                        walk == 3 ? 1 : 0, s),
                                       "edge-parallel g-SpMM launch");
        if (st != GNNK_OK) return st;
        // empty rows: the fill role of the row engine alone
        EngineArgs F = A;
        SchedDev& sc = F.sch;
        sc.n_seg = 0;
        sc.n_hub = 0;
        sc.n_big = sc.n_nz;
        sc.w_big_end = 0;
        sc.w_small_end = 0;
        sc.w_total = (int32_t)((d.n_rows - d.n_nz + (int64_t)geo.G * sc.fill_rows_per_group - 1) /
                               ((int64_t)geo.G * sc.fill_rows_per_group));
        return GNNK_LAUNCH(launch_spmm(F, dtype, geo.vec, false, opk, SP_DYN, 0, s), "empty-row fill launch");
    }
    if (A.sch.n_seg > 0) {
        A.partial = sc.take((size_t)A.sch.n_seg * geo.D * 8);
        if (!A.partial) return scratch_fail(sc);
    }
    gnnk_status st = (fused_dw && *fused_dw)
                         ? GNNK_LAUNCH(launch_spmm_dw(A, dtype, geo.vec, pk.spec, pk.gc, s),
                                         "g-SpMM launch (with the edge gradient)")
                         : GNNK_LAUNCH(launch_spmm(A, dtype, geo.vec, false, opk, pk.spec, pk.gc, s),
                                         "g-SpMM launch");
    if (st == GNNK_OK && A.sch.n_hub > 0)
        st = GNNK_LAUNCH(launch_spmm_combine(A, dtype, geo.vec, false, s), "g-SpMM combine launch");
    return st;
}

gnnk_status run_sddmm(gnnk_graph* g, EngineArgs& A, const Geo& geo, int dtype, int opk, hipStream_t s, Scratch& sc) {
    // the in-CSR's finer segments (c3 u_dot_v 3.33 -> 3.19 ms): a g-SDDMM
    // leaves no partials, and more of each hub row runs in narrow pieces
    const Dir& d = g->in_fine;
    A.csr = csr_of(g, d);
    set_geo(A, geo);
    A.sch = schedule(d, geo, false);
    // narrow rows (16 or more lane groups, a batch of 64 or more edges) put
    // two wavefronts on each hub segment: it holds few batches, and a
    // wavefront's fixed start (segment, row value, first ids) then overlaps
    // with another's gathers
    {
        const int64_t o = options().sddmm_split;
        const int ks = (int)(o > 0 ? o : (geo.G >= 16 ? 2 : 1));
        if (ks > 1 && A.sch.n_seg > 0) {
            const int64_t extra = (int64_t)A.sch.n_seg * (ks - 1);
            if ((int64_t)A.sch.w_total + extra > INT32_MAX) return fail(GNNK_EUNSUPPORTED, "too many wavefronts");
            A.sch.seg_split = ks;
            A.sch.w_big_end += (int32_t)extra;
            A.sch.w_small_end += (int32_t)extra;
            A.sch.w_total += (int32_t)extra;
        }
    }
    const Pick pk = pick_sddmm(g, A, geo, dtype, opk);
    const bool multi = A.out.reduce && geo.nchunk > 1;
    if (multi) {
        // running per-edge sums between the passes of a row wider than the wavefront
        A.xacc = reinterpret_cast<double*>(sc.take((size_t)g->n_edges * 8));
        if (!A.xacc) return scratch_fail(sc);
    }
    if (pick_walk(d, multi)) {
        set_edge_chunks(A, g->n_edges, geo);
        return GNNK_LAUNCH(launch_sddmm_edge(A, g->n_edges, dtype, geo.vec, opk, pk.spec, pk.gc, s),
                             "edge-parallel g-SDDMM launch");
    }
    return GNNK_LAUNCH(launch_sddmm(A, dtype, geo.vec, opk, pk.spec, pk.gc, s), "g-SDDMM launch");
}

int32_t tgt_in(int t) { return t == GNNK_SRC ? T_NBR : (t == GNNK_EDGE ? T_EDGE : T_SELF); }   // in-CSR walk
int32_t tgt_out(int t) { return t == GNNK_SRC ? T_SELF : (t == GNNK_EDGE ? T_EDGE : T_NBR); }  // reverse walk

// Heads [h0, h0 + hc) of a (rows, Hm, F) tensor (a view: same rows and row
// stride); a tensor broadcast over heads is shared by every slice.
gnnk_tensor head_slice(const gnnk_tensor* t, int Hm, int h0, int hc) {
    gnnk_tensor s = *t;
    if (t->heads == Hm && Hm > 1) {
        const size_t es = t->dtype == GNNK_BF16 ? 2 : 4;
        if (s.data) s.data = static_cast<char*>(t->data) + (size_t)h0 * t->feat * es;
        s.heads = hc;
    }
    return s;
}

// Heads per slice of a call with a per-head sum (an output holding one value
// per head of an (Hm, Fm) message, Fm > 1) that would need more than one pass
// of the wavefront: Fm / vec lanes per head, 64 lanes per pass; one head per
// slice when a head alone is wider (its sum then runs over several passes).
// 0: the call runs whole.
int heads_per_slice(int Hm, int Fm, std::initializer_list<const gnnk_tensor*> all,
                    std::initializer_list<const gnnk_tensor*> outs, const void* int_array = nullptr) {
    if (Hm <= 1 || Fm <= 1) return 0;
    bool per_head = false;
    for (const gnnk_tensor* t : outs)
        if (t && t->heads == Hm && t->feat == 1) per_head = true;
    if (!per_head) return 0;
    std::vector<Member> ms;
    for (const gnnk_tensor* t : all)
        if (t) ms.push_back({t, K_FULL});
    Geo geo;
    if (choose_geo(Hm, Fm, ms, {int_array}, geo) != GNNK_OK || geo.merged || geo.nchunk == 1) return 0;
    return std::max(1, 64 / (Fm / geo.vec));
}

}  // namespace

// gspmm with its scratch from `sc` (the buffer lent for the stream, or the
// static buffer of gspmm_noalloc); checks every argument before it takes
// scratch or launches anything
gnnk_status gspmm_impl(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                       const gnnk_tensor* rhs, gnnk_tensor* out, int32_t* arg_lhs, int32_t* arg_rhs,
                       hipStream_t stream, Scratch& sc) {
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (op < GNNK_COPY_LHS || op > GNNK_DIV) return fail(GNNK_EINVAL, "gspmm op must be COPY_LHS..DIV");
    if (reduce < GNNK_SUM || reduce > GNNK_MIN) return fail(GNNK_EINVAL, "bad reduce");
    const bool use_l = op != GNNK_COPY_RHS, use_r = op != GNNK_COPY_LHS;
    if (use_l != (lhs != nullptr) || use_r != (rhs != nullptr))
        return fail(GNNK_EINVAL, "lhs is required unless COPY_RHS and rhs unless COPY_LHS (and absent otherwise)");
    if ((use_l && !tensor_ok(lhs)) || (use_r && !tensor_ok(rhs)) || !tensor_ok(out))
        return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({lhs, rhs, out})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    if ((use_l && lhs->rows != g->n_src) || (use_r && rhs->rows != g->n_edges) || out->rows != g->n_dst)
        return fail(GNNK_EINVAL, "row counts must be num_src (lhs), num_edges (rhs), num_dst (out)");
    const bool cmp = reduce == GNNK_MAX || reduce == GNNK_MIN;
    if (!cmp && (arg_lhs || arg_rhs)) return fail(GNNK_EUNSUPPORTED, "arg arrays are only produced by MAX/MIN");
    int Hm, Fm;
    if (!use_r) { Hm = lhs->heads; Fm = lhs->feat; }
    else if (!use_l) { Hm = rhs->heads; Fm = rhs->feat; }
    else { Hm = std::max(lhs->heads, rhs->heads); Fm = std::max(lhs->feat, rhs->feat); }
    if (out->heads != Hm || out->feat != Fm) return fail(GNNK_EINVAL, "out must have the message shape (%d, %d)", Hm, Fm);
    std::vector<Member> ms;
    if (use_l) ms.push_back({lhs, K_FULL});
    if (use_r) ms.push_back({rhs, K_FULL});
    ms.push_back({out, K_FULL});
    Geo geo;
    gnnk_status st = choose_geo(Hm, Fm, ms, {arg_lhs, arg_rhs}, geo);
    if (st != GNNK_OK) return st;
    if (g->n_dst == 0) return GNNK_OK;
    EngineArgs A{};
    size_t k = 0;
    OperandDev ol = use_l ? operand(lhs, ms[k++].kind, T_NBR) : OperandDev{};
    OperandDev orr = use_r ? operand(rhs, ms[k++].kind, T_EDGE) : OperandDev{};
    int opk;
    if (op == GNNK_COPY_LHS) { A.a = ol; opk = 0; }
    else if (op == GNNK_COPY_RHS) { A.a = orr; opk = 0; }
    else {
        A.a = ol;
        A.b = orr;
        opk = op == GNNK_MUL ? 1 : 2;
        A.op = op == GNNK_ADD ? M_ADD : (op == GNNK_SUB ? M_SUB : (op == GNNK_MUL ? M_MUL : M_DIV));
    }
    A.out.data = out->data;
    A.out.stride = out->row_stride;
    A.out.red = 1;
    A.out.reduce = 0;
    A.flags = (reduce == GNNK_MEAN ? F_OWN_MEAN : 0) | (reduce == GNNK_MIN ? F_IS_MIN : 0);
    // passes that gather node rows take the in-CSR's finer segments (c3
    // copy_u/mean 2.59 -> 2.46 ms, c4 copy_u/sum 3.59 -> 3.24 ms); copy_e
    // reductions keep the coarser ones, on which they run faster
    const bool gathers = (A.a.target == T_NBR && A.a.full) || (A.b.data && A.b.target == T_NBR && A.b.full);
    const Dir& d = gathers ? g->in_fine : g->in;
    if (!cmp) return run_spmm_sum(g, d, A, geo, dtype_code(out), opk, stream, sc);
    A.arg_nbr = arg_lhs;
    A.arg_edge = arg_rhs;
    A.csr = csr_of(g, d);
    set_geo(A, geo);
    A.sch = schedule(d, geo, true);
    if (A.sch.n_seg > 0) {
        A.partial = sc.take((size_t)A.sch.n_seg * geo.D * 12);
        if (!A.partial) return scratch_fail(sc);
    }
    const Pick pk = pick_spmm(g, d, A, geo, dtype_code(out), opk, true);
    st = GNNK_LAUNCH(launch_spmm(A, dtype_code(out), geo.vec, true, opk, pk.spec, pk.gc, stream), "g-SpMM launch");
    if (st == GNNK_OK && A.sch.n_hub > 0)
        st = GNNK_LAUNCH(launch_spmm_combine(A, dtype_code(out), geo.vec, true, stream), "g-SpMM combine launch");
    return st;
}

}  // namespace gnnk

using namespace gnnk;

extern "C" {

gnnk_status gspmm(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                  const gnnk_tensor* rhs, gnnk_tensor* out, int32_t* arg_lhs, int32_t* arg_rhs,
                  hipStream_t stream) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    Scratch sc = scratch_of(g, stream);
    return gspmm_impl(g, op, reduce, lhs, rhs, out, arg_lhs, arg_rhs, stream, sc);
}

gnnk_status gspmm_noalloc(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                          const gnnk_tensor* rhs, gnnk_tensor* out, int32_t* arg_lhs, int32_t* arg_rhs,
                          hipStream_t stream) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    Scratch sc;
    gnnk_status st = static_scratch(stream, sc);
    if (st != GNNK_OK) return st;
    st = gspmm_impl(g, op, reduce, lhs, rhs, out, arg_lhs, arg_rhs, stream, sc);
    if (st == GNNK_ENOMEM && sc.used > sc.bytes)
        return fail(GNNK_ENOMEM, "gspmm_noalloc: the call needs at least %zu bytes of scratch, more than the %zu of "
                    "the fixed buffer (gspmm takes a lent buffer of any size)", sc.used, sc.bytes);
    return st;
}

gnnk_status graph_scratch_bytes(gnnk_graph_t g, int64_t max_cols, int32_t flags, size_t* bytes) {
    clear_error();
    if (!g || !bytes) return fail(GNNK_EINVAL, "NULL argument");
    if (max_cols < 1 || max_cols > ((int64_t)1 << 31)) return fail(GNNK_EINVAL, "max_cols must be in [1, 2^31]");
    if (flags & ~(GNNK_SCRATCH_ARGMAX | GNNK_SCRATCH_WIDE_SUMS)) return fail(GNNK_EINVAL, "unknown flags");
    auto al = [](size_t n) { return (n + 255) / 256 * 256; };
    const size_t C = (size_t)max_cols, E = (size_t)g->n_edges;
    const size_t si = (size_t)g->in.n_seg, so = (size_t)std::max(g->out.n_seg, g->out_fine.n_seg);
    const size_t sif = (size_t)g->in_fine.n_seg;
    // sums and their gradients: fp64 partials of hub segments (any table)
    size_t need = al(std::max({si, sif, so}) * C * 8);
    // max / min: value, edge and neighbour per segment and column
    need = std::max(need, al(std::max(si, sif) * C * 12));
    // fused attention: partial states of segments, and the row state of hub
    // rows when the attention is written
    need = std::max(need, al(si * 3 * C * 8 + (size_t)g->in.n_hub * 2 * C * 8));
    // its backward: a record per destination and head (heads <= columns),
    // the accumulators of a head run in column chunks, then the larger of
    // the two passes' segment partials
    need = std::max(need, al((size_t)g->n_dst * C * 16) + al((size_t)g->n_dst * 16) + al((size_t)g->n_src * 8) +
                              al(std::max(si * 3 * C * 8, so * 2 * C * 8) + 8));
    if (flags & GNNK_SCRATCH_ARGMAX)  // winner masks, then the reverse pass's partials
        need = std::max(need, al(E * ((C + 31) / 32) * 4) + al(so * C * 8));
    if (flags & GNNK_SCRATCH_WIDE_SUMS)  // running fp64 sum per edge between passes
        need = std::max(need, al(E * 8));
    if (options().schedule >= 2) {
        // edge-parallel walks: two partial rows per sub-chunk of at least 64
        // positions, or one per row with atomics
        const size_t n_sub = (E + 63) / 64;
        need = std::max(need, al(std::max(2 * n_sub, (size_t)std::max(g->n_src, g->n_dst)) * C * 8));
    }
    *bytes = need;
    return GNNK_OK;
}

gnnk_status gsddmm(gnnk_graph_t g, gnnk_binop op, const gnnk_tensor* lhs, gnnk_target lhs_target,
                   const gnnk_tensor* rhs, gnnk_target rhs_target, gnnk_tensor* out, hipStream_t stream) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (op < GNNK_COPY_LHS || op > GNNK_DOT) return fail(GNNK_EINVAL, "bad op");
    if (lhs_target < GNNK_SRC || lhs_target > GNNK_DST || rhs_target < GNNK_SRC || rhs_target > GNNK_DST)
        return fail(GNNK_EINVAL, "bad target");
    const bool use_l = op != GNNK_COPY_RHS, use_r = op != GNNK_COPY_LHS;
    if (use_l != (lhs != nullptr) || use_r != (rhs != nullptr))
        return fail(GNNK_EINVAL, "lhs is required unless COPY_RHS and rhs unless COPY_LHS (and absent otherwise)");
    if ((use_l && !tensor_ok(lhs)) || (use_r && !tensor_ok(rhs)) || !tensor_ok(out))
        return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({lhs, rhs, out})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    if ((use_l && lhs->rows != rows_of_target(g, lhs_target)) || (use_r && rhs->rows != rows_of_target(g, rhs_target)) ||
        out->rows != g->n_edges)
        return fail(GNNK_EINVAL, "row counts do not match the targets / num_edges");
    int Hm, Fm;
    if (!use_r) { Hm = lhs->heads; Fm = lhs->feat; }
    else if (!use_l) { Hm = rhs->heads; Fm = rhs->feat; }
    else { Hm = std::max(lhs->heads, rhs->heads); Fm = std::max(lhs->feat, rhs->feat); }
    if (op == GNNK_DOT) {
        if (out->heads != Hm || out->feat != 1) return fail(GNNK_EINVAL, "dot output must be (E, %d, 1)", Hm);
    } else if (out->heads != Hm || out->feat != Fm) {
        return fail(GNNK_EINVAL, "out must have the message shape (%d, %d)", Hm, Fm);
    }
    if (const int hs = heads_per_slice(Hm, Fm, {lhs, rhs, out}, {out})) {
        // per-head dots wider than one pass: slices of heads, one call each
        for (int h0 = 0; h0 < Hm; h0 += hs) {
            const int hc = std::min(hs, Hm - h0);
            gnnk_tensor l = use_l ? head_slice(lhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor r = use_r ? head_slice(rhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor o = head_slice(out, Hm, h0, hc);
            gnnk_status st = gsddmm(g, op, use_l ? &l : nullptr, lhs_target, use_r ? &r : nullptr, rhs_target, &o,
                                    stream);
            if (st != GNNK_OK) return st;
        }
        return GNNK_OK;
    }
    std::vector<Member> ms;
    if (use_l) ms.push_back({lhs, K_FULL});
    if (use_r) ms.push_back({rhs, K_FULL});
    ms.push_back({out, K_FULL});
    Geo geo;
    gnnk_status st = choose_geo(Hm, Fm, ms, {}, geo);
    if (st != GNNK_OK) return st;
    if (g->n_edges == 0) return GNNK_OK;
    EngineArgs A{};
    size_t k = 0;
    OperandDev ol = use_l ? operand(lhs, ms[k++].kind, tgt_in(lhs_target)) : OperandDev{};
    OperandDev orr = use_r ? operand(rhs, ms[k++].kind, tgt_in(rhs_target)) : OperandDev{};
    st = out_desc(out, ms[k].kind, geo, A.out);
    if (st != GNNK_OK) return st;
    int opk;
    if (op == GNNK_COPY_LHS) { A.a = ol; opk = 0; }
    else if (op == GNNK_COPY_RHS) { A.a = orr; opk = 0; }
    else {
        A.a = ol;
        A.b = orr;
        opk = (op == GNNK_MUL || op == GNNK_DOT) ? 1 : 2;
        A.op = op == GNNK_ADD ? M_ADD : (op == GNNK_SUB ? M_SUB : (op == GNNK_DIV ? M_DIV : M_MUL));
    }
    Scratch sc = scratch_of(g, stream);
    return run_sddmm(g, A, geo, dtype_code(out), opk, stream, sc);
}

// arg_ld: elements per row of arg_rhs (-1: H * F of the call; a head slice
// keeps the stride of the whole array)
static gnnk_status spmm_backward(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                                 const gnnk_tensor* rhs, const int32_t* arg_rhs, const gnnk_tensor* grad_out,
                                 gnnk_tensor* grad_lhs, gnnk_tensor* grad_rhs, hipStream_t stream, int64_t arg_ld) {
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (op < GNNK_COPY_LHS || op > GNNK_DIV) return fail(GNNK_EINVAL, "gspmm op must be COPY_LHS..DIV");
    if (reduce < GNNK_SUM || reduce > GNNK_MIN) return fail(GNNK_EINVAL, "bad reduce");
    const bool use_l = op != GNNK_COPY_RHS, use_r = op != GNNK_COPY_LHS;
    const bool cmp = reduce == GNNK_MAX || reduce == GNNK_MIN;
    if (use_l != (lhs != nullptr) || use_r != (rhs != nullptr))
        return fail(GNNK_EINVAL, "lhs is required unless COPY_RHS and rhs unless COPY_LHS (and absent otherwise)");
    if ((grad_lhs && !use_l) || (grad_rhs && !use_r)) return fail(GNNK_EINVAL, "gradient of an unused operand");
    if ((use_l && !tensor_ok(lhs)) || (use_r && !tensor_ok(rhs)) || !tensor_ok(grad_out) ||
        (grad_lhs && !tensor_ok(grad_lhs)) || (grad_rhs && !tensor_ok(grad_rhs)))
        return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({lhs, rhs, grad_out, grad_lhs, grad_rhs})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    if ((use_l && lhs->rows != g->n_src) || (use_r && rhs->rows != g->n_edges) || grad_out->rows != g->n_dst)
        return fail(GNNK_EINVAL, "row counts must be num_src (lhs), num_edges (rhs), num_dst (grad_out)");
    if (cmp && !arg_rhs) return fail(GNNK_EINVAL, "MAX/MIN backward needs arg_rhs (edge ids)");
    int Hm, Fm;
    if (!use_r) { Hm = lhs->heads; Fm = lhs->feat; }
    else if (!use_l) { Hm = rhs->heads; Fm = rhs->feat; }
    else { Hm = std::max(lhs->heads, rhs->heads); Fm = std::max(lhs->feat, rhs->feat); }
    if (grad_out->heads != Hm || grad_out->feat != Fm) return fail(GNNK_EINVAL, "grad_out must have the message shape");
    if (grad_lhs && (grad_lhs->rows != g->n_src || grad_lhs->heads != lhs->heads || grad_lhs->feat != lhs->feat))
        return fail(GNNK_EINVAL, "grad_lhs must have lhs's shape");
    if (grad_rhs && (grad_rhs->rows != g->n_edges || grad_rhs->heads != rhs->heads || grad_rhs->feat != rhs->feat))
        return fail(GNNK_EINVAL, "grad_rhs must have rhs's shape");
    const int64_t ld = arg_ld >= 0 ? arg_ld : (int64_t)Hm * Fm;
    if (const int hs = heads_per_slice(Hm, Fm, {lhs, rhs, grad_out, grad_lhs, grad_rhs}, {grad_lhs, grad_rhs}, arg_rhs)) {
        // per-head gradients wider than one pass: slices of heads, one call each
        for (int h0 = 0; h0 < Hm; h0 += hs) {
            const int hc = std::min(hs, Hm - h0);
            gnnk_tensor l = use_l ? head_slice(lhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor r = use_r ? head_slice(rhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor go = head_slice(grad_out, Hm, h0, hc);
            gnnk_tensor gl = grad_lhs ? head_slice(grad_lhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor gr = grad_rhs ? head_slice(grad_rhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_status st = spmm_backward(g, op, reduce, use_l ? &l : nullptr, use_r ? &r : nullptr,
                                           arg_rhs ? arg_rhs + (size_t)h0 * Fm : nullptr, &go,
                                           grad_lhs ? &gl : nullptr, grad_rhs ? &gr : nullptr, stream, ld);
            if (st != GNNK_OK) return st;
        }
        return GNNK_OK;
    }
    const int dt = dtype_code(grad_out);
    const int32_t scale_flags = (reduce == GNNK_MEAN ? F_SCALE_A_DEG : 0) | (cmp ? F_MASK_A : 0);
    bool dw_done = false;
    const Scratch lent = scratch_of(g, stream);

    if (grad_lhs && g->n_src > 0) {
        // Lemma complex_dspmm_dx: a g-SpMM on the reverse graph, message dZ[v] * d phi / d x
        std::vector<Member> ms{{grad_out, K_FULL}};
        if (op == GNNK_MUL || op == GNNK_DIV) ms.push_back({rhs, K_FULL});
        ms.push_back({grad_lhs, K_FULL});
        Geo geo;
        gnnk_status st = choose_geo(Hm, Fm, ms, {arg_rhs}, geo);
        if (st != GNNK_OK) return st;
        EngineArgs A{};
        A.a = operand(grad_out, ms[0].kind, T_NBR);
        int opk = 0;
        if (op == GNNK_MUL || op == GNNK_DIV) {
            A.b = operand(rhs, ms[1].kind, T_EDGE);
            opk = op == GNNK_MUL ? 1 : 2;
            A.op = op == GNNK_MUL ? M_MUL : M_DIV;
        }
        st = out_desc(grad_lhs, ms.back().kind, geo, A.out);
        if (st != GNNK_OK) return st;
        A.flags = scale_flags;
        A.deg = g->in.deg;
        A.mask_arg = arg_rhs;
        A.mask_ld = ld;
        Scratch sc = lent;
        if (cmp && g->n_edges > 0) {
            // the argmax scatter as a masked g-SpMM on the reverse graph: the
            // winning columns of each edge are marked once in a bit mask laid
            // out in reverse-CSR order, so the walk reads 4 bytes per 32
            // columns per edge instead of the arg array of its destination
            const int32_t words = (int32_t)((geo.D + 31) / 32);
            uint32_t* bits = reinterpret_cast<uint32_t*>(sc.take((size_t)g->n_edges * words * 4));
            if (!bits) return scratch_fail(sc);
            hipError_t le = hipSuccess;
            if (planning()) {
                // nothing is launched while planning
            } else if (g->identity_eids && g->n_edges <= 64 * g->in.n_nz) {
                // rows of the in-CSR (mean in-degree up to 64): the positions
                // of a row's edges are read in order and each edge's mask is
                // stored whole.  Longer rows win few of their columns per
                // edge: there one lookup and one word per winning column
                // moves less (on the 114.6M-edge graph, mean in-degree 513 at
                // D = 128, the whole call takes 3.31 ms against 3.60; on the
                // 61.9M-edge graph, 25 at D = 100, 4.91 against 5.26 ms)
                WinnerRowsArgs W{};
                W.arg = arg_rhs;
                W.ld = ld;
                W.D = (int32_t)geo.D;
                W.words = words;
                W.ptr = g->in.ptr;
                W.perm = g->in.perm;
                W.seg = g->in.seg;
                W.n_seg = g->in.n_seg;
                W.n_hub = g->in.n_hub;
                W.n_small = g->in.n_nz - g->in.n_hub;
                W.pos = g->out.pos;
                W.bits = bits;
                le = launch_winner_rows(W, g->ptr64, g->n_edges, stream);
            } else {
                le = launch_winner_bits(arg_rhs, g->n_dst, (int32_t)geo.D, ld, g->out.pos, bits, g->n_edges, words,
                                        stream);
            }
            st = launch_status(le, "winner mask launch");
            if (st != GNNK_OK) return st;
            A.flags = (scale_flags & ~F_MASK_A) | F_BITS_A;
            A.mask_arg = reinterpret_cast<const int32_t*>(bits);
            A.mask_ld = words;
        }
        // u_mul_e/sum with a per-head or per-edge weight: the weight's
        // gradient dZ[v] . X[u] can come from the same reverse pass (the
        // pass has dZ[v] in its lanes and X[u] is the row's own), written at
        // the edge id, one scattered record per edge.  A g-SDDMM of its own
        // over the in-CSR writes the records in order but gathers X again.
        // On the 114.6M-edge graph at 128 columns: with 8 heads the two
        // passes take 5.06 + 3.76 ms against 9.26 ms fused (32-byte
        // records); with one weight per edge 5.06 + 3.00 against 7.55 fused
        // (4-byte records).  So by default only a one-column weight is fused.
        const int64_t fz = options().fused_dw;
        const bool want_dw = (fz == 1 || (fz < 0 && rhs && rhs->heads == 1)) && grad_rhs && g->n_edges > 0 &&
                             op == GNNK_MUL && reduce == GNNK_SUM && rhs->feat == 1 &&
                             (rhs->heads == Hm || rhs->heads == 1) && lhs->heads == Hm && lhs->feat == Fm;
        if (want_dw) {
            A.x2 = lhs->data;
            A.x2_stride = lhs->row_stride;
            A.out2 = grad_rhs->data;
            A.out2_stride = grad_rhs->row_stride;
            A.per_head2 = rhs->heads > 1 ? 1 : 0;
            A.red2 = A.per_head2 ? Fm / geo.vec : (int32_t)geo.NV;
        }
        // node rows gathered in the finer segments; the argmax scatter, which
        // reads its masks in order and gathers few rows, keeps the coarse ones
        st = run_spmm_sum(g, cmp ? g->out : g->out_fine, A, geo, dt, opk, stream, sc, want_dw ? &dw_done : nullptr);
        if (st != GNNK_OK) return st;
    }
    if (grad_rhs && g->n_edges > 0 && !dw_done) {
        // the lemma on dL/dW of g-SpMM: a g-SDDMM, message dZ[v] * d phi / d w
        std::vector<Member> ms{{grad_out, K_FULL}};
        if (op == GNNK_MUL || op == GNNK_DIV) ms.push_back({lhs, K_FULL});
        if (op == GNNK_DIV) ms.push_back({rhs, K_FULL});
        ms.push_back({grad_rhs, K_FULL});
        Geo geo;
        gnnk_status st = choose_geo(Hm, Fm, ms, {arg_rhs}, geo);
        if (st != GNNK_OK) return st;
        EngineArgs A{};
        A.a = operand(grad_out, ms[0].kind, T_SELF);
        int opk = 0;
        if (op == GNNK_MUL) {
            A.b = operand(lhs, ms[1].kind, T_NBR);
            opk = 1;
            A.op = M_MUL;
        } else if (op == GNNK_DIV) {
            A.b = operand(lhs, ms[1].kind, T_NBR);
            A.c = operand(rhs, ms[2].kind, T_EDGE);
            opk = 2;
            A.op = M_NEGDIV2;
        }
        st = out_desc(grad_rhs, ms.back().kind, geo, A.out);
        if (st != GNNK_OK) return st;
        A.flags = scale_flags | (op == GNNK_SUB ? F_NEGATE : 0);
        A.deg = g->in.deg;
        A.mask_arg = arg_rhs;
        A.mask_ld = ld;
        // the passes run in stream order: this one reuses the scratch from its start
        Scratch sc = lent;
        st = run_sddmm(g, A, geo, dt, opk, stream, sc);
        if (st != GNNK_OK) return st;
    }
    return GNNK_OK;
}

gnnk_status gspmm_backward(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                           const gnnk_tensor* rhs, const int32_t* arg_lhs, const int32_t* arg_rhs,
                           const gnnk_tensor* grad_out, gnnk_tensor* grad_lhs, gnnk_tensor* grad_rhs,
                           hipStream_t stream) {
    clear_error();
    (void)arg_lhs;
    return planned(g, stream, [&] {
        return spmm_backward(g, op, reduce, lhs, rhs, arg_rhs, grad_out, grad_lhs, grad_rhs, stream, -1);
    });
}

static gnnk_status sddmm_backward(gnnk_graph_t g, gnnk_binop op, const gnnk_tensor* lhs, gnnk_target lhs_target,
                                  const gnnk_tensor* rhs, gnnk_target rhs_target, const gnnk_tensor* grad_out,
                                  gnnk_tensor* grad_lhs, gnnk_tensor* grad_rhs, hipStream_t stream) {
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (op < GNNK_COPY_LHS || op > GNNK_DOT) return fail(GNNK_EINVAL, "bad op");
    if (lhs_target < GNNK_SRC || lhs_target > GNNK_DST || rhs_target < GNNK_SRC || rhs_target > GNNK_DST)
        return fail(GNNK_EINVAL, "bad target");
    const bool use_l = op != GNNK_COPY_RHS, use_r = op != GNNK_COPY_LHS;
    const bool binary = use_l && use_r;
    if (use_l != (lhs != nullptr) || use_r != (rhs != nullptr))
        return fail(GNNK_EINVAL, "lhs is required unless COPY_RHS and rhs unless COPY_LHS (and absent otherwise)");
    if ((grad_lhs && !use_l) || (grad_rhs && !use_r)) return fail(GNNK_EINVAL, "gradient of an unused operand");
    if ((use_l && !tensor_ok(lhs)) || (use_r && !tensor_ok(rhs)) || !tensor_ok(grad_out) ||
        (grad_lhs && !tensor_ok(grad_lhs)) || (grad_rhs && !tensor_ok(grad_rhs)))
        return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({lhs, rhs, grad_out, grad_lhs, grad_rhs})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    if ((use_l && lhs->rows != rows_of_target(g, lhs_target)) || (use_r && rhs->rows != rows_of_target(g, rhs_target)) ||
        grad_out->rows != g->n_edges)
        return fail(GNNK_EINVAL, "row counts do not match the targets / num_edges");
    int Hm, Fm;
    if (!use_r) { Hm = lhs->heads; Fm = lhs->feat; }
    else if (!use_l) { Hm = rhs->heads; Fm = rhs->feat; }
    else { Hm = std::max(lhs->heads, rhs->heads); Fm = std::max(lhs->feat, rhs->feat); }
    if (grad_out->heads != Hm || grad_out->feat != (op == GNNK_DOT ? 1 : Fm))
        return fail(GNNK_EINVAL, "grad_out must have the output shape");
    if (grad_lhs && (grad_lhs->rows != lhs->rows || grad_lhs->heads != lhs->heads || grad_lhs->feat != lhs->feat))
        return fail(GNNK_EINVAL, "grad_lhs must have lhs's shape");
    if (grad_rhs && (grad_rhs->rows != rhs->rows || grad_rhs->heads != rhs->heads || grad_rhs->feat != rhs->feat))
        return fail(GNNK_EINVAL, "grad_rhs must have rhs's shape");
    if (const int hs = heads_per_slice(Hm, Fm, {lhs, rhs, grad_out, grad_lhs, grad_rhs}, {grad_lhs, grad_rhs})) {
        // per-head gradients wider than one pass: slices of heads, one call each
        for (int h0 = 0; h0 < Hm; h0 += hs) {
            const int hc = std::min(hs, Hm - h0);
            gnnk_tensor l = use_l ? head_slice(lhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor r = use_r ? head_slice(rhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor go = head_slice(grad_out, Hm, h0, hc);
            gnnk_tensor gl = grad_lhs ? head_slice(grad_lhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_tensor gr = grad_rhs ? head_slice(grad_rhs, Hm, h0, hc) : gnnk_tensor{};
            gnnk_status st = sddmm_backward(g, op, use_l ? &l : nullptr, lhs_target, use_r ? &r : nullptr,
                                            rhs_target, &go, grad_lhs ? &gl : nullptr, grad_rhs ? &gr : nullptr,
                                            stream);
            if (st != GNNK_OK) return st;
        }
        return GNNK_OK;
    }
    const int dt = dtype_code(grad_out);

    for (int which = 0; which < 2; ++which) {
        gnnk_tensor* gx = which == 0 ? grad_lhs : grad_rhs;
        if (!gx || gx->rows == 0) continue;
        const int tx = which == 0 ? lhs_target : rhs_target;
        // the other operand enters the derivative of mul / div / dot
        std::vector<Member> ms{{grad_out, K_FULL}};
        EngineArgs A{};
        int opk = 0;
        int32_t flags = 0;
        auto tg = [&](int t) { return tx == GNNK_EDGE || tx == GNNK_DST ? tgt_in(t) : tgt_out(t); };
        const bool muldot = op == GNNK_MUL || op == GNNK_DOT;
        // operands b and c of the derivative message, with their own targets
        const gnnk_tensor* bt = nullptr;
        const gnnk_tensor* ct = nullptr;
        int b_target = 0, c_target = 0;
        if (which == 0) {
            if (binary && (muldot || op == GNNK_DIV)) {
                bt = rhs; b_target = rhs_target;
                opk = muldot ? 1 : 2;
                A.op = muldot ? M_MUL : M_DIV;
            }
        } else {
            if (binary && muldot) {
                bt = lhs; b_target = lhs_target;
                opk = 1;
                A.op = M_MUL;
            } else if (op == GNNK_DIV) {
                bt = lhs; b_target = lhs_target;
                ct = rhs; c_target = rhs_target;
                opk = 2;
                A.op = M_NEGDIV2;
            } else if (op == GNNK_SUB) {
                flags |= F_NEGATE;
            }
        }
        // a product is commutative (one IEEE multiplication either way): the
        // node operand goes first, the layout of the fast kernels
        const bool swap = bt && A.op == M_MUL;
        if (swap) ms.insert(ms.begin(), {bt, K_FULL});
        else if (bt) ms.push_back({bt, K_FULL});
        if (ct) ms.push_back({ct, K_FULL});
        ms.push_back({gx, K_FULL});
        Geo geo;
        gnnk_status st = choose_geo(Hm, Fm, ms, {}, geo);
        if (st != GNNK_OK) return st;
        if (swap) {
            A.a = operand(bt, ms[0].kind, tg(b_target));
            A.b = operand(grad_out, ms[1].kind, tg(GNNK_EDGE));
        } else {
            A.a = operand(grad_out, ms[0].kind, tg(GNNK_EDGE));
            if (bt) A.b = operand(bt, ms[1].kind, tg(b_target));
        }
        if (ct) A.c = operand(ct, ms[2].kind, tg(c_target));
        st = out_desc(gx, ms.back().kind, geo, A.out);
        if (st != GNNK_OK) return st;
        A.flags = flags;
        Scratch sc = scratch_of(g, stream);
        // a pass that gathers node rows (the other operand of mul/div/dot)
        // takes its CSR's finer segments; copy_e sums the coarse ones
        const bool gathers = (A.a.target == T_NBR && A.a.full) || (A.b.data && A.b.target == T_NBR && A.b.full);
        if (tx == GNNK_EDGE) st = run_sddmm(g, A, geo, dt, opk, stream, sc);
        else st = run_spmm_sum(g, tx == GNNK_SRC ? (gathers ? g->out_fine : g->out) : (gathers ? g->in_fine : g->in),
                               A, geo, dt, opk, stream, sc);
        if (st != GNNK_OK) return st;
    }
    return GNNK_OK;
}

gnnk_status gsddmm_backward(gnnk_graph_t g, gnnk_binop op, const gnnk_tensor* lhs, gnnk_target lhs_target,
                            const gnnk_tensor* rhs, gnnk_target rhs_target, const gnnk_tensor* grad_out,
                            gnnk_tensor* grad_lhs, gnnk_tensor* grad_rhs, hipStream_t stream) {
    clear_error();
    return planned(g, stream, [&] {
        return sddmm_backward(g, op, lhs, lhs_target, rhs, rhs_target, grad_out, grad_lhs, grad_rhs, stream);
    });
}

static gnnk_status softmax_common(gnnk_graph_t g, const gnnk_tensor* a, const gnnk_tensor* b, gnnk_tensor* out,
                                  bool backward, hipStream_t stream) {
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (!tensor_ok(a) || (b && !tensor_ok(b)) || !tensor_ok(out)) return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({a, b, out})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    for (const gnnk_tensor* t : {a, b, (const gnnk_tensor*)out}) {
        if (!t) continue;
        if (t->rows != g->n_edges || t->heads != a->heads || t->feat != a->feat)
            return fail(GNNK_EINVAL, "edge tensors must be (num_edges, H, F) of one shape");
    }
    std::vector<Member> ms{{a, K_FULL}, {out, K_FULL}};
    if (b) ms.push_back({b, K_FULL});
    Geo geo;
    gnnk_status st = choose_geo(a->heads, a->feat, ms, {}, geo);
    if (st != GNNK_OK) return st;
    if (g->n_edges == 0) return GNNK_OK;
    EngineArgs A{};
    A.a = operand(a, K_FULL, T_EDGE);
    if (b) A.b = operand(b, K_FULL, T_EDGE);
    A.out.data = out->data;
    A.out.stride = out->row_stride;
    A.out.red = 1;
    A.out.reduce = 0;
    A.csr = csr_of(g, g->in);
    set_geo(A, geo);
    // a workgroup of its own for every row of more than 2048 in-edges (or
    // the graph's segment size, when larger); shorter rows by one wavefront
    // or lane group, whatever the segment size
    A.sch = schedule(g->in, geo, false, std::max<int64_t>(g->seg_edges, 2048));
    return GNNK_LAUNCH(launch_softmax(A, dtype_code(a), geo.vec, backward, stream), "edge softmax launch");
}

gnnk_status edge_softmax(gnnk_graph_t g, const gnnk_tensor* score, gnnk_tensor* out, hipStream_t stream) {
    clear_error();
    return softmax_common(g, score, nullptr, out, false, stream);
}

gnnk_status edge_softmax_backward(gnnk_graph_t g, const gnnk_tensor* out, const gnnk_tensor* grad_out,
                                  gnnk_tensor* grad_score, hipStream_t stream) {
    clear_error();
    if (!grad_out) return fail(GNNK_EINVAL, "grad_out is NULL");
    return softmax_common(g, out, grad_out, grad_score, true, stream);
}

// (num_dst, H, 2) fp32 per-row statistics of the fused attention
static bool stats_ok(const gnnk_graph* g, const gnnk_tensor* st, int H) {
    return tensor_ok(st) && st->dtype == GNNK_F32 && st->rows == g->n_dst && st->heads == H && st->feat == 2;
}

gnnk_status gat_aggregate(gnnk_graph_t g, const gnnk_tensor* feat, const gnnk_tensor* el, const gnnk_tensor* er,
                          float slope, gnnk_tensor* out, gnnk_tensor* attn, gnnk_tensor* stats, hipStream_t stream) {
    clear_error();
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (!tensor_ok(feat) || !tensor_ok(el) || !tensor_ok(er) || !tensor_ok(out) || (attn && !tensor_ok(attn)))
        return fail(GNNK_EINVAL, "malformed tensor");
    if (stats && !stats_ok(g, stats, feat->heads)) return fail(GNNK_EINVAL, "stats must be (num_dst, H, 2) fp32");
    if (!same_dtype({feat, el, er, out, attn})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    const int H = feat->heads, F = feat->feat;
    if (feat->rows != g->n_src || el->rows != g->n_src || er->rows != g->n_dst || out->rows != g->n_dst)
        return fail(GNNK_EINVAL, "row counts must be num_src (feat, el) and num_dst (er, out)");
    if (el->heads != H || el->feat != 1 || er->heads != H || er->feat != 1 || out->heads != H || out->feat != F)
        return fail(GNNK_EINVAL, "shapes must be feat (H, F), el and er (H, 1), out (H, F)");
    if (attn && (attn->rows != g->n_edges || attn->heads != H || attn->feat != 1))
        return fail(GNNK_EINVAL, "attn must be (num_edges, H, 1)");
    // el and er broadcast over features: keep heads separate (F per head)
    std::vector<Member> ms{{feat, K_FULL}, {el, K_FULL}, {out, K_FULL}};
    Geo geo;
    gnnk_status st = choose_geo(H, F, ms, {}, geo, true);
    if (st != GNNK_OK) return st;
    if (g->n_dst == 0) return GNNK_OK;
    EngineArgs A{};
    A.a = operand(feat, K_FULL, T_NBR);
    A.b = operand(el, ms[1].kind, T_NBR);
    A.op = M_MUL;
    A.out.data = out->data;
    A.out.stride = out->row_stride;
    A.out.red = 1;
    A.csr = csr_of(g, g->in);
    set_geo(A, geo);
    A.sch = schedule(g->in, geo, true);
    const int dt = dtype_code(out);
    const size_t part = (size_t)A.sch.n_seg * 3 * geo.D * 8, ml = attn ? (size_t)A.sch.n_hub * 2 * geo.D * 8 : 0;
    void* row_ml = nullptr;
    if (part + ml > 0) {
        Scratch sc = scratch_of(g, stream);
        char* p = reinterpret_cast<char*>(sc.take(part + ml));
        if (!p) return scratch_fail(sc);
        A.partial = p;
        row_ml = ml ? p + part : nullptr;
    }
    const int es = dt == 1 ? 2 : 4;
    const bool fast = !options().no_fast && fast_geo(geo, dt) && fits32(A.a, g->n_src, es) &&
                      fits32(A.b, g->n_src, es);
    return GNNK_LAUNCH(launch_gat(A, er->data, er->row_stride, attn ? attn->data : nullptr,
                                    attn ? attn->row_stride : 0, slope, row_ml,
                                    stats ? reinterpret_cast<float*>(stats->data) : nullptr,
                                    stats ? stats->row_stride : 0, dt, geo.vec, fast ? geo.G : 0, stream),
                         "fused attention launch");
}

// One run of the fused attention backward's kernels over one head slice
// whose heads fit a pass of the wavefront (or one column chunk of a wider
// head: chunk 1-3, with the accumulators acc_dst / acc_src; chunk 0 for
// whole heads).  passes: 1 pass A, 2 pass B, 3 both.  rec: the records of
// pass A read by pass B; the segment partials are carved from sc.
static gnnk_status gat_bwd_run(gnnk_graph_t g, const gnnk_tensor* feat, const gnnk_tensor* el, const gnnk_tensor* er,
                               float slope, const gnnk_tensor* stats, const gnnk_tensor* grad_out,
                               gnnk_tensor* grad_feat, gnnk_tensor* grad_el, gnnk_tensor* grad_er, hipStream_t stream,
                               Scratch& sc, float4* rec, int chunk, int passes, double* acc_dst, double* acc_src) {
    const int H = feat->heads, F = feat->feat;
    std::vector<Member> ms{{feat, K_FULL}, {el, K_FULL}, {grad_out, K_FULL}};
    Geo geo;
    gnnk_status st = choose_geo(H, F, ms, {}, geo, true);
    if (st != GNNK_OK) return st;
    if (geo.nchunk != 1) return fail(GNNK_EUNSUPPORTED, "fused attention backward: a slice wider than one pass");
    const int dt = dtype_code(grad_out);
    EngineArgs ain{}, aout{};
    ain.a = operand(feat, K_FULL, T_NBR);
    ain.b = operand(el, ms[1].kind, T_NBR);
    ain.op = M_MUL;
    ain.csr = csr_of(g, g->in);
    set_geo(ain, geo);
    ain.sch = schedule(g->in, geo, true);
    aout.csr = csr_of(g, g->out_fine);
    set_geo(aout, geo);
    aout.sch = schedule(g->out_fine, geo, true);
    const size_t pa = (size_t)ain.sch.n_seg * 3 * H * 8, pb = (size_t)aout.sch.n_seg * (geo.D + H) * 8;
    double* part = reinterpret_cast<double*>(sc.take(std::max(pa, pb) + 8));
    if (!part) return scratch_fail(sc);
    GatBwdArgs B{};
    B.er = er->data;
    B.er_stride = er->row_stride;
    B.stats = reinterpret_cast<const float*>(stats->data);
    B.stats_stride = stats->row_stride;
    B.dz = grad_out->data;
    B.dz_stride = grad_out->row_stride;
    B.d_er = grad_er ? grad_er->data : nullptr;
    B.d_er_stride = grad_er ? grad_er->row_stride : 0;
    B.d_el = grad_el ? grad_el->data : nullptr;
    B.d_el_stride = grad_el ? grad_el->row_stride : 0;
    B.d_feat = grad_feat ? grad_feat->data : nullptr;
    B.d_feat_stride = grad_feat ? grad_feat->row_stride : 0;
    B.el = el->data;
    B.el_stride = el->row_stride;
    B.feat = feat->data;
    B.feat_stride = feat->row_stride;
    B.rec = rec;
    B.part = part;
    B.slope = slope;
    B.H = H;
    B.chunk = chunk;
    B.passes = passes;
    B.acc_dst = acc_dst;
    B.acc_src = acc_src;
    const int es = dt == 1 ? 2 : 4;
    const bool fast = !options().no_fast && fast_geo(geo, dt) && fits32(ain.a, g->n_src, es) &&
                      fits32(ain.b, g->n_src, es);
    return GNNK_LAUNCH(launch_gat_backward(ain, aout, B, dt, geo.vec, fast ? geo.G : 0, stream),
                         "fused attention backward launch");
}

// columns [c0, c0 + cw) of a one-head (rows, 1, F) tensor (a view: same rows
// and row stride)
static gnnk_tensor col_slice(const gnnk_tensor* t, int c0, int cw) {
    gnnk_tensor s = *t;
    const size_t es = t->dtype == GNNK_BF16 ? 2 : 4;
    if (s.data) s.data = static_cast<char*>(t->data) + (size_t)c0 * es;
    s.feat = cw;
    return s;
}

static gnnk_status gat_backward(gnnk_graph_t g, const gnnk_tensor* feat, const gnnk_tensor* el,
                                const gnnk_tensor* er, float slope, const gnnk_tensor* stats,
                                const gnnk_tensor* grad_out, gnnk_tensor* grad_feat, gnnk_tensor* grad_el,
                                gnnk_tensor* grad_er, hipStream_t stream) {
    if (!g) return fail(GNNK_EINVAL, "NULL graph");
    if (!tensor_ok(feat) || !tensor_ok(el) || !tensor_ok(er) || !tensor_ok(grad_out) || !stats ||
        (grad_feat && !tensor_ok(grad_feat)) || (grad_el && !tensor_ok(grad_el)) || (grad_er && !tensor_ok(grad_er)))
        return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({feat, el, er, grad_out, grad_feat, grad_el, grad_er}))
        return fail(GNNK_EINVAL, "all tensors but stats must share one dtype");
    const int H = feat->heads, F = feat->feat;
    if (!stats_ok(g, stats, H)) return fail(GNNK_EINVAL, "stats must be (num_dst, H, 2) fp32");
    if (feat->rows != g->n_src || el->rows != g->n_src || er->rows != g->n_dst || grad_out->rows != g->n_dst)
        return fail(GNNK_EINVAL, "row counts must be num_src (feat, el) and num_dst (er, grad_out)");
    if (el->heads != H || el->feat != 1 || er->heads != H || er->feat != 1 || grad_out->heads != H ||
        grad_out->feat != F)
        return fail(GNNK_EINVAL, "shapes must be feat (H, F), el and er (H, 1), grad_out (H, F)");
    auto same = [](const gnnk_tensor* a, const gnnk_tensor* b) {
        return !a || (a->rows == b->rows && a->heads == b->heads && a->feat == b->feat);
    };
    if (!same(grad_feat, feat) || !same(grad_el, el) || !same(grad_er, er))
        return fail(GNNK_EINVAL, "each gradient must have its operand's shape");
    std::vector<Member> ms{{feat, K_FULL}, {el, K_FULL}, {grad_out, K_FULL}};
    Geo geo;
    gnnk_status st = choose_geo(H, F, ms, {}, geo, true);
    if (st != GNNK_OK) return st;
    Scratch sc = scratch_of(g, stream);
    if (geo.nchunk == 1) {
        float4* rec = reinterpret_cast<float4*>(sc.take((size_t)g->n_dst * H * 16));
        if (!rec) return scratch_fail(sc);
        return gat_bwd_run(g, feat, el, er, slope, stats, grad_out, grad_feat, grad_el, grad_er, stream, sc, rec, 0, 3,
                           nullptr, nullptr);
    }
    // a head's dot products are reduced across the lanes of one pass: rows
    // wider than a pass run as slices of heads (heads are independent), and
    // a head wider than a pass in column chunks of one pass each
    const int lanes = F / geo.vec;
    const int hs = lanes <= 64 ? 64 / lanes : 1;
    const int cw = lanes <= 64 ? F : 64 * geo.vec;
    const int nc = (F + cw - 1) / cw;
    float4* rec = reinterpret_cast<float4*>(sc.take((size_t)g->n_dst * hs * 16));
    double* acc_dst = nullptr;
    double* acc_src = nullptr;
    if (rec && nc > 1) {
        acc_dst = reinterpret_cast<double*>(sc.take((size_t)g->n_dst * 2 * 8));
        acc_src = reinterpret_cast<double*>(sc.take((size_t)g->n_src * 8));
    }
    if (!rec || (nc > 1 && (!acc_dst || !acc_src))) return scratch_fail(sc);
    const size_t base = sc.used;
    for (int h0 = 0; h0 < H; h0 += hs) {
        const int hc = std::min(hs, H - h0);
        gnnk_tensor f = head_slice(feat, H, h0, hc), l = head_slice(el, H, h0, hc), r = head_slice(er, H, h0, hc);
        gnnk_tensor sts = head_slice(stats, H, h0, hc), go = head_slice(grad_out, H, h0, hc);
        gnnk_tensor gf = grad_feat ? head_slice(grad_feat, H, h0, hc) : gnnk_tensor{};
        gnnk_tensor gl = grad_el ? head_slice(grad_el, H, h0, hc) : gnnk_tensor{};
        gnnk_tensor gr = grad_er ? head_slice(grad_er, H, h0, hc) : gnnk_tensor{};
        gnnk_tensor* pgf = grad_feat ? &gf : nullptr;
        gnnk_tensor* pgl = grad_el ? &gl : nullptr;
        gnnk_tensor* pgr = grad_er ? &gr : nullptr;
        if (nc == 1) {
            sc.used = base;  // the slices run in stream order and reuse the partials
            st = gat_bwd_run(g, &f, &l, &r, slope, &sts, &go, pgf, pgl, pgr, stream, sc, rec, 0, 3, nullptr,
                             nullptr);
            if (st != GNNK_OK) return st;
            continue;
        }
        // one head in column chunks: every chunk of pass A, then every chunk
        // of pass B (which reads the records the last chunk of pass A wrote)
        for (int pass = 1; pass <= 2; ++pass) {
            for (int k = 0; k < nc; ++k) {
                const int c0 = k * cw, w = std::min(cw, F - c0);
                gnnk_tensor fc = col_slice(&f, c0, w), zc = col_slice(&go, c0, w);
                gnnk_tensor gfc = grad_feat ? col_slice(&gf, c0, w) : gnnk_tensor{};
                const int chunk = k == 0 ? 1 : (k == nc - 1 ? 3 : 2);
                sc.used = base;
                st = gat_bwd_run(g, &fc, &l, &r, slope, &sts, &zc, grad_feat ? &gfc : nullptr, pgl, pgr, stream, sc,
                                 rec, chunk, pass, acc_dst, acc_src);
                if (st != GNNK_OK) return st;
            }
        }
    }
    return GNNK_OK;
}

gnnk_status gat_aggregate_backward(gnnk_graph_t g, const gnnk_tensor* feat, const gnnk_tensor* el,
                                   const gnnk_tensor* er, float slope, const gnnk_tensor* stats,
                                   const gnnk_tensor* grad_out, gnnk_tensor* grad_feat, gnnk_tensor* grad_el,
                                   gnnk_tensor* grad_er, hipStream_t stream) {
    clear_error();
    return planned(g, stream, [&] {
        return gat_backward(g, feat, el, er, slope, stats, grad_out, grad_feat, grad_el, grad_er, stream);
    });
}

static gnnk_status leaky_common(const gnnk_tensor* x, const gnnk_tensor* dy, gnnk_tensor* y, float slope,
                                bool backward, hipStream_t stream) {
    if (!tensor_ok(x) || (backward && !tensor_ok(dy)) || !tensor_ok(y)) return fail(GNNK_EINVAL, "malformed tensor");
    if (!same_dtype({x, dy, y})) return fail(GNNK_EINVAL, "all tensors must share one dtype");
    if (y->rows != x->rows || y->heads != x->heads || y->feat != x->feat ||
        (dy && (dy->rows != x->rows || dy->heads != x->heads || dy->feat != x->feat)))
        return fail(GNNK_EINVAL, "tensors must have one shape");
    hipError_t e = launch_leaky(x->data, dy ? dy->data : nullptr, y->data, x->rows, x->heads * x->feat,
                                x->row_stride, dy ? dy->row_stride : 0, y->row_stride, slope, dtype_code(x), backward,
                                stream);
    return launch_status(e, "leaky relu launch");
}

gnnk_status edge_leaky_relu(const gnnk_tensor* x, gnnk_tensor* y, float slope, hipStream_t stream) {
    clear_error();
    return leaky_common(x, nullptr, y, slope, false, stream);
}

gnnk_status edge_leaky_relu_backward(const gnnk_tensor* x, const gnnk_tensor* dy, gnnk_tensor* dx, float slope,
                                     hipStream_t stream) {
    clear_error();
    if (!dy) return fail(GNNK_EINVAL, "dy is NULL");
    return leaky_common(x, dy, dx, slope, true, stream);
}

}  // extern "C"
