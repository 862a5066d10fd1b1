/*
 * Oracle for generalized SpMM / SDDMM message passing.  TEST INFRASTRUCTURE
 * ONLY: loaded by the tests, the smoke check and the benchmark's CPU-baseline
 * leg, never by the GPU library.  Shares no code with the GPU path.
 *
 * Each function is the plain definition it cites, as a single-threaded loop:
 *   - g-SDDMM:  m_e = phi(x_u, y_v, w_e) for every edge (u, e, v)
 *               (Section 3, definition of generalized SDDMM);
 *   - g-SpMM:   z_v = rho{ phi(x_u, w_e) : (u, e, v) in E }, a reduction over
 *               the in-edges of v (Section 3, definition of generalized SpMM);
 *   - gradients: the chain-rule sums in the proofs of the lemmas behind
 *               Theorem 1 (Appendix B): dX sums over the out-edges of u (the
 *               reverse graph), dY over the in-edges of v, dW per edge.
 * Edges of a node are visited in ascending edge id.  Sums are taken in double
 * and rounded once to the output type (fp32: one IEEE rounding; bf16: to fp32,
 * then to bf16 round-to-nearest-even; fp64 outputs are not rounded).
 *
 * Readings where the paper is silent (all are listed with the design notes):
 *   - an empty reduction gives 0, and argmax/argmin index -1;
 *   - max/min compare messages in the precision a message tensor would hold
 *     (fp32 for fp32 and bf16 inputs, fp64 for fp64); the first (smallest)
 *     edge id wins a tie, and the whole gradient goes to that edge;
 *   - mean divides by the in-degree counting multi-edges;
 *   - operands broadcast per dimension: a head or feature extent of 1 is
 *     repeated to the other operand's extent; gradients to a broadcast operand
 *     are summed over the repeated positions;
 *   - edge_softmax normalises over the in-edges of each destination, per
 *     column, after subtracting that group's maximum;
 *   - leaky ReLU is x > 0 ? x : slope * x, and its derivative at 0 is slope.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* element access                                                           */

/* bf16 -> double: the bf16 pattern is the top half of an fp32 pattern */
static double bf16_to_double(uint16_t h) {
    uint32_t b = (uint32_t)h << 16;
    float f;
    memcpy(&f, &b, 4);
    return (double)f;
}

/* fp32 -> bf16, round to nearest, ties to even, by comparing the two
 * neighbouring bf16 values around f exactly in double. */
static uint16_t float_to_bf16(float f) {
    uint32_t b;
    memcpy(&b, &f, 4);
    if ((b & 0x7F800000u) == 0x7F800000u) return (uint16_t)((b >> 16) | ((b & 0xFFFFu) ? 0x40u : 0u));
    uint16_t lo = (uint16_t)(b >> 16);                 /* truncated toward zero */
    if ((b & 0xFFFFu) == 0) return lo;                 /* exactly representable */
    uint16_t hi = (uint16_t)(lo + 1);                  /* next bf16 away from zero */
    /* IEEE 754 overflow: the neighbour past the largest finite value is taken
     * at magnitude 2^128, as if the exponent range were unbounded */
    double vhi = ((hi & 0x7F80u) == 0x7F80u) ? copysign(0x1.0p128, (double)f) : bf16_to_double(hi);
    double dl = fabs((double)f - bf16_to_double(lo));
    double dh = fabs(vhi - (double)f);
    if (dl < dh) return lo;
    if (dh < dl) return hi;
    return (lo & 1u) ? hi : lo;                        /* tie: even mantissa */
}

void oracle_round_bf16(int64_t n, const float* in, uint16_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = float_to_bf16(in[i]);
}

static int64_t off(const or_tensor* t, int64_t row, int64_t h, int64_t f) {
    return row * t->stride + (t->heads == 1 ? 0 : h) * t->feat + (t->feat == 1 ? 0 : f);
}

static double ld(const or_tensor* t, int64_t row, int64_t h, int64_t f) {
    int64_t i = off(t, row, h, f);
    switch (t->dtype) {
        case OR_F32: return (double)((const float*)t->data)[i];
        case OR_BF16: return bf16_to_double(((const uint16_t*)t->data)[i]);
        default: return ((const double*)t->data)[i];
    }
}

static void st(or_tensor* t, int64_t row, int64_t h, int64_t f, double v) {
    int64_t i = row * t->stride + h * t->feat + f;
    switch (t->dtype) {
        case OR_F32: ((float*)t->data)[i] = (float)v; break;
        case OR_BF16: ((uint16_t*)t->data)[i] = float_to_bf16((float)v); break;
        default: ((double*)t->data)[i] = v; break;
    }
}

/* value as a message tensor of this dtype would hold it */
static double as_stored(int dtype, double v) { return dtype == OR_F64 ? v : (double)(float)v; }

static int dtype_ok(const or_tensor* t) {
    return t && t->data && (t->dtype == OR_F32 || t->dtype == OR_BF16 || t->dtype == OR_F64) && t->heads >= 1 &&
           t->feat >= 1 && t->stride >= t->heads * t->feat;
}

/* operand extents must equal the message extent or be 1 */
static int fits(const or_tensor* t, int64_t H, int64_t F) {
    return (t->heads == H || t->heads == 1) && (t->feat == F || t->feat == 1);
}

/* ------------------------------------------------------------------------ */
/* adjacency: in-lists and out-lists in ascending edge id (counting sort)   */

typedef struct {
    int64_t* ptr; /* n + 1 */
    int64_t* eid; /* E */
} adj;

static int build_adj(const or_graph* g, int by_src, adj* a) {
    int64_t n = by_src ? g->n_src : g->n_dst;
    const int32_t* key = by_src ? g->src : g->dst;
    a->ptr = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
    a->eid = (int64_t*)malloc((size_t)(g->n_edges > 0 ? g->n_edges : 1) * sizeof(int64_t));
    if (!a->ptr || !a->eid) return -1;
    for (int64_t e = 0; e < g->n_edges; ++e) {
        if (key[e] < 0 || key[e] >= n) return -2;
        a->ptr[key[e] + 1]++;
    }
    for (int64_t i = 0; i < n; ++i) a->ptr[i + 1] += a->ptr[i];
    int64_t* fill = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    if (!fill) return -1;
    memcpy(fill, a->ptr, (size_t)n * sizeof(int64_t));
    for (int64_t e = 0; e < g->n_edges; ++e) a->eid[fill[key[e]]++] = e; /* ascending e within a node */
    free(fill);
    return 0;
}

static void free_adj(adj* a) {
    free(a->ptr);
    free(a->eid);
}

static int graph_ok(const or_graph* g) {
    if (!g || g->n_src < 0 || g->n_dst < 0 || g->n_edges < 0) return 0;
    if (g->n_edges > 0 && (!g->src || !g->dst)) return 0;
    for (int64_t e = 0; e < g->n_edges; ++e)
        if (g->src[e] < 0 || g->src[e] >= g->n_src || g->dst[e] < 0 || g->dst[e] >= g->n_dst) return 0;
    return 1;
}

int oracle_degrees(const or_graph* g, int64_t* in_deg, int64_t* out_deg) {
    if (!graph_ok(g)) return -1;
    if (in_deg) memset(in_deg, 0, (size_t)g->n_dst * sizeof(int64_t));
    if (out_deg) memset(out_deg, 0, (size_t)g->n_src * sizeof(int64_t));
    for (int64_t e = 0; e < g->n_edges; ++e) {
        if (in_deg) in_deg[g->dst[e]]++;
        if (out_deg) out_deg[g->src[e]]++;
    }
    return 0;
}

/* In-CSR (rows = destinations, indices = sources) or, with reverse != 0, the
 * CSR of the reverse graph (rows = sources, indices = destinations); eids
 * keep the original edge ids (Appendix B, definition of the reverse graph). */
int oracle_csr(const or_graph* g, int reverse, int64_t* indptr, int32_t* indices, int32_t* eids) {
    if (!graph_ok(g)) return -1;
    adj a;
    if (build_adj(g, reverse, &a)) { free_adj(&a); return -1; }
    int64_t n = reverse ? g->n_src : g->n_dst;
    for (int64_t i = 0; i <= n; ++i) indptr[i] = a.ptr[i];
    for (int64_t p = 0; p < g->n_edges; ++p) {
        int64_t e = a.eid[p];
        indices[p] = reverse ? g->dst[e] : g->src[e];
        eids[p] = (int32_t)e;
    }
    free_adj(&a);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* message functions                                                        */

static double phi(int op, double x, double w) {
    switch (op) {
        case OR_COPY_LHS: return x;
        case OR_COPY_RHS: return w;
        case OR_ADD: return x + w;
        case OR_SUB: return x - w;
        case OR_MUL: return x * w;
        case OR_DIV: return x / w;
        default: return NAN;
    }
}

static int op_uses_lhs(int op) { return op != OR_COPY_RHS; }
static int op_uses_rhs(int op) { return op != OR_COPY_LHS; }

/* message extent of an op over its operands */
static int msg_shape(int op, const or_tensor* l, const or_tensor* r, int64_t* H, int64_t* F) {
    if (op == OR_COPY_LHS) { *H = l->heads; *F = l->feat; return 0; }
    if (op == OR_COPY_RHS) { *H = r->heads; *F = r->feat; return 0; }
    *H = l->heads > r->heads ? l->heads : r->heads;
    *F = l->feat > r->feat ? l->feat : r->feat;
    return (fits(l, *H, *F) && fits(r, *H, *F)) ? 0 : -1;
}

/* ------------------------------------------------------------------------ */
/* g-SpMM (Section 3): z_v = rho over the in-edges of v of phi(x_u, w_e)     */

int oracle_gspmm(const or_graph* g, int op, int reduce, const or_tensor* lhs, const or_tensor* rhs,
                 or_tensor* out, int32_t* arg_u, int32_t* arg_e, const int64_t* rows, int64_t n_rows) {
    if (!graph_ok(g) || !dtype_ok(out) || op < OR_COPY_LHS || op > OR_DIV || reduce < OR_SUM || reduce > OR_MIN)
        return -1;
    if (op_uses_lhs(op) && (!dtype_ok(lhs) || lhs->rows != g->n_src)) return -1;
    if (op_uses_rhs(op) && (!dtype_ok(rhs) || rhs->rows != g->n_edges)) return -1;
    int64_t H, F;
    if (msg_shape(op, lhs, rhs, &H, &F) || out->heads != H || out->feat != F ||
        out->rows != (rows ? n_rows : g->n_dst))
        return -1;
    adj in;
    if (build_adj(g, 0, &in)) { free_adj(&in); return -1; }
    int64_t cnt = rows ? n_rows : g->n_dst;
    for (int64_t k = 0; k < cnt; ++k) {
        int64_t v = rows ? rows[k] : k;
        if (v < 0 || v >= g->n_dst) { free_adj(&in); return -1; }
        int64_t b = in.ptr[v], e_end = in.ptr[v + 1], deg = e_end - b;
        for (int64_t h = 0; h < H; ++h)
            for (int64_t f = 0; f < F; ++f) {
                int64_t col = h * F + f;
                if (reduce == OR_SUM || reduce == OR_MEAN) {
                    double acc = 0.0;
                    for (int64_t p = b; p < e_end; ++p) {
                        int64_t e = in.eid[p];
                        double x = op_uses_lhs(op) ? ld(lhs, g->src[e], h, f) : 0.0;
                        double w = op_uses_rhs(op) ? ld(rhs, e, h, f) : 0.0;
                        acc += phi(op, x, w);
                    }
                    if (deg == 0) acc = 0.0;
                    else if (reduce == OR_MEAN) acc = acc / (double)deg;
                    st(out, k, h, f, acc);
                } else {
                    double best = 0.0;
                    int64_t be = -1;
                    for (int64_t p = b; p < e_end; ++p) {
                        int64_t e = in.eid[p];
                        double x = op_uses_lhs(op) ? ld(lhs, g->src[e], h, f) : 0.0;
                        double w = op_uses_rhs(op) ? ld(rhs, e, h, f) : 0.0;
                        double m = as_stored(out->dtype, phi(op, x, w));
                        int better = (reduce == OR_MAX) ? (m > best) : (m < best);
                        if (be < 0 || better) { best = m; be = e; }
                    }
                    st(out, k, h, f, be < 0 ? 0.0 : best);
                    if (arg_e) arg_e[k * H * F + col] = (int32_t)be;
                    if (arg_u) arg_u[k * H * F + col] = be < 0 ? -1 : g->src[be];
                }
            }
    }
    free_adj(&in);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* g-SDDMM (Section 3): m_e = phi(lhs at its target, rhs at its target)      */

static int64_t target_row(int target, int64_t u, int64_t e, int64_t v) {
    return target == OR_SRC ? u : (target == OR_DST ? v : e);
}

static int64_t target_rows(const or_graph* g, int target) {
    return target == OR_SRC ? g->n_src : (target == OR_DST ? g->n_dst : g->n_edges);
}

int oracle_gsddmm(const or_graph* g, int op, const or_tensor* lhs, int lhs_target, const or_tensor* rhs,
                  int rhs_target, or_tensor* out, const int64_t* edges, int64_t n_sel) {
    if (!graph_ok(g) || !dtype_ok(out) || op < OR_COPY_LHS || op > OR_DOT) return -1;
    if (lhs_target < OR_SRC || lhs_target > OR_DST || rhs_target < OR_SRC || rhs_target > OR_DST) return -1;
    if (op_uses_lhs(op) && (!dtype_ok(lhs) || lhs->rows != target_rows(g, lhs_target))) return -1;
    if (op_uses_rhs(op) && (!dtype_ok(rhs) || rhs->rows != target_rows(g, rhs_target))) return -1;
    int64_t H, F;
    if (op == OR_DOT) {
        if (msg_shape(OR_MUL, lhs, rhs, &H, &F) || out->heads != H || out->feat != 1) return -1;
    } else if (msg_shape(op, lhs, rhs, &H, &F) || out->heads != H || out->feat != F) {
        return -1;
    }
    if (out->rows != (edges ? n_sel : g->n_edges)) return -1;
    int64_t cnt = edges ? n_sel : g->n_edges;
    for (int64_t k = 0; k < cnt; ++k) {
        int64_t e = edges ? edges[k] : k;
        if (e < 0 || e >= g->n_edges) return -1;
        int64_t u = g->src[e], v = g->dst[e];
        int64_t rl = target_row(lhs_target, u, e, v), rr = target_row(rhs_target, u, e, v);
        for (int64_t h = 0; h < H; ++h) {
            if (op == OR_DOT) {
                double acc = 0.0;
                for (int64_t f = 0; f < F; ++f) acc += ld(lhs, rl, h, f) * ld(rhs, rr, h, f);
                st(out, k, h, 0, acc);
            } else {
                for (int64_t f = 0; f < F; ++f) {
                    double x = op_uses_lhs(op) ? ld(lhs, rl, h, f) : 0.0;
                    double w = op_uses_rhs(op) ? ld(rhs, rr, h, f) : 0.0;
                    st(out, k, h, f, phi(op, x, w));
                }
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* g-SpMM backward (Appendix B: the lemma on dL/dW of g-SpMM and lemma      */
/* complex_dspmm_dx).  With g'_{v,e} = dL/dz_v * d rho / d m_e:              */
/*   dL/dx_u = sum over out-edges (u, e, v) of g'_{v,e} * d phi / d x_u      */
/*   dL/dw_e = g'_{v,e} * d phi / d w_e                                      */
/* d rho / d m_e is 1 for sum, 1/deg(v) for mean, and for max/min the        */
/* indicator that e is the recorded arg edge.                                 */

static double dz_scaled(int reduce, const or_tensor* dz, const int32_t* arg_e, int64_t v, int64_t e, int64_t deg,
                        int64_t h, int64_t f, int64_t H, int64_t F) {
    double d = ld(dz, v, h, f);
    if (reduce == OR_MEAN) return d / (double)deg;
    if (reduce == OR_MAX || reduce == OR_MIN) return arg_e[v * H * F + h * F + f] == (int32_t)e ? d : 0.0;
    return d;
}

/* d phi / d x and d phi / d w, already multiplied by the incoming gradient gz */
static double dphi_dx(int op, double gz, double x, double w) {
    (void)x;
    switch (op) {
        case OR_COPY_LHS: case OR_ADD: case OR_SUB: return gz;
        case OR_MUL: return gz * w;
        case OR_DIV: return gz / w;
        default: return 0.0;
    }
}

static double dphi_dw(int op, double gz, double x, double w) {
    switch (op) {
        case OR_COPY_RHS: case OR_ADD: return gz;
        case OR_SUB: return -gz;
        case OR_MUL: return gz * x;
        case OR_DIV: return -gz * x / (w * w);
        default: return 0.0;
    }
}

int oracle_gspmm_backward(const or_graph* g, int op, int reduce, const or_tensor* lhs, const or_tensor* rhs,
                          const int32_t* arg_e, const or_tensor* grad_out, or_tensor* grad_lhs,
                          or_tensor* grad_rhs, const int64_t* sel, int64_t n_sel) {
    if (!graph_ok(g) || !dtype_ok(grad_out) || op < OR_COPY_LHS || op > OR_DIV || reduce < OR_SUM ||
        reduce > OR_MIN)
        return -1;
    if ((reduce == OR_MAX || reduce == OR_MIN) && !arg_e) return -1;
    if (op_uses_lhs(op) && (!dtype_ok(lhs) || lhs->rows != g->n_src)) return -1;
    if (op_uses_rhs(op) && (!dtype_ok(rhs) || rhs->rows != g->n_edges)) return -1;
    if (grad_lhs && (!op_uses_lhs(op) || !dtype_ok(grad_lhs) || grad_lhs->rows != (sel ? n_sel : g->n_src) ||
                     grad_lhs->heads != lhs->heads || grad_lhs->feat != lhs->feat))
        return -1;
    if (grad_rhs && (!op_uses_rhs(op) || !dtype_ok(grad_rhs) || grad_rhs->rows != (sel ? n_sel : g->n_edges) ||
                     grad_rhs->heads != rhs->heads || grad_rhs->feat != rhs->feat))
        return -1;
    if (sel && grad_lhs && grad_rhs) return -1; /* sampled mode computes one gradient */
    int64_t H, F;
    if (msg_shape(op, lhs, rhs, &H, &F) || grad_out->heads != H || grad_out->feat != F ||
        grad_out->rows != g->n_dst)
        return -1;
    adj in, outl;
    if (build_adj(g, 0, &in) || build_adj(g, 1, &outl)) { free_adj(&in); free_adj(&outl); return -1; }
    int rc = 0;
    if (grad_lhs) {
        int64_t cnt = sel ? n_sel : g->n_src;
        for (int64_t k = 0; k < cnt && !rc; ++k) {
            int64_t u = sel ? sel[k] : k;
            if (u < 0 || u >= g->n_src) { rc = -1; break; }
            for (int64_t hl = 0; hl < lhs->heads; ++hl)
                for (int64_t fl = 0; fl < lhs->feat; ++fl) {
                    double acc = 0.0;
                    for (int64_t p = outl.ptr[u]; p < outl.ptr[u + 1]; ++p) {
                        int64_t e = outl.eid[p], v = g->dst[e], deg = in.ptr[v + 1] - in.ptr[v];
                        for (int64_t h = 0; h < H; ++h) {
                            if (lhs->heads != 1 && h != hl) continue;
                            for (int64_t f = 0; f < F; ++f) {
                                if (lhs->feat != 1 && f != fl) continue;
                                double gz = dz_scaled(reduce, grad_out, arg_e, v, e, deg, h, f, H, F);
                                double x = ld(lhs, u, h, f);
                                double w = op_uses_rhs(op) ? ld(rhs, e, h, f) : 0.0;
                                acc += dphi_dx(op, gz, x, w);
                            }
                        }
                    }
                    st(grad_lhs, k, hl, fl, acc);
                }
        }
    }
    if (grad_rhs && !rc) {
        int64_t cnt = sel ? n_sel : g->n_edges;
        for (int64_t k = 0; k < cnt; ++k) {
            int64_t e = sel ? sel[k] : k;
            if (e < 0 || e >= g->n_edges) { rc = -1; break; }
            int64_t u = g->src[e], v = g->dst[e], deg = in.ptr[v + 1] - in.ptr[v];
            for (int64_t hr = 0; hr < rhs->heads; ++hr)
                for (int64_t fr = 0; fr < rhs->feat; ++fr) {
                    double acc = 0.0;
                    for (int64_t h = 0; h < H; ++h) {
                        if (rhs->heads != 1 && h != hr) continue;
                        for (int64_t f = 0; f < F; ++f) {
                            if (rhs->feat != 1 && f != fr) continue;
                            double gz = dz_scaled(reduce, grad_out, arg_e, v, e, deg, h, f, H, F);
                            double x = op_uses_lhs(op) ? ld(lhs, u, h, f) : 0.0;
                            double w = ld(rhs, e, h, f);
                            acc += dphi_dw(op, gz, x, w);
                        }
                    }
                    st(grad_rhs, k, hr, fr, acc);
                }
        }
    }
    free_adj(&in);
    free_adj(&outl);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* g-SDDMM backward (Appendix B: the lemma on dL/dW of g-SDDMM and lemma     */
/* rev).  An operand on the source side collects over the out-edges of its   */
/* node, on the destination side over the in-edges, on the edge side from    */
/* its own edge only.                                                        */

/* derivative of lhs (which = 0) or rhs (which = 1) times the incoming gm */
static double dsddmm(int op, int which, double gm, double l, double r) {
    if (which == 0) {
        switch (op) {
            case OR_COPY_LHS: case OR_ADD: case OR_SUB: return gm;
            case OR_MUL: case OR_DOT: return gm * r;
            case OR_DIV: return gm / r;
            default: return 0.0;
        }
    }
    switch (op) {
        case OR_COPY_RHS: case OR_ADD: return gm;
        case OR_SUB: return -gm;
        case OR_MUL: case OR_DOT: return gm * l;
        case OR_DIV: return -gm * l / (r * r);
        default: return 0.0;
    }
}

int oracle_gsddmm_backward(const or_graph* g, int op, const or_tensor* lhs, int lhs_target, const or_tensor* rhs,
                           int rhs_target, const or_tensor* grad_out, or_tensor* grad_lhs, or_tensor* grad_rhs,
                           const int64_t* sel, int64_t n_sel) {
    if (!graph_ok(g) || !dtype_ok(grad_out) || op < OR_COPY_LHS || op > OR_DOT) return -1;
    if (lhs_target < OR_SRC || lhs_target > OR_DST || rhs_target < OR_SRC || rhs_target > OR_DST) return -1;
    int uses_l = op_uses_lhs(op), uses_r = op_uses_rhs(op);
    /* dot and the binary ops read both operands (the derivative needs the other one) */
    if ((uses_l || grad_rhs) && op != OR_COPY_RHS && (!dtype_ok(lhs) || lhs->rows != target_rows(g, lhs_target)))
        return -1;
    if ((uses_r || grad_lhs) && op != OR_COPY_LHS && (!dtype_ok(rhs) || rhs->rows != target_rows(g, rhs_target)))
        return -1;
    if (grad_lhs && (!uses_l || !dtype_ok(grad_lhs) || grad_lhs->rows != (sel ? n_sel : lhs->rows) ||
                     grad_lhs->heads != lhs->heads || grad_lhs->feat != lhs->feat))
        return -1;
    if (grad_rhs && (!uses_r || !dtype_ok(grad_rhs) || grad_rhs->rows != (sel ? n_sel : rhs->rows) ||
                     grad_rhs->heads != rhs->heads || grad_rhs->feat != rhs->feat))
        return -1;
    if (sel && grad_lhs && grad_rhs) return -1;
    int64_t H, F;
    if (msg_shape(op == OR_DOT ? OR_MUL : op, lhs, rhs, &H, &F)) return -1;
    if (grad_out->rows != g->n_edges || grad_out->heads != H || grad_out->feat != (op == OR_DOT ? 1 : F)) return -1;
    adj in, outl;
    if (build_adj(g, 0, &in) || build_adj(g, 1, &outl)) { free_adj(&in); free_adj(&outl); return -1; }
    int rc = 0;
    for (int which = 0; which < 2 && !rc; ++which) {
        or_tensor* gt = which == 0 ? grad_lhs : grad_rhs;
        const or_tensor* self = which == 0 ? lhs : rhs;
        int target = which == 0 ? lhs_target : rhs_target;
        if (!gt) continue;
        int64_t cnt = sel ? n_sel : self->rows;
        for (int64_t k = 0; k < cnt; ++k) {
            int64_t row = sel ? sel[k] : k;
            if (row < 0 || row >= self->rows) { rc = -1; break; }
            /* the edges whose message reads this row of the operand */
            const int64_t* list;
            int64_t nl, one = row;
            if (target == OR_SRC) { list = outl.eid + outl.ptr[row]; nl = outl.ptr[row + 1] - outl.ptr[row]; }
            else if (target == OR_DST) { list = in.eid + in.ptr[row]; nl = in.ptr[row + 1] - in.ptr[row]; }
            else { list = &one; nl = 1; }
            for (int64_t hs = 0; hs < self->heads; ++hs)
                for (int64_t fs = 0; fs < self->feat; ++fs) {
                    double acc = 0.0;
                    for (int64_t i = 0; i < nl; ++i) {
                        int64_t e = list[i], u = g->src[e], v = g->dst[e];
                        int64_t rl = target_row(lhs_target, u, e, v), rr = target_row(rhs_target, u, e, v);
                        for (int64_t h = 0; h < H; ++h) {
                            if (self->heads != 1 && h != hs) continue;
                            for (int64_t f = 0; f < F; ++f) {
                                if (self->feat != 1 && f != fs) continue;
                                double gm = ld(grad_out, e, h, op == OR_DOT ? 0 : f);
                                double l = (op != OR_COPY_RHS) ? ld(lhs, rl, h, f) : 0.0;
                                double r = (op != OR_COPY_LHS) ? ld(rhs, rr, h, f) : 0.0;
                                acc += dsddmm(op, which, gm, l, r);
                            }
                        }
                    }
                    st(gt, k, hs, fs, acc);
                }
        }
    }
    free_adj(&in);
    free_adj(&outl);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* edge softmax over the in-edges of each destination, per column.  With a   */
/* row selection, outputs are written compactly: the in-edges of rows[0],   */
/* then of rows[1], ..., each in ascending edge id, and out_eids (if given)  */
/* receives the edge id of every written row.                                */

static int64_t sel_edges(const adj* in, const int64_t* rows, int64_t n_rows) {
    int64_t t = 0;
    for (int64_t k = 0; k < n_rows; ++k) t += in->ptr[rows[k] + 1] - in->ptr[rows[k]];
    return t;
}

int oracle_edge_softmax(const or_graph* g, const or_tensor* score, or_tensor* out, const int64_t* rows,
                        int64_t n_rows, int64_t* out_eids) {
    if (!graph_ok(g) || !dtype_ok(score) || !dtype_ok(out) || score->rows != g->n_edges ||
        out->heads != score->heads || out->feat != score->feat)
        return -1;
    adj in;
    if (build_adj(g, 0, &in)) { free_adj(&in); return -1; }
    int64_t cnt = rows ? n_rows : g->n_dst;
    for (int64_t k = 0; k < cnt; ++k)
        if (rows && (rows[k] < 0 || rows[k] >= g->n_dst)) { free_adj(&in); return -1; }
    if (out->rows != (rows ? sel_edges(&in, rows, n_rows) : g->n_edges)) { free_adj(&in); return -1; }
    int64_t q = 0;
    for (int64_t k = 0; k < cnt; ++k) {
        int64_t v = rows ? rows[k] : k, b = in.ptr[v], end = in.ptr[v + 1];
        for (int64_t h = 0; h < score->heads; ++h)
            for (int64_t f = 0; f < score->feat; ++f) {
                double m = -INFINITY, den = 0.0;
                for (int64_t p = b; p < end; ++p) {
                    double s = ld(score, in.eid[p], h, f);
                    if (s > m) m = s;
                }
                for (int64_t p = b; p < end; ++p) den += exp(ld(score, in.eid[p], h, f) - m);
                for (int64_t p = b; p < end; ++p) {
                    int64_t e = in.eid[p];
                    st(out, rows ? q + (p - b) : e, h, f, exp(ld(score, e, h, f) - m) / den);
                }
            }
        if (rows && out_eids)
            for (int64_t p = b; p < end; ++p) out_eids[q + (p - b)] = in.eid[p];
        q += end - b;
    }
    free_adj(&in);
    return 0;
}

/* d a_e / d s: ds_e = a_e (g_e - sum over the group of a * g); the selection
 * works as in oracle_edge_softmax, and out / grad_out are read at edge ids. */
int oracle_edge_softmax_backward(const or_graph* g, const or_tensor* out, const or_tensor* grad_out,
                                 or_tensor* grad_score, const int64_t* rows, int64_t n_rows, int64_t* out_eids) {
    if (!graph_ok(g) || !dtype_ok(out) || !dtype_ok(grad_out) || !dtype_ok(grad_score) ||
        out->rows != g->n_edges || grad_out->rows != g->n_edges || grad_out->heads != out->heads ||
        grad_out->feat != out->feat || grad_score->heads != out->heads || grad_score->feat != out->feat)
        return -1;
    adj in;
    if (build_adj(g, 0, &in)) { free_adj(&in); return -1; }
    int64_t cnt = rows ? n_rows : g->n_dst;
    for (int64_t k = 0; k < cnt; ++k)
        if (rows && (rows[k] < 0 || rows[k] >= g->n_dst)) { free_adj(&in); return -1; }
    if (grad_score->rows != (rows ? sel_edges(&in, rows, n_rows) : g->n_edges)) { free_adj(&in); return -1; }
    int64_t q = 0;
    for (int64_t k = 0; k < cnt; ++k) {
        int64_t v = rows ? rows[k] : k, b = in.ptr[v], end = in.ptr[v + 1];
        for (int64_t h = 0; h < out->heads; ++h)
            for (int64_t f = 0; f < out->feat; ++f) {
                double s = 0.0;
                for (int64_t p = b; p < end; ++p) s += ld(out, in.eid[p], h, f) * ld(grad_out, in.eid[p], h, f);
                for (int64_t p = b; p < end; ++p) {
                    int64_t e = in.eid[p];
                    st(grad_score, rows ? q + (p - b) : e, h, f, ld(out, e, h, f) * (ld(grad_out, e, h, f) - s));
                }
            }
        if (rows && out_eids)
            for (int64_t p = b; p < end; ++p) out_eids[q + (p - b)] = in.eid[p];
        q += end - b;
    }
    free_adj(&in);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* leaky ReLU on edge scores                                                 */

int oracle_leaky_relu(const or_tensor* x, or_tensor* y, float slope) {
    if (!dtype_ok(x) || !dtype_ok(y) || x->rows != y->rows || x->heads != y->heads || x->feat != y->feat) return -1;
    for (int64_t r = 0; r < x->rows; ++r)
        for (int64_t h = 0; h < x->heads; ++h)
            for (int64_t f = 0; f < x->feat; ++f) {
                double v = ld(x, r, h, f);
                st(y, r, h, f, v > 0.0 ? v : (double)slope * v);
            }
    return 0;
}

int oracle_leaky_relu_backward(const or_tensor* x, const or_tensor* dy, or_tensor* dx, float slope) {
    if (!dtype_ok(x) || !dtype_ok(dy) || !dtype_ok(dx) || x->rows != dy->rows || x->rows != dx->rows ||
        x->heads != dy->heads || x->heads != dx->heads || x->feat != dy->feat || x->feat != dx->feat)
        return -1;
    for (int64_t r = 0; r < x->rows; ++r)
        for (int64_t h = 0; h < x->heads; ++h)
            for (int64_t f = 0; f < x->feat; ++f) {
                double d = ld(dy, r, h, f);
                st(dx, r, h, f, ld(x, r, h, f) > 0.0 ? d : (double)slope * d);
            }
    return 0;
}
