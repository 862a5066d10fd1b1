/*
 * gnnk: generalized sparse message-passing kernels for MI355X (gfx950).
 *
 * C ABI of the GPU library libgnnk.so.  It implements the two primitives that
 * Section 3 of "Deep Graph Library: A Graph-Centric, Highly-Performant Package
 * for Graph Neural Networks" (arXiv 1909.01315) reduces message passing to:
 *
 *   g-SDDMM  m_e = phi(x_u, y_v, w_e)                 for every edge (u, e, v)
 *   g-SpMM   z_v = rho{ phi(x_u, w_e) : (u, e, v) }   over the in-edges of v
 *
 * and their gradients, which by Theorem 1 are again a g-SDDMM on the graph
 * (edge gradients) and g-SpMMs on the graph or on the reverse graph (node
 * gradients).  Edge softmax and the leaky ReLU of attention layers are
 * provided on the same graph structure.
 *
 * Conventions shared by every call:
 *  - Every call returns a gnnk_status and never throws.  On failure
 *    gnnk_last_error() describes the cause (thread-local, valid until the next
 *    gnnk call on the same thread).
 *  - Device pointers: all tensor and index pointers are device memory owned by
 *    the caller; the library never frees them.  A NULL tensor pointer means
 *    "absent" where the argument is documented nullable.
 *  - Work is enqueued on `stream` and runs asynchronously; calls return before
 *    the kernels finish.  Only graph_create_* and graph_validate synchronise.
 *    No call allocates device memory (Section 4.2: the framework allocates):
 *    the graph's derived arrays live in a workspace the caller provides, and
 *    the scratch memory some compute calls need is lent by the caller per
 *    stream (graph_attach_scratch).  A sequence of compute calls can
 *    therefore be captured into a HIP graph as it is.
 *  - Outputs are fully overwritten, never accumulated into.  Inputs may alias
 *    each other; outputs must not alias inputs or each other.
 *  - Edge tensors are indexed by edge id.  Node tensors by node id.
 *  - Index ranges are not checked on the compute path; use graph_validate.
 *  - All floating-point tensors of one call share one dtype.  Sums and dot
 *    products accumulate in fp64 and are rounded once to the output dtype
 *    (bf16 outputs: to fp32, then to bf16 round-to-nearest-even).
 *  - Rows of any width: a sum over the features of a message (DOT, or the
 *    gradient of an operand broadcast over features) wider than one pass of a
 *    wavefront (64 lanes of 4 fp32 or 8 bf16 values) adds its passes in fp64
 *    in order, and per-head sums of such rows run as slices of heads.
 *  - A handle is immutable after creation: calls on several streams may use
 *    it at once, each stream with its own lent scratch buffer.
 */
#ifndef GNNK_H
#define GNNK_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GNNK_OK = 0,
    GNNK_EINVAL = 1,       /* invalid argument: enum, shape, broadcast, NULL */
    GNNK_EUNSUPPORTED = 2, /* legal combination that is not implemented */
    GNNK_EHIP = 3,         /* HIP runtime or launch error */
    GNNK_ERANGE = 4,       /* graph_validate: an index is out of range */
    GNNK_ENOMEM = 5        /* workspace too small or allocation failed */
} gnnk_status;

typedef enum { GNNK_I32 = 0, GNNK_I64 = 1 } gnnk_itype;
typedef enum { GNNK_F32 = 0, GNNK_BF16 = 1 } gnnk_ftype;

/* message functions phi: copy_u = COPY_LHS, copy_e = COPY_RHS, and the binary
 * ops on (lhs, rhs); DOT reduces the feature dimension (g-SDDMM only). */
typedef enum {
    GNNK_COPY_LHS = 0,
    GNNK_COPY_RHS = 1,
    GNNK_ADD = 2,
    GNNK_SUB = 3,
    GNNK_MUL = 4,
    GNNK_DIV = 5,
    GNNK_DOT = 6
} gnnk_binop;

/* reduce functions rho of g-SpMM */
typedef enum { GNNK_SUM = 0, GNNK_MEAN = 1, GNNK_MAX = 2, GNNK_MIN = 3 } gnnk_reduce;

/* where a g-SDDMM operand lives: u (source node), e (edge), v (destination) */
typedef enum { GNNK_SRC = 0, GNNK_EDGE = 1, GNNK_DST = 2 } gnnk_target;

/* A dense (rows, heads, feat) tensor, row-major, with a row stride in
 * elements (>= heads * feat, < 2^31).  Broadcasting (Appendix E's multi-head forms):
 * an operand may be (H, F), (H, 1) or (1, 1) against an (H, F) message. */
typedef struct {
    void* data;
    int64_t rows;
    int32_t heads;
    int32_t feat;
    int64_t row_stride;
    int32_t dtype; /* gnnk_ftype */
    int32_t reserved;
} gnnk_tensor;

typedef struct gnnk_graph* gnnk_graph_t; /* opaque, immutable after creation */

/* Host-side description of a graph handle (no GPU access). */
typedef struct {
    int64_t num_src, num_dst, num_edges;
    int32_t ptr_type;       /* gnnk_itype of the CSR row offsets */
    int32_t identity_eids;  /* 1 when edge id == in-CSR position */
    int64_t max_in_degree, max_out_degree;
    int64_t empty_dst_rows, empty_src_rows;
    int64_t seg_edges;      /* edges per segment of a hub row of the in-CSR */
    int64_t hub_dst_rows, hub_src_rows;   /* rows longer than their CSR's segment size */
    int64_t segments_in, segments_out;    /* segments of those rows */
    size_t workspace_bytes;
    int64_t seg_edges_out;  /* edges per segment of a hub row of the reverse graph's CSR */
    int64_t seg_edges_gather; /* the same for the reverse passes that gather node rows */
    int64_t segments_gather;  /* the segments of that finer table */
    int64_t seg_edges_in_gather; /* the in-CSR's finer segments, for the passes that gather node rows */
    int64_t segments_in_gather;  /* the segments of that table */
} gnnk_graph_info;

/* ------------------------------------------------------------------------ */
/* Graph structure (Section 4.1: CSR for g-SpMM forward, the reverse graph's
 * CSR for backward, edge ids kept; Appendix B, definition of the reverse
 * graph).  A handle holds the in-CSR (rows = destinations), the out-CSR of
 * the reverse graph (rows = sources, with the original edge ids), in- and
 * out-degrees, rows sorted by degree for scheduling, and the segment tables
 * of rows longer than seg_edges.  Derived arrays live in a caller-allocated
 * device workspace of graph_workspace_bytes() bytes, which the caller keeps
 * alive (with any borrowed index arrays) until graph_destroy.  Building runs
 * on the device, on `stream`: stable radix sorts of (row, edge id) pairs, so
 * each row lists its edges in ascending edge id, row offsets by binary search
 * in the sorted rows, and rows ordered by descending degree (ties by row id).
 * The segments of long rows are also ordered by the neighbour ids they cover
 * (the halves of their first and last neighbour id, summed; a stable sort):
 * calls take them in that order, so that where rows list their neighbours in
 * ascending order (an edge list sorted by destination, then source) the
 * segments processed at the same time gather from one slice of the neighbour
 * table.  The order never changes a result: segment partials are combined in
 * table order.
 * The call synchronises `stream` twice (after checking the input, and to read
 * back the sorted degrees); it allocates no device memory (its temporaries
 * are part of the workspace). */

/* Upper bound of the workspace for a graph of this size; ptr_t is the width
 * of the CSR row offsets the handle builds (either width for any size).
 * Node counts must be below 2^31 - 1 and num_edges at most 2^31 - 2^16 - 1
 * (edge ids and CSR positions are int32, and the walks step positions past a
 * row's end before testing them); GNNK_EINVAL otherwise. */
gnnk_status graph_workspace_bytes(int64_t num_src, int64_t num_dst, int64_t num_edges, gnnk_itype ptr_t,
                                  size_t* bytes);

/* From an edge list in edge-id order: edge e goes src[e] -> dst[e] (device
 * int32 arrays of num_edges entries, only read during the call).  Edges of a
 * destination keep ascending edge id in the in-CSR, edges of a source keep
 * ascending edge id in the out-CSR.  Multi-edges and self-loops are legal; an
 * endpoint out of range returns GNNK_EINVAL. */
gnnk_status graph_create_coo(int64_t num_src, int64_t num_dst, int64_t num_edges, const int32_t* src,
                             const int32_t* dst, gnnk_itype ptr_t, void* workspace, size_t ws_bytes,
                             hipStream_t stream, gnnk_graph_t* out);

/* From an in-CSR: indptr (num_dst + 1 entries of ptr_t), indices (num_edges
 * int32 source ids) and eids (num_edges int32 edge ids, or NULL when the edge
 * id is the position).  These device arrays are borrowed, not copied: keep
 * them unchanged until graph_destroy.  Rows must be ascending in position
 * (indptr non-decreasing, indptr[0] == 0, indptr[num_dst] == num_edges),
 * indices below num_src, and eids a permutation of 0..num_edges-1; any
 * violation returns GNNK_EINVAL and builds nothing. */
gnnk_status graph_create_csr(int64_t num_src, int64_t num_dst, int64_t num_edges, const void* indptr,
                             gnnk_itype ptr_t, const int32_t* indices, const int32_t* eids, void* workspace,
                             size_t ws_bytes, hipStream_t stream, gnnk_graph_t* out);

/* Host-side facts about a handle. */
gnnk_status graph_info(gnnk_graph_t g, gnnk_graph_info* info);

/* In-degrees (num_dst int32) and out-degrees (num_src int32), written to
 * caller device memory on `stream` (the batched g.in_degree of Section 4.1). */
gnnk_status graph_in_degrees(gnnk_graph_t g, int32_t* out, hipStream_t stream);
gnnk_status graph_out_degrees(gnnk_graph_t g, int32_t* out, hipStream_t stream);

/* Copy the in-CSR (reverse = 0) or the reverse graph's CSR (reverse = 1) into
 * caller device buffers: indptr (rows + 1 entries of the handle's ptr type),
 * indices (num_edges int32), eids (num_edges int32; for reverse = 0 with
 * identity ids this is 0..E-1).  Any of the three may be NULL. */
gnnk_status graph_csr_export(gnnk_graph_t g, int reverse, void* indptr, int32_t* indices, int32_t* eids,
                             hipStream_t stream);

/* Check every stored index against its range; synchronises `stream`.
 * Returns GNNK_ERANGE if any index is out of range. */
gnnk_status graph_validate(gnnk_graph_t g, hipStream_t stream);

/* Free the handle (a host object; the workspace and every lent scratch
 * buffer stay the caller's, to be released once the kernels queued on them
 * have finished). */
gnnk_status graph_destroy(gnnk_graph_t g);

/* ------------------------------------------------------------------------ */
/* Scratch memory of compute calls.  Some calls need device memory beyond
 * their inputs and outputs: fp64 partial results of the segments of hub
 * rows (g-SpMM sum/mean/max/min and their gradients, the fused attention),
 * the winner masks of the max/min backward, the per-(destination, head)
 * records of the fused attention backward, per-edge fp64 running sums of
 * reductions wider than one pass of a wavefront, and the partial rows of the
 * edge-parallel schedules.  The caller lends it, per stream: a call that
 * needs scratch uses the buffer attached to the handle for the stream it is
 * issued on, front to back; with none, or one too small, it returns
 * GNNK_ENOMEM before launching anything, and gnnk_scratch_needed() tells the
 * bytes it asked for.  Calls on one stream run in stream order and share its
 * buffer; calls on different streams use different buffers.  The contents
 * of a buffer need not be initialised and are not preserved between
 * calls. */

enum {
    GNNK_SCRATCH_ARGMAX = 1,     /* include the max/min backward (winner masks: E * ceil(cols / 32) * 4 bytes) */
    GNNK_SCRATCH_WIDE_SUMS = 2   /* include sums over more than 64 lanes of a row (E * 8 bytes) */
};

/* Bytes of scratch that any call on this handle with messages of at most
 * max_cols columns (heads * feat) needs, under the options set now; flags
 * add the two kinds above. */
gnnk_status graph_scratch_bytes(gnnk_graph_t g, int64_t max_cols, int32_t flags, size_t* bytes);

/* Lend buf (device memory, 256-byte aligned, `bytes` bytes) to the handle for
 * the calls issued on `stream`, replacing any earlier buffer of that stream;
 * buf == NULL or bytes == 0 takes the stream's buffer back.  Host-side only:
 * no GPU work.  The caller keeps the buffer alive, unchanged by other work,
 * until the calls queued on `stream` with it have finished (releasing it to
 * an allocator ordered on that stream is enough).  At most 16 streams per
 * handle (GNNK_EINVAL beyond). */
gnnk_status graph_attach_scratch(gnnk_graph_t g, hipStream_t stream, void* buf, size_t bytes);

/* Bytes of scratch the last call on this thread that returned GNNK_ENOMEM for
 * lack of scratch asked for (0 after any other outcome): the whole call's
 * need, so the same call with a buffer of that many bytes gets its scratch.
 * A call made of several passes (gradient pairs, the max/min backward, slices
 * of heads, the fused attention backward) is checked whole, arguments and
 * scratch, before its first pass is launched. */
gnnk_status gnnk_scratch_needed(size_t* bytes);

/* ------------------------------------------------------------------------ */
/* g-SpMM (Section 3, definition of generalized SpMM):
 *   out[v] = reduce over in-edges (u, e, v) of op(lhs[u], rhs[e])
 * op: COPY_LHS | COPY_RHS | ADD | SUB | MUL | DIV (not DOT).
 * lhs: num_src rows (NULL iff op == COPY_RHS); rhs: num_edges rows (NULL iff
 * op == COPY_LHS); out: num_dst rows of the broadcast (H, F) shape.
 * reduce: SUM, MEAN (divides by the in-degree, multi-edges counted), MAX, MIN.
 * A destination with no in-edge gets 0.
 * MAX/MIN: messages are formed in fp32 and compared exactly; the smallest edge
 * id wins a tie.  arg_lhs (source id) and arg_rhs (edge id) are nullable dense
 * (num_dst, H, F) int32 arrays, -1 for empty destinations.
 * Scratch: fp64 partials of hub-row segments, segments x H * F x 8 bytes
 * (12 for MAX/MIN).
 * Errors: GNNK_EINVAL on a bad op/reduce, shapes or dtypes; GNNK_EUNSUPPORTED
 * for arg arrays with SUM/MEAN. */
gnnk_status gspmm(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                  const gnnk_tensor* rhs, gnnk_tensor* out, int32_t* arg_lhs, int32_t* arg_rhs,
                  hipStream_t stream);

/* gspmm for callers that cannot allocate at all (code under HIP graph
 * capture with no buffer to lend, tight serving loops, harnesses that forbid
 * allocation): the same operation, arguments and results as gspmm, with its
 * scratch taken from a fixed buffer of 64 MiB that the library holds on each
 * GPU it runs on (from the first call on that GPU until the process ends)
 * instead of a lent one; no buffer needs to be attached.  The caller still
 * provides inputs and outputs.  A call whose scratch would exceed 64 MiB
 * (segments x H * F x 8 bytes, x 12 for MAX/MIN) returns GNNK_ENOMEM before
 * launching anything.  Every call on one GPU shares that GPU's buffer: calls
 * that overlap in time on one GPU (on different streams, or from several
 * threads without ordering) race and give undefined results; calls ordered
 * on one stream are safe.  Nothing in the buffer needs to start at zero. */
gnnk_status gspmm_noalloc(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                          const gnnk_tensor* rhs, gnnk_tensor* out, int32_t* arg_lhs, int32_t* arg_rhs,
                          hipStream_t stream);

/* g-SDDMM (Section 3, definition of generalized SDDMM):
 *   out[e] = op(lhs[t_l(e)], rhs[t_r(e)]) for every edge (u, e, v),
 * t(e) being u, e or v by the operand's target.  ADD/SUB/MUL/DIV are single
 * fp32 operations; DOT is the fp64-accumulated inner product over the feature
 * dimension, giving (E, H, 1) (the per-head attention score of Appendix E);
 * COPY_LHS / COPY_RHS copy one operand.  out: num_edges rows. */
gnnk_status gsddmm(gnnk_graph_t g, gnnk_binop op, const gnnk_tensor* lhs, gnnk_target lhs_target,
                   const gnnk_tensor* rhs, gnnk_target rhs_target, gnnk_tensor* out, hipStream_t stream);

/* Gradients of gspmm (Theorem 1; Appendix B, the lemma on dL/dW of g-SpMM and
 * lemma complex_dspmm_dx).  With g'_e = grad_out[v] scaled by d rho/d m_e
 * (1 for SUM, 1/deg(v) for MEAN, for MAX/MIN 1 iff e is arg_rhs[v]):
 *   grad_lhs[u] = sum over out-edges (u, e, v) of g'_e * d phi/d lhs   (a
 *                 g-SpMM on the reverse graph)
 *   grad_rhs[e] = g'_e * d phi/d rhs                                   (a
 *                 g-SDDMM on the graph)
 * both summed over broadcast positions when the operand is broadcast.
 * lhs/rhs as in the forward call; grad_out: num_dst rows of the message
 * shape.  arg_rhs is required for MAX/MIN (the edge ids written by gspmm);
 * arg_lhs is accepted and unused.  grad_lhs / grad_rhs are nullable.  MAX/MIN
 * run without atomics (a masked reverse g-SpMM and a masked g-SDDMM). */
gnnk_status gspmm_backward(gnnk_graph_t g, gnnk_binop op, gnnk_reduce reduce, const gnnk_tensor* lhs,
                           const gnnk_tensor* rhs, const int32_t* arg_lhs, const int32_t* arg_rhs,
                           const gnnk_tensor* grad_out, gnnk_tensor* grad_lhs, gnnk_tensor* grad_rhs,
                           hipStream_t stream);

/* Gradients of gsddmm (Appendix B, the lemma on dL/dW of g-SDDMM and lemma
 * rev): an operand on the source side collects over its node's out-edges
 * (reverse graph), on the destination side over its in-edges, on the edge side
 * from its own edge.  grad_out: num_edges rows of the output shape.
 * grad_lhs / grad_rhs are nullable and take their operand's shape. */
gnnk_status gsddmm_backward(gnnk_graph_t g, gnnk_binop op, const gnnk_tensor* lhs, gnnk_target lhs_target,
                            const gnnk_tensor* rhs, gnnk_target rhs_target, const gnnk_tensor* grad_out,
                            gnnk_tensor* grad_lhs, gnnk_tensor* grad_rhs, hipStream_t stream);

/* Edge softmax (the attention normalisation applied to Appendix E's edge
 * scores): for each destination v and column c,
 *   out[e, c] = exp(score[e, c] - max) / sum over in-edges of v of exp(. - max).
 * score and out: num_edges rows, same shape.  Edges of a destination with one
 * in-edge get exactly 1.  Uses no scratch memory (a destination with many
 * in-edges is reduced within one workgroup). */
gnnk_status edge_softmax(gnnk_graph_t g, const gnnk_tensor* score, gnnk_tensor* out, hipStream_t stream);

/* grad_score[e] = out[e] * (grad_out[e] - sum over in-edges e' of dst(e) of
 * out[e'] * grad_out[e']), where out is the softmax result.  No scratch
 * memory, as for edge_softmax. */
gnnk_status edge_softmax_backward(gnnk_graph_t g, const gnnk_tensor* out, const gnnk_tensor* grad_out,
                                  gnnk_tensor* grad_score, hipStream_t stream);

/* Leaky ReLU on an edge (or any) tensor: y = x > 0 ? x : slope * x (one fp32
 * operation), and its backward dx = x > 0 ? dy : slope * dy. */
gnnk_status edge_leaky_relu(const gnnk_tensor* x, gnnk_tensor* y, float slope, hipStream_t stream);
gnnk_status edge_leaky_relu_backward(const gnnk_tensor* x, const gnnk_tensor* dy, gnnk_tensor* dx, float slope,
                                     hipStream_t stream);

/* Fused graph attention: the multi-head attention layer of Appendix E (a
 * g-SDDMM u_add_v producing per-head edge scores, leaky ReLU, softmax over
 * the in-edges of each destination, then a g-SpMM u_mul_e/sum) in one pass
 * over each destination's in-edges, without writing the scores:
 *   s[e, h]   = leaky(el[u, h] + er[v, h])      (fp32, as edge_leaky_relu)
 *   out[v, h] = sum over in-edges of softmax_v(s)[e, h] * feat[u, h, :]
 * feat: (num_src, H, F); el: (num_src, H, 1); er: (num_dst, H, 1); out:
 * (num_dst, H, F).  attn (nullable, (num_edges, H, 1)) receives the softmax,
 * which the unfused backward (gspmm_backward, edge_softmax_backward, ...)
 * needs.  stats (nullable, (num_dst, H, 2), always fp32) receives per
 * destination and head the maximum score m and the reciprocal 1/l of the
 * sum l of exp(s - m), from which gat_aggregate_backward recomputes the
 * attention (a = exp(s - m) * (1/l), as attn holds it); rows without
 * in-edges get (0, 0).  The running maximum is tracked per destination and
 * head and the fp64 sums are rescaled when it grows; destinations without
 * in-edges get 0.  Errors: GNNK_EINVAL on shapes or dtypes. */
gnnk_status gat_aggregate(gnnk_graph_t g, const gnnk_tensor* feat, const gnnk_tensor* el, const gnnk_tensor* er,
                          float slope, gnnk_tensor* out, gnnk_tensor* attn, gnnk_tensor* stats, hipStream_t stream);

/* Backward of gat_aggregate (Theorem 1's gradients of the g-SpMM and the
 * g-SDDMM, chained through the softmax and the leaky ReLU) without any
 * tensor of num_edges elements: with a the attention recomputed from stats,
 * da = grad_out[v, h, :] . feat[u, h, :] and lk the leaky ReLU's derivative
 * at el[u, h] + er[v, h] (the slope at 0 and below),
 *   grad_feat[u, h, :] = sum over out-edges of a * grad_out[v, h, :]
 *   grad_el[u, h]      = sum over out-edges of a * (da - S[v, h]) * lk
 *   grad_er[v, h]      = sum over in-edges of a * (da - S[v, h]) * lk
 * where S[v, h] = sum over in-edges of a * da; every sum in fp64, rounded
 * once.  feat, el, er, slope and stats as passed to (and written by)
 * gat_aggregate; grad_out (num_dst, H, F); the three gradients are nullable
 * and take their operand's shape; all tensors but stats share one dtype.
 * Rows of several heads wider than one pass of a wavefront (64 lanes of vec
 * values, vec being 4 fp32 or 8 bf16 as F and the row strides allow) run as
 * slices of heads; a single head wider than a pass runs in column chunks of
 * one pass, S, P and d_el being sums of per-chunk parts carried in fp64
 * between the chunks.  Scratch: 16 bytes per (destination, head), per-segment
 * partials of hub rows, and for a head in column chunks 16 bytes per
 * destination and 8 per source.  Errors: GNNK_EINVAL on shapes or dtypes. */
gnnk_status gat_aggregate_backward(gnnk_graph_t g, const gnnk_tensor* feat, const gnnk_tensor* el,
                                   const gnnk_tensor* er, float slope, const gnnk_tensor* stats,
                                   const gnnk_tensor* grad_out, gnnk_tensor* grad_feat, gnnk_tensor* grad_el,
                                   gnnk_tensor* grad_er, hipStream_t stream);
/* ------------------------------------------------------------------------ */
/* Tuning knobs, for schedule comparisons (forcing node- or edge-balanced
 * schedules; the paper's Table 1 states both are valid for commutative and
 * associative reducers).  Process-wide; "seg_edges" applies to graphs created
 * afterwards, the others to calls issued afterwards.  Keys:
 *   "seg_edges"   edges per hub-row segment: 0 (default) chooses per graph
 *                 the next power of two of num_edges / 8192 within [64, 512]
 *                 for the in-CSR and of num_edges / 2048 within [64, 2048]
 *                 for the reverse graph's CSR, and for the passes of either
 *                 CSR that gather node rows (and every g-SDDMM) of
 *                 num_edges / 16384 within [64, 256]
 *                 (small graphs split their long rows across more
 *                 wavefronts); otherwise a fixed value in [32, 2^30] for all
 *   "no_split"    1: never split a row across waves (hub rows run whole)
 *   "sddmm_split" wavefronts per hub-row segment of a g-SDDMM, each taking
 *                 whole batches of it: 0 (default) two where a batch holds
 *                 64 or more edges (16 or more lane groups), else one;
 *                 otherwise 1-8 (results do not depend on it)
 *   "small_deg"   rows of at most this many edges take one lane group each
 *                 and share a wavefront (-1 = auto: 32, or the lane groups
 *                 per wavefront if more; none when a wavefront is one group)
 *   "schedule"    0 auto (the row engine), 1 the row engine (node-parallel over the degree-
 *                 sorted rows), 2 the edge-parallel walk over the COO form
 *                 (equal edges per lane group; split rows combined in a fixed
 *                 order), 3 edge-parallel with fp64 atomics for split rows
 *                 (summation order not fixed).  Edge-parallel covers g-SpMM
 *                 sum/mean and g-SDDMM; max/min, edge softmax and outputs
 *                 summed over broadcast positions use the row engine.
 *   "edge_chunk"  positions per lane group of edge-parallel walks (0 auto)
 *   "no_fast"     1: run every call on the kernels that read operand layouts
 *                 at run time (no compile-time specialised walks)
 *   "fused_dw"    where the weight gradient of u_mul_e/sum (a per-head or
 *                 per-edge weight, both gradients asked for) is formed:
 *                 1: by the reverse pass that forms dX (one scattered record
 *                 per edge); 0: by a g-SDDMM pass of its own over the in-CSR;
 *                 -1 (default): fused for a weight of one column per edge,
 *                 a pass of its own for per-head weights
 * Returns GNNK_EINVAL for an unknown key or value. */
gnnk_status gnnk_set_option(const char* key, int64_t value);

const char* gnnk_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GNNK_H */
