/*
 * Reference ("oracle") implementation of generalized SpMM / SDDMM message
 * passing, for tests only.
 *
 * TEST INFRASTRUCTURE: only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  The GPU library never
 * includes, links or calls it, and it includes nothing from the GPU library.
 *
 * Everything here is a plain single-threaded loop over the definitions of
 * Section 3 (g-SDDMM and g-SpMM) and Appendix B (Theorem 1 and its lemmas,
 * the reverse graph).  Floating point is accumulated in double and rounded
 * once to the output type.
 *
 * Graph input: an edge list; edge e goes from src[e] to dst[e] (the paper's
 * (u, e, v) triple).  Multi-edges and self-loops are allowed.
 */
#ifndef GNN_ORACLE_H
#define GNN_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { OR_F32 = 0, OR_BF16 = 1, OR_F64 = 2 };
enum { OR_COPY_LHS = 0, OR_COPY_RHS = 1, OR_ADD = 2, OR_SUB = 3, OR_MUL = 4, OR_DIV = 5, OR_DOT = 6 };
enum { OR_SUM = 0, OR_MEAN = 1, OR_MAX = 2, OR_MIN = 3 };
enum { OR_SRC = 0, OR_EDGE = 1, OR_DST = 2 };

/* A (rows, heads, feat) tensor with a row stride in elements.  heads == 1 and
 * feat == 1 broadcast against the other operand. */
typedef struct {
    void* data;
    int32_t dtype;
    int32_t pad;
    int64_t rows;
    int64_t heads;
    int64_t feat;
    int64_t stride;
} or_tensor;

typedef struct {
    int64_t n_src, n_dst, n_edges;
    const int32_t* src;
    const int32_t* dst;
} or_graph;

/* All functions return 0 on success, a negative code on invalid arguments.
 * A selection (rows / edges / sel, with its count) restricts the work to the
 * listed output rows; output row k then holds the result for entry k (the
 * output tensor has n_sel rows), so full-size graphs can be checked on a
 * sample.  arg arrays are dense (out rows, heads, feat) int32. */

int oracle_degrees(const or_graph* g, int64_t* in_deg, int64_t* out_deg);
int oracle_csr(const or_graph* g, int reverse, int64_t* indptr, int32_t* indices, int32_t* eids);

int oracle_gspmm(const or_graph* g, int op, int reduce, const or_tensor* lhs, const or_tensor* rhs,
                 or_tensor* out, int32_t* arg_u, int32_t* arg_e, const int64_t* rows, int64_t n_rows);
int oracle_gsddmm(const or_graph* g, int op, const or_tensor* lhs, int lhs_target, const or_tensor* rhs,
                  int rhs_target, or_tensor* out, const int64_t* edges, int64_t n_sel);
int oracle_gspmm_backward(const or_graph* g, int op, int reduce, const or_tensor* lhs, const or_tensor* rhs,
                          const int32_t* arg_e, const or_tensor* grad_out, or_tensor* grad_lhs,
                          or_tensor* grad_rhs, const int64_t* sel, int64_t n_sel);
int oracle_gsddmm_backward(const or_graph* g, int op, const or_tensor* lhs, int lhs_target, const or_tensor* rhs,
                           int rhs_target, const or_tensor* grad_out, or_tensor* grad_lhs, or_tensor* grad_rhs,
                           const int64_t* sel, int64_t n_sel);
int oracle_edge_softmax(const or_graph* g, const or_tensor* score, or_tensor* out, const int64_t* rows,
                        int64_t n_rows, int64_t* out_eids);
int oracle_edge_softmax_backward(const or_graph* g, const or_tensor* out, const or_tensor* grad_out,
                                 or_tensor* grad_score, const int64_t* rows, int64_t n_rows, int64_t* out_eids);
int oracle_leaky_relu(const or_tensor* x, or_tensor* y, float slope);
int oracle_leaky_relu_backward(const or_tensor* x, const or_tensor* dy, or_tensor* dx, float slope);
void oracle_round_bf16(int64_t n, const float* in, uint16_t* out);

#ifdef __cplusplus
}
#endif
#endif
