// Internal declarations of the gnnk GPU library (host and device side).
//
// Geometry of a call.  A message row of D = H * F columns is split into
// vectors of VEC consecutive columns (VEC divides F, so a vector never spans
// two heads); NV = D / VEC vectors.  L = lanes per edge (power of two, at most
// 64, L >= NV unless the row is processed in chunks of 64 vectors), and a
// 64-lane wavefront holds G = 64 / L lane groups, each working on one edge at
// a time.
//
// Schedule of a row traversal (an in-CSR or the reverse graph's CSR).  Rows
// are kept sorted by descending degree (perm).  A call splits them into:
//   hub rows   degree > seg_edges: cut into segments of seg_edges edges, one
//              wavefront per segment, partial results combined afterwards in
//              segment order;
//   big rows   one wavefront per row, the G lane groups striding its edges;
//   small rows degree <= small_deg: each lane group owns one row;
//   empty rows degree 0: filled with the empty-reduction value.
// Every role sits in one launch; block b takes the roles of its wavefronts in
// that order, so the longest work items start first.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gnnk {

enum OperandTarget : int32_t { T_NBR = 0, T_EDGE = 1, T_SELF = 2 };

#ifndef GNNK_ENGINE_UNR
#define GNNK_ENGINE_UNR 4
#endif
constexpr int ENGINE_UNR = GNNK_ENGINE_UNR;  // edges in flight per lane group and batch

// message kinds (fused op of up to three operands a, b, c)
enum MsgOp : int32_t {
    M_COPY_A = 0,   // a
    M_ADD = 1,      // a + b
    M_SUB = 2,      // a - b
    M_MUL = 3,      // a * b
    M_DIV = 4,      // a / b
    M_NEGDIV2 = 5,  // -(a * b) / (c * c)   (gradient of a division w.r.t. its divisor)
    M_RSUB = 6,     // b - a
};

struct OperandDev {
    const void* data;   // nullptr when absent
    int64_t stride;     // row stride, elements
    int32_t hmul;       // element offset per head for a broadcast-over-feature operand (1 or 0)
    int32_t full;       // 1: operand has the message feature extent (per-lane vector load)
    int32_t target;     // OperandTarget
    int32_t pad;
};

struct OutDev {
    void* data;
    int64_t stride;
    int32_t reduce;     // 1: the output is summed over broadcast positions (operand of shape (H,1) or (1,1))
    int32_t red;        // lanes summed into one output element (after each lane sums its VEC columns)
    int32_t per_head;   // with reduce: 1 -> one value per head, 0 -> one value per row
    int32_t pad;
};

struct CsrDev {
    const void* ptr;        // row offsets (int32 or int64)
    const int32_t* idx;     // neighbour of each position
    const int32_t* eid;     // edge id of each position, nullptr = identity
    const int32_t* perm;    // rows by descending degree
    const int4* seg;        // {row, begin, end, hub index} per segment of a hub row
    // segment taken by hub-segment wavefront w: segments in the order of the
    // neighbour ids they cover, so that the segments of different rows that
    // run at the same time gather from one slice of the neighbour table
    const int32_t* seg_order;
    const int32_t* hub_off; // first segment of each hub row (hub rows = perm[0, n_hub)), n_hub + 1 entries
    const int32_t* row;     // row of each position (the COO form of the same CSR)
    const int4* segw;       // seg[seg_order[w]] with its table index: {row, begin, end, seg_order[w]}
    const int4* rowt;       // {perm[k], begin, end, 0}: the rows in degree order with their positions
    int32_t ptr64;
    int32_t pad;
};

struct SchedDev {
    int32_t n_seg;          // waves of segments
    int32_t n_hub;          // hub rows (perm[0, n_hub))
    int32_t n_big;          // rows with one wavefront each end at perm[n_big)
    int32_t n_nz;           // non-empty rows end at perm[n_nz)
    int32_t n_rows;
    int32_t w_big_end;      // wave index where big rows end
    int32_t w_small_end;    // wave index where small rows end
    int32_t w_total;        // total waves
    int32_t fill_rows_per_group;
    int32_t seg_split;      // g-SDDMM: wavefronts per hub segment (0 or 1: one); n_seg counts segments
};

struct GeomDev {
    int32_t F;       // feature extent of the message (canonical)
    int32_t NV;      // vectors per message row
    int32_t L;       // lanes per edge
    int32_t log2L;
    int32_t G;       // lane groups per wavefront
    int32_t nchunk;  // chunks of 64 vectors (NV > 64)
};

// flags of a row-engine call
enum : int32_t {
    F_MASK_A = 1,       // a is zeroed unless arg[row of a][col] == edge id
    F_SCALE_A_DEG = 2,  // a is divided by the degree of a's row (mean backward)
    F_OWN_MEAN = 4,     // the reduced value is divided by the row's own degree
    F_NEGATE = 8,       // the output is negated
    F_IS_MIN = 16,      // max/min reductions: minimum
    F_BITS_A = 32,      // a is zeroed unless its column's bit is set in the winner mask of the position
};

// EXT: extra treatment of operand a in backward passes
enum : int {
    EXT_NONE = 0,
    EXT_SCALE = 1,  // a / deg(row of a)
    EXT_MASK = 2,   // a where arg[row of a][col] == edge id
    EXT_BITS = 3,   // a where bit col of the winner mask at this CSR position is set
};

inline int ext_of(int32_t flags) {
    if (flags & F_BITS_A) return EXT_BITS;
    return (flags & F_MASK_A) ? EXT_MASK : ((flags & F_SCALE_A_DEG) ? EXT_SCALE : EXT_NONE);
}

struct EngineArgs {
    CsrDev csr;
    SchedDev sch;
    GeomDev geo;
    OperandDev a, b, c;
    OutDev out;
    int32_t* arg_nbr;        // max/min: neighbour id of the winner (nullable)
    int32_t* arg_edge;       // max/min: edge id of the winner (nullable)
    const int32_t* mask_arg; // F_MASK_A: edge-id array (rows of a's target, D columns);
                             // F_BITS_A: winner bits, mask_ld 32-bit words per CSR position
    const int32_t* deg;      // F_SCALE_A_DEG: degree per row of a's target
    void* partial;           // hub-row partials (fp64 sums, or fp32 value + int32 edge + int32 nbr)
    int64_t partial_stride;  // elements per segment row (D)
    int32_t op;              // MsgOp
    int32_t flags;
    int64_t mask_ld;         // row stride of mask_arg
    int32_t log2hb;          // coalesced b: log2 of the values per edge (heads, or 1 per row)
    int32_t sub_edges;       // edge-parallel walks: positions per lane group (a sub-chunk)
    int32_t n_sub;           // edge-parallel walks: number of sub-chunks
    int32_t pad2;
    // fused edge gradient of a reverse-graph g-SpMM (u_mul_e/sum backward):
    // out2[edge] = sum over runs of red2 lanes of a . x2[row], per head or per row
    const void* x2;          // the walked row's own operand (lhs of the forward), full rows
    int64_t x2_stride;
    void* out2;              // per-edge output (grad of the edge weight)
    int64_t out2_stride;
    int32_t red2;            // lanes summed per output value (a power of two)
    int32_t per_head2;       // 1: one value per head, 0: one per edge
    // g-SDDMM whose per-edge sum over the whole row spans several passes of
    // the wavefront (nchunk > 1): fp64 running sum per edge between passes
    double* xacc;
};

// Operand layouts with kernels specialised at compile time (the host picks
// one when a call matches it and the lane-group count is 1, 2 or 4; SP_DYN
// reads every layout from the descriptors).
enum SpecId : int32_t {
    SP_DYN = 0,
    SP_CU = 1,       // a: neighbour row, full                 (copy_u, and dZ in node gradients)
    SP_UE_H = 2,     // a: neighbour row; b: edge, one per head (u_mul_e with attention weights)
    SP_UE_H_CB = 3,  //   the same, b read coalesced (identity edge ids)
    SP_UE_R = 4,     // a: neighbour row; b: edge, one per row  (u_mul_e with a scalar edge weight)
    SP_UE_R_CB = 5,  //   the same, b read coalesced
    SP_UV = 6,       // a: neighbour row; b: own row            (g-SDDMM u_op_v)
    SP_VU = 7,       // a: own row; b: neighbour row            (edge gradient dZ[v] . X[u])
};

// ----- host-side launchers (spmm.hip, sddmm.hip, edge.hip, gat.hip, softmax.hip, misc.hip) -----
// dtype: 0 fp32, 1 bf16; opk: 0 copy-a, 1 mul-ab, 2 generic; gc: lane groups
// of a fast spec
bool fast_vec(int dtype, int vec);
hipError_t launch_spmm(const EngineArgs& a, int dtype, int vec, bool maxmin, int opk, int spec, int gc,
                       hipStream_t s);
// u_mul_e/sum backward in one reverse pass: dX as launch_spmm with spec
// SP_UE_H or SP_UE_R (gc 1, 2 or 4), and the edge gradient into a.out2
hipError_t launch_spmm_dw(const EngineArgs& a, int dtype, int vec, int spec, int gc, hipStream_t s);
hipError_t launch_spmm_combine(const EngineArgs& a, int dtype, int vec, bool maxmin, hipStream_t s);
// edge-parallel (COO) walks, edge.hip: mode 0 = partials of split rows combined
// in order afterwards, mode 1 = fp64 atomics into scratch (a.partial, rows x D)
hipError_t launch_spmm_edge(const EngineArgs& a, int64_t n_pos, int64_t n_rows, int dtype, int vec, int opk, int spec,
                            int gc, int mode, hipStream_t s);
hipError_t launch_sddmm_edge(const EngineArgs& a, int64_t n_pos, int dtype, int vec, int opk, int spec, int gc,
                             hipStream_t s);
// fused attention, gat.hip (a: feat at the neighbour, b: el at the neighbour;
// row_ml: n_hub x 2 x D doubles when attn is written)
hipError_t launch_gat(const EngineArgs& a, const void* er, int64_t er_stride, void* attn, int64_t attn_stride,
                      float slope, void* row_ml, float* stats, int64_t stats_stride, int dtype, int vec, int gc,
                      hipStream_t s);
// backward of the fused attention, gat.hip: pass A walks the in-CSR (ain: a =
// feat, b = el at the neighbour), pass B the reverse graph's CSR (aout)
struct GatBwdArgs {
    const void* er;          // (N_dst, H) T
    int64_t er_stride;
    const float* stats;      // (N_dst, H, 2) fp32 from the forward
    int64_t stats_stride;
    const void* dz;          // (N_dst, H, F) T
    int64_t dz_stride;
    void* d_er;              // (N_dst, H) T, nullable
    int64_t d_er_stride;
    void* d_el;              // (N_src, H) T, nullable
    int64_t d_el_stride;
    void* d_feat;            // (N_src, H, F) T, nullable
    int64_t d_feat_stride;
    const void* el;          // (N_src, H) T
    int64_t el_stride;
    const void* feat;        // (N_src, H, F) T
    int64_t feat_stride;
    float4* rec;             // (N_dst, H): er, max, 1 / sum, S
    double* part;            // hub segments: pass A 3 x H, pass B D + H doubles per segment
    float slope;
    int32_t H;
    // A head wider than one pass of the wavefront runs in column chunks: the
    // sums S and P of pass A and d_el of pass B are linear in the per-chunk
    // dot products, so each chunk adds its share into fp64 accumulators and
    // the last chunk finishes.  chunk: 0 a whole head; 1 the first chunk
    // (stores), 2 a middle one (adds), 3 the last (adds and writes).
    int32_t chunk;
    int32_t passes;          // 1: pass A only, 2: pass B only, 3: both
    double* acc_dst;         // (N_dst, H) x {S, P} of the chunks so far
    double* acc_src;         // (N_src, H): d_el of the chunks so far
};
hipError_t launch_gat_backward(const EngineArgs& ain, const EngineArgs& aout, const GatBwdArgs& b, int dtype, int vec,
                               int gc, hipStream_t s);
hipError_t launch_fill_rows(const void* ptr, int ptr64, int64_t n_rows, int64_t n_edges, int32_t* row,
                            hipStream_t s);
hipError_t launch_sddmm(const EngineArgs& a, int dtype, int vec, int opk, int spec, int gc, hipStream_t s);
hipError_t launch_softmax(const EngineArgs& a, int dtype, int vec, bool backward, hipStream_t s);
hipError_t launch_leaky(const void* x, const void* dy, void* y, int64_t rows, int32_t cols, int64_t sx,
                        int64_t sdy, int64_t sy, float slope, int dtype, bool backward, hipStream_t s);
hipError_t launch_validate(const int32_t* idx, int64_t n, int64_t bound, int32_t* flag, hipStream_t s);
hipError_t launch_validate_ptr(const void* ptr, int ptr64, int64_t n_rows, int64_t n_edges, int32_t* flag,
                               hipStream_t s);
hipError_t launch_iota(int32_t* out, int64_t n, hipStream_t s);
// pos[perm[q]] = q for q < n
hipError_t launch_inverse(const int32_t* perm, int64_t n, int32_t* pos, hipStream_t s);
// Winner masks of max/min: bits[pos_of_edge[e] * words + c / 32] has bit c % 32
// set iff arg_e[v * ld + c] == e for some row v and column c < D (zeroed first).
hipError_t launch_winner_bits(const int32_t* arg_e, int64_t n_rows, int32_t D, int64_t ld,
                              const int32_t* pos_of_edge, uint32_t* bits, int64_t n_edges, int32_t words,
                              hipStream_t s);
// The same masks built row by row (winner_rows_kernel) for a graph with
// identity edge ids: units are the n_seg hub segments of the in-CSR, then its
// rows perm[n_hub .. n_hub + n_small).  An arg names an edge of its own row
// or nothing.
struct WinnerRowsArgs {
    const int32_t* arg;   // (n_dst rows, ld) winning edge ids
    int64_t ld;
    int32_t D, words;
    const void* ptr;      // in-CSR row offsets (int32 or int64)
    const int32_t* perm;  // rows by descending degree
    const int4* seg;      // hub segments (row, begin, end, k)
    int64_t n_seg, n_hub, n_small;
    const int32_t* pos;   // reverse-CSR position of each edge id
    uint32_t* bits;       // n_edges * words, zeroed here first
};
hipError_t launch_winner_rows(const WinnerRowsArgs& a, int ptr64, int64_t n_edges, hipStream_t s);
hipError_t launch_copy_ptr(const void* src, int src64, void* dst, int dst64, int64_t n, hipStream_t s);

// ----- device construction of the graph formats (build.hip) -----
// key[k] = idx[seg[k].begin] / 2 + idx[seg[k].end - 1] / 2 for k < n_seg
hipError_t launch_seg_keys(const int4* seg, int64_t n_seg, const int32_t* idx, uint32_t* key, hipStream_t s);
hipError_t launch_seg_wave(const int4* seg, const int32_t* order, int64_t n_seg, int4* segw, hipStream_t s);
hipError_t launch_row_table(const void* ptr, int ptr64, const int32_t* perm, int64_t n_rows, int4* rowt,
                            hipStream_t s);
// bits needed for keys in [0, max_key]
int key_bits(uint64_t max_key);
// uint32 words of scratch radix_sort_pairs needs for n pairs
size_t radix_scratch_words(int64_t n);
// Stable sort of (key, value) pairs by the low `bits` bits of the key; vals_in
// == nullptr stands for 0..n-1.  Inputs are only read; the result lands in
// keys_out/vals_out; tmp_keys/tmp_vals (n entries each) and scratch are
// clobbered.  No buffer may alias another.
hipError_t radix_sort_pairs(const uint32_t* keys_in, const uint32_t* vals_in, int64_t n, int bits,
                            uint32_t* keys_out, uint32_t* vals_out, uint32_t* tmp_keys, uint32_t* tmp_vals,
                            uint32_t* scratch, hipStream_t s);
// ptr[r] = first position of the sorted keys that is >= r, r in [0, n_rows]
hipError_t launch_ptr_from_keys(const uint32_t* keys, int64_t n_keys, int64_t n_rows, void* ptr, int ptr64,
                                hipStream_t s);
// deg[r] = ptr[r + 1] - ptr[r]; deg_key[r] = cap - deg[r]
hipError_t launch_degrees(const void* ptr, int ptr64, int64_t n_rows, int32_t* deg, uint32_t* deg_key, uint32_t cap,
                          hipStream_t s);
// out[p] = table[idx[p]]
hipError_t launch_gather(const int32_t* table, const uint32_t* idx, int64_t n, int32_t* out, hipStream_t s);
// flag |= bit unless eid[p] == p for every p
hipError_t launch_check_identity(const int32_t* eid, int64_t n, int32_t* flag, int32_t bit, hipStream_t s);
// flag |= bit unless eid is a permutation of 0..n-1 (counts: n words of scratch)
hipError_t launch_check_permutation(const int32_t* eid, int64_t n, uint32_t* counts, int32_t* flag, int32_t bit,
                                    hipStream_t s);
// src_of_e[eid[p]] = idx[p], dst_of_e[eid[p]] = row[p]
hipError_t launch_edge_ends(const int32_t* idx, const int32_t* eid, const int32_t* row, int64_t n, int32_t* src_of_e,
                            int32_t* dst_of_e, hipStream_t s);
// segments of the hub rows perm[0, n_hub), starting at seg[hub_off[k]]
hipError_t launch_hub_segments(const void* ptr, int ptr64, const int32_t* perm, const int32_t* hub_off, int64_t n_hub,
                               int64_t seg_edges, int4* seg, hipStream_t s);

}  // namespace gnnk
