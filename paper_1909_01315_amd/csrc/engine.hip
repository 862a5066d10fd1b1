// Row-engine kernels of the gnnk library (gfx950, wave64).
//
// g-SpMM reduces over the edges of a CSR row (Section 3, definition of
// generalized SpMM): the in-CSR for the forward pass, the reverse graph's CSR
// for node gradients (Theorem 1).  g-SDDMM writes one output per edge
// (definition of generalized SDDMM) and walks the in-CSR row by row, so the
// destination-side operand is read once per destination.  Edge softmax and
// its backward reduce per destination and then write per edge.
//
// All three share one schedule (see internal.h): hub rows cut into segments,
// a wavefront per big row, a lane group per small row, empty rows filled, all
// in one launch ordered from the longest work item to the shortest.  A lane
// holds VEC consecutive columns of the message row and loads them with one
// vector load; the G lane groups of a wavefront stride the edges of a row and
// are combined in a fixed order (xor shuffles), so results are deterministic.
// Sums accumulate in fp64; max/min compare fp32 messages exactly and break
// ties toward the smaller edge id.  No atomics.
#include "internal.h"

namespace gnnk {

constexpr int WAVE = 64;
constexpr int WPB = 4;  // wavefronts per block
constexpr int UNR = 4;  // edges in flight per lane group

typedef uint16_t bf16_t;

__device__ __forceinline__ int64_t row_ptr(const CsrDev& c, int64_t r) {
    return c.ptr64 ? reinterpret_cast<const int64_t*>(c.ptr)[r] : (int64_t) reinterpret_cast<const int32_t*>(c.ptr)[r];
}

// ---------------------------------------------------------------------------
// element IO: VEC consecutive elements <-> float registers

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t f2bf(float f) {
    uint32_t b = __float_as_uint(f);
    b += 0x7FFFu + ((b >> 16) & 1u);  // round to nearest, ties to even (finite inputs)
    return b >> 16;
}

template <typename T, int VEC>
struct IO;

template <int VEC>
struct IO<float, VEC> {
    static __device__ __forceinline__ void load(const float* p, float* v) {
        if constexpr (VEC == 4) {
            float4 x = *reinterpret_cast<const float4*>(p);
            v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        } else if constexpr (VEC == 2) {
            float2 x = *reinterpret_cast<const float2*>(p);
            v[0] = x.x; v[1] = x.y;
        } else {
            v[0] = *p;
        }
    }
    static __device__ __forceinline__ float load1(const float* p) { return *p; }
    static __device__ __forceinline__ void store(float* p, const float* v) {
        if constexpr (VEC == 4) {
            *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
        } else if constexpr (VEC == 2) {
            *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
        } else {
            *p = v[0];
        }
    }
    static __device__ __forceinline__ void store1(float* p, float v) { *p = v; }
};

template <int VEC>
struct IO<bf16_t, VEC> {
    static __device__ __forceinline__ void load(const bf16_t* p, float* v) {
        if constexpr (VEC == 8) {
            uint4 x = *reinterpret_cast<const uint4*>(p);
            v[0] = bf_lo(x.x); v[1] = bf_hi(x.x); v[2] = bf_lo(x.y); v[3] = bf_hi(x.y);
            v[4] = bf_lo(x.z); v[5] = bf_hi(x.z); v[6] = bf_lo(x.w); v[7] = bf_hi(x.w);
        } else if constexpr (VEC == 4) {
            uint2 x = *reinterpret_cast<const uint2*>(p);
            v[0] = bf_lo(x.x); v[1] = bf_hi(x.x); v[2] = bf_lo(x.y); v[3] = bf_hi(x.y);
        } else if constexpr (VEC == 2) {
            uint32_t x = *reinterpret_cast<const uint32_t*>(p);
            v[0] = bf_lo(x); v[1] = bf_hi(x);
        } else {
            v[0] = bf_lo(*p);
        }
    }
    static __device__ __forceinline__ float load1(const bf16_t* p) { return bf_lo(*p); }
    static __device__ __forceinline__ void store(bf16_t* p, const float* v) {
        if constexpr (VEC == 8) {
            uint4 x;
            x.x = f2bf(v[0]) | (f2bf(v[1]) << 16); x.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
            x.z = f2bf(v[4]) | (f2bf(v[5]) << 16); x.w = f2bf(v[6]) | (f2bf(v[7]) << 16);
            *reinterpret_cast<uint4*>(p) = x;
        } else if constexpr (VEC == 4) {
            uint2 x;
            x.x = f2bf(v[0]) | (f2bf(v[1]) << 16); x.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
            *reinterpret_cast<uint2*>(p) = x;
        } else if constexpr (VEC == 2) {
            *reinterpret_cast<uint32_t*>(p) = f2bf(v[0]) | (f2bf(v[1]) << 16);
        } else {
            *p = (bf16_t)f2bf(v[0]);
        }
    }
    static __device__ __forceinline__ void store1(bf16_t* p, float v) { *p = (bf16_t)f2bf(v); }
};

template <int VEC>
__device__ __forceinline__ void load_i32(const int32_t* p, int32_t* v) {
    if constexpr (VEC >= 4 && VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            int4 x = reinterpret_cast<const int4*>(p)[q];
            v[4 * q] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
        }
    } else if constexpr (VEC == 2) {
        int2 x = *reinterpret_cast<const int2*>(p);
        v[0] = x.x; v[1] = x.y;
    } else {
        v[0] = *p;
    }
}

template <int VEC>
__device__ __forceinline__ void store_i32(int32_t* p, const int32_t* v) {
    if constexpr (VEC >= 4 && VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q)
            reinterpret_cast<int4*>(p)[q] = make_int4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    } else if constexpr (VEC == 2) {
        *reinterpret_cast<int2*>(p) = make_int2(v[0], v[1]);
    } else {
        *p = v[0];
    }
}

// ---------------------------------------------------------------------------
// cross-lane helpers (64-bit values move as two 32-bit shuffles)

__device__ __forceinline__ double shfl_xor_d(double x, int m) {
    int2 v = *reinterpret_cast<int2*>(&x);
    v.x = __shfl_xor(v.x, m, WAVE);
    v.y = __shfl_xor(v.y, m, WAVE);
    return *reinterpret_cast<double*>(&v);
}

__device__ __forceinline__ double shfl_d(double x, int src) {
    int2 v = *reinterpret_cast<int2*>(&x);
    v.x = __shfl(v.x, src, WAVE);
    v.y = __shfl(v.y, src, WAVE);
    return *reinterpret_cast<double*>(&v);
}

// Sum over aligned runs of `red` consecutive lanes starting at multiples of
// `red` within each lane group of L lanes; the first lane of a run gets the
// total (other lanes hold partial sums).  All lanes must call it.
__device__ __forceinline__ double seg_sum(double v, int lane_in_group, int red) {
    int pos = lane_in_group % red;
    int lane = __lane_id();
    for (int s = 1; s < red; s <<= 1) {
        double o = shfl_d(v, lane + s < WAVE ? lane + s : lane);
        if ((pos & (2 * s - 1)) == 0 && pos + s < red) v += o;
    }
    return v;
}

// ---------------------------------------------------------------------------
// operands

__device__ __forceinline__ int64_t row_of(int32_t target, int64_t nb, int64_t ed, int64_t self) {
    return target == T_NBR ? nb : (target == T_EDGE ? ed : self);
}

template <typename T, int VEC>
__device__ __forceinline__ void load_operand(const OperandDev& o, int64_t row, int col0, int h, float* v) {
    const T* base = reinterpret_cast<const T*>(o.data) + row * o.stride;
    if (o.full) {
        IO<T, VEC>::load(base + col0, v);
    } else {
        float x = IO<T, VEC>::load1(base + h * o.hmul);
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = x;
    }
}

// message of one edge for this lane's VEC columns, in fp64 (sums, SDDMM)
template <typename T, int VEC, int OPK>
__device__ __forceinline__ void message_f64(const EngineArgs& A, int64_t nb, int64_t ed, int64_t self, int col0,
                                            int h, double* m) {
    float a[VEC];
    const int64_t ar = row_of(A.a.target, nb, ed, self);
    load_operand<T, VEC>(A.a, ar, col0, h, a);
    double ad[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) ad[i] = a[i];
    if (A.flags & F_SCALE_A_DEG) {
        double d = (double)A.deg[ar];
#pragma unroll
        for (int i = 0; i < VEC; ++i) ad[i] = ad[i] / d;
    }
    if (A.flags & F_MASK_A) {
        int32_t k[VEC];
        load_i32<VEC>(A.mask_arg + ar * A.mask_ld + col0, k);
#pragma unroll
        for (int i = 0; i < VEC; ++i) ad[i] = (k[i] == (int32_t)ed) ? ad[i] : 0.0;
    }
    if constexpr (OPK == 0) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) m[i] = ad[i];
    } else {
        float b[VEC];
        load_operand<T, VEC>(A.b, row_of(A.b.target, nb, ed, self), col0, h, b);
        if constexpr (OPK == 1) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) m[i] = ad[i] * (double)b[i];
        } else {
            switch (A.op) {
                case M_COPY_A:
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = ad[i];
                    break;
                case M_ADD:
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = ad[i] + (double)b[i];
                    break;
                case M_SUB:
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = ad[i] - (double)b[i];
                    break;
                case M_RSUB:
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = (double)b[i] - ad[i];
                    break;
                case M_MUL:
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = ad[i] * (double)b[i];
                    break;
                case M_DIV:
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = ad[i] / (double)b[i];
                    break;
                default: {  // M_NEGDIV2
                    float c[VEC];
                    load_operand<T, VEC>(A.c, row_of(A.c.target, nb, ed, self), col0, h, c);
#pragma unroll
                    for (int i = 0; i < VEC; ++i) m[i] = -ad[i] * (double)b[i] / ((double)c[i] * (double)c[i]);
                }
            }
        }
    }
}

// message for max/min: one fp32 operation, as a message tensor would hold it
template <typename T, int VEC, int OPK>
__device__ __forceinline__ void message_f32(const EngineArgs& A, int64_t nb, int64_t ed, int64_t self, int col0,
                                            int h, float* m) {
    float a[VEC];
    load_operand<T, VEC>(A.a, row_of(A.a.target, nb, ed, self), col0, h, a);
    if constexpr (OPK == 0) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) m[i] = a[i];
    } else {
        float b[VEC];
        load_operand<T, VEC>(A.b, row_of(A.b.target, nb, ed, self), col0, h, b);
        int op = OPK == 1 ? (int)M_MUL : A.op;
        switch (op) {
            case M_ADD:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = a[i] + b[i];
                break;
            case M_SUB:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = a[i] - b[i];
                break;
            case M_MUL:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = a[i] * b[i];
                break;
            case M_DIV:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = a[i] / b[i];
                break;
            default:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = a[i];
        }
    }
}

// ---------------------------------------------------------------------------
// output of one reduced row (sums)

template <typename T, int VEC>
__device__ __forceinline__ void write_sum_row(const EngineArgs& A, int64_t row, bool active, int lig, int col0,
                                              int h, double* acc, int64_t deg, bool write_lane) {
    if (A.flags & F_OWN_MEAN) {
        double d = deg > 0 ? (double)deg : 1.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = acc[i] / d;
    }
    if (A.flags & F_NEGATE) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = -acc[i];
    }
    if (!A.out.reduce) {
        if (active && write_lane && row >= 0) {
            float v[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = (float)acc[i];
            IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + row * A.out.stride + col0, v);
        }
    } else {
        double s = 0.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) s += acc[i];
        s = seg_sum(active ? s : 0.0, lig, A.out.red);
        if (active && write_lane && row >= 0 && (lig % A.out.red) == 0) {
            int64_t o = A.out.per_head ? h : 0;
            IO<T, VEC>::store1(reinterpret_cast<T*>(A.out.data) + row * A.out.stride + o, (float)s);
        }
    }
}

// ---------------------------------------------------------------------------
// edge batches.  The loops below have no divergent branches: slots past the
// row end read the row's first position instead (always in bounds) and their
// results are discarded with selects, inactive lanes read column 0.

__device__ __forceinline__ void batch_ids(const CsrDev& C, int64_t b, int64_t e, int64_t p0, int64_t stride,
                                          bool* ok, int64_t* nb, int64_t* ed) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        const int64_t p = p0 + (int64_t)u * stride;
        ok[u] = p < e;
        const int64_t pc = ok[u] ? p : b;
        nb[u] = C.idx[pc];
        ed[u] = C.eid ? (int64_t)C.eid[pc] : pc;
    }
}

// ---------------------------------------------------------------------------
// g-SpMM, sums

template <typename T, int VEC, int OPK>
__device__ __forceinline__ void spmm_sum_edges(const EngineArgs& A, int64_t self, int64_t b, int64_t e, int start,
                                               int stride, int col0, int h, double* acc) {
    for (int64_t p0 = b + start; p0 < e; p0 += (int64_t)stride * UNR) {
        int64_t nb[UNR], ed[UNR];
        bool ok[UNR];
        batch_ids(A.csr, b, e, p0, stride, ok, nb, ed);
        double m[UNR][VEC];
#pragma unroll
        for (int u = 0; u < UNR; ++u) message_f64<T, VEC, OPK>(A, nb[u], ed[u], self, col0, h, m[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u)
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] += ok[u] ? m[u][i] : 0.0;
    }
}

template <typename T, int VEC, int OPK>
__global__ __launch_bounds__(256) void spmm_sum_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    const int64_t D = (int64_t)geo.NV * VEC;

    if (w < A.sch.w_big_end) {
        // one wavefront: a segment of a hub row, or a whole big row
        int64_t r, b, e;
        int slot = -1;
        if (w < A.sch.n_seg) {
            int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z; slot = w;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            double acc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
            spmm_sum_edges<T, VEC, OPK>(A, r, b, e, g, geo.G, col0, h, acc);
            for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += shfl_xor_d(acc[i], s);
            if (slot >= 0) {
                if (g == 0 && active) {
                    double* P = reinterpret_cast<double*>(A.partial) + (int64_t)slot * A.partial_stride + col0;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) P[i] = acc[i];
                }
            } else {
                write_sum_row<T, VEC>(A, r, active, lig, col0, h, acc, e - b, g == 0);
            }
        }
    } else if (w < A.sch.w_small_end) {
        // small rows: each lane group owns one row
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            double acc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
            spmm_sum_edges<T, VEC, OPK>(A, r >= 0 ? r : 0, b, e, 0, 1, col0, h, acc);
            write_sum_row<T, VEC>(A, r, active, lig, col0, h, acc, e - b, true);
        }
    } else {
        // empty rows: the empty reduction is 0
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * geo.G + g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * geo.L + lig;
                const bool active = j < geo.NV;
                const int col0 = j * VEC;
                const int h = col0 / geo.F;
                double acc[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
                // no negation or mean for the empty reduction
                if (!A.out.reduce) {
                    if (active && r >= 0) {
                        float v[VEC];
#pragma unroll
                        for (int i = 0; i < VEC; ++i) v[i] = 0.0f;
                        IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + col0, v);
                    }
                } else if (active && r >= 0 && (lig % A.out.red) == 0) {
                    int64_t o = A.out.per_head ? h : 0;
                    IO<T, VEC>::store1(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + o, 0.0f);
                }
            }
        }
    }
    (void)D;
}

// combine the segment partials of hub rows, in segment order
template <typename T, int VEC>
__global__ __launch_bounds__(256) void spmm_sum_combine_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    const int64_t k = (int64_t)w * geo.G + g;
    if ((int64_t)w * geo.G >= A.sch.n_hub) return;  // wave-uniform
    const bool row_ok = k < A.sch.n_hub;
    const int64_t r = row_ok ? A.csr.perm[k] : -1;
    const int s0 = row_ok ? A.csr.hub_off[k] : 0;
    const int s1 = row_ok ? A.csr.hub_off[k + 1] : 0;
    const int64_t deg = row_ok ? row_ptr(A.csr, r + 1) - row_ptr(A.csr, r) : 0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + lig;
        const bool active = j < geo.NV && row_ok;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        double acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
        for (int s = s0; s < s1; ++s) {
            const double* P = reinterpret_cast<const double*>(A.partial) + (int64_t)s * A.partial_stride + col0;
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] += P[i];
        }
        write_sum_row<T, VEC>(A, r, active, lig, col0, h, acc, deg, true);
    }
}

// ---------------------------------------------------------------------------
// g-SpMM, max / min with the winning edge and neighbour

// candidate (m, e) replaces (best, be): strictly better, or equal with a
// smaller edge id, or nothing recorded yet.  Bitwise operators keep it
// branch-free.
__device__ __forceinline__ bool better(float m, int32_t e, float best, int32_t be, bool is_min) {
    const bool strict = is_min ? (m < best) : (m > best);
    const bool tie = (m == best) & (e < be);
    return (be < 0) | strict | tie;
}

template <typename T, int VEC, int OPK>
__device__ __forceinline__ void spmm_cmp_edges(const EngineArgs& A, int64_t self, int64_t b, int64_t e, int start,
                                               int stride, int col0, int h, float* best, int32_t* be,
                                               int32_t* bn) {
    const bool is_min = (A.flags & F_IS_MIN) != 0;
    for (int64_t p0 = b + start; p0 < e; p0 += (int64_t)stride * UNR) {
        int64_t nb[UNR], ed[UNR];
        bool ok[UNR];
        batch_ids(A.csr, b, e, p0, stride, ok, nb, ed);
        float m[UNR][VEC];
#pragma unroll
        for (int u = 0; u < UNR; ++u) message_f32<T, VEC, OPK>(A, nb[u], ed[u], self, col0, h, m[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                const bool upd = ok[u] & better(m[u][i], (int32_t)ed[u], best[i], be[i], is_min);
                best[i] = upd ? m[u][i] : best[i];
                be[i] = upd ? (int32_t)ed[u] : be[i];
                bn[i] = upd ? (int32_t)nb[u] : bn[i];
            }
        }
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void write_cmp_row(const EngineArgs& A, int64_t row, bool active, int col0,
                                              const float* best, const int32_t* be, const int32_t* bn) {
    if (!active || row < 0) return;
    float v[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) v[i] = be[i] < 0 ? 0.0f : best[i];
    IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + row * A.out.stride + col0, v);
    const int64_t D = (int64_t)A.geo.NV * VEC;
    if (A.arg_edge) store_i32<VEC>(A.arg_edge + row * D + col0, be);
    if (A.arg_nbr) store_i32<VEC>(A.arg_nbr + row * D + col0, bn);
}

template <typename T, int VEC, int OPK>
__global__ __launch_bounds__(256) void spmm_cmp_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    const int64_t D = (int64_t)geo.NV * VEC;
    const bool is_min = (A.flags & F_IS_MIN) != 0;

    if (w < A.sch.w_big_end) {
        int64_t r, b, e;
        int slot = -1;
        if (w < A.sch.n_seg) {
            int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z; slot = w;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            float best[VEC];
            int32_t be[VEC], bn[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
            spmm_cmp_edges<T, VEC, OPK>(A, r, b, e, g, geo.G, col0, h, best, be, bn);
            for (int s = geo.L; s < WAVE; s <<= 1) {
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    const float ob = __shfl_xor(best[i], s, WAVE);
                    const int32_t oe = __shfl_xor(be[i], s, WAVE);
                    const int32_t on = __shfl_xor(bn[i], s, WAVE);
                    const bool upd = (oe >= 0) & better(ob, oe, best[i], be[i], is_min);
                    best[i] = upd ? ob : best[i];
                    be[i] = upd ? oe : be[i];
                    bn[i] = upd ? on : bn[i];
                }
            }
            if (slot >= 0) {
                if (g == 0 && active) {
                    float* PV = reinterpret_cast<float*>(A.partial) + (int64_t)slot * D + col0;
                    int32_t* PE = reinterpret_cast<int32_t*>(A.partial) + (int64_t)A.sch.n_seg * D +
                                  (int64_t)slot * D + col0;
                    int32_t* PN = PE + (int64_t)A.sch.n_seg * D;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) { PV[i] = best[i]; PE[i] = be[i]; PN[i] = bn[i]; }
                }
            } else if (g == 0) {
                write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn);
            }
        }
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            float best[VEC];
            int32_t be[VEC], bn[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
            spmm_cmp_edges<T, VEC, OPK>(A, r >= 0 ? r : 0, b, e, 0, 1, col0, h, best, be, bn);
            write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn);
        }
    } else {
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * geo.G + g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * geo.L + lig;
                const bool active = j < geo.NV;
                float best[VEC];
                int32_t be[VEC], bn[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
                write_cmp_row<T, VEC>(A, r, active, j * VEC, best, be, bn);
            }
        }
    }
}

template <typename T, int VEC>
__global__ __launch_bounds__(256) void spmm_cmp_combine_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    const int64_t k = (int64_t)w * geo.G + g;
    if ((int64_t)w * geo.G >= A.sch.n_hub) return;
    const bool row_ok = k < A.sch.n_hub;
    const int64_t r = row_ok ? A.csr.perm[k] : -1;
    const int s0 = row_ok ? A.csr.hub_off[k] : 0;
    const int s1 = row_ok ? A.csr.hub_off[k + 1] : 0;
    const int64_t D = (int64_t)geo.NV * VEC;
    const bool is_min = (A.flags & F_IS_MIN) != 0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + lig;
        const bool active = j < geo.NV && row_ok;
        const int col0 = active ? j * VEC : 0;
        float best[VEC];
        int32_t be[VEC], bn[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
        for (int s = s0; s < s1; ++s) {
            const float* PV = reinterpret_cast<const float*>(A.partial) + (int64_t)s * D + col0;
            const int32_t* PE = reinterpret_cast<const int32_t*>(A.partial) + (int64_t)A.sch.n_seg * D +
                                (int64_t)s * D + col0;
            const int32_t* PN = PE + (int64_t)A.sch.n_seg * D;
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                const float pv = PV[i];
                const int32_t pe = PE[i], pn = PN[i];
                const bool upd = (pe >= 0) & better(pv, pe, best[i], be[i], is_min);
                best[i] = upd ? pv : best[i];
                be[i] = upd ? pe : be[i];
                bn[i] = upd ? pn : bn[i];
            }
        }
        write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn);
    }
}

// ---------------------------------------------------------------------------
// g-SDDMM: per-edge outputs, rows of the in-CSR (or the reverse CSR)

template <typename T, int VEC, int OPK>
__device__ __forceinline__ void sddmm_edges(const EngineArgs& A, int64_t self, int64_t b, int64_t e, int64_t n_iter,
                                            int start, int stride, int lig, int col0, int h, bool active) {
    const CsrDev& C = A.csr;
    // n_iter is uniform over the wavefront so the lane reductions line up
    for (int64_t it = 0; it < n_iter; it += UNR) {
        int64_t nb[UNR], ed[UNR];
        bool ok[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t p = b + start + (it + u) * (int64_t)stride;
            ok[u] = ((it + u) < n_iter) & (p < e);
            const int64_t pc = ok[u] ? p : b;
            nb[u] = C.idx[pc];
            ed[u] = C.eid ? (int64_t)C.eid[pc] : pc;
        }
        double m[UNR][VEC];
#pragma unroll
        for (int u = 0; u < UNR; ++u) message_f64<T, VEC, OPK>(A, nb[u], ed[u], self, col0, h, m[u]);
        if (!A.out.reduce) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                if (ok[u] & active) {
                    float v[VEC];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) v[i] = (float)((A.flags & F_NEGATE) ? -m[u][i] : m[u][i]);
                    IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + ed[u] * A.out.stride + col0, v);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                double s = 0.0;
#pragma unroll
                for (int i = 0; i < VEC; ++i) s += m[u][i];
                s = seg_sum(active ? s : 0.0, lig, A.out.red);
                if (ok[u] & active & ((lig % A.out.red) == 0)) {
                    if (A.flags & F_NEGATE) s = -s;
                    const int64_t o = A.out.per_head ? h : 0;
                    IO<T, VEC>::store1(reinterpret_cast<T*>(A.out.data) + ed[u] * A.out.stride + o, (float)s);
                }
            }
        }
    }
}

template <typename T, int VEC, int OPK>
__global__ __launch_bounds__(256) void sddmm_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    if (w >= A.sch.w_small_end) return;
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    int64_t r, b, e, n_iter;
    int start, stride;
    if (w < A.sch.w_big_end) {
        if (w < A.sch.n_seg) {
            int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        start = g;
        stride = geo.G;
        n_iter = (e - b + geo.G - 1) / geo.G;
    } else {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + g;
        r = -1; b = 0; e = 0;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        start = 0;
        stride = 1;
        // the first group of the wave has the longest row (rows sorted by degree)
        const int64_t k0 = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G;
        const int64_t r0 = A.csr.perm[k0];
        n_iter = row_ptr(A.csr, r0 + 1) - row_ptr(A.csr, r0);
    }
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        sddmm_edges<T, VEC, OPK>(A, r >= 0 ? r : 0, b, e, n_iter, start, stride, lig, col0, h, active);
    }
}

// ---------------------------------------------------------------------------
// edge softmax over the in-edges of each destination, per column.
// Forward: max, then sum of exp(s - max) in fp64, then a = exp(s - max) / sum.
// Backward: S = sum of a * g in fp64, then ds = a * (g - S).
// Hub rows: the first launch leaves per-segment (max, sum) or S partials, the
// second combines them in segment order and writes the segment's edges.

template <typename T, int VEC>
__device__ __forceinline__ void ld_edge(const OperandDev& o, int64_t ed, int col0, float* v) {
    IO<T, VEC>::load(reinterpret_cast<const T*>(o.data) + ed * o.stride + col0, v);
}

template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_max(const EngineArgs& A, int64_t b, int64_t e, int start, int stride,
                                                 int col0, float* mx) {
    for (int64_t p = b + start; p < e; p += stride) {
        const int64_t ed = A.csr.eid ? (int64_t)A.csr.eid[p] : p;
        float s[VEC];
        ld_edge<T, VEC>(A.a, ed, col0, s);
#pragma unroll
        for (int i = 0; i < VEC; ++i) mx[i] = fmaxf(mx[i], s[i]);
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_sum(const EngineArgs& A, int64_t b, int64_t e, int start, int stride,
                                                 int col0, const float* mx, double* sum, bool backward) {
    for (int64_t p = b + start; p < e; p += stride) {
        const int64_t ed = A.csr.eid ? (int64_t)A.csr.eid[p] : p;
        float s[VEC];
        ld_edge<T, VEC>(A.a, ed, col0, s);
        if (backward) {
            float gg[VEC];
            ld_edge<T, VEC>(A.b, ed, col0, gg);
#pragma unroll
            for (int i = 0; i < VEC; ++i) sum[i] += (double)s[i] * (double)gg[i];
        } else {
#pragma unroll
            for (int i = 0; i < VEC; ++i) sum[i] += (double)expf(s[i] - mx[i]);
        }
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_write(const EngineArgs& A, int64_t b, int64_t e, int start,
                                                   int stride, int col0, bool active, const float* mx,
                                                   const double* sum, bool backward) {
    for (int64_t p = b + start; p < e; p += stride) {
        const int64_t ed = A.csr.eid ? (int64_t)A.csr.eid[p] : p;
        float s[VEC], v[VEC];
        ld_edge<T, VEC>(A.a, ed, col0, s);
        if (backward) {
            float gg[VEC];
            ld_edge<T, VEC>(A.b, ed, col0, gg);
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = (float)((double)s[i] * ((double)gg[i] - sum[i]));
        } else {
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = (float)((double)expf(s[i] - mx[i]) / sum[i]);
        }
        if (active) IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + ed * A.out.stride + col0, v);
    }
}

template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(256) void softmax_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    if (w >= A.sch.w_small_end) return;
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    const int64_t D = (int64_t)geo.NV * VEC;
    bool coop = w < A.sch.w_big_end;
    int64_t r = -1, b = 0, e = 0;
    int slot = -1;
    if (coop) {
        if (w < A.sch.n_seg) {
            int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z; slot = w;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
    } else {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + g;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
    }
    const int start = coop ? g : 0, stride = coop ? geo.G : 1;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + lig;
        const bool active = j < geo.NV && r >= 0;
        const int col0 = j < geo.NV ? j * VEC : 0;
        float mx[VEC];
        double sum[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) { mx[i] = -INFINITY; sum[i] = 0.0; }
        if (!BWD) {
            softmax_pass_max<T, VEC>(A, b, e, start, stride, col0, mx);
            if (coop)
                for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                    for (int i = 0; i < VEC; ++i) mx[i] = fmaxf(mx[i], __shfl_xor(mx[i], s, WAVE));
        }
        softmax_pass_sum<T, VEC>(A, b, e, start, stride, col0, mx, sum, BWD);
        if (coop)
            for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                for (int i = 0; i < VEC; ++i) sum[i] += shfl_xor_d(sum[i], s);
        if (slot >= 0) {
            if (g == 0 && active) {
                double* P = reinterpret_cast<double*>(A.partial) + (int64_t)slot * 2 * D;
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    P[col0 + i] = (double)mx[i];
                    P[D + col0 + i] = sum[i];
                }
            }
        } else {
            softmax_pass_write<T, VEC>(A, b, e, start, stride, col0, active, mx, sum, BWD);
        }
    }
}

// hub rows: combine the segment partials of the row, then write this segment
template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(256) void softmax_finish_kernel(EngineArgs A) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = blockIdx.x * WPB + (threadIdx.x >> 6);
    if (w >= A.sch.n_seg) return;
    const GeomDev& geo = A.geo;
    const int g = lane >> geo.log2L;
    const int lig = lane & (geo.L - 1);
    const int64_t D = (int64_t)geo.NV * VEC;
    const int4 sg = A.csr.seg[w];
    const int s0 = A.csr.hub_off[sg.w], s1 = A.csr.hub_off[sg.w + 1];
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        float mx[VEC];
        double sum[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) { mx[i] = -INFINITY; sum[i] = 0.0; }
        const double* P = reinterpret_cast<const double*>(A.partial);
        if (!BWD) {
            for (int s = s0; s < s1; ++s)
#pragma unroll
                for (int i = 0; i < VEC; ++i) mx[i] = fmaxf(mx[i], (float)P[(int64_t)s * 2 * D + col0 + i]);
        }
        for (int s = s0; s < s1; ++s) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                double part = P[(int64_t)s * 2 * D + D + col0 + i];
                if (!BWD) {
                    const float ms = (float)P[(int64_t)s * 2 * D + col0 + i];
                    part *= (double)expf(ms - mx[i]);  // rescale the segment's sum to the row maximum
                }
                sum[i] += part;
            }
        }
        softmax_pass_write<T, VEC>(A, sg.y, sg.z, g, geo.G, col0, active, mx, sum, BWD);
    }
}

// ---------------------------------------------------------------------------
// leaky ReLU (elementwise), validation, small helpers

template <typename T, bool BWD>
__global__ void leaky_kernel(const T* x, const T* dy, T* y, int64_t rows, int32_t cols, int64_t sx, int64_t sdy,
                             int64_t sy, float slope) {
    const int64_t n = rows * (int64_t)cols;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / cols, c = i - r * cols;
        float xv = IO<T, 1>::load1(x + r * sx + c);
        float out;
        if (BWD) {
            float d = IO<T, 1>::load1(dy + r * sdy + c);
            out = xv > 0.0f ? d : slope * d;
        } else {
            out = xv > 0.0f ? xv : slope * xv;
        }
        IO<T, 1>::store1(y + r * sy + c, out);
    }
}

__global__ void validate_kernel(const int32_t* idx, int64_t n, int64_t bound, int32_t* flag) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        int32_t v = idx[i];
        if (v < 0 || v >= bound) atomicOr(flag, 1);
    }
}

template <typename P>
__global__ void validate_ptr_kernel(const P* ptr, int64_t n_rows, int64_t n_edges, int32_t* flag) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i <= n_rows;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t v = ptr[i];
        bool bad = v < 0 || v > n_edges || (i == 0 && v != 0) || (i == n_rows && v != n_edges) ||
                   (i < n_rows && ptr[i + 1] < v);
        if (bad) atomicOr(flag, 2);
    }
}

__global__ void iota_kernel(int32_t* out, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        out[i] = (int32_t)i;
}

__global__ void copy_ptr_kernel(const void* src, int src64, void* dst, int dst64, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t v = src64 ? reinterpret_cast<const int64_t*>(src)[i] : reinterpret_cast<const int32_t*>(src)[i];
        if (dst64) reinterpret_cast<int64_t*>(dst)[i] = v;
        else reinterpret_cast<int32_t*>(dst)[i] = (int32_t)v;
    }
}

// ---------------------------------------------------------------------------
// launchers

static inline unsigned blocks_for_waves(int64_t waves) { return (unsigned)((waves + WPB - 1) / WPB); }

static inline unsigned grid_1d(int64_t n) {
    int64_t b = (n + 255) / 256;
    if (b > 65536) b = 65536;
    return (unsigned)(b > 0 ? b : 1);
}

#define GNNK_VEC_DISPATCH_F32(VEC_, ...)     \
    switch (VEC_) {                          \
        case 4: { constexpr int V = 4; __VA_ARGS__; } break; \
        case 2: { constexpr int V = 2; __VA_ARGS__; } break; \
        default: { constexpr int V = 1; __VA_ARGS__; } break; \
    }

#define GNNK_VEC_DISPATCH_BF16(VEC_, ...)    \
    switch (VEC_) {                          \
        case 8: { constexpr int V = 8; __VA_ARGS__; } break; \
        case 4: { constexpr int V = 4; __VA_ARGS__; } break; \
        case 2: { constexpr int V = 2; __VA_ARGS__; } break; \
        default: { constexpr int V = 1; __VA_ARGS__; } break; \
    }

#define GNNK_OPK_DISPATCH(OPK_, ...)         \
    switch (OPK_) {                          \
        case 0: { constexpr int K = 0; __VA_ARGS__; } break; \
        case 1: { constexpr int K = 1; __VA_ARGS__; } break; \
        default: { constexpr int K = 2; __VA_ARGS__; } break; \
    }

hipError_t launch_spmm(const EngineArgs& a, int dtype, int vec, bool maxmin, int opk, hipStream_t s) {
    if (a.sch.w_total <= 0) return hipSuccess;
    dim3 grid(blocks_for_waves(a.sch.w_total)), block(WAVE * WPB);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, GNNK_OPK_DISPATCH(opk, {
            if (maxmin) hipLaunchKernelGGL((spmm_cmp_kernel<float, V, K>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((spmm_sum_kernel<float, V, K>), grid, block, 0, s, a);
        }))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, GNNK_OPK_DISPATCH(opk, {
            if (maxmin) hipLaunchKernelGGL((spmm_cmp_kernel<bf16_t, V, K>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((spmm_sum_kernel<bf16_t, V, K>), grid, block, 0, s, a);
        }))
    }
    return hipGetLastError();
}

hipError_t launch_spmm_combine(const EngineArgs& a, int dtype, int vec, bool maxmin, hipStream_t s) {
    if (a.sch.n_hub <= 0) return hipSuccess;
    int64_t waves = (a.sch.n_hub + a.geo.G - 1) / a.geo.G;
    dim3 grid(blocks_for_waves(waves)), block(WAVE * WPB);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, {
            if (maxmin) hipLaunchKernelGGL((spmm_cmp_combine_kernel<float, V>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((spmm_sum_combine_kernel<float, V>), grid, block, 0, s, a);
        })
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, {
            if (maxmin) hipLaunchKernelGGL((spmm_cmp_combine_kernel<bf16_t, V>), grid, block, 0, s, a);
            else hipLaunchKernelGGL((spmm_sum_combine_kernel<bf16_t, V>), grid, block, 0, s, a);
        })
    }
    return hipGetLastError();
}

hipError_t launch_sddmm(const EngineArgs& a, int dtype, int vec, int opk, hipStream_t s) {
    if (a.sch.w_small_end <= 0) return hipSuccess;
    dim3 grid(blocks_for_waves(a.sch.w_small_end)), block(WAVE * WPB);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, GNNK_OPK_DISPATCH(opk, {
            hipLaunchKernelGGL((sddmm_kernel<float, V, K>), grid, block, 0, s, a);
        }))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, GNNK_OPK_DISPATCH(opk, {
            hipLaunchKernelGGL((sddmm_kernel<bf16_t, V, K>), grid, block, 0, s, a);
        }))
    }
    return hipGetLastError();
}

hipError_t launch_softmax(const EngineArgs& a, int dtype, int vec, bool backward, hipStream_t s) {
    if (a.sch.w_small_end <= 0) return hipSuccess;
    dim3 grid(blocks_for_waves(a.sch.w_small_end)), block(WAVE * WPB);
    dim3 fgrid(blocks_for_waves(a.sch.n_seg));
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, {
            if (backward) {
                hipLaunchKernelGGL((softmax_kernel<float, V, true>), grid, block, 0, s, a);
                if (a.sch.n_seg > 0)
                    hipLaunchKernelGGL((softmax_finish_kernel<float, V, true>), fgrid, block, 0, s, a);
            } else {
                hipLaunchKernelGGL((softmax_kernel<float, V, false>), grid, block, 0, s, a);
                if (a.sch.n_seg > 0)
                    hipLaunchKernelGGL((softmax_finish_kernel<float, V, false>), fgrid, block, 0, s, a);
            }
        })
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, {
            if (backward) {
                hipLaunchKernelGGL((softmax_kernel<bf16_t, V, true>), grid, block, 0, s, a);
                if (a.sch.n_seg > 0)
                    hipLaunchKernelGGL((softmax_finish_kernel<bf16_t, V, true>), fgrid, block, 0, s, a);
            } else {
                hipLaunchKernelGGL((softmax_kernel<bf16_t, V, false>), grid, block, 0, s, a);
                if (a.sch.n_seg > 0)
                    hipLaunchKernelGGL((softmax_finish_kernel<bf16_t, V, false>), fgrid, block, 0, s, a);
            }
        })
    }
    return hipGetLastError();
}

hipError_t launch_leaky(const void* x, const void* dy, void* y, int64_t rows, int32_t cols, int64_t sx,
                        int64_t sdy, int64_t sy, float slope, int dtype, bool backward, hipStream_t s) {
    int64_t n = rows * (int64_t)cols;
    if (n <= 0) return hipSuccess;
    dim3 grid(grid_1d(n)), block(256);
    if (dtype == 0) {
        if (backward)
            hipLaunchKernelGGL((leaky_kernel<float, true>), grid, block, 0, s, (const float*)x, (const float*)dy,
                               (float*)y, rows, cols, sx, sdy, sy, slope);
        else
            hipLaunchKernelGGL((leaky_kernel<float, false>), grid, block, 0, s, (const float*)x, (const float*)dy,
                               (float*)y, rows, cols, sx, sdy, sy, slope);
    } else {
        if (backward)
            hipLaunchKernelGGL((leaky_kernel<bf16_t, true>), grid, block, 0, s, (const bf16_t*)x,
                               (const bf16_t*)dy, (bf16_t*)y, rows, cols, sx, sdy, sy, slope);
        else
            hipLaunchKernelGGL((leaky_kernel<bf16_t, false>), grid, block, 0, s, (const bf16_t*)x,
                               (const bf16_t*)dy, (bf16_t*)y, rows, cols, sx, sdy, sy, slope);
    }
    return hipGetLastError();
}

hipError_t launch_validate(const int32_t* idx, int64_t n, int64_t bound, int32_t* flag, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(validate_kernel, dim3(grid_1d(n)), dim3(256), 0, s, idx, n, bound, flag);
    return hipGetLastError();
}

hipError_t launch_validate_ptr(const void* ptr, int ptr64, int64_t n_rows, int64_t n_edges, int32_t* flag,
                               hipStream_t s) {
    dim3 grid(grid_1d(n_rows + 1)), block(256);
    if (ptr64)
        hipLaunchKernelGGL((validate_ptr_kernel<int64_t>), grid, block, 0, s, (const int64_t*)ptr, n_rows, n_edges,
                           flag);
    else
        hipLaunchKernelGGL((validate_ptr_kernel<int32_t>), grid, block, 0, s, (const int32_t*)ptr, n_rows, n_edges,
                           flag);
    return hipGetLastError();
}

hipError_t launch_iota(int32_t* out, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(iota_kernel, dim3(grid_1d(n)), dim3(256), 0, s, out, n);
    return hipGetLastError();
}

hipError_t launch_copy_ptr(const void* src, int src64, void* dst, int dst64, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(copy_ptr_kernel, dim3(grid_1d(n)), dim3(256), 0, s, src, src64, dst, dst64, n);
    return hipGetLastError();
}

}  // namespace gnnk
