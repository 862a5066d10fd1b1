// Edge-parallel (COO) walks: the load-balanced alternative to the row
// engine (Table 1 of the paper: both are valid for commutative and
// associative reducers; Appendix E compares them).  The positions of a CSR
// are cut into sub-chunks of sub_edges consecutive positions, one per lane
// group, so every lane group handles the same number of edges whatever the
// degree distribution.  The row of a position comes from the COO row array.
//
// g-SpMM (sum, mean) is a segmented reduction along the sub-chunk: a lane
// group accumulates while the row stays the same and flushes at each row
// change.  A row that lies inside the sub-chunk is written directly.  A row
// that crosses a sub-chunk boundary leaves partials:
//   mode 0 (deterministic): in sub-chunk k, the first row when it started
//     before k ("head" slot of k), the last row when it started inside k and
//     goes on after k ("tail" slot of k).  Then spmm_edge_fix_kernel, once
//     per split row, in the sub-chunk where the row ends, adds the tail of
//     the sub-chunk where it starts and the heads of the following ones in
//     sub-chunk order;
//   mode 1 (atomic, order not fixed): fp64 atomic adds into a zeroed
//     rows x D scratch, then spmm_edge_finish_kernel rounds the split rows.
// g-SDDMM has no reduction: every position is independent, so the positions
// are dealt out flat, consecutive ones to consecutive lane groups, and both
// endpoints are read per edge (no row-level reuse of the destination
// operand, which is what the row engine gains on CSR).
#include "walk.h"

namespace gnnk {

// positions [sb, se) of sub-chunk k
__device__ __forceinline__ void sub_range(const EngineArgs& A, int64_t k, int64_t n_pos, int32_t& sb, int32_t& se) {
    const int64_t b = k * (int64_t)A.sub_edges;
    sb = (int32_t)(b < n_pos ? b : n_pos);
    se = (int32_t)(b + A.sub_edges < n_pos ? b + A.sub_edges : n_pos);
}

// Per-lane ids and rows of UNR consecutive positions p0 .. p0 + UNR - 1,
// clamped to sb past se.
__device__ __forceinline__ void coo_ids(const CsrDev& C, int32_t sb, int32_t se, int32_t p0, bool* ok, int32_t* nb,
                                        int32_t* ed, int32_t* rw, int32_t* ps) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        const int32_t p = p0 + u;
        ok[u] = p < se;
        const int32_t pc = ok[u] ? p : sb;
        ps[u] = pc;
        nb[u] = C.idx[pc];
        ed[u] = C.eid ? C.eid[pc] : pc;
        rw[u] = C.row[pc];
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void write_row_final(const EngineArgs& A, int32_t r, int col0, bool active, double* acc,
                                                int64_t deg) {
    if (A.flags & F_OWN_MEAN) {
        const double d = deg > 0 ? (double)deg : 1.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = acc[i] / d;
    }
    if (A.flags & F_NEGATE) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = -acc[i];
    }
    if (active) {
        float v[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = (float)acc[i];
        IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + (uint64_t)(uint32_t)r * (uint32_t)A.out.stride + col0, v);
    }
}

template <typename T, int VEC, int OPK, int EXT, class S, int MODE>
__global__ __launch_bounds__(256) void spmm_edge_kernel(EngineArgs A, int64_t n_pos) {
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int G = S::GC > 0 ? S::GC : geo.G;
    const int L = WAVE / G;
    const int64_t k = (int64_t)wave_id() * G + ln.g;
    if (k >= A.n_sub) return;  // whole lane groups leave; no cross-lane work below
    int32_t sb, se;
    sub_range(A, k, n_pos, sb, se);
    if (sb >= se) return;
    using SN = Spec<S::AT, S::AK, S::BT, S::BK, S::GC, false, false>;
    const int64_t D = (int64_t)geo.NV * VEC;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        double acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
        int32_t cur = A.csr.row[sb];
        auto flush = [&](int32_t r) {
            const int64_t rb = row_ptr(A.csr, r), re = row_ptr(A.csr, r + 1);
            if (rb >= sb && re <= se) {
                write_row_final<T, VEC>(A, r, col0, active, acc, re - rb);
            } else if (active) {
                if constexpr (MODE == 1) {
                    double* P = reinterpret_cast<double*>(A.partial) + (int64_t)r * D + col0;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) unsafeAtomicAdd(P + i, acc[i]);
                } else {
                    const int64_t slot = 2 * k + (rb < sb ? 0 : 1);
                    double* P = reinterpret_cast<double*>(A.partial) + slot * D + col0;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) P[i] = acc[i];
                }
            }
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
        };
        Pre<VEC> pre;
        int32_t nb[UNR], ed[UNR], rw[UNR], ps[UNR];
        bool ok[UNR];
        for (int32_t p0 = sb; p0 < se; p0 += UNR) {
            coo_ids(A.csr, sb, se, p0, ok, nb, ed, rw, ps);
            Raw<VEC> r[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) fetch_bits<VEC, EXT>(A, ps[u], col0, r[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT, SN>(A, nb[u], ed[u], rw[u], col0, h, pre, r[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                if (ok[u]) {
                    if (rw[u] != cur) {
                        flush(cur);
                        cur = rw[u];
                    }
                    double m[VEC];
                    combine_f64<VEC, OPK, EXT>(A, r[u], ed[u], m);
#pragma unroll
                    for (int i = 0; i < VEC; ++i) acc[i] += m[i];
                }
            }
        }
        flush(cur);
    }
}

// mode 0: the split rows, each once, in the sub-chunk where the row ends
template <typename T, int VEC>
__global__ __launch_bounds__(256) void spmm_edge_fix_kernel(EngineArgs A, int64_t n_pos) {
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int64_t k = (int64_t)wave_id() * geo.G + ln.g;
    if (k >= A.n_sub) return;
    int32_t sb, se;
    sub_range(A, k, n_pos, sb, se);
    if (sb >= se) return;
    const int32_t r = A.csr.row[sb];
    const int64_t rb = row_ptr(A.csr, r), re = row_ptr(A.csr, r + 1);
    if (!(rb < sb && re <= se)) return;  // not a split row that ends here
    const int64_t k0 = rb / A.sub_edges;  // the sub-chunk where the row starts
    const int64_t D = (int64_t)geo.NV * VEC;
    const double* P = reinterpret_cast<const double*>(A.partial);
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        double acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = P[(2 * k0 + 1) * D + col0 + i];
        for (int64_t q = k0 + 1; q <= k; ++q)
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] += P[(2 * q) * D + col0 + i];
        write_row_final<T, VEC>(A, r, col0, active, acc, re - rb);
    }
}

// mode 1: zero the scratch rows of split rows before the atomics
template <int VEC>
__global__ __launch_bounds__(256) void spmm_edge_zero_kernel(EngineArgs A, int64_t n_rows) {
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int64_t r = (int64_t)wave_id() * geo.G + ln.g;
    if (r >= n_rows) return;
    const int64_t rb = row_ptr(A.csr, r), re = row_ptr(A.csr, r + 1);
    if (re == rb || rb / A.sub_edges == (re - 1) / A.sub_edges) return;  // not split
    const int64_t D = (int64_t)geo.NV * VEC;
    double* P = reinterpret_cast<double*>(A.partial) + r * D;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        if (j < geo.NV)
#pragma unroll
            for (int i = 0; i < VEC; ++i) P[j * VEC + i] = 0.0;
    }
}

// mode 1: round the accumulated split rows
template <typename T, int VEC>
__global__ __launch_bounds__(256) void spmm_edge_finish_kernel(EngineArgs A, int64_t n_rows) {
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int64_t r = (int64_t)wave_id() * geo.G + ln.g;
    if (r >= n_rows) return;
    const int64_t rb = row_ptr(A.csr, r), re = row_ptr(A.csr, r + 1);
    if (re == rb || rb / A.sub_edges == (re - 1) / A.sub_edges) return;  // empty, or inside one sub-chunk
    const int64_t D = (int64_t)geo.NV * VEC;
    const double* P = reinterpret_cast<const double*>(A.partial) + r * D;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        double acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = P[col0 + i];
        write_row_final<T, VEC>(A, (int32_t)r, col0, active, acc, re - rb);
    }
}

// ids of slot u of lane group g in a step of G * UNR positions from q: slot
// u of every group lies on G consecutive positions q + u * G + g, so one
// store instruction of the wavefront covers consecutive outputs; slots past
// n_pos read position q (in bounds) and are dropped
__device__ __forceinline__ void flat_ids(const CsrDev& C, int64_t q, int64_t n_pos, int G, int g, bool* ok,
                                         int32_t* nb, int32_t* ed, int32_t* rw, int32_t* ps) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        const int64_t p = q + (int64_t)u * G + g;
        ok[u] = p < n_pos;
        const int32_t pc = (int32_t)(ok[u] ? p : q);
        ps[u] = pc;
        nb[u] = C.idx[pc];
        ed[u] = C.eid ? C.eid[pc] : pc;
        rw[u] = C.row[pc];
    }
}

// g-SDDMM, one output per position, both endpoints read per edge.  The
// positions are dealt out flat: a wavefront takes G * UNR consecutive ones
// per step (grid-stride), so every lane group has the same work and the
// outputs of a step are written as one contiguous stretch (with identity
// edge ids).  No reduction crosses lane groups, so no sub-chunks are needed.
template <typename T, int VEC, int OPK, int EXT, int RM, class S>
__global__ __launch_bounds__(256) void sddmm_edge_kernel(EngineArgs A, int64_t n_pos) {
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int G = S::GC > 0 ? S::GC : geo.G;
    const int L = WAVE / G;
    const int64_t per = (int64_t)G * UNR;
    const int64_t stride = (int64_t)gridDim.x * WPB * per;
    using SN = Spec<S::AT, S::AK, S::BT, S::BK, S::GC, false, false>;
    const bool neg = (A.flags & F_NEGATE) != 0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        Pre<VEC> pre;
        int32_t nb[UNR], ed[UNR], rw[UNR], ps[UNR];
        bool ok[UNR];
        for (int64_t q = (int64_t)wave_id() * per; q < n_pos; q += stride) {
            flat_ids(A.csr, q, n_pos, G, ln.g, ok, nb, ed, rw, ps);
            Raw<VEC> r[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) fetch_bits<VEC, EXT>(A, ps[u], col0, r[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT, SN>(A, nb[u], ed[u], rw[u], col0, h, pre, r[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                double m[VEC];
                combine_f64<VEC, OPK, EXT>(A, r[u], ed[u], m);
                T* row = reinterpret_cast<T*>(A.out.data) + (uint64_t)(uint32_t)ed[u] * (uint32_t)A.out.stride;
                const bool reduce = RM < 0 ? A.out.reduce != 0 : RM > 0;
                if (!reduce) {
                    if (ok[u] & active) {
                        float v[VEC];
#pragma unroll
                        for (int i = 0; i < VEC; ++i) v[i] = (float)(neg ? -m[i] : m[i]);
                        IO<T, VEC>::store(row + col0, v);
                    }
                } else {
                    double s = 0.0;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) s += m[i];
                    const int red = A.out.red;
                    s = active ? s : 0.0;
                    if constexpr (RM > 0) s = run_sum(s, red);
                    else s = (red & (red - 1)) == 0 ? run_sum(s, red) : seg_sum(s, ln.lig, red);
                    const bool writer = RM > 0 ? ((ln.lig & (red - 1)) == 0) : ((ln.lig % red) == 0);
                    if (ok[u] & active & writer) {
                        const int o = A.out.per_head ? h : 0;
                        IO<T, VEC>::store1(row + o, (float)(neg ? -s : s));
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// launchers

namespace {

template <int GC, bool CB>
using SpUEH = Spec<T_NBR, OK_FULL, T_EDGE, OK_HEAD, GC, CB>;
template <int GC, bool CB>
using SpUER = Spec<T_NBR, OK_FULL, T_EDGE, OK_ROW, GC, CB>;
template <int GC>
using SpCU = Spec<T_NBR, OK_FULL, DYN, DYN, GC, false>;
template <int C>
using SpUV = Spec<T_NBR, OK_FULL, T_SELF, OK_FULL, C, false>;
template <int C>
using SpVU = Spec<T_SELF, OK_FULL, T_NBR, OK_FULL, C, false>;

template <typename T, int V, int M>
void spmm_edge_t(const EngineArgs& a, int64_t n_pos, int opk, int ext, int spec, int gc, dim3 grid, dim3 block,
                 hipStream_t s) {
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        if (spec != SP_DYN) {
            auto go = [&](auto cgc) {
                constexpr int C = decltype(cgc)::value;
                if (spec == SP_CU) {
                    GNNK_EXT_DISPATCH(ext, {
                        hipLaunchKernelGGL((spmm_edge_kernel<T, V, 0, X, SpCU<C>, M>), grid, block, 0, s, a, n_pos);
                    })
                } else if (spec == SP_UE_H || spec == SP_UE_H_CB) {
                    hipLaunchKernelGGL((spmm_edge_kernel<T, V, 1, EXT_NONE, SpUEH<C, false>, M>), grid, block, 0, s,
                                       a, n_pos);
                } else {
                    hipLaunchKernelGGL((spmm_edge_kernel<T, V, 1, EXT_NONE, SpUER<C, false>, M>), grid, block, 0, s,
                                       a, n_pos);
                }
            };
            GNNK_GC_DISPATCH(gc, go(std::integral_constant<int, C>{}))
            return;
        }
    }
    GNNK_OPK_DISPATCH(opk, GNNK_EXT_DISPATCH(ext, {
        hipLaunchKernelGGL((spmm_edge_kernel<T, V, K, X, SpecDyn, M>), grid, block, 0, s, a, n_pos);
    }))
}

template <typename T, int V>
void sddmm_edge_t(const EngineArgs& a, int64_t n_pos, int opk, int ext, int spec, int gc, dim3 grid, dim3 block,
                  hipStream_t s) {
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        if (spec == SP_UV || spec == SP_VU) {
            const bool rm = a.out.reduce != 0;
            auto go = [&](auto cgc) {
                constexpr int C = decltype(cgc)::value;
                if (spec == SP_VU) {
                    if (rm) hipLaunchKernelGGL((sddmm_edge_kernel<T, V, 1, EXT_NONE, 1, SpVU<C>>), grid, block, 0, s, a, n_pos);
                    else hipLaunchKernelGGL((sddmm_edge_kernel<T, V, 1, EXT_NONE, 0, SpVU<C>>), grid, block, 0, s, a, n_pos);
                } else if (opk == 1) {
                    if (rm) hipLaunchKernelGGL((sddmm_edge_kernel<T, V, 1, EXT_NONE, 1, SpUV<C>>), grid, block, 0, s, a, n_pos);
                    else hipLaunchKernelGGL((sddmm_edge_kernel<T, V, 1, EXT_NONE, 0, SpUV<C>>), grid, block, 0, s, a, n_pos);
                } else {
                    hipLaunchKernelGGL((sddmm_edge_kernel<T, V, 2, EXT_NONE, 0, SpUV<C>>), grid, block, 0, s, a, n_pos);
                }
            };
            GNNK_GC_DISPATCH(gc, go(std::integral_constant<int, C>{}))
            return;
        }
    }
    GNNK_OPK_DISPATCH(opk, GNNK_EXT3_DISPATCH(ext, {
        hipLaunchKernelGGL((sddmm_edge_kernel<T, V, K, X, -1, SpecDyn>), grid, block, 0, s, a, n_pos);
    }))
}

template <typename T, int V>
void spmm_edge_all(const EngineArgs& a, int64_t n_pos, int64_t n_rows, int opk, int ext, int spec, int gc, int mode,
                   hipStream_t s) {
    const dim3 block(WAVE * WPB);
    const dim3 grid(blocks_for_waves((a.n_sub + a.geo.G - 1) / a.geo.G));
    const dim3 rgrid(blocks_for_waves((n_rows + a.geo.G - 1) / a.geo.G));
    if (mode == 1) {
        if (n_rows > 0) hipLaunchKernelGGL((spmm_edge_zero_kernel<V>), rgrid, block, 0, s, a, n_rows);
        spmm_edge_t<T, V, 1>(a, n_pos, opk, ext, spec, gc, grid, block, s);
        if (n_rows > 0) hipLaunchKernelGGL((spmm_edge_finish_kernel<T, V>), rgrid, block, 0, s, a, n_rows);
    } else {
        spmm_edge_t<T, V, 0>(a, n_pos, opk, ext, spec, gc, grid, block, s);
        hipLaunchKernelGGL((spmm_edge_fix_kernel<T, V>), grid, block, 0, s, a, n_pos);
    }
}

}  // namespace

hipError_t launch_spmm_edge(const EngineArgs& a, int64_t n_pos, int64_t n_rows, int dtype, int vec, int opk, int spec,
                            int gc, int mode, hipStream_t s) {
    if (a.n_sub <= 0) return hipSuccess;
    const int ext = ext_of(a.flags);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, spmm_edge_all<float, V>(a, n_pos, n_rows, opk, ext, spec, gc, mode, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, spmm_edge_all<bf16_t, V>(a, n_pos, n_rows, opk, ext, spec, gc, mode, s))
    }
    return hipGetLastError();
}

hipError_t launch_sddmm_edge(const EngineArgs& a, int64_t n_pos, int dtype, int vec, int opk, int spec, int gc,
                             hipStream_t s) {
    if (n_pos <= 0) return hipSuccess;
    const int ext = ext_of(a.flags);
    const dim3 block(WAVE * WPB);
    // one step of G * UNR positions per wavefront, at most 16384 blocks
    // (grid-stride beyond)
    const int64_t waves = (n_pos + (int64_t)a.geo.G * UNR - 1) / ((int64_t)a.geo.G * UNR);
    const dim3 grid(blocks_for_waves(waves < 16384 * WPB ? waves : 16384 * WPB));
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, sddmm_edge_t<float, V>(a, n_pos, opk, ext, spec, gc, grid, block, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, sddmm_edge_t<bf16_t, V>(a, n_pos, opk, ext, spec, gc, grid, block, s))
    }
    return hipGetLastError();
}

}  // namespace gnnk
