// g-SpMM kernels (Section 3, definition of generalized SpMM): each output row
// reduces the messages of the edges of one CSR row -- the in-CSR for the
// forward pass, the reverse graph's CSR for node gradients (Theorem 1).
//
// One launch covers every role of the degree-sorted schedule (internal.h):
// hub segments (partials to scratch), a wavefront per big row (lane groups
// stride the edges and are combined by xor shuffles in fixed order), a lane
// group per small row, and the empty-row fill.  Sums accumulate in fp64; max
// and min compare fp32 messages and break ties toward the smaller edge id.
// The edge loop loads the next batch's indices while the current batch's
// gathers are in flight.
#include "device.h"

namespace gnnk {

// ---------------------------------------------------------------------------
// sums

template <typename T, int VEC, int OPK, int EXT>
__device__ __forceinline__ void spmm_sum_edges(const EngineArgs& A, int32_t self, int64_t b, int64_t e, int start,
                                               int stride, int col0, int h, double* acc) {
    const int64_t step = (int64_t)stride * UNR;
    int64_t p0 = b + start;
    if (p0 >= e) return;
    int32_t nb[UNR], ed[UNR];
    bool ok[UNR];
    batch_ids(A.csr, b, e, p0, stride, ok, nb, ed);
    for (; p0 < e; p0 += step) {
        Raw<VEC> r[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT>(A, nb[u], ed[u], self, col0, h, r[u]);
        bool okc[UNR];
        int32_t edc[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            okc[u] = ok[u];
            edc[u] = ed[u];
        }
        batch_ids(A.csr, b, e, p0 + step, stride, ok, nb, ed);  // next batch, overlapping the gathers
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            double m[VEC];
            combine_f64<VEC, OPK, EXT>(A, r[u], edc[u], m);
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] += okc[u] ? m[i] : 0.0;
        }
    }
}

template <typename T, int VEC, int OPK, int EXT>
__global__ __launch_bounds__(256) void spmm_sum_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);

    if (w < A.sch.w_big_end) {
        // one wavefront: a segment of a hub row, or a whole big row
        int64_t r, b, e;
        int slot = -1;
        if (w < A.sch.n_seg) {
            const int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z; slot = w;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            double acc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
            spmm_sum_edges<T, VEC, OPK, EXT>(A, (int32_t)r, b, e, ln.g, geo.G, col0, h, acc);
            for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += shfl_xor_d(acc[i], s);
            if (slot >= 0) {
                if (ln.g == 0 && active) {
                    double* P = reinterpret_cast<double*>(A.partial) + (int64_t)slot * A.partial_stride + col0;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) P[i] = acc[i];
                }
            } else {
                write_sum_row<T, VEC>(A, r, active, ln.lig, col0, h, acc, e - b, ln.g == 0);
            }
        }
    } else if (w < A.sch.w_small_end) {
        // small rows: each lane group owns one row
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            double acc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
            spmm_sum_edges<T, VEC, OPK, EXT>(A, r >= 0 ? (int32_t)r : 0, b, e, 0, 1, col0, h, acc);
            write_sum_row<T, VEC>(A, r, active, ln.lig, col0, h, acc, e - b, true);
        }
    } else {
        // empty rows: the empty reduction is 0 (no mean, no negation)
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * geo.G + ln.g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * geo.L + ln.lig;
                const bool active = j < geo.NV;
                const int col0 = active ? j * VEC : 0;
                const int h = col0 / geo.F;
                if (!A.out.reduce) {
                    if (active && r >= 0) {
                        float v[VEC];
#pragma unroll
                        for (int i = 0; i < VEC; ++i) v[i] = 0.0f;
                        IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + col0, v);
                    }
                } else if (active && r >= 0 && (ln.lig % A.out.red) == 0) {
                    const int64_t o = A.out.per_head ? h : 0;
                    IO<T, VEC>::store1(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + o, 0.0f);
                }
            }
        }
    }
}

// combine the segment partials of hub rows, in segment order
template <typename T, int VEC>
__global__ __launch_bounds__(256) void spmm_sum_combine_kernel(EngineArgs A) {
    const int w = wave_id();
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    if ((int64_t)w * geo.G >= A.sch.n_hub) return;  // wave-uniform
    const int64_t k = (int64_t)w * geo.G + ln.g;
    const bool row_ok = k < A.sch.n_hub;
    const int64_t r = row_ok ? A.csr.perm[k] : -1;
    const int s0 = row_ok ? A.csr.hub_off[k] : 0;
    const int s1 = row_ok ? A.csr.hub_off[k + 1] : 0;
    const int64_t deg = row_ok ? row_ptr(A.csr, r + 1) - row_ptr(A.csr, r) : 0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
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
        write_sum_row<T, VEC>(A, r, active, ln.lig, col0, h, acc, deg, true);
    }
}

// ---------------------------------------------------------------------------
// max / min with the winning edge and neighbour

template <typename T, int VEC, int OPK>
__device__ __forceinline__ void spmm_cmp_edges(const EngineArgs& A, int32_t self, int64_t b, int64_t e, int start,
                                               int stride, int col0, int h, float* best, int32_t* be,
                                               int32_t* bn) {
    const bool is_min = (A.flags & F_IS_MIN) != 0;
    const int64_t step = (int64_t)stride * UNR;
    int64_t p0 = b + start;
    if (p0 >= e) return;
    int32_t nb[UNR], ed[UNR];
    bool ok[UNR];
    batch_ids(A.csr, b, e, p0, stride, ok, nb, ed);
    for (; p0 < e; p0 += step) {
        Raw<VEC> r[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT_NONE>(A, nb[u], ed[u], self, col0, h, r[u]);
        bool okc[UNR];
        int32_t edc[UNR], nbc[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            okc[u] = ok[u];
            edc[u] = ed[u];
            nbc[u] = nb[u];
        }
        batch_ids(A.csr, b, e, p0 + step, stride, ok, nb, ed);
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            float m[VEC];
            combine_f32<VEC, OPK>(A, r[u], m);
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                const bool upd = okc[u] & better(m[i], edc[u], best[i], be[i], is_min);
                best[i] = upd ? m[i] : best[i];
                be[i] = upd ? edc[u] : be[i];
                bn[i] = upd ? nbc[u] : bn[i];
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
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int64_t D = (int64_t)geo.NV * VEC;
    const bool is_min = (A.flags & F_IS_MIN) != 0;

    if (w < A.sch.w_big_end) {
        int64_t r, b, e;
        int slot = -1;
        if (w < A.sch.n_seg) {
            const int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z; slot = w;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            float best[VEC];
            int32_t be[VEC], bn[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
            spmm_cmp_edges<T, VEC, OPK>(A, (int32_t)r, b, e, ln.g, geo.G, col0, h, best, be, bn);
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
                if (ln.g == 0 && active) {
                    float* PV = reinterpret_cast<float*>(A.partial) + (int64_t)slot * D + col0;
                    int32_t* PE = reinterpret_cast<int32_t*>(A.partial) + (int64_t)A.sch.n_seg * D +
                                  (int64_t)slot * D + col0;
                    int32_t* PN = PE + (int64_t)A.sch.n_seg * D;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) { PV[i] = best[i]; PE[i] = be[i]; PN[i] = bn[i]; }
                }
            } else if (ln.g == 0) {
                write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn);
            }
        }
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * geo.L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            float best[VEC];
            int32_t be[VEC], bn[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
            spmm_cmp_edges<T, VEC, OPK>(A, r >= 0 ? (int32_t)r : 0, b, e, 0, 1, col0, h, best, be, bn);
            write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn);
        }
    } else {
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * geo.G + ln.g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * geo.L + ln.lig;
                const bool active = j < geo.NV;
                float best[VEC];
                int32_t be[VEC], bn[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
                write_cmp_row<T, VEC>(A, r, active, active ? j * VEC : 0, best, be, bn);
            }
        }
    }
}

template <typename T, int VEC>
__global__ __launch_bounds__(256) void spmm_cmp_combine_kernel(EngineArgs A) {
    const int w = wave_id();
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    if ((int64_t)w * geo.G >= A.sch.n_hub) return;
    const int64_t k = (int64_t)w * geo.G + ln.g;
    const bool row_ok = k < A.sch.n_hub;
    const int64_t r = row_ok ? A.csr.perm[k] : -1;
    const int s0 = row_ok ? A.csr.hub_off[k] : 0;
    const int s1 = row_ok ? A.csr.hub_off[k + 1] : 0;
    const int64_t D = (int64_t)geo.NV * VEC;
    const bool is_min = (A.flags & F_IS_MIN) != 0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
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
// launchers

hipError_t launch_spmm(const EngineArgs& a, int dtype, int vec, bool maxmin, int opk, hipStream_t s) {
    if (a.sch.w_total <= 0) return hipSuccess;
    const dim3 grid(blocks_for_waves(a.sch.w_total)), block(WAVE * WPB);
    const int ext = ext_of(a.flags);
    if (maxmin) {
        if (dtype == 0) {
            GNNK_VEC_DISPATCH_F32(vec, GNNK_OPK_DISPATCH(opk, {
                hipLaunchKernelGGL((spmm_cmp_kernel<float, V, K>), grid, block, 0, s, a);
            }))
        } else {
            GNNK_VEC_DISPATCH_BF16(vec, GNNK_OPK_DISPATCH(opk, {
                hipLaunchKernelGGL((spmm_cmp_kernel<bf16_t, V, K>), grid, block, 0, s, a);
            }))
        }
    } else {
        if (dtype == 0) {
            GNNK_VEC_DISPATCH_F32(vec, GNNK_OPK_DISPATCH(opk, GNNK_EXT_DISPATCH(ext, {
                hipLaunchKernelGGL((spmm_sum_kernel<float, V, K, X>), grid, block, 0, s, a);
            })))
        } else {
            GNNK_VEC_DISPATCH_BF16(vec, GNNK_OPK_DISPATCH(opk, GNNK_EXT_DISPATCH(ext, {
                hipLaunchKernelGGL((spmm_sum_kernel<bf16_t, V, K, X>), grid, block, 0, s, a);
            })))
        }
    }
    return hipGetLastError();
}

hipError_t launch_spmm_combine(const EngineArgs& a, int dtype, int vec, bool maxmin, hipStream_t s) {
    if (a.sch.n_hub <= 0) return hipSuccess;
    const int64_t waves = (a.sch.n_hub + a.geo.G - 1) / a.geo.G;
    const dim3 grid(blocks_for_waves(waves)), block(WAVE * WPB);
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

}  // namespace gnnk
