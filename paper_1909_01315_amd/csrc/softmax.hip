// Edge softmax over the in-edges of each destination, per column (the
// attention normalisation applied to the per-edge scores of Appendix D), and
// its backward.  Forward: one pass keeps the running max m and the fp64 sum
// of exp(s - m), rescaled whenever m grows; a second pass writes
// a = exp(s - max) / sum.  Backward: S = sum of a * g in fp64, then
// ds = a * (g - S).  Rows use the degree-sorted schedule; hub rows leave
// per-segment (max, sum) or S partials and a second launch combines them in
// segment order and writes the segment's edges.
#include <type_traits>

#include "device.h"

namespace gnnk {

template <typename T, int VEC>
__device__ __forceinline__ void ld_edge(const OperandDev& o, int64_t ed, int col0, float* v) {
    IO<T, VEC>::load(reinterpret_cast<const T*>(o.data) + ed * o.stride + col0, v);
}
// the write pass reads each edge for the last time: nontemporal where a
// wavefront's lane groups take consecutive edges of one row, so that an
// instruction reads whole lines (c3 softmax 2.22 -> 2.18 ms, its backward
// 3.55 -> 3.47 ms).  A lane group walking a row alone (stride 1) reads
// each line several times in a row, and the first pass of every row keeps
// plain loads, so that short rows are read again from L2.
template <typename T, int VEC>
__device__ __forceinline__ void ld_edge_last(const OperandDev& o, int64_t ed, int col0, float* v, bool nt) {
    if (nt) IO<T, VEC>::load_nt(reinterpret_cast<const T*>(o.data) + ed * o.stride + col0, v);
    else IO<T, VEC>::load(reinterpret_cast<const T*>(o.data) + ed * o.stride + col0, v);
}

// running (max, sum of exp(s - max)) over the edges of a lane group
template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_online(const EngineArgs& A, int64_t b, int64_t e, int start, int stride,
                                                    int col0, float* mx, double* sum) {
    for (int64_t p = b + start; p < e; p += stride) {
        const int64_t ed = A.csr.eid ? (int64_t)A.csr.eid[p] : p;
        float s[VEC];
        ld_edge<T, VEC>(A.a, ed, col0, s);
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            const float mn = fmaxf(mx[i], s[i]);
            const double f = (double)exp_le0(fminf(mx[i], s[i]) - mn);
            sum[i] = s[i] > mx[i] ? sum[i] * f + 1.0 : sum[i] + f;
            mx[i] = mn;
        }
    }
}

// merge another (max, sum) pair into this one
__device__ __forceinline__ void softmax_merge(float& m, double& s, float om, double os) {
    const float mn = fmaxf(m, om);
    const double f1 = m == -INFINITY ? 0.0 : (double)exp_le0(m - mn);
    const double f2 = om == -INFINITY ? 0.0 : (double)exp_le0(om - mn);
    s = s * f1 + os * f2;
    m = mn;
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
            for (int i = 0; i < VEC; ++i) sum[i] += (double)exp_le0(s[i] - mx[i]);
        }
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_write(const EngineArgs& A, int64_t b, int64_t e, int start,
                                                   int stride, int col0, bool active, const float* mx,
                                                   const double* sum, bool backward) {
    // forward: a = exp(s - max) times the reciprocal of the fp64 sum, both
    // rounded to fp32 (3 roundings, well inside the fp32 tolerance)
    float inv[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) inv[i] = backward ? 0.0f : (float)(1.0 / sum[i]);
    for (int64_t p = b + start; p < e; p += stride) {
        const int64_t ed = A.csr.eid ? (int64_t)A.csr.eid[p] : p;
        float s[VEC], v[VEC];
        ld_edge_last<T, VEC>(A.a, ed, col0, s, stride > 1);
        if (backward) {
            float gg[VEC];
            ld_edge_last<T, VEC>(A.b, ed, col0, gg, stride > 1);
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = (float)((double)s[i] * ((double)gg[i] - sum[i]));
        } else {
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = exp_le0(s[i] - mx[i]) * inv[i];
        }
        if (active) {
            T* o = reinterpret_cast<T*>(A.out.data) + ed * A.out.stride + col0;
            if (stride > 1) IO<T, VEC>::store_nt(o, v);
            else IO<T, VEC>::store(o, v);
        }
    }
}

template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(256) void softmax_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.w_small_end) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int g = ln.g, lig = ln.lig;
    const int64_t D = (int64_t)geo.NV * VEC;
    bool coop = w < A.sch.w_big_end;
    int64_t r = -1, b = 0, e = 0;
    int slot = -1;
    if (coop) {
        if (w < A.sch.n_seg) {
            const int si = A.csr.seg_order[w];
            const int4 s = A.csr.seg[si];
            r = s.x; b = s.y; e = s.z; slot = si;
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
            softmax_pass_online<T, VEC>(A, b, e, start, stride, col0, mx, sum);
            if (coop)
                for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                    for (int i = 0; i < VEC; ++i)
                        softmax_merge(mx[i], sum[i], __shfl_xor(mx[i], s, WAVE), shfl_xor_d(sum[i], s));
        } else {
            softmax_pass_sum<T, VEC>(A, b, e, start, stride, col0, mx, sum, BWD);
            if (coop)
                for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                    for (int i = 0; i < VEC; ++i) sum[i] += shfl_xor_d(sum[i], s);
        }
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

// hub rows: combine the segment partials of each row once, in segment
// order (one lane group per hub row), into the row's (max, sum) after the
// segment partials
template <int VEC, bool BWD>
__global__ __launch_bounds__(256) void softmax_rows_kernel(EngineArgs A) {
    const int w = wave_id();
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    if ((int64_t)w * geo.G >= A.sch.n_hub) return;  // wave-uniform
    const int64_t k = (int64_t)w * geo.G + ln.g;
    if (k >= A.sch.n_hub) return;
    const int64_t D = (int64_t)geo.NV * VEC;
    const int s0 = A.csr.hub_off[k], s1 = A.csr.hub_off[k + 1];
    double* P = reinterpret_cast<double*>(A.partial);
    double* R = P + ((int64_t)A.sch.n_seg + k) * 2 * D;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        if (j >= geo.NV) continue;
        const int col0 = j * VEC;
        float mx[VEC];
        double sum[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) { mx[i] = -INFINITY; sum[i] = 0.0; }
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
                    part *= (double)exp_le0(ms - mx[i]);  // rescale the segment's sum to the row maximum
                }
                sum[i] += part;
            }
        }
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            R[col0 + i] = (double)mx[i];
            R[D + col0 + i] = sum[i];
        }
    }
}

// hub rows: write this segment with its row's combined (max, sum)
template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(256) void softmax_finish_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.n_seg) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int g = ln.g, lig = ln.lig;
    const int64_t D = (int64_t)geo.NV * VEC;
    const int4 sg = A.csr.seg[A.csr.seg_order[w]];
    const double* R = reinterpret_cast<const double*>(A.partial) + ((int64_t)A.sch.n_seg + sg.w) * 2 * D;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        float mx[VEC];
        double sum[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            mx[i] = (float)R[col0 + i];
            sum[i] = R[D + col0 + i];
        }
        softmax_pass_write<T, VEC>(A, sg.y, sg.z, g, geo.G, col0, active, mx, sum, BWD);
    }
}


hipError_t launch_softmax(const EngineArgs& a, int dtype, int vec, bool backward, hipStream_t s) {
    if (a.sch.w_small_end <= 0) return hipSuccess;
    dim3 grid(blocks_for_waves(a.sch.w_small_end)), block(WAVE * WPB);
    dim3 fgrid(blocks_for_waves(a.sch.n_seg));
    dim3 rgrid(blocks_for_waves((a.sch.n_hub + a.geo.G - 1) / a.geo.G));
    // pass over all rows (hub segments leave partials), then for hub rows the
    // per-row combine and the write pass of each segment
    auto run = [&](auto tv, auto vv, auto bv) {
        using T = decltype(tv);
        constexpr int V = decltype(vv)::value;
        constexpr bool B = decltype(bv)::value;
        hipLaunchKernelGGL((softmax_kernel<T, V, B>), grid, block, 0, s, a);
        if (a.sch.n_seg > 0) {
            hipLaunchKernelGGL((softmax_rows_kernel<V, B>), rgrid, block, 0, s, a);
            hipLaunchKernelGGL((softmax_finish_kernel<T, V, B>), fgrid, block, 0, s, a);
        }
    };
    using BT = std::true_type;
    using BF = std::false_type;
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, {
            if (backward) run(float{}, std::integral_constant<int, V>{}, BT{});
            else run(float{}, std::integral_constant<int, V>{}, BF{});
        })
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, {
            if (backward) run(bf16_t{}, std::integral_constant<int, V>{}, BT{});
            else run(bf16_t{}, std::integral_constant<int, V>{}, BF{});
        })
    }
    return hipGetLastError();
}

}  // namespace gnnk
