// Edge softmax over the in-edges of each destination, per column (the
// attention normalisation applied to the per-edge scores of Appendix E), and
// its backward.  Forward: one pass keeps the running max m and the fp64 sum
// of exp(s - m), rescaled whenever m grows; a second pass writes
// a = exp(s - max) / sum.  Backward: S = sum of a * g in fp64, then
// ds = a * (g - S).  Rows use the degree-sorted schedule.  A hub row takes
// one block of wavefronts that merge their partials through LDS in wavefront
// order and write the row at once, so the second read of its scores comes
// from the caches rather than HBM (one launch for all hub rows instead of
// segment partials, a combine and a write launch: c3 softmax 2.22 -> 1.80
// ms, its backward 3.50 -> 2.70 ms).
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

// Each pass takes a lane group's edges in groups of SM_UNROLL: the group's
// loads are issued together (one lane keeps several loads in flight, which
// a wavefront or block walking one long row needs to cover the memory
// latency) and its edges are then consumed in edge order, so the results are
// those of the edge-by-edge loop.
constexpr int SM_UNROLL = 4;

__device__ __forceinline__ int64_t edge_at(const EngineArgs& A, int64_t p) {
    return A.csr.eid ? (int64_t)A.csr.eid[p] : p;
}

template <int VEC>
__device__ __forceinline__ void online_step(float* mx, double* sum, const float* s) {
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
        // a score of -inf (a masked edge) adds exp(-inf) = 0; while the
        // running max is still -inf too, -inf - (-inf) would give NaN
        const float mn = fmaxf(mx[i], s[i]);
        const double f = mn == -INFINITY ? 0.0 : (double)exp_le0(fminf(mx[i], s[i]) - mn);
        sum[i] = s[i] > mx[i] ? sum[i] * f + 1.0 : sum[i] + f;
        mx[i] = mn;
    }
}

// U scores at once: the running sum is rescaled once to the new maximum
// (the batch's and the old one's), then the batch's terms are added, about
// 60% of the instructions of U single steps (c3 softmax forward ran close to
// its VALU issue limit).  A column whose scores are all -inf so far keeps
// (-inf, 0).
template <int VEC, int U>
__device__ __forceinline__ void online_batch(float* mx, double* sum, const float (*s)[VEC]) {
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
        float mb = s[0][i];
#pragma unroll
        for (int u = 1; u < U; ++u) mb = fmaxf(mb, s[u][i]);
        const float mn = fmaxf(mx[i], mb);
        double acc = mx[i] == -INFINITY ? 0.0 : sum[i] * (double)exp_le0(mx[i] - mn);
#pragma unroll
        for (int u = 0; u < U; ++u) acc += (double)exp_le0(s[u][i] - mn);
        const bool live = mn != -INFINITY;
        sum[i] = live ? acc : sum[i];
        mx[i] = mn;
    }
}

// running (max, sum of exp(s - max)) over the edges of a lane group
template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_online(const EngineArgs& A, int64_t b, int64_t e, int start, int stride,
                                                    int col0, float* mx, double* sum) {
    constexpr int U = SM_UNROLL;
    int64_t p = b + start;
    for (; p + (int64_t)(U - 1) * stride < e; p += (int64_t)U * stride) {
        float s[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) ld_edge<T, VEC>(A.a, edge_at(A, p + (int64_t)u * stride), col0, s[u]);
        online_batch<VEC, U>(mx, sum, s);
    }
    for (; p < e; p += stride) {
        float s[VEC];
        ld_edge<T, VEC>(A.a, edge_at(A, p), col0, s);
        online_step<VEC>(mx, sum, s);
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

// backward: S = sum of a * g over the edges of a lane group
template <typename T, int VEC>
__device__ __forceinline__ void softmax_pass_dot(const EngineArgs& A, int64_t b, int64_t e, int start, int stride,
                                                 int col0, double* sum) {
    constexpr int U = SM_UNROLL;
    int64_t p = b + start;
    for (; p + (int64_t)(U - 1) * stride < e; p += (int64_t)U * stride) {
        float s[U][VEC], gg[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t ed = edge_at(A, p + (int64_t)u * stride);
            ld_edge<T, VEC>(A.a, ed, col0, s[u]);
            ld_edge<T, VEC>(A.b, ed, col0, gg[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int i = 0; i < VEC; ++i) sum[i] += (double)s[u][i] * (double)gg[u][i];
    }
    for (; p < e; p += stride) {
        const int64_t ed = edge_at(A, p);
        float s[VEC], gg[VEC];
        ld_edge<T, VEC>(A.a, ed, col0, s);
        ld_edge<T, VEC>(A.b, ed, col0, gg);
#pragma unroll
        for (int i = 0; i < VEC; ++i) sum[i] += (double)s[i] * (double)gg[i];
    }
}

// the output of one edge from its loaded operands
template <typename T, int VEC>
__device__ __forceinline__ void softmax_out(const EngineArgs& A, int64_t ed, int col0, bool active, bool nt,
                                            const float* s, const float* gg, const float* mx, const double* sum,
                                            const float* inv, bool backward) {
    float v[VEC];
    if (backward) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = (float)((double)s[i] * ((double)gg[i] - sum[i]));
    } else {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = exp_le0(s[i] - mx[i]) * inv[i];
    }
    if (active) {
        T* o = reinterpret_cast<T*>(A.out.data) + ed * A.out.stride + col0;
        if (nt) IO<T, VEC>::store_nt(o, v);
        else IO<T, VEC>::store(o, v);
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
    const bool nt = stride > 1;
    constexpr int U = SM_UNROLL;
    int64_t p = b + start;
    for (; p + (int64_t)(U - 1) * stride < e; p += (int64_t)U * stride) {
        float s[U][VEC], gg[U][VEC];
        int64_t ed[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            ed[u] = edge_at(A, p + (int64_t)u * stride);
            ld_edge_last<T, VEC>(A.a, ed[u], col0, s[u], nt);
            if (backward) ld_edge_last<T, VEC>(A.b, ed[u], col0, gg[u], nt);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) softmax_out<T, VEC>(A, ed[u], col0, active, nt, s[u], gg[u], mx, sum, inv, backward);
    }
    for (; p < e; p += stride) {
        const int64_t ed = edge_at(A, p);
        float s[VEC], gg[VEC];
        ld_edge_last<T, VEC>(A.a, ed, col0, s, nt);
        if (backward) ld_edge_last<T, VEC>(A.b, ed, col0, gg, nt);
        softmax_out<T, VEC>(A, ed, col0, active, nt, s, gg, mx, sum, inv, backward);
    }
}

// The same passes with the first K unrolled steps of each lane kept in
// registers between them: the write pass takes those edges' operands (the
// backward's attention and its gradient) from the registers instead of
// reading them again.  A lane walks the same positions in the same order in
// both passes, so the results are those of the uncached passes, bit for bit.
// The backward (two operands, eight fp32 values per edge and lane at VEC = 4)
// keeps two steps: c3 softmax backward 2.63 -> 2.53 ms on the hub rows, 2.54
// -> 2.49 ms with the other rows too.  The forward keeps none: one to four
// steps made it slower (1.80 -> 1.98-2.05 ms; the registers cost more
// occupancy than the second read costs), and wider lanes (VEC = 8) would
// spill.
__host__ __device__ constexpr int hub_cache_steps(bool backward, int vec) { return backward && vec <= 4 ? 2 : 0; }

template <typename T, int VEC, int K>
struct RowCache {
    float s[K > 0 ? K : 1][SM_UNROLL][VEC];
    float g[K > 0 ? K : 1][SM_UNROLL][VEC];
    int n;  // unrolled steps held
};

template <typename T, int VEC, int K, bool BWD>
__device__ __forceinline__ void softmax_pass_first_cached(const EngineArgs& A, int64_t b, int64_t e, int start,
                                                          int stride, int col0, float* mx, double* sum,
                                                          RowCache<T, VEC, K>& c) {
    constexpr int U = SM_UNROLL;
    int64_t p = b + start;
    c.n = 0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (c.n == k && p + (int64_t)(U - 1) * stride < e) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t ed = edge_at(A, p + (int64_t)u * stride);
                ld_edge<T, VEC>(A.a, ed, col0, c.s[k][u]);
                if (BWD) ld_edge<T, VEC>(A.b, ed, col0, c.g[k][u]);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!BWD) {
                    online_step<VEC>(mx, sum, c.s[k][u]);
                } else {
#pragma unroll
                    for (int i = 0; i < VEC; ++i) sum[i] += (double)c.s[k][u][i] * (double)c.g[k][u][i];
                }
            }
            p += (int64_t)U * stride;
            c.n = k + 1;
        }
    }
    // the rest of the lane's positions: the uncached pass from p
    if (!BWD) softmax_pass_online<T, VEC>(A, p, e, 0, stride, col0, mx, sum);
    else softmax_pass_dot<T, VEC>(A, p, e, 0, stride, col0, sum);
}

template <typename T, int VEC, int K>
__device__ __forceinline__ void softmax_pass_write_cached(const EngineArgs& A, int64_t b, int64_t e, int start,
                                                          int stride, int col0, bool active, const float* mx,
                                                          const double* sum, bool backward,
                                                          const RowCache<T, VEC, K>& c) {
    constexpr int U = SM_UNROLL;
    float inv[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) inv[i] = backward ? 0.0f : (float)(1.0 / sum[i]);
    const bool nt = stride > 1;
    int64_t p = b + start;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (k < c.n) {
#pragma unroll
            for (int u = 0; u < U; ++u)
                softmax_out<T, VEC>(A, edge_at(A, p + (int64_t)u * stride), col0, active, nt, c.s[k][u], c.g[k][u],
                                    mx, sum, inv, backward);
            p += (int64_t)U * stride;
        }
    }
    softmax_pass_write<T, VEC>(A, p, e, 0, stride, col0, active, mx, sum, backward);
}

// rows after the hub rows: a wavefront per big row (its lane groups stride
// over the row and merge by shuffles), a lane group per small row
template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(256) void softmax_kernel(EngineArgs A) {
    // the hub segments' wave indices are not launched
    const int w = wave_id() + A.sch.n_seg;
    if (w >= A.sch.w_small_end) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int g = ln.g, lig = ln.lig;
    const bool coop = w < A.sch.w_big_end;
    int64_t r = -1, b = 0, e = 0;
    if (coop) {
        const int4 t = A.csr.rowt[A.sch.n_hub + (w - A.sch.n_seg)];
        r = t.x; b = t.y; e = t.z;
    } else {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + g;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
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
        constexpr int KC = hub_cache_steps(BWD, VEC);
        RowCache<T, VEC, KC> rc;
        if constexpr (KC > 0) softmax_pass_first_cached<T, VEC, KC, BWD>(A, b, e, start, stride, col0, mx, sum, rc);
        if (!BWD) {
            softmax_pass_online<T, VEC>(A, b, e, start, stride, col0, mx, sum);
            if (coop)
                for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                    for (int i = 0; i < VEC; ++i)
                        softmax_merge(mx[i], sum[i], __shfl_xor(mx[i], s, WAVE), shfl_xor_d(sum[i], s));
        } else {
            if constexpr (KC == 0) softmax_pass_dot<T, VEC>(A, b, e, start, stride, col0, sum);
            if (coop)
                for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                    for (int i = 0; i < VEC; ++i) sum[i] += shfl_xor_d(sum[i], s);
        }
        if constexpr (KC > 0) softmax_pass_write_cached<T, VEC, KC>(A, b, e, start, stride, col0, active, mx, sum, BWD, rc);
        else softmax_pass_write<T, VEC>(A, b, e, start, stride, col0, active, mx, sum, BWD);
    }
}

// wavefronts per hub row: c3 (114.6M edges, (E,8) fp32) softmax takes
// 2.03 / 1.80 / 2.87 ms with 4 / 8 / 16 (backward 2.97 / 2.70 / 2.78 ms)
constexpr int HUB_WAVES = 8;


// hub row perm[blockIdx.x]: the lane groups of all HUB_WAVES wavefronts
// stride over the row; each wavefront merges its lane groups by shuffles,
// then every wavefront merges the wavefronts' partials from LDS in wavefront
// order (all reach the same values) and writes its share of the row
template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(WAVE * HUB_WAVES) void softmax_hub_kernel(EngineArgs A) {
    __shared__ float smx[HUB_WAVES][WAVE];
    __shared__ double ssum[HUB_WAVES][WAVE];
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int wv = threadIdx.x >> 6;
    const int4 t = A.csr.rowt[blockIdx.x];
    const int64_t b = uniform64(t.y), e = uniform64(t.z);
    const int start = wv * geo.G + ln.g, stride = HUB_WAVES * geo.G;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        float mx[VEC];
        double sum[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) { mx[i] = -INFINITY; sum[i] = 0.0; }
        constexpr int KC = hub_cache_steps(BWD, VEC);
        RowCache<T, VEC, KC> rc;
        if constexpr (KC > 0) {
            softmax_pass_first_cached<T, VEC, KC, BWD>(A, b, e, start, stride, col0, mx, sum, rc);
        } else {
            if (!BWD) softmax_pass_online<T, VEC>(A, b, e, start, stride, col0, mx, sum);
            else softmax_pass_dot<T, VEC>(A, b, e, start, stride, col0, sum);
        }
        if (!BWD) {
            for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                for (int i = 0; i < VEC; ++i)
                    softmax_merge(mx[i], sum[i], __shfl_xor(mx[i], s, WAVE), shfl_xor_d(sum[i], s));
        } else {
            for (int s = geo.L; s < WAVE; s <<= 1)
#pragma unroll
                for (int i = 0; i < VEC; ++i) sum[i] += shfl_xor_d(sum[i], s);
        }
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            __syncthreads();  // the previous column's readers are done
            if (ln.g == 0) {
                smx[wv][ln.lig] = mx[i];
                ssum[wv][ln.lig] = sum[i];
            }
            __syncthreads();
            float m = smx[0][ln.lig];
            double t = ssum[0][ln.lig];
            for (int k = 1; k < HUB_WAVES; ++k) {
                if (!BWD) softmax_merge(m, t, smx[k][ln.lig], ssum[k][ln.lig]);
                else t += ssum[k][ln.lig];
            }
            mx[i] = m;
            sum[i] = t;
        }
        if constexpr (KC > 0) softmax_pass_write_cached<T, VEC, KC>(A, b, e, start, stride, col0, active, mx, sum, BWD, rc);
        else softmax_pass_write<T, VEC>(A, b, e, start, stride, col0, active, mx, sum, BWD);
    }
}

hipError_t launch_softmax(const EngineArgs& a, int dtype, int vec, bool backward, hipStream_t s) {
    const int64_t rest = (int64_t)a.sch.w_small_end - a.sch.n_seg;  // waves after the hub segments
    // a block per hub row, then the other rows
    auto run = [&](auto tv, auto vv, auto bv) {
        using T = decltype(tv);
        constexpr int V = decltype(vv)::value;
        constexpr bool B = decltype(bv)::value;
        if (a.sch.n_hub > 0)
            hipLaunchKernelGGL((softmax_hub_kernel<T, V, B>), dim3(a.sch.n_hub), dim3(WAVE * HUB_WAVES), 0, s, a);
        if (rest > 0) hipLaunchKernelGGL((softmax_kernel<T, V, B>), dim3(blocks_for_waves(rest)), dim3(WAVE * WPB), 0, s, a);
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
