// Fused graph attention: the u_add_v -> leaky ReLU -> edge softmax ->
// u_mul_e/sum chain (the multi-head attention layer of Appendix D, written
// there as a g-SDDMM followed by a g-SpMM) in one pass over each
// destination's in-edges:
//
//   s_e = leaky(el[u, h] + er[v, h])            (two single fp32 operations)
//   out[v, h, :] = sum_e exp(s_e - m) feat[u, h, :] / sum_e exp(s_e - m)
//
// with m the running maximum of s over the edges seen so far: when m grows,
// the fp64 sums so far are rescaled by exp(m_old - m_new) (online softmax),
// so no edge tensor is read or written between the steps.  Optionally the
// attention a_e = exp(s_e - m) / sum is written (the softmax output the
// backward pass needs), by a second walk over the row once m and the sum
// are final.  Rows use the degree-sorted roles of the row engine; hub rows
// leave per-segment (m, sum, acc) partials merged in segment order.
#include "walk.h"

namespace gnnk {

struct GatArgs {
    const void* er;       // (N_dst, H) per-head destination score
    int64_t er_stride;
    void* attn;           // (E, H) attention out, nullable
    int64_t attn_stride;
    float slope;
    int32_t pad;
    void* row_ml;         // hub rows: final (m, sum) per column, 2 x D doubles per hub row
};

// online state of one lane for its VEC columns
template <int VEC>
struct Online {
    float m;
    double l;
    double acc[VEC];
    __device__ __forceinline__ void init() {
        m = -INFINITY;
        l = 0.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
    }
    // add one edge with score s and source row x
    __device__ __forceinline__ void add(float s, const float* x) {
        const float mn = fmaxf(m, s);
        const double f = (double)exp_le0(fminf(m, s) - mn);
        const bool up = s > m;
        const double c_old = up ? f : 1.0;
        const double c_new = up ? 1.0 : f;
        l = l * c_old + c_new;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = acc[i] * c_old + c_new * (double)x[i];
        m = mn;
    }
    // merge another state (in segment or lane-group order)
    __device__ __forceinline__ void merge(float om, double ol, const double* oacc) {
        const float mn = fmaxf(m, om);
        const double f1 = m == -INFINITY ? 0.0 : (double)exp_le0(m - mn);
        const double f2 = om == -INFINITY ? 0.0 : (double)exp_le0(om - mn);
        l = l * f1 + ol * f2;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = acc[i] * f1 + oacc[i] * f2;
        m = mn;
    }
};

template <typename T>
__device__ __forceinline__ float gat_score(float el, float er, float slope) {
    const float s = el + er;
    return s > 0.0f ? s : slope * s;
}

template <typename T, int VEC>
__device__ __forceinline__ float load_er(const GatArgs& G, int32_t v, int h) {
    return IO<T, VEC>::load1(reinterpret_cast<const T*>(G.er) + (uint64_t)(uint32_t)v * (uint32_t)G.er_stride + h);
}

// write a_e for the edges b + start, b + start + stride, ... < e of a row,
// given the final (m, sum) of the lane's head (one writer lane per head)
template <typename T, int VEC>
__device__ __forceinline__ void gat_write_attn(const EngineArgs& A, const GatArgs& G, int64_t b64, int64_t e64,
                                               int64_t start, int stride, int lig, int h, bool active, float er_h,
                                               float m, double l) {
    const int per_head = A.geo.F / VEC;  // lanes of one head
    const bool writer = active & (lig % per_head == 0);
    const int32_t b = (int32_t)b64, e = (int32_t)e64;
    const T* el = reinterpret_cast<const T*>(A.b.data);
    T* out = reinterpret_cast<T*>(G.attn);
    const float inv = (float)(1.0 / l);
    for (int32_t p0 = b + (int32_t)start; p0 < e; p0 += stride * UNR) {
        int32_t nb[UNR], ed[UNR], ps[UNR];
        bool ok[UNR];
        batch_ids(A.csr, b, e, p0, stride, ok, nb, ed, ps);
        float x[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u)
            x[u] = IO<T, 1>::load1(el + (uint64_t)(uint32_t)nb[u] * (uint32_t)A.b.stride + h);
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const float s = gat_score<T>(x[u], er_h, G.slope);
            if (ok[u] & writer)
                IO<T, 1>::store1(out + (uint64_t)(uint32_t)ed[u] * (uint32_t)G.attn_stride + h,
                                 exp_le0(s - m) * inv);
        }
    }
}

template <typename T, int VEC, class S, bool ATTN>
__global__ __launch_bounds__(256) void gat_kernel(EngineArgs A, GatArgs G) {
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int Gn = S::GC > 0 ? S::GC : geo.G;
    const int L = WAVE / Gn;
    const int64_t D = (int64_t)geo.NV * VEC;

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
        r = uniform64(r);
        b = uniform64(b);
        e = uniform64(e);
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            const float er_h = load_er<T, VEC>(G, (int32_t)r, h);
            Online<VEC> st;
            st.init();
            Pre<VEC> pre;
            auto sink = [&](const Raw<VEC>& rw, int32_t, int32_t, bool ok) {
                if (ok) st.add(gat_score<T>(rw.b[0], er_h, G.slope), rw.a);
            };
            walk_row<T, VEC, 1, EXT_NONE, S>(A, (int32_t)r, b, e, ln.g, Gn, col0, h, pre, sink);
            for (int s = L; s < WAVE; s <<= 1) {
                double oacc[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) oacc[i] = shfl_xor_d(st.acc[i], s);
                st.merge(__shfl_xor(st.m, s, WAVE), shfl_xor_d(st.l, s), oacc);
            }
            if (slot >= 0) {
                if (ln.g == 0 && active) {
                    double* P = reinterpret_cast<double*>(A.partial) + (int64_t)slot * 3 * D;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) {
                        P[col0 + i] = (double)st.m;
                        P[D + col0 + i] = st.l;
                        P[2 * D + col0 + i] = st.acc[i];
                    }
                }
            } else {
                if (ln.g == 0 && active) {
                    float v[VEC];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) v[i] = (float)(st.acc[i] / st.l);
                    IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + col0, v);
                }
                if constexpr (ATTN) gat_write_attn<T, VEC>(A, G, b, e, ln.g, Gn, ln.lig, h, active, er_h, st.m, st.l);
            }
        }
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * Gn + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            r = A.csr.perm[k];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        const int32_t self = r >= 0 ? (int32_t)r : 0;
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            const float er_h = r >= 0 ? load_er<T, VEC>(G, self, h) : 0.0f;
            Online<VEC> st;
            st.init();
            Pre<VEC> pre;
            auto sink = [&](const Raw<VEC>& rw, int32_t, int32_t, bool ok) {
                if (ok) st.add(gat_score<T>(rw.b[0], er_h, G.slope), rw.a);
            };
            walk_lane<T, VEC, 1, EXT_NONE, S>(A, self, b, e, col0, h, pre, sink);
            if (r >= 0 && active) {
                float v[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[i] = (float)(st.acc[i] / st.l);
                IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + col0, v);
            }
            if constexpr (ATTN)
                if (r >= 0) gat_write_attn<T, VEC>(A, G, b, e, 0, 1, ln.lig, h, active, er_h, st.m, st.l);
        }
    } else {
        // empty rows: no edge, output 0
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * Gn + ln.g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * L + ln.lig;
                if (j < geo.NV && r >= 0) {
                    float v[VEC];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) v[i] = 0.0f;
                    IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + j * VEC, v);
                }
            }
        }
    }
}

// hub rows: merge the segment partials in order and write the row; keep the
// row's final (m, sum) for the attention writes
template <typename T, int VEC>
__global__ __launch_bounds__(256) void gat_combine_kernel(EngineArgs A, GatArgs G) {
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
    const double* P = reinterpret_cast<const double*>(A.partial);
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV && row_ok;
        const int col0 = active ? j * VEC : 0;
        if (!active) continue;
        Online<VEC> st;
        st.init();
        for (int s = s0; s < s1; ++s) {
            const double* Q = P + (int64_t)s * 3 * D;
            double oacc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) oacc[i] = Q[2 * D + col0 + i];
            st.merge((float)Q[col0], Q[D + col0], oacc);
        }
        float v[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = (float)(st.acc[i] / st.l);
        IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + r * A.out.stride + col0, v);
        if (G.attn) {
            double* ML = reinterpret_cast<double*>(G.row_ml) + k * 2 * D;
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                ML[col0 + i] = (double)st.m;
                ML[D + col0 + i] = st.l;
            }
        }
    }
}

// hub rows with attention out: each segment writes its edges' a_e
template <typename T, int VEC>
__global__ __launch_bounds__(256) void gat_attn_segments_kernel(EngineArgs A, GatArgs G) {
    const int w = wave_id();
    if (w >= A.sch.n_seg) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    const int64_t D = (int64_t)geo.NV * VEC;
    const int4 sg = A.csr.seg[w];
    const double* ML = reinterpret_cast<const double*>(G.row_ml) + (int64_t)sg.w * 2 * D;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        const float er_h = load_er<T, VEC>(G, sg.x, h);
        gat_write_attn<T, VEC>(A, G, sg.y, sg.z, ln.g, geo.G, ln.lig, h, active, er_h, (float)ML[col0],
                               ML[D + col0]);
    }
}

namespace {

template <typename T, int V, bool ATTN>
void gat_launch_t(const EngineArgs& a, const GatArgs& g, int gc, hipStream_t s) {
    const dim3 grid(blocks_for_waves(a.sch.w_total)), block(WAVE * WPB);
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        if (gc > 0) {
            GNNK_GC_DISPATCH(gc, {
                hipLaunchKernelGGL((gat_kernel<T, V, Spec<T_NBR, OK_FULL, T_NBR, OK_HEAD, C, false>, ATTN>), grid,
                                   block, 0, s, a, g);
            })
            return;
        }
    }
    hipLaunchKernelGGL((gat_kernel<T, V, Spec<T_NBR, OK_FULL, T_NBR, OK_HEAD, 0, false>, ATTN>), grid, block, 0, s,
                       a, g);
}

template <typename T, int V>
void gat_all(const EngineArgs& a, const GatArgs& g, int gc, hipStream_t s) {
    if (g.attn) gat_launch_t<T, V, true>(a, g, gc, s);
    else gat_launch_t<T, V, false>(a, g, gc, s);
    if (a.sch.n_hub > 0) {
        const dim3 block(WAVE * WPB);
        const dim3 cgrid(blocks_for_waves((a.sch.n_hub + a.geo.G - 1) / a.geo.G));
        hipLaunchKernelGGL((gat_combine_kernel<T, V>), cgrid, block, 0, s, a, g);
        if (g.attn)
            hipLaunchKernelGGL((gat_attn_segments_kernel<T, V>), dim3(blocks_for_waves(a.sch.n_seg)), block, 0, s,
                               a, g);
    }
}

}  // namespace

hipError_t launch_gat(const EngineArgs& a, const void* er, int64_t er_stride, void* attn, int64_t attn_stride,
                      float slope, void* row_ml, int dtype, int vec, int gc, hipStream_t s) {
    if (a.sch.w_total <= 0) return hipSuccess;
    GatArgs g{er, er_stride, attn, attn_stride, slope, 0, row_ml};
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, gat_all<float, V>(a, g, gc, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, gat_all<bf16_t, V>(a, g, gc, s))
    }
    return hipGetLastError();
}

}  // namespace gnnk
