// Fused graph attention: the u_add_v -> leaky ReLU -> edge softmax ->
// u_mul_e/sum chain (the multi-head attention layer of Appendix E, written
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
    float* stats;         // (N_dst, H, 2) fp32: max score and 1 / sum per head, nullable
    int64_t stats_stride;
};

// the per-head statistics of a destination row: the max score and the
// reciprocal of the sum of exp(score - max), rounded to fp32 as the
// attention written by this kernel uses it
__device__ __forceinline__ void gat_write_stats(const GatArgs& G, int64_t row, int h, float m, double l) {
    if (!G.stats) return;
    float* p = G.stats + row * G.stats_stride + 2 * h;
    p[0] = l > 0.0 ? m : 0.0f;
    p[1] = l > 0.0 ? (float)(1.0 / l) : 0.0f;
}

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
        // a score of -inf adds nothing; while the running max is still -inf
        // too, -inf - (-inf) would give NaN
        const float mn = fmaxf(m, s);
        const double f = mn == -INFINITY ? 0.0 : (double)exp_le0(fminf(m, s) - mn);
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
            const int4 s = A.csr.segw[w];
            r = s.x; b = s.y; e = s.z; slot = s.w;
        } else {
            const int4 t = A.csr.rowt[A.sch.n_hub + (w - A.sch.n_seg)];
            r = t.x; b = t.y; e = t.z;
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
                    if (col0 % geo.F == 0) gat_write_stats(G, r, h, st.m, st.l);
                }
                if constexpr (ATTN) gat_write_attn<T, VEC>(A, G, b, e, ln.g, Gn, ln.lig, h, active, er_h, st.m, st.l);
            }
        }
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * Gn + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
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
                if (col0 % geo.F == 0) gat_write_stats(G, r, h, st.m, st.l);
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
                    if ((j * VEC) % geo.F == 0) gat_write_stats(G, r, (j * VEC) / geo.F, 0.0f, 0.0);
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
        if (col0 % geo.F == 0) gat_write_stats(G, r, col0 / geo.F, st.m, st.l);
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
    const int4 sg = A.csr.seg[A.csr.seg_order[w]];
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

// ---------------------------------------------------------------------------
// backward of the fused attention
//
// With s_e = leaky(el[u] + er[v]) per head, a_e = softmax over the in-edges
// of v of s_e, and out[v] = sum over in-edges of a_e feat[u] (per head):
//   da_e      = dZ[v] . feat[u]                        (per head)
//   ds_e      = a_e (da_e - S_v) lk_e                  lk_e = leaky'(el[u] + er[v])
//   S_v       = sum_in a_e da_e
//   d_er[v]   = sum_in ds_e = P_v - S_v Q_v           P_v = sum_in a_e da_e lk_e, Q_v = sum_in a_e lk_e
//   d_el[u]   = sum_out ds_e
//   d_feat[u] = sum_out a_e dZ[v]
// (the chain rule through the four steps, Theorem 1's gradients of g-SpMM
// and g-SDDMM).  a_e is recomputed from the forward's per-row max and
// 1 / sum, so no tensor of E x H elements is read or written.  Pass A walks
// the in-CSR: S, P, Q per destination and head in fp64, d_er, and a record
// {er, max, 1 / sum, S} per (destination, head) for pass B.  Pass B walks the
// reverse graph's CSR and gathers dZ[v] and that record per edge.


// sum of a per-lane value over the `red` lanes of one head (aligned runs in
// the lane group); the total is exact in the head's first lane
__device__ __forceinline__ double head_sum(double v, int lig, int red) {
    return (red & (red - 1)) == 0 ? run_sum(v, red) : seg_sum(v, lig, red);
}

// head_sum with the lanes per head fixed at compile time (RED > 0: a power
// of two, no per-step branches) or read at run time (RED = 0)
template <int RED>
__device__ __forceinline__ double head_sum_t(double v, int lig, int red) {
    if constexpr (RED > 0) return run_sum_c<RED>(v);
    else return head_sum(v, lig, red);
}

// the attention of one edge, recomputed as the forward computes it
__device__ __forceinline__ float gat_attention(float el, float er, float slope, float m, float il, bool& pos) {
    const float s = el + er;
    pos = s > 0.0f;
    return exp_le0((pos ? s : slope * s) - m) * il;
}

template <typename T>
__device__ __forceinline__ void gat_finish_dst(const GatBwdArgs& B, int64_t v, int h, float er_h, float m, float il,
                                               double S, double P, double Q) {
    if (B.chunk) {
        // S and P of this column chunk: stored by the first, added by the
        // others in chunk order; Q does not depend on the columns
        double* ac = B.acc_dst + (v * B.H + h) * 2;
        if (B.chunk > 1) {
            S += ac[0];
            P += ac[1];
        }
        if (B.chunk < 3) {
            ac[0] = S;
            ac[1] = P;
            return;
        }
    }
    if (B.d_er) IO<T, 1>::store1(reinterpret_cast<T*>(B.d_er) + v * B.d_er_stride + h, (float)(P - S * Q));
    B.rec[v * B.H + h] = make_float4(er_h, m, il, (float)S);
}

// pass A: one destination row (a hub segment, a row by the wavefront, or a
// row by this lane group)
template <typename T, int VEC, class S, bool WAVE_ROW, int RED>
__device__ __forceinline__ void gat_bwd_dst_row(const EngineArgs& A, const GatBwdArgs& B, const Lanes& ln, int Gn,
                                                int64_t r, int64_t b, int64_t e, int slot) {
    const GeomDev& geo = A.geo;
    const int L = WAVE / Gn;
    const int red = RED > 0 ? RED : geo.F / VEC;
    const bool active = ln.lig < geo.NV;
    const int col0 = active ? ln.lig * VEC : 0;
    const int h = col0 / geo.F;
    const bool head_lane = active && (col0 % geo.F) == 0;
    const int32_t self = r >= 0 ? (int32_t)r : 0;
    float dz[VEC];
    IO<T, VEC>::load(reinterpret_cast<const T*>(B.dz) + (int64_t)self * B.dz_stride + col0, dz);
    double dzd[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) dzd[i] = dz[i];
    const float er_h = IO<T, 1>::load1(reinterpret_cast<const T*>(B.er) + (int64_t)self * B.er_stride + h);
    const float m = B.stats[(int64_t)self * B.stats_stride + 2 * h];
    const float il = B.stats[(int64_t)self * B.stats_stride + 2 * h + 1];
    double sS = 0.0, sP = 0.0, sQ = 0.0;
    Pre<VEC> pre;
    auto sink = [&](const Raw<VEC>& rw, int32_t, int32_t, bool ok) {
        bool pos;
        const double a = gat_attention(rw.b[0], er_h, B.slope, m, il, pos);
        double dp = 0.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) dp = fma((double)rw.a[i], dzd[i], dp);
        const double da = head_sum_t<RED>(dp, ln.lig, red);
        const double lk = pos ? 1.0 : (double)B.slope;
        const double ad = a * da;
        sS += ok ? ad : 0.0;
        sP += ok ? ad * lk : 0.0;
        sQ += ok ? a * lk : 0.0;
    };
    if constexpr (WAVE_ROW) {
        walk_row<T, VEC, 1, EXT_NONE, S>(A, self, b, e, ln.g, Gn, col0, h, pre, sink);
        for (int s = L; s < WAVE; s <<= 1) {
            sS += shfl_xor_d(sS, s);
            sP += shfl_xor_d(sP, s);
            sQ += shfl_xor_d(sQ, s);
        }
        if (ln.g != 0 || !head_lane) return;
        if (slot >= 0) {
            double* p = B.part + (int64_t)slot * 3 * B.H;
            p[h] = sS;
            p[B.H + h] = sP;
            p[2 * B.H + h] = sQ;
        } else {
            gat_finish_dst<T>(B, r, h, er_h, m, il, sS, sP, sQ);
        }
    } else {
        walk_lane<T, VEC, 1, EXT_NONE, S>(A, self, b, e, col0, h, pre, sink);
        if (r >= 0 && head_lane) gat_finish_dst<T>(B, r, h, er_h, m, il, sS, sP, sQ);
    }
}

template <typename T, int VEC, class S, int RED>
__global__ __launch_bounds__(256) void gat_bwd_dst_kernel(EngineArgs A, GatBwdArgs B) {
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int Gn = S::GC > 0 ? S::GC : geo.G;
    if (w < A.sch.w_big_end) {
        int64_t r, b, e;
        int slot = -1;
        if (w < A.sch.n_seg) {
            const int4 sg = A.csr.segw[w];
            r = sg.x; b = sg.y; e = sg.z; slot = sg.w;
        } else {
            const int4 t = A.csr.rowt[A.sch.n_hub + (w - A.sch.n_seg)];
            r = t.x; b = t.y; e = t.z;
        }
        gat_bwd_dst_row<T, VEC, S, true, RED>(A, B, ln, Gn, uniform64(r), uniform64(b), uniform64(e), slot);
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * Gn + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
        }
        gat_bwd_dst_row<T, VEC, S, false, RED>(A, B, ln, Gn, r, b, e, -1);
    } else if (B.d_er) {
        // rows without in-edges: d_er = 0 (no edge reads their record)
        const int64_t k0 = A.sch.n_nz + ((int64_t)(w - A.sch.w_small_end) * Gn + ln.g) * A.sch.fill_rows_per_group;
        const int col0 = ln.lig * VEC;
        if (ln.lig < geo.NV && col0 % geo.F == 0) {
            for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
                const int64_t k = k0 + q;
                if (k < A.sch.n_rows)
                    IO<T, 1>::store1(reinterpret_cast<T*>(B.d_er) + (int64_t)A.csr.perm[k] * B.d_er_stride +
                                         col0 / geo.F, 0.0f);
            }
        }
    }
}

// pass A, hub rows: one thread per (hub row, head), segments in order
template <typename T>
__global__ __launch_bounds__(256) void gat_bwd_dst_combine_kernel(EngineArgs A, GatBwdArgs B) {
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int64_t k = t / B.H;
    const int h = (int)(t % B.H);
    if (k >= A.sch.n_hub) return;
    const int64_t r = A.csr.perm[k];
    const int s0 = A.csr.hub_off[k], s1 = A.csr.hub_off[k + 1];
    double sS = 0.0, sP = 0.0, sQ = 0.0;
    for (int s = s0; s < s1; ++s) {
        const double* p = B.part + (int64_t)s * 3 * B.H;
        sS += p[h];
        sP += p[B.H + h];
        sQ += p[2 * B.H + h];
    }
    const float er_h = IO<T, 1>::load1(reinterpret_cast<const T*>(B.er) + r * B.er_stride + h);
    const float m = B.stats[r * B.stats_stride + 2 * h];
    const float il = B.stats[r * B.stats_stride + 2 * h + 1];
    gat_finish_dst<T>(B, r, h, er_h, m, il, sS, sP, sQ);
}

// pass B: the out-edges [b, e) of one source row, positions b + start,
// b + start + stride, ...; the next batch's destination ids load while this
// batch's gathers are in flight
template <typename T, int VEC, class F>
__device__ __forceinline__ void gat_walk_out(const EngineArgs& A, const GatBwdArgs& B, int64_t b64, int64_t e64,
                                             int64_t start, int stride, int col0, int h, F& consume) {
    const int32_t b = (int32_t)b64, e = (int32_t)e64;
    const int32_t step = stride * UNR;
    int32_t p0 = b + (int32_t)start;
    if (p0 >= e) return;
    int32_t nb[UNR];
    bool ok[UNR];
    auto ids = [&](int32_t q0) {
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int32_t p = q0 + u * stride;
            ok[u] = p < e;
            nb[u] = A.csr.idx[ok[u] ? p : b];
        }
    };
    ids(p0);
    const T* dz = reinterpret_cast<const T*>(B.dz);
    for (; p0 < e; p0 += step) {
        float z[UNR][VEC];
        float4 rc[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            IO<T, VEC>::load(dz + (int64_t)nb[u] * B.dz_stride + col0, z[u]);
            rc[u] = B.rec[(int64_t)nb[u] * B.H + h];
        }
        bool okc[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) okc[u] = ok[u];
        ids(p0 + step);
#pragma unroll
        for (int u = 0; u < UNR; ++u) consume(z[u], rc[u], okc[u]);
    }
}

template <typename T, int VEC>
__device__ __forceinline__ void gat_write_src(const GatBwdArgs& B, int64_t u, int col0, int h, bool active,
                                              bool head_lane, const double* df, double dl) {
    if (B.d_feat && active) {
        float v[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = (float)df[i];
        IO<T, VEC>::store(reinterpret_cast<T*>(B.d_feat) + u * B.d_feat_stride + col0, v);
    }
    if (B.d_el && head_lane) {
        if (B.chunk) {
            // this column chunk's share of d_el, added in chunk order
            double* ac = B.acc_src + u * B.H + h;
            if (B.chunk > 1) dl += *ac;
            if (B.chunk < 3) {
                *ac = dl;
                return;
            }
        }
        IO<T, 1>::store1(reinterpret_cast<T*>(B.d_el) + u * B.d_el_stride + h, (float)dl);
    }
}

// pass B: one source row (a hub segment, a row by the wavefront, or a row by
// this lane group)
template <typename T, int VEC, bool WAVE_ROW, int RED>
__device__ __forceinline__ void gat_bwd_src_row(const EngineArgs& A, const GatBwdArgs& B, const Lanes& ln,
                                                int64_t r, int64_t b, int64_t e, int slot) {
    const GeomDev& geo = A.geo;
    const int red = RED > 0 ? RED : geo.F / VEC;
    const bool active = ln.lig < geo.NV;
    const int col0 = active ? ln.lig * VEC : 0;
    const int h = col0 / geo.F;
    const bool head_lane = active && (col0 % geo.F) == 0;
    const int64_t self = r >= 0 ? r : 0;
    float x[VEC];
    IO<T, VEC>::load(reinterpret_cast<const T*>(B.feat) + self * B.feat_stride + col0, x);
    double xd[VEC], df[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
        xd[i] = x[i];
        df[i] = 0.0;
    }
    const float el_h = IO<T, 1>::load1(reinterpret_cast<const T*>(B.el) + self * B.el_stride + h);
    double dl = 0.0;
    // d_el = sum of a (da - S) lk: a head in column chunks adds the a S lk
    // part with its first chunk only (da is summed chunk by chunk)
    const bool with_s = B.chunk <= 1;
    auto sink = [&](const float* z, const float4& rc, bool ok) {
        bool pos;
        const double a = gat_attention(el_h, rc.x, B.slope, rc.y, rc.z, pos);
        double dp = 0.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) dp = fma((double)z[i], xd[i], dp);
        const double da = head_sum_t<RED>(dp, ln.lig, red);
        const double lk = pos ? 1.0 : (double)B.slope;
        const double ak = ok ? a : 0.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) df[i] = fma(ak, (double)z[i], df[i]);
        dl += ak * (da - (with_s ? (double)rc.w : 0.0)) * lk;
    };
    if constexpr (WAVE_ROW) {
        const int L = geo.L;
        gat_walk_out<T, VEC>(A, B, b, e, ln.g, geo.G, col0, h, sink);
        for (int s = L; s < WAVE; s <<= 1) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) df[i] += shfl_xor_d(df[i], s);
            dl += shfl_xor_d(dl, s);
        }
        if (ln.g != 0) return;
        if (slot >= 0) {
            const int64_t D = (int64_t)geo.NV * VEC;
            double* p = B.part + (int64_t)slot * (D + B.H);
            if (active) {
#pragma unroll
                for (int i = 0; i < VEC; ++i) p[col0 + i] = df[i];
            }
            if (head_lane) p[D + h] = dl;
        } else {
            gat_write_src<T, VEC>(B, r, col0, h, active, head_lane, df, dl);
        }
    } else {
        gat_walk_out<T, VEC>(A, B, b, e, 0, 1, col0, h, sink);
        if (r >= 0) gat_write_src<T, VEC>(B, r, col0, h, active, head_lane, df, dl);
    }
}

template <typename T, int VEC, int RED>
__global__ __launch_bounds__(256) void gat_bwd_src_kernel(EngineArgs A, GatBwdArgs B) {
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    if (w < A.sch.w_big_end) {
        int64_t r, b, e;
        int slot = -1;
        if (w < A.sch.n_seg) {
            const int4 sg = A.csr.segw[w];
            r = sg.x; b = sg.y; e = sg.z; slot = sg.w;
        } else {
            const int4 t = A.csr.rowt[A.sch.n_hub + (w - A.sch.n_seg)];
            r = t.x; b = t.y; e = t.z;
        }
        gat_bwd_src_row<T, VEC, true, RED>(A, B, ln, uniform64(r), uniform64(b), uniform64(e), slot);
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
        }
        gat_bwd_src_row<T, VEC, false, RED>(A, B, ln, r, b, e, -1);
    } else {
        // sources without out-edges: zero gradients
        const int64_t k0 = A.sch.n_nz + ((int64_t)(w - A.sch.w_small_end) * geo.G + ln.g) * A.sch.fill_rows_per_group;
        const bool active = ln.lig < geo.NV;
        const int col0 = active ? ln.lig * VEC : 0;
        const double zero[VEC] = {};
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            if (k < A.sch.n_rows)
                gat_write_src<T, VEC>(B, A.csr.perm[k], col0, col0 / geo.F, active, active && col0 % geo.F == 0,
                                      zero, 0.0);
        }
    }
}

// pass B, hub rows: partials of the row's segments summed in order
template <typename T, int VEC>
__global__ __launch_bounds__(256) void gat_bwd_src_combine_kernel(EngineArgs A, GatBwdArgs B) {
    const int w = wave_id();
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    if ((int64_t)w * geo.G >= A.sch.n_hub) return;
    const int64_t k = (int64_t)w * geo.G + ln.g;
    if (k >= A.sch.n_hub) return;
    const int64_t r = A.csr.perm[k];
    const int s0 = A.csr.hub_off[k], s1 = A.csr.hub_off[k + 1];
    const int64_t D = (int64_t)geo.NV * VEC;
    const bool active = ln.lig < geo.NV;
    const int col0 = active ? ln.lig * VEC : 0;
    const int h = col0 / geo.F;
    const bool head_lane = active && (col0 % geo.F) == 0;
    double df[VEC], dl = 0.0;
#pragma unroll
    for (int i = 0; i < VEC; ++i) df[i] = 0.0;
    for (int s = s0; s < s1; ++s) {
        const double* p = B.part + (int64_t)s * (D + B.H);
#pragma unroll
        for (int i = 0; i < VEC; ++i) df[i] += p[col0 + i];
        dl += p[D + h];
    }
    gat_write_src<T, VEC>(B, r, col0, h, active, head_lane, df, dl);
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

template <typename T, int V, int RED>
void gat_bwd_red(const EngineArgs& ain, const EngineArgs& aout, const GatBwdArgs& B, int gc, hipStream_t s) {
    const dim3 block(WAVE * WPB);
    if ((B.passes & 1) && ain.sch.w_total > 0) {
        const dim3 grid(blocks_for_waves(ain.sch.w_total));
        bool done = false;
        if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
            if (gc > 0) {
                GNNK_GC_DISPATCH(gc, {
                    hipLaunchKernelGGL((gat_bwd_dst_kernel<T, V, Spec<T_NBR, OK_FULL, T_NBR, OK_HEAD, C, false>, RED>),
                                       grid, block, 0, s, ain, B);
                })
                done = true;
            }
        }
        if (!done)
            hipLaunchKernelGGL((gat_bwd_dst_kernel<T, V, Spec<T_NBR, OK_FULL, T_NBR, OK_HEAD, 0, false>, RED>), grid,
                               block, 0, s, ain, B);
        if (ain.sch.n_hub > 0) {
            const int64_t n = (int64_t)ain.sch.n_hub * B.H;
            hipLaunchKernelGGL((gat_bwd_dst_combine_kernel<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                               ain, B);
        }
    }
    if ((B.passes & 2) && aout.sch.w_total > 0 && (B.d_feat || B.d_el)) {
        hipLaunchKernelGGL((gat_bwd_src_kernel<T, V, RED>), dim3(blocks_for_waves(aout.sch.w_total)), block, 0, s,
                           aout, B);
        if (aout.sch.n_hub > 0)
            hipLaunchKernelGGL((gat_bwd_src_combine_kernel<T, V>),
                               dim3(blocks_for_waves((aout.sch.n_hub + aout.geo.G - 1) / aout.geo.G)), block, 0, s,
                               aout, B);
    }
}

// both passes with the lanes per head (F / V) as a compile-time constant
// when it is 2-16, else read at run time
template <typename T, int V>
void gat_bwd_all(const EngineArgs& ain, const EngineArgs& aout, const GatBwdArgs& B, int gc, hipStream_t s) {
    switch (ain.geo.F / V) {
        case 2: gat_bwd_red<T, V, 2>(ain, aout, B, gc, s); return;
        case 4: gat_bwd_red<T, V, 4>(ain, aout, B, gc, s); return;
        case 8: gat_bwd_red<T, V, 8>(ain, aout, B, gc, s); return;
        case 16: gat_bwd_red<T, V, 16>(ain, aout, B, gc, s); return;
        default: gat_bwd_red<T, V, 0>(ain, aout, B, gc, s); return;
    }
}

}  // namespace

hipError_t launch_gat(const EngineArgs& a, const void* er, int64_t er_stride, void* attn, int64_t attn_stride,
                      float slope, void* row_ml, float* stats, int64_t stats_stride, int dtype, int vec, int gc,
                      hipStream_t s) {
    if (a.sch.w_total <= 0) return hipSuccess;
    GatArgs g{er, er_stride, attn, attn_stride, slope, 0, row_ml, stats, stats_stride};
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, gat_all<float, V>(a, g, gc, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, gat_all<bf16_t, V>(a, g, gc, s))
    }
    return hipGetLastError();
}

hipError_t launch_gat_backward(const EngineArgs& ain, const EngineArgs& aout, const GatBwdArgs& b, int dtype, int vec,
                               int gc, hipStream_t s) {
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, gat_bwd_all<float, V>(ain, aout, b, gc, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, gat_bwd_all<bf16_t, V>(ain, aout, b, gc, s))
    }
    return hipGetLastError();
}

}  // namespace gnnk
