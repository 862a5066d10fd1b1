// g-SDDMM kernel (Section 3, definition of generalized SDDMM): one output per
// edge, op(lhs at its target, rhs at its target).  Edges are walked row by
// row over the in-CSR (rows = destinations) with the degree-sorted schedule,
// so a destination-side operand is read once per destination and hub rows are
// split across wavefronts.  The same kernel computes the edge gradients of
// g-SpMM (the lemma on dL/dW of g-SpMM) and of g-SDDMM.  Elementwise ops are
// single fp32 operations (computed in fp64, rounded once); dot products and
// sums over broadcast positions accumulate in fp64.
#include "walk.h"

namespace gnnk {

// Output of one edge: VEC columns (RM = 0), or the sum over runs of
// out.red lanes (a head for dot, or the whole row): RM = 1 for power-of-two
// runs (DPP within 16-lane rows), RM > 1 for runs of exactly RM lanes known at
// compile time (no per-step branches), RM = -1 reads the mode at run time.  A
// whole-row sum of a row wider than one pass (nchunk > 1: one lane group,
// lane 0 writes every edge) keeps its running fp64 total per edge in xacc
// between passes ch and writes the output in the last one.
template <typename T, int VEC, int OPK, int EXT, int RM, bool WAVE_ROW>
struct SddmmSink {
    const EngineArgs& A;
    int lig, col0, h, ch;
    bool active;

    // Runs of four lanes and batches of four edges per lane group (a per-head
    // dot of 16 fp32 columns): a full batch's four partial sums are reduced
    // and scattered together, a 4 x 4 transpose in two DPP steps after which
    // lane q of a run holds the total of slot q, and one store instruction
    // writes the four outputs.  Per batch that is 3 fp64 additions and 6
    // lane moves per lane instead of 8 and 16, and one store path instead of
    // four (c3 u_dot_v and the d attention pass were bound by VALU issue).
    // The sums pair up as run_sum_c<4> pairs them for each slot, lanes {0, 1}
    // and {2, 3} and then the two pairs, so the results are bit-identical.
    static constexpr bool kBatch = RM == 4 && UNR == 4;

    __device__ __forceinline__ void batch(const Raw<VEC>* rw, const int32_t* ed) {
        double s[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            double m[VEC];
            combine_f64<VEC, OPK, EXT>(A, rw[u], ed[u], m);
            double t = 0.0;
#pragma unroll
            for (int i = 0; i < VEC; ++i) t += m[i];
            s[u] = t;
        }
        // Where the row's vectors come in whole runs of four (per-head dots,
        // rows of a multiple of four vectors) every run is active or inactive
        // as a whole and needs no masking.  A whole-row sum of three vectors
        // (runs of four lanes, the fourth outside the row) zeroes the lane
        // outside the row, whose loads repeat the row's first vector.
        if ((A.geo.NV & 3) != 0) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) s[u] = active ? s[u] : 0.0;
        }
        const int q = lig & 3;
        const bool odd = (q & 1) != 0, hi = (q & 2) != 0;
        // with lane q ^ 1: keep the two slots of q's parity, hand over the others
        const double k0 = (odd ? s[1] : s[0]) + dpp_d<DPP_QUAD_1032>(odd ? s[0] : s[1]);
        const double k1 = (odd ? s[3] : s[2]) + dpp_d<DPP_QUAD_1032>(odd ? s[2] : s[3]);
        // with lane q ^ 2: keep slot q
        const double tot = (hi ? k1 : k0) + dpp_d<DPP_QUAD_2301>(hi ? k0 : k1);
        // slot q's edge by two selects (no branches)
        const int32_t e01 = odd ? ed[1] : ed[0], e23 = odd ? ed[3] : ed[2];
        const int32_t e = hi ? e23 : e01;
        // every lane of a run that holds a vector of the row stores its slot,
        // also a lane outside the row in a partly active run
        const bool run_active = ch * A.geo.L + (lig & ~3) < A.geo.NV;
        if (run_active) {
            T* row = reinterpret_cast<T*>(A.out.data) + (uint64_t)(uint32_t)e * (uint32_t)A.out.stride;
            const bool neg = (A.flags & F_NEGATE) != 0;
            IO<T, VEC>::store1(row + (A.out.per_head ? h : 0), (float)(neg ? -tot : tot));
        }
    }

    __device__ __forceinline__ void operator()(const Raw<VEC>& rw, int32_t ed, int32_t, bool ok) {
        double m[VEC];
        combine_f64<VEC, OPK, EXT>(A, rw, ed, m);
        const bool neg = (A.flags & F_NEGATE) != 0;
        T* row = reinterpret_cast<T*>(A.out.data) + (uint64_t)(uint32_t)ed * (uint32_t)A.out.stride;
        const bool reduce = RM < 0 ? A.out.reduce != 0 : RM > 0;
        if (!reduce) {
            if (ok & active) {
                float v[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[i] = (float)(neg ? -m[i] : m[i]);
                // written once, never read by this kernel: nontemporal vector
                // stores keep the gathered node rows in L2 (c3 u_add_v 1.83 ->
                // 1.59 ms) where the wavefront's lane groups write consecutive
                // edges (whole lines per instruction); a lane group on a row of
                // its own and single-value stores of reduced outputs stay plain
                if constexpr (WAVE_ROW) IO<T, VEC>::store_nt(row + col0, v);
                else IO<T, VEC>::store(row + col0, v);
            }
        } else {
            double s = 0.0;
#pragma unroll
            for (int i = 0; i < VEC; ++i) s += m[i];
            const int red = A.out.red;
            s = active ? s : 0.0;
            if constexpr (RM > 1) s = run_sum_c<RM>(s);
            else if constexpr (RM == 1) s = run_sum(s, red);
            else s = (red & (red - 1)) == 0 ? run_sum(s, red) : seg_sum(s, lig, red);
            const bool writer = RM > 1 ? ((lig & (RM - 1)) == 0)
                                       : (RM == 1 ? ((lig & (red - 1)) == 0) : ((lig % red) == 0));
            // (runtime-layout kernels only: the host picks them for such rows)
            if (RM < 0 && A.geo.nchunk > 1 && (ok & active & writer)) {
                double* x = A.xacc + (uint32_t)ed;
                if (ch > 0) s += *x;
                if (ch + 1 < A.geo.nchunk) {
                    *x = s;
                    return;
                }
            }
            if (ok & active & writer) {
                const int o = A.out.per_head ? h : 0;
                IO<T, VEC>::store1(row + o, (float)(neg ? -s : s));
            }
        }
    }
};

// the edges of one row: by the whole wavefront (WAVE_ROW, uniform bounds) or
// by this lane group alone
template <typename T, int VEC, int OPK, int EXT, int RM, class S, bool WAVE_ROW>
__device__ __forceinline__ void sddmm_row(const EngineArgs& A, const Lanes& ln, int G, int L, int64_t r, int64_t b,
                                          int64_t e) {
    const GeomDev& geo = A.geo;
    const int32_t self = r >= 0 ? (int32_t)r : 0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        Pre<VEC> pre;
        if (r >= 0) load_pre<T, VEC, OPK, S>(A, self, col0, h, pre);
        SddmmSink<T, VEC, OPK, EXT, RM, WAVE_ROW> sink{A, ln.lig, col0, h, ch, active};
        if constexpr (WAVE_ROW) walk_row<T, VEC, OPK, EXT, S>(A, self, b, e, ln.g, G, col0, h, pre, sink);
        else walk_lane<T, VEC, OPK, EXT, S>(A, self, b, e, col0, h, pre, sink);
    }
}

template <typename T, int VEC, int OPK, int EXT, int RM, class S>
__global__ __launch_bounds__(256) void sddmm_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.w_small_end) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int G = S::GC > 0 ? S::GC : geo.G;
    const int L = WAVE / G;
    if (w < A.sch.w_big_end) {
        int64_t r, b, e;
        const int ks = A.sch.seg_split > 1 ? A.sch.seg_split : 1;
        const int nsw = A.sch.n_seg * ks;  // hub-segment wavefronts
        if (w < nsw) {
            const int4 s = A.csr.segw[w / ks];
            r = s.x; b = s.y; e = s.z;
            if (ks > 1) {
                // part w % ks of the segment, cut at whole batches
                const int64_t nbt = (int64_t)G * ENGINE_UNR;
                const int64_t step = ((e - b + ks - 1) / ks + nbt - 1) / nbt * nbt;
                const int64_t b2 = b + (int64_t)(w % ks) * step;
                b = b2 < e ? b2 : e;
                e = b2 + step < e ? b2 + step : e;
            }
        } else {
            const int4 t = A.csr.rowt[A.sch.n_hub + (w - nsw)];
            r = t.x; b = t.y; e = t.z;
        }
        sddmm_row<T, VEC, OPK, EXT, RM, S, true>(A, ln, G, L, uniform64(r), uniform64(b), uniform64(e));
    } else {
        int64_t r = -1, b = 0, e = 0;
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * G + ln.g;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
        }
        sddmm_row<T, VEC, OPK, EXT, RM, S, false>(A, ln, G, L, r, b, e);
    }
}

namespace {

template <int C>
using SpUV = Spec<T_NBR, OK_FULL, T_SELF, OK_FULL, C, false>;
template <int C>
using SpVU = Spec<T_SELF, OK_FULL, T_NBR, OK_FULL, C, false>;

template <typename T, int V, int C, int R>
void launch_sddmm_rm(const EngineArgs& a, int spec, dim3 grid, dim3 block, hipStream_t s) {
    if (spec == SP_VU) hipLaunchKernelGGL((sddmm_kernel<T, V, 1, EXT_NONE, R, SpVU<C>>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((sddmm_kernel<T, V, 1, EXT_NONE, R, SpUV<C>>), grid, block, 0, s, a);
}

// red: lanes per reduced output (0: no reduction); a run of 2-64 lanes that
// fits the lane group is a compile-time constant of the kernel
template <typename T, int V, int C>
void launch_sddmm_fast(const EngineArgs& a, int opk, int spec, int red, dim3 grid, dim3 block, hipStream_t s) {
    if (spec != SP_VU && opk != 1) {
        hipLaunchKernelGGL((sddmm_kernel<T, V, 2, EXT_NONE, 0, SpUV<C>>), grid, block, 0, s, a);
        return;
    }
    constexpr int L = 64 / C;
    switch (red) {
        case 0: launch_sddmm_rm<T, V, C, 0>(a, spec, grid, block, s); return;
        case 2: if constexpr (L >= 2) { launch_sddmm_rm<T, V, C, 2>(a, spec, grid, block, s); return; } break;
        case 4: if constexpr (L >= 4) { launch_sddmm_rm<T, V, C, 4>(a, spec, grid, block, s); return; } break;
        case 8: if constexpr (L >= 8) { launch_sddmm_rm<T, V, C, 8>(a, spec, grid, block, s); return; } break;
        case 16: if constexpr (L >= 16) { launch_sddmm_rm<T, V, C, 16>(a, spec, grid, block, s); return; } break;
        case 32: if constexpr (L >= 32) { launch_sddmm_rm<T, V, C, 32>(a, spec, grid, block, s); return; } break;
        case 64: if constexpr (L >= 64) { launch_sddmm_rm<T, V, C, 64>(a, spec, grid, block, s); return; } break;
        default: break;
    }
    launch_sddmm_rm<T, V, C, 1>(a, spec, grid, block, s);
}

template <typename T, int V>
void launch_sddmm_t(const EngineArgs& a, int opk, int ext, int spec, int gc, dim3 grid, dim3 block, hipStream_t s) {
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        if (spec == SP_UV || spec == SP_VU) {
            const int red = a.out.reduce ? a.out.red : 0;
            GNNK_GC_DISPATCH(gc, launch_sddmm_fast<T, V, C>(a, opk, spec, red, grid, block, s))
            return;
        }
    }
    GNNK_OPK_DISPATCH(opk, GNNK_EXT3_DISPATCH(ext, {
        hipLaunchKernelGGL((sddmm_kernel<T, V, K, X, -1, SpecDyn>), grid, block, 0, s, a);
    }))
}

}  // namespace

hipError_t launch_sddmm(const EngineArgs& a, int dtype, int vec, int opk, int spec, int gc, hipStream_t s) {
    if (a.sch.w_small_end <= 0) return hipSuccess;
    const dim3 grid(blocks_for_waves(a.sch.w_small_end)), block(WAVE * WPB);
    const int ext = ext_of(a.flags);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, launch_sddmm_t<float, V>(a, opk, ext, spec, gc, grid, block, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, launch_sddmm_t<bf16_t, V>(a, opk, ext, spec, gc, grid, block, s))
    }
    return hipGetLastError();
}

}  // namespace gnnk
