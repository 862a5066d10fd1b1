// g-SDDMM kernel (Section 3, definition of generalized SDDMM): one output per
// edge, op(lhs at its target, rhs at its target).  Edges are walked row by
// row over the in-CSR (rows = destinations) with the degree-sorted schedule,
// so a destination-side operand is read once per destination and hub rows are
// split across wavefronts.  The same kernel computes the edge gradients of
// g-SpMM (the lemma on dL/dW of g-SpMM) and of g-SDDMM.  Elementwise ops are
// single fp32 operations (computed in fp64, rounded once); dot products and
// sums over broadcast positions accumulate in fp64.
#include "device.h"

namespace gnnk {

template <typename T, int VEC, int OPK, int EXT>
__device__ __forceinline__ void sddmm_edges(const EngineArgs& A, int32_t self, int64_t b, int64_t e, int64_t n_iter,
                                            int start, int stride, int lig, int col0, int h, bool active) {
    const CsrDev& C = A.csr;
    // n_iter is uniform over the wavefront so the lane reductions line up
    for (int64_t it = 0; it < n_iter; it += UNR) {
        int32_t nb[UNR], ed[UNR];
        bool ok[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t p = b + start + (it + u) * (int64_t)stride;
            ok[u] = ((it + u) < n_iter) & (p < e);
            const int64_t pc = ok[u] ? p : b;
            nb[u] = C.idx[pc];
            ed[u] = C.eid ? C.eid[pc] : (int32_t)pc;
        }
        Raw<VEC> r[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT>(A, nb[u], ed[u], self, col0, h, r[u]);
        if (!A.out.reduce) {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                double m[VEC];
                combine_f64<VEC, OPK, EXT>(A, r[u], ed[u], m);
                if (ok[u] & active) {
                    float v[VEC];
#pragma unroll
                    for (int i = 0; i < VEC; ++i) v[i] = (float)((A.flags & F_NEGATE) ? -m[i] : m[i]);
                    IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + (int64_t)ed[u] * A.out.stride + col0, v);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                double m[VEC];
                combine_f64<VEC, OPK, EXT>(A, r[u], ed[u], m);
                double s = 0.0;
#pragma unroll
                for (int i = 0; i < VEC; ++i) s += m[i];
                s = seg_sum(active ? s : 0.0, lig, A.out.red);
                if (ok[u] & active & ((lig % A.out.red) == 0)) {
                    if (A.flags & F_NEGATE) s = -s;
                    const int64_t o = A.out.per_head ? h : 0;
                    IO<T, VEC>::store1(reinterpret_cast<T*>(A.out.data) + (int64_t)ed[u] * A.out.stride + o,
                                       (float)s);
                }
            }
        }
    }
}

template <typename T, int VEC, int OPK, int EXT>
__global__ __launch_bounds__(256) void sddmm_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.w_small_end) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of(geo);
    int64_t r, b, e, n_iter;
    int start, stride;
    if (w < A.sch.w_big_end) {
        if (w < A.sch.n_seg) {
            const int4 s = A.csr.seg[w];
            r = s.x; b = s.y; e = s.z;
        } else {
            r = A.csr.perm[A.sch.n_hub + (w - A.sch.n_seg)];
            b = row_ptr(A.csr, r);
            e = row_ptr(A.csr, r + 1);
        }
        start = ln.g;
        stride = geo.G;
        n_iter = (e - b + geo.G - 1) / geo.G;
    } else {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * geo.G + ln.g;
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
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        sddmm_edges<T, VEC, OPK, EXT>(A, r >= 0 ? (int32_t)r : 0, b, e, n_iter, start, stride, ln.lig, col0, h,
                                      active);
    }
}

hipError_t launch_sddmm(const EngineArgs& a, int dtype, int vec, int opk, hipStream_t s) {
    if (a.sch.w_small_end <= 0) return hipSuccess;
    const dim3 grid(blocks_for_waves(a.sch.w_small_end)), block(WAVE * WPB);
    const int ext = ext_of(a.flags);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, GNNK_OPK_DISPATCH(opk, GNNK_EXT_DISPATCH(ext, {
            hipLaunchKernelGGL((sddmm_kernel<float, V, K, X>), grid, block, 0, s, a);
        })))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, GNNK_OPK_DISPATCH(opk, GNNK_EXT_DISPATCH(ext, {
            hipLaunchKernelGGL((sddmm_kernel<bf16_t, V, K, X>), grid, block, 0, s, a);
        })))
    }
    return hipGetLastError();
}

}  // namespace gnnk
