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
#include <type_traits>

#include "walk.h"

namespace gnnk {

// ---------------------------------------------------------------------------
// sums

// DW: also write, per edge, the dot of a (dZ[v]) with the row's own x2
// (X[u]) over runs of red2 lanes -- the edge-weight gradient of u_mul_e/sum,
// computed in the reverse pass that gathers dZ[v] anyway
// (DW: 0 none; 1 runs of A.red2 lanes read at run time; 2-64 runs of DW
// lanes fixed at compile time, with no per-step branches)
template <typename T, int VEC, int DW>
struct EdgeDot {
    float x[VEC];
    __device__ __forceinline__ void load(const EngineArgs& A, int32_t self, int col0) {
        if constexpr (DW) IO<T, VEC>::load(reinterpret_cast<const T*>(A.x2) + (int64_t)self * A.x2_stride + col0, x);
    }
    __device__ __forceinline__ void put(const EngineArgs& A, const Raw<VEC>& rw, int32_t ed, bool ok, int lig,
                                        int h, bool active) {
        if constexpr (DW) {
            double dp = 0.0;
#pragma unroll
            for (int i = 0; i < VEC; ++i) dp = fma((double)rw.a[i], (double)x[i], dp);
            const int red = DW > 1 ? DW : A.red2;
            if constexpr (DW > 1) dp = run_sum_c<DW>(dp);
            else dp = run_sum(dp, red);
            if (ok & active & ((lig & (red - 1)) == 0))
                IO<T, 1>::store1_nt(reinterpret_cast<T*>(A.out2) + (int64_t)ed * A.out2_stride +
                                        (A.per_head2 ? h : 0), (float)dp);
        }
    }
};

template <typename T, int VEC, int OPK, int EXT, class S, int DW = 0>
__global__ __launch_bounds__(256) void spmm_sum_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int G = S::GC > 0 ? S::GC : geo.G;
    const int L = WAVE / G;

    if (w < A.sch.w_big_end) {
        // one wavefront: a segment of a hub row, or a whole big row
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
        double carry = 0.0;
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            double acc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
            Pre<VEC> pre;
            load_pre<T, VEC, OPK, S>(A, (int32_t)r, col0, h, pre);
            EdgeDot<T, VEC, DW> dw;
            dw.load(A, (int32_t)r, col0);
            auto sink = [&](const Raw<VEC>& rw, int32_t ed, int32_t, bool ok) {
                // winner masks: most slots of a wavefront won no column at all
                if constexpr (EXT == EXT_BITS)
                    if (__ballot(rw.kb != 0u) == 0ull) return;
                double m[VEC];
                combine_f64<VEC, OPK, EXT>(A, rw, ed, m);
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += ok ? m[i] : 0.0;
                dw.put(A, rw, ed, ok, ln.lig, h, active);
            };
            if constexpr (EXT == EXT_BITS)
                walk_winners<T, VEC, OPK, S>(A, (int32_t)r, b, e, ln.g, G, col0, h, pre, sink);
            else
                walk_row<T, VEC, OPK, EXT, S>(A, (int32_t)r, b, e, ln.g, G, col0, h, pre, sink);
            sum_groups<S::GC, VEC>(geo, acc);
            if (slot >= 0) {
                if (ln.g == 0 && active) {
                    double* P = reinterpret_cast<double*>(A.partial) + (int64_t)slot * A.partial_stride + col0;
#pragma unroll
                    for (int i = 0; i < VEC; ++i) P[i] = acc[i];
                }
            } else {
                write_sum_row<T, VEC>(A, r, active, ln.lig, col0, h, acc, e - b, ln.g == 0, !S::FAST, ch, &carry);
            }
        }
    } else if (w < A.sch.w_small_end) {
        // small rows: each lane group owns one row
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * G + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
        }
        const int32_t self = r >= 0 ? (int32_t)r : 0;
        double carry = 0.0;
        for (int ch = 0; ch < geo.nchunk; ++ch) {
            const int j = ch * L + ln.lig;
            const bool active = j < geo.NV;
            const int col0 = active ? j * VEC : 0;
            const int h = col0 / geo.F;
            double acc[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
            Pre<VEC> pre;
            load_pre<T, VEC, OPK, S>(A, self, col0, h, pre);
            EdgeDot<T, VEC, DW> dw;
            dw.load(A, self, col0);
            auto sink = [&](const Raw<VEC>& rw, int32_t ed, int32_t, bool ok) {
                // winner masks: most slots of a wavefront won no column at all
                if constexpr (EXT == EXT_BITS)
                    if (__ballot(rw.kb != 0u) == 0ull) return;
                double m[VEC];
                combine_f64<VEC, OPK, EXT>(A, rw, ed, m);
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += ok ? m[i] : 0.0;
                dw.put(A, rw, ed, ok, ln.lig, h, active);
            };
            walk_lane<T, VEC, OPK, EXT, S>(A, self, b, e, col0, h, pre, sink);
            write_sum_row<T, VEC>(A, r, active, ln.lig, col0, h, acc, e - b, true, !S::FAST, ch, &carry);
        }
    } else {
        // empty rows: the empty reduction is 0 (no mean, no negation)
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * G + ln.g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * L + ln.lig;
                const bool active = j < geo.NV;
                const int col0 = active ? j * VEC : 0;
                const int h = col0 / geo.F;
                if (S::FAST || !A.out.reduce) {
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

// combine the segment partials of hub rows, in segment order.  A lane walks
// its row's segments COMB_UNR at a time with the loads issued together: the
// longest rows have hundreds of segments, and one load in flight per lane
// left the combine waiting on each in turn.
constexpr int COMB_UNR = 8;

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
    double carry = 0.0;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * geo.L + ln.lig;
        const bool active = j < geo.NV && row_ok;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        double acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0;
        const double* P0 = reinterpret_cast<const double*>(A.partial) + col0;
        int s = s0;
        // COMB_UNR segments' loads in flight at once, added in segment order
        for (; s + COMB_UNR <= s1; s += COMB_UNR) {
            double v[COMB_UNR][VEC];
#pragma unroll
            for (int u = 0; u < COMB_UNR; ++u)
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[u][i] = P0[(int64_t)(s + u) * A.partial_stride + i];
#pragma unroll
            for (int u = 0; u < COMB_UNR; ++u)
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += v[u][i];
        }
        for (; s < s1; ++s) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] += P0[(int64_t)s * A.partial_stride + i];
        }
        write_sum_row<T, VEC>(A, r, active, ln.lig, col0, h, acc, deg, true, true, ch, &carry);
    }
}

// ---------------------------------------------------------------------------
// max / min with the winning edge and neighbour

// identity of max / min: a running best starts here, so the first message
// that is not -inf (+inf for min) replaces it by a strict comparison
__device__ __forceinline__ float cmp_identity(bool is_min) { return is_min ? INFINITY : -INFINITY; }

// Output of one row.  first: the row's first CSR position (-1 for an empty
// row).  With identity edge ids (ids == positions) be holds positions and a
// row whose messages are all -inf (+inf for min) kept be = -1: its first edge
// wins, as a scan with strict comparisons from the first edge gives; the
// neighbour of the winner is read from the CSR here.  With explicit edge ids
// be and bn come from the walk.
template <typename T, int VEC>
__device__ __forceinline__ void write_cmp_row(const EngineArgs& A, int64_t row, bool active, int col0, float* best,
                                              int32_t* be, int32_t* bn, int64_t first) {
    if (!active || row < 0) return;
    if (A.csr.eid == nullptr) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            if (be[i] < 0 && first >= 0) be[i] = (int32_t)first;
            bn[i] = be[i] >= 0 ? A.csr.idx[be[i]] : -1;
        }
    }
    float v[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) v[i] = be[i] < 0 ? 0.0f : best[i];
    // value and arg arrays are written once: nontemporal where a lane group
    // writes whole lines of its row (8 lanes or more; c4 copy_u/max with arg
    // edge 4.72 -> 4.48 ms, its three outputs being 2.9 GB), plain below that
    const int64_t D = (int64_t)A.geo.NV * VEC;
    T* out = reinterpret_cast<T*>(A.out.data) + row * A.out.stride + col0;
    if (A.geo.L >= 8) {
        IO<T, VEC>::store_nt(out, v);
        if (A.arg_edge) store_i32<VEC>(A.arg_edge + row * D + col0, be);
        if (A.arg_nbr) store_i32<VEC>(A.arg_nbr + row * D + col0, bn);
    } else {
        IO<T, VEC>::store(out, v);
        if (A.arg_edge) store_i32<VEC, false>(A.arg_edge + row * D + col0, be);
        if (A.arg_nbr) store_i32<VEC, false>(A.arg_nbr + row * D + col0, bn);
    }
}

// Running max/min of one lane group.  The group sees its edges in ascending
// position.  TIES = false (identity edge ids): ascending position is
// ascending edge id, so a strict comparison keeps the smallest id among
// equal messages, and only the value and the position are tracked.  TIES =
// true (explicit ids, in any order) tests the smaller id explicitly and
// tracks the edge and the neighbour.
template <int VEC, int OPK, bool TIES, bool MIN>
struct CmpSink {
    const EngineArgs& A;
    float best[VEC];
    int32_t be[VEC], bn[VEC];
    __device__ __forceinline__ void operator()(const Raw<VEC>& rw, int32_t ed, int32_t nb, bool ok) {
        float m[VEC];
        combine_f32<VEC, OPK>(A, rw, m);
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
            if constexpr (TIES) {
                const bool upd = ok & better(m[i], ed, best[i], be[i], MIN);
                best[i] = upd ? m[i] : best[i];
                be[i] = upd ? ed : be[i];
                bn[i] = upd ? nb : bn[i];
            } else {
                const bool upd = ok & (MIN ? (m[i] < best[i]) : (m[i] > best[i]));
                best[i] = upd ? m[i] : best[i];
                be[i] = upd ? ed : be[i];
            }
        }
    }
};

// max/min over the edges of one row: by the whole wavefront (WAVE_ROW,
// uniform bounds; hub segments leave partials) or by this lane group alone
template <typename T, int VEC, int OPK, class S, bool WAVE_ROW>
__device__ __forceinline__ void cmp_row(const EngineArgs& A, const Lanes& ln, int G, int L, int64_t r, int64_t b,
                                        int64_t e, int slot) {
    const GeomDev& geo = A.geo;
    const int64_t D = (int64_t)geo.NV * VEC;
    const bool is_min = (A.flags & F_IS_MIN) != 0;
    const bool ties = A.csr.eid != nullptr;
    const int32_t self = r >= 0 ? (int32_t)r : 0;
    const int64_t first = e > b ? b : -1;
    for (int ch = 0; ch < geo.nchunk; ++ch) {
        const int j = ch * L + ln.lig;
        const bool active = j < geo.NV;
        const int col0 = active ? j * VEC : 0;
        const int h = col0 / geo.F;
        float best[VEC];
        int32_t be[VEC], bn[VEC];
        Pre<VEC> pre;
        auto run = [&](auto& sk) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) { sk.best[i] = cmp_identity(is_min); sk.be[i] = -1; sk.bn[i] = -1; }
            if constexpr (WAVE_ROW) walk_row<T, VEC, OPK, EXT_NONE, S>(A, self, b, e, ln.g, G, col0, h, pre, sk);
            else walk_lane<T, VEC, OPK, EXT_NONE, S>(A, self, b, e, col0, h, pre, sk);
#pragma unroll
            for (int i = 0; i < VEC; ++i) { best[i] = sk.best[i]; be[i] = sk.be[i]; bn[i] = sk.bn[i]; }
        };
        if (ties) {
            if (is_min) { CmpSink<VEC, OPK, true, true> sk{A, {}, {}, {}}; run(sk); }
            else { CmpSink<VEC, OPK, true, false> sk{A, {}, {}, {}}; run(sk); }
        } else {
            if (is_min) { CmpSink<VEC, OPK, false, true> sk{A, {}, {}, {}}; run(sk); }
            else { CmpSink<VEC, OPK, false, false> sk{A, {}, {}, {}}; run(sk); }
        }
        if constexpr (!WAVE_ROW) {
            write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn, first);
        } else {
            for (int s = L; s < WAVE; s <<= 1) {
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
                write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn, first);
            }
        }
    }
}

template <typename T, int VEC, int OPK, class S>
__global__ __launch_bounds__(256) void spmm_cmp_kernel(EngineArgs A) {
    const int w = wave_id();
    if (w >= A.sch.w_total) return;
    const GeomDev& geo = A.geo;
    const Lanes ln = lanes_of<S::GC>(geo);
    const int G = S::GC > 0 ? S::GC : geo.G;
    const int L = WAVE / G;

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
        cmp_row<T, VEC, OPK, S, true>(A, ln, G, L, uniform64(r), uniform64(b), uniform64(e), slot);
    } else if (w < A.sch.w_small_end) {
        const int64_t k = A.sch.n_big + (int64_t)(w - A.sch.w_big_end) * G + ln.g;
        int64_t r = -1, b = 0, e = 0;
        if (k < A.sch.n_nz) {
            const int4 t = A.csr.rowt[k];
            r = t.x; b = t.y; e = t.z;
        }
        cmp_row<T, VEC, OPK, S, false>(A, ln, G, L, r, b, e, -1);
    } else {
        const int64_t k0 = A.sch.n_nz +
                           ((int64_t)(w - A.sch.w_small_end) * G + ln.g) * A.sch.fill_rows_per_group;
        for (int q = 0; q < A.sch.fill_rows_per_group; ++q) {
            const int64_t k = k0 + q;
            const int64_t r = k < A.sch.n_rows ? A.csr.perm[k] : -1;
            for (int ch = 0; ch < geo.nchunk; ++ch) {
                const int j = ch * L + ln.lig;
                const bool active = j < geo.NV;
                float best[VEC];
                int32_t be[VEC], bn[VEC];
#pragma unroll
                for (int i = 0; i < VEC; ++i) { best[i] = 0.0f; be[i] = -1; bn[i] = -1; }
                write_cmp_row<T, VEC>(A, r, active, active ? j * VEC : 0, best, be, bn, -1);
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
        const float* PV0 = reinterpret_cast<const float*>(A.partial) + col0;
        const int32_t* PE0 = reinterpret_cast<const int32_t*>(A.partial) + (int64_t)A.sch.n_seg * D + col0;
        const int32_t* PN0 = PE0 + (int64_t)A.sch.n_seg * D;
        auto take = [&](float pv, int32_t pe, int32_t pn, int i) {
            const bool upd = (pe >= 0) & better(pv, pe, best[i], be[i], is_min);
            best[i] = upd ? pv : best[i];
            be[i] = upd ? pe : be[i];
            bn[i] = upd ? pn : bn[i];
        };
        int s = s0;
        // COMB_UNR segments' loads in flight at once, compared in segment order
        for (; s + COMB_UNR <= s1; s += COMB_UNR) {
            float pv[COMB_UNR][VEC];
            int32_t pe[COMB_UNR][VEC], pn[COMB_UNR][VEC];
#pragma unroll
            for (int u = 0; u < COMB_UNR; ++u)
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    const int64_t o = (int64_t)(s + u) * D + i;
                    pv[u][i] = PV0[o];
                    pe[u][i] = PE0[o];
                    pn[u][i] = PN0[o];
                }
#pragma unroll
            for (int u = 0; u < COMB_UNR; ++u)
#pragma unroll
                for (int i = 0; i < VEC; ++i) take(pv[u][i], pe[u][i], pn[u][i], i);
        }
        for (; s < s1; ++s) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                const int64_t o = (int64_t)s * D + i;
                take(PV0[o], PE0[o], PN0[o], i);
            }
        }
        write_cmp_row<T, VEC>(A, r, active, col0, best, be, bn, row_ok ? row_ptr(A.csr, r) : -1);
    }
}

// ---------------------------------------------------------------------------
// launchers

bool fast_vec(int dtype, int vec) { return dtype == 0 ? vec == 4 : (vec == 4 || vec == 8); }

namespace {

template <int GC, bool CB>
using SpUEH = Spec<T_NBR, OK_FULL, T_EDGE, OK_HEAD, GC, CB>;
template <int GC, bool CB>
using SpUER = Spec<T_NBR, OK_FULL, T_EDGE, OK_ROW, GC, CB>;
template <int GC>
using SpCU = Spec<T_NBR, OK_FULL, DYN, DYN, GC, false>;

template <typename T, int V>
void launch_sum_t(const EngineArgs& a, int opk, int ext, int spec, int gc, dim3 grid, dim3 block, hipStream_t s) {
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        if (spec != SP_DYN) {
            GNNK_GC_DISPATCH(gc, {
                switch (spec) {
                    case SP_CU:
                        GNNK_EXT_DISPATCH(ext, {
                            hipLaunchKernelGGL((spmm_sum_kernel<T, V, 0, X, SpCU<C>>), grid, block, 0, s, a);
                        })
                        break;
                    case SP_UE_H:
                        hipLaunchKernelGGL((spmm_sum_kernel<T, V, 1, EXT_NONE, SpUEH<C, false>>), grid, block, 0, s, a);
                        break;
                    case SP_UE_H_CB:
                        hipLaunchKernelGGL((spmm_sum_kernel<T, V, 1, EXT_NONE, SpUEH<C, true>>), grid, block, 0, s, a);
                        break;
                    case SP_UE_R:
                        hipLaunchKernelGGL((spmm_sum_kernel<T, V, 1, EXT_NONE, SpUER<C, false>>), grid, block, 0, s, a);
                        break;
                    default:
                        hipLaunchKernelGGL((spmm_sum_kernel<T, V, 1, EXT_NONE, SpUER<C, true>>), grid, block, 0, s, a);
                        break;
                }
            })
            return;
        }
    }
    GNNK_OPK_DISPATCH(opk, GNNK_EXT_DISPATCH(ext, {
        hipLaunchKernelGGL((spmm_sum_kernel<T, V, K, X, SpecDyn>), grid, block, 0, s, a);
    }))
}

template <typename T, int V>
void launch_cmp_t(const EngineArgs& a, int opk, int spec, int gc, dim3 grid, dim3 block, hipStream_t s) {
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        if (spec == SP_CU) {
            GNNK_GC_DISPATCH(gc, { hipLaunchKernelGGL((spmm_cmp_kernel<T, V, 0, SpCU<C>>), grid, block, 0, s, a); })
            return;
        }
    }
    GNNK_OPK_DISPATCH(opk, { hipLaunchKernelGGL((spmm_cmp_kernel<T, V, K, SpecDyn>), grid, block, 0, s, a); })
}

template <typename T, int V>
void launch_dw_t(const EngineArgs& a, int spec, int gc, dim3 grid, dim3 block, hipStream_t s) {
    if constexpr ((sizeof(T) == 4 && V == 4) || (sizeof(T) == 2 && (V == 4 || V == 8))) {
        // the edge gradient's lane runs (a.red2) as a compile-time constant
        // when they are 2-32 lanes long (the host fuses only runs that fit
        // the lane group), else read at run time
        auto launch = [&](auto cg, auto rg) {
            constexpr int C = decltype(cg)::value;
            constexpr int R = decltype(rg)::value;
            if (spec == SP_UE_H)
                hipLaunchKernelGGL((spmm_sum_kernel<T, V, 1, EXT_NONE, SpUEH<C, false>, R>), grid, block, 0, s, a);
            else
                hipLaunchKernelGGL((spmm_sum_kernel<T, V, 1, EXT_NONE, SpUER<C, false>, R>), grid, block, 0, s, a);
        };
        auto go = [&](auto cg) {
            constexpr int L = 64 / decltype(cg)::value;
            switch (a.red2) {
                case 2: if constexpr (L >= 2) { launch(cg, std::integral_constant<int, 2>{}); return; } break;
                case 4: if constexpr (L >= 4) { launch(cg, std::integral_constant<int, 4>{}); return; } break;
                case 8: if constexpr (L >= 8) { launch(cg, std::integral_constant<int, 8>{}); return; } break;
                case 16: if constexpr (L >= 16) { launch(cg, std::integral_constant<int, 16>{}); return; } break;
                case 32: if constexpr (L >= 32) { launch(cg, std::integral_constant<int, 32>{}); return; } break;
                default: break;
            }
            launch(cg, std::integral_constant<int, 1>{});
        };
        if (gc == 1) go(std::integral_constant<int, 1>{});
        else if (gc == 2) go(std::integral_constant<int, 2>{});
        else go(std::integral_constant<int, 4>{});
    }
}

}  // namespace

hipError_t launch_spmm_dw(const EngineArgs& a, int dtype, int vec, int spec, int gc, hipStream_t s) {
    if (a.sch.w_total <= 0) return hipSuccess;
    const dim3 grid(blocks_for_waves(a.sch.w_total)), block(WAVE * WPB);
    if (dtype == 0) {
        GNNK_VEC_DISPATCH_F32(vec, launch_dw_t<float, V>(a, spec, gc, grid, block, s))
    } else {
        GNNK_VEC_DISPATCH_BF16(vec, launch_dw_t<bf16_t, V>(a, spec, gc, grid, block, s))
    }
    return hipGetLastError();
}

hipError_t launch_spmm(const EngineArgs& a, int dtype, int vec, bool maxmin, int opk, int spec, int gc,
                       hipStream_t s) {
    if (a.sch.w_total <= 0) return hipSuccess;
    const dim3 grid(blocks_for_waves(a.sch.w_total)), block(WAVE * WPB);
    const int ext = ext_of(a.flags);
    if (maxmin) {
        if (dtype == 0) {
            GNNK_VEC_DISPATCH_F32(vec, launch_cmp_t<float, V>(a, opk, spec, gc, grid, block, s))
        } else {
            GNNK_VEC_DISPATCH_BF16(vec, launch_cmp_t<bf16_t, V>(a, opk, spec, gc, grid, block, s))
        }
    } else {
        if (dtype == 0) {
            GNNK_VEC_DISPATCH_F32(vec, launch_sum_t<float, V>(a, opk, ext, spec, gc, grid, block, s))
        } else {
            GNNK_VEC_DISPATCH_BF16(vec, launch_sum_t<bf16_t, V>(a, opk, ext, spec, gc, grid, block, s))
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
