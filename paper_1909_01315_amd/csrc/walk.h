// Edge walks of the row engine.
//
// walk_row(): the whole wavefront works on the positions [b, e) of one CSR
// row (a hub segment or a big row).  Lane group g takes the positions
// b + g, b + g + G, ...; a batch is UNR consecutive positions per group, so
// G * UNR consecutive positions per wavefront.
//
// Under a fast spec (G known at compile time) full batches have no per-slot
// selects.  With G <= 4 the neighbour and edge ids of a batch come from
// scalar loads issued one batch ahead (waited on through the scalar counter,
// so they never wait behind the vector gathers); with G >= 8 (a scalar
// batch would need 32-128 scalar registers) every lane loads its group's
// ids, the next batch's after this batch's gathers.  A per-edge head or row
// value of b (the attention weights) is read with one coalesced load per
// batch and moved to its lanes with ds_bpermute.  The last, partial batch and every
// batch of a runtime-G call read their ids per lane, clamp positions past
// the row end to the row start (always in bounds) and drop those slots.
//
// walk_lane(): one lane group walks its own row (the small-row role).
//
// Both call consume(const Raw& r, int32_t edge_id, int32_t nbr_id, bool ok)
// for every edge of the lane group in ascending position order.
#pragma once

#include <type_traits>

#include "device.h"

namespace gnnk {

template <int NBT>
struct Ids {
    int32_t nb[NBT];
    int32_t ed[NBT];
};

typedef int v4i __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(4))) v4i* cint4_ptr;

// ids of positions [q, q + NBT): scalar loads (q is uniform)
template <int NBT>
__device__ __forceinline__ void sload_ids(const CsrDev& C, int64_t q, Ids<NBT>& s) {
    static_assert(NBT % 4 == 0, "batches hold a multiple of 4 positions");
    cint4_ptr pn = (cint4_ptr)(C.idx + q);
#pragma unroll
    for (int k = 0; k < NBT / 4; ++k) {
        const v4i v = pn[k];
        s.nb[4 * k] = v.x; s.nb[4 * k + 1] = v.y; s.nb[4 * k + 2] = v.z; s.nb[4 * k + 3] = v.w;
    }
    if (C.eid) {
        cint4_ptr pe = (cint4_ptr)(C.eid + q);
#pragma unroll
        for (int k = 0; k < NBT / 4; ++k) {
            const v4i v = pe[k];
            s.ed[4 * k] = v.x; s.ed[4 * k + 1] = v.y; s.ed[4 * k + 2] = v.z; s.ed[4 * k + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < NBT; ++k) s.ed[k] = (int32_t)(q + k);
    }
}

// the value of slot u of lane group g among GC candidates held in scalars
// (read through readfirstlane so the choice stays a register select and
// never becomes an indexed access to a private array)
template <int GC>
__device__ __forceinline__ int32_t pick(const int32_t* v, int u, int g) {
    if constexpr (GC == 1) {
        return __builtin_amdgcn_readfirstlane(v[u]);
    } else if constexpr (GC == 2) {
        // the two candidates as one 64-bit scalar shifted by 0 or 32 bits in
        // each lane: one VALU instruction with one scalar operand, where a
        // select between two scalars first moves both into the lanes
        const uint32_t x0 = (uint32_t)__builtin_amdgcn_readfirstlane(v[2 * u]);
        const uint32_t x1 = (uint32_t)__builtin_amdgcn_readfirstlane(v[2 * u + 1]);
        const uint64_t pr = ((uint64_t)x1 << 32) | x0;
        return (int32_t)(uint32_t)(pr >> ((g & 1) << 5));
    } else {
        static_assert(GC == 4, "scalar id batches serve 1, 2 or 4 lane groups");
        const uint32_t x0 = (uint32_t)__builtin_amdgcn_readfirstlane(v[4 * u]);
        const uint32_t x1 = (uint32_t)__builtin_amdgcn_readfirstlane(v[4 * u + 1]);
        const uint32_t x2 = (uint32_t)__builtin_amdgcn_readfirstlane(v[4 * u + 2]);
        const uint32_t x3 = (uint32_t)__builtin_amdgcn_readfirstlane(v[4 * u + 3]);
        const int sh = (g & 1) << 5;
        const int32_t lo = (int32_t)(uint32_t)((((uint64_t)x1 << 32) | x0) >> sh);
        const int32_t hi = (int32_t)(uint32_t)((((uint64_t)x3 << 32) | x2) >> sh);
        return (g & 2) ? hi : lo;
    }
}

// Issue the loads of one full batch at position q (uniform), slot u of
// lane group g being position q + g + GC * u with ids nb[u], ed[u].
template <typename T, int VEC, int OPK, int EXT, class S>
__device__ __forceinline__ void issue_slots(const EngineArgs& A, const int32_t* nb, const int32_t* ed, int64_t q,
                                            int g, int32_t self, int col0, int h, const Pre<VEC>& pre, Raw<VEC>* r,
                                            float& cbv) {
    constexpr int GC = S::GC;
#pragma unroll
    for (int u = 0; u < UNR; ++u) fetch_bits<VEC, EXT>(A, (int32_t)q + g + GC * u, col0, r[u]);
#pragma unroll
    for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT, S>(A, nb[u], ed[u], self, col0, h, pre, r[u]);
    if constexpr (S::CB && OPK >= 1) {
        // lane l reads element (l mod Hb) of edge q + l / Hb; lanes past the
        // batch read the batch's first value
        constexpr int NBT = GC * UNR;
        const int lane = __lane_id();
        const int hb = A.log2hb;
        const int l = lane < (NBT << hb) ? lane : 0;
        const T* p = reinterpret_cast<const T*>(A.b.data) + q * A.b.stride;
        cbv = IO<T, 1>::load1(p + (uint32_t)(l >> hb) * (uint32_t)A.b.stride + (l & ((1 << hb) - 1)));
    }
}

// the same with the ids taken from the scalar batch (GC <= 4)
template <typename T, int VEC, int OPK, int EXT, class S>
__device__ __forceinline__ void issue_batch(const EngineArgs& A, const Ids<S::GC * UNR>& s, int64_t q, int g,
                                            int32_t self, int col0, int h, const Pre<VEC>& pre, Raw<VEC>* r,
                                            int32_t* nb, int32_t* ed, float& cbv) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) nb[u] = pick<S::GC>(s.nb, u, g);
    if (A.csr.eid == nullptr) {
        // identity edge ids: the slot's position, by arithmetic rather than
        // moving the batch's scalar ids into the lanes (12 fewer VALU
        // instructions per batch where edges are written or read by id)
#pragma unroll
        for (int u = 0; u < UNR; ++u) ed[u] = (int32_t)q + g + S::GC * u;
    } else {
#pragma unroll
        for (int u = 0; u < UNR; ++u) ed[u] = pick<S::GC>(s.ed, u, g);
    }
    issue_slots<T, VEC, OPK, EXT, S>(A, nb, ed, q, g, self, col0, h, pre, r, cbv);
}

// per-lane ids of a full batch (GC >= 8: a scalar batch would need too many
// scalar registers); every lane of group g reads its group's ids
__device__ __forceinline__ void vload_ids(const CsrDev& C, int64_t q, int g, int GC, int32_t* nb, int32_t* ed) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        const int32_t p = (int32_t)q + g + GC * u;
        nb[u] = C.idx[p];
        ed[u] = C.eid ? C.eid[p] : p;
    }
}

// A consumer that takes a whole full batch at once says so with a constant
// member kBatch = true and a method batch(r, ed) (partial batches still go
// edge by edge).
template <class F, class = void>
struct TakesBatch : std::false_type {};
template <class F>
struct TakesBatch<F, std::void_t<decltype(F::kBatch)>> : std::integral_constant<bool, F::kBatch> {};

// Hand the edges of a full batch to consume (b of a CB spec arrives by
// ds_bpermute from the coalesced load).
template <int VEC, int OPK, class S, class F>
__device__ __forceinline__ void take_batch(const EngineArgs& A, Raw<VEC>* r, const int32_t* nb, const int32_t* ed,
                                           float cbv, int g, int h, F& consume) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        if constexpr (S::CB && OPK >= 1) {
            const int src = ((g + S::GC * u) << A.log2hb) + (S::BK == OK_HEAD ? h : 0);
            const float x = __shfl(cbv, src, WAVE);
#pragma unroll
            for (int i = 0; i < VEC; ++i) r[u].b[i] = x;
        }
    }
    if constexpr (TakesBatch<F>::value) {
        consume.batch(r, ed);
    } else {
#pragma unroll
        for (int u = 0; u < UNR; ++u) consume(r[u], ed[u], nb[u], true);
    }
}

// Per-lane ids of one batch: positions p0 + u * stride, clamped to b past e.
// Positions fit in 32 bits (edge ids are int32).
__device__ __forceinline__ void batch_ids(const CsrDev& C, int32_t b, int32_t e, int32_t p0, int32_t stride,
                                          bool* ok, int32_t* nb, int32_t* ed, int32_t* ps) {
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
        const int32_t p = p0 + u * stride;
        ok[u] = p < e;
        const int32_t pc = ok[u] ? p : b;
        ps[u] = pc;
        nb[u] = C.idx[pc];
        ed[u] = C.eid ? C.eid[pc] : pc;
    }
}

// Per-lane batches over positions b + start, b + start + stride, ... < e,
// the next batch's ids loaded while the current batch's gathers are in
// flight.  No CB for these (the b operand is read per slot).
template <typename T, int VEC, int OPK, int EXT, class S, class F>
__device__ __forceinline__ void walk_strided(const EngineArgs& A, int32_t self, int64_t b64, int64_t e64,
                                             int64_t start, int stride, int col0, int h, const Pre<VEC>& pre,
                                             F& consume) {
    using SN = Spec<S::AT, S::AK, S::BT, S::BK, S::GC, false>;
    const int32_t b = (int32_t)b64, e = (int32_t)e64;
    const int32_t step = stride * UNR;
    int32_t p0 = b + (int32_t)start;
    if (p0 >= e) return;
    int32_t nb[UNR], ed[UNR], ps[UNR];
    bool ok[UNR];
    batch_ids(A.csr, b, e, p0, stride, ok, nb, ed, ps);
    for (; p0 < e; p0 += step) {
        Raw<VEC> r[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) fetch_bits<VEC, EXT>(A, ps[u], col0, r[u]);
#pragma unroll
        for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT, SN>(A, nb[u], ed[u], self, col0, h, pre, r[u]);
        bool okc[UNR];
        int32_t edc[UNR], nbc[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            okc[u] = ok[u];
            edc[u] = ed[u];
            nbc[u] = nb[u];
        }
        batch_ids(A.csr, b, e, p0 + step, stride, ok, nb, ed, ps);  // next batch, overlapping the gathers
#pragma unroll
        for (int u = 0; u < UNR; ++u) consume(r[u], edc[u], nbc[u], okc[u]);
    }
}

// The wavefront walks [b, e) of one row (see the file comment).  b and e
// must be wave-uniform.
template <typename T, int VEC, int OPK, int EXT, class S, class F>
__device__ __forceinline__ void walk_row(const EngineArgs& A, int32_t self, int64_t b, int64_t e, int g, int G,
                                         int col0, int h, const Pre<VEC>& pre, F& consume) {
    if constexpr (!S::FAST) {
        walk_strided<T, VEC, OPK, EXT, S>(A, self, b, e, g, G, col0, h, pre, consume);
    } else {
        constexpr int NBT = S::GC * UNR;
        const int64_t nfull = (e - b) / NBT;
        if constexpr (S::GC <= 4) {
            // one batch in flight per wavefront; the next batch's ids load
            // (scalar) while this batch's gathers are in flight
            if (nfull > 0) {
                Ids<NBT> ia;
                sload_ids<NBT>(A.csr, b, ia);
                for (int64_t i = 0; i < nfull; ++i) {
                    const int64_t q = b + i * NBT;
                    Raw<VEC> ra[UNR];
                    int32_t na[UNR], ea[UNR];
                    float ca = 0.0f;
                    issue_batch<T, VEC, OPK, EXT, S>(A, ia, q, g, self, col0, h, pre, ra, na, ea, ca);
                    if (i + 1 < nfull) sload_ids<NBT>(A.csr, q + NBT, ia);
                    take_batch<VEC, OPK, S>(A, ra, na, ea, ca, g, h, consume);
                }
            }
        } else {
            // ids per lane, the next batch's loaded after this batch's gathers
            if (nfull > 0) {
                int32_t na[UNR], ea[UNR];
                vload_ids(A.csr, b, g, S::GC, na, ea);
                for (int64_t i = 0; i < nfull; ++i) {
                    const int64_t q = b + i * NBT;
                    Raw<VEC> ra[UNR];
                    float ca = 0.0f;
                    issue_slots<T, VEC, OPK, EXT, S>(A, na, ea, q, g, self, col0, h, pre, ra, ca);
                    int32_t nc[UNR], ec[UNR];
#pragma unroll
                    for (int u = 0; u < UNR; ++u) {
                        nc[u] = na[u];
                        ec[u] = ea[u];
                    }
                    if (i + 1 < nfull) vload_ids(A.csr, q + NBT, g, S::GC, na, ea);
                    take_batch<VEC, OPK, S>(A, ra, nc, ec, ca, g, h, consume);
                }
            }
        }
        const int64_t t0 = b + nfull * NBT;
        if (t0 < e) walk_strided<T, VEC, OPK, EXT, S>(A, self, b, e, t0 - b + g, S::GC, col0, h, pre, consume);
    }
}

// Winner-mask walk (the max/min backward, EXT_BITS): the wavefront reads the
// masks of 64 positions of [b, e) at once (lane i: every word of position
// p0 + i), keeps the positions where any column won, packs them in
// ascending order into the low lanes (ds_permute of a stable partition),
// and hands only those to the lane groups: slot u of group g is kept
// position k + g + G * u.  On a graph whose rows are much longer than D,
// most positions win no column, and this skips them at 64 per mask load.
// b and e must be wave-uniform; every lane must take part.
template <typename T, int VEC, int OPK, class S, class F>
__device__ __forceinline__ void walk_winners(const EngineArgs& A, int32_t self, int64_t b64, int64_t e64, int g,
                                             int G, int col0, int h, const Pre<VEC>& pre, F& consume) {
    using SN = Spec<S::AT, S::AK, S::BT, S::BK, S::GC, false>;
    const int32_t b = (int32_t)b64, e = (int32_t)e64;
    const uint32_t* M = reinterpret_cast<const uint32_t*>(A.mask_arg);
    const uint32_t words = (uint32_t)A.mask_ld;
    const int lane = __lane_id();
    for (int32_t p0 = b; p0 < e; p0 += WAVE) {
        const int32_t p = p0 + lane;
        uint32_t any = 0u;
        // the position's ids load with its mask words, so that the kept
        // positions' gathers wait on one round trip, not two
        int32_t pn = 0, pe = 0;
        if (p < e) {
            const uint32_t* w = M + (uint64_t)(uint32_t)p * words;
            pn = A.csr.idx[p];
            pe = A.csr.eid ? A.csr.eid[p] : p;
            for (uint32_t j = 0; j < words; ++j) any |= w[j];
        }
        const uint64_t m = __ballot(any != 0u);
        if (m == 0ull) continue;
        const int n = __popcll(m);
        // kept lanes below this one; kept positions go to lanes 0..n-1 in
        // order, the others after them (a permutation of the 64 lanes)
        const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        const int dst = any != 0u ? below : n + (lane - below);
        const int32_t cpos = __builtin_amdgcn_ds_permute(dst << 2, p);
        const int32_t cnb = __builtin_amdgcn_ds_permute(dst << 2, pn);
        const int32_t ced = __builtin_amdgcn_ds_permute(dst << 2, pe);
        for (int k = 0; k < n; k += G * UNR) {
            int32_t nb[UNR], ed[UNR], ps[UNR];
            bool ok[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int q = k + g + G * u;
                ok[u] = q < n;
                // a slot past the kept positions takes kept position 0 (n > 0
                // here), whose ids are in range; it is dropped by ok
                const int qs = ok[u] ? q : 0;
                const int32_t pq = __shfl(cpos, qs, WAVE);
                ps[u] = ok[u] ? pq : b;
                nb[u] = __shfl(cnb, qs, WAVE);
                ed[u] = __shfl(ced, qs, WAVE);
            }
            Raw<VEC> r[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) fetch_bits<VEC, EXT_BITS>(A, ps[u], col0, r[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) fetch<T, VEC, OPK, EXT_BITS, SN>(A, nb[u], ed[u], self, col0, h, pre, r[u]);
#pragma unroll
            for (int u = 0; u < UNR; ++u) consume(r[u], ed[u], nb[u], ok[u]);
        }
    }
}

// One lane group walks its own row [b, e) (b == e for no row).
template <typename T, int VEC, int OPK, int EXT, class S, class F>
__device__ __forceinline__ void walk_lane(const EngineArgs& A, int32_t self, int64_t b, int64_t e, int col0, int h,
                                          const Pre<VEC>& pre, F& consume) {
    walk_strided<T, VEC, OPK, EXT, S>(A, self, b, e, 0, 1, col0, h, pre, consume);
}

}  // namespace gnnk
