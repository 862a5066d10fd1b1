// Device-side building blocks shared by the gnnk kernels (gfx950, wave64):
// vector IO of fp32/bf16 rows, cross-lane reductions, operand fetch and the
// message arithmetic, edge batches, and the row output.
//
// Conventions that keep every kernel deterministic and branch-free in its
// edge loop: a lane holds VEC consecutive columns of the message row; edge
// batches read clamped (always in-bounds) positions and drop the extra slots
// with selects; inactive lanes read column 0 and never write.
#pragma once

#include "internal.h"

namespace gnnk {

constexpr int WAVE = 64;
constexpr int WPB = 4;  // wavefronts per block
constexpr int UNR = ENGINE_UNR;  // edges in flight per lane group

typedef uint16_t bf16_t;

__device__ __forceinline__ int64_t row_ptr(const CsrDev& c, int64_t r) {
    return c.ptr64 ? reinterpret_cast<const int64_t*>(c.ptr)[r] : (int64_t) reinterpret_cast<const int32_t*>(c.ptr)[r];
}

// ---------------------------------------------------------------------------
// element IO: VEC consecutive elements <-> float registers

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t f2bf(float f) {
    uint32_t b = __float_as_uint(f);
    b += 0x7FFFu + ((b >> 16) & 1u);  // round to nearest, ties to even (finite inputs)
    return b >> 16;
}

template <typename T, int VEC>
struct IO;

template <int VEC>
struct IO<float, VEC> {
    static __device__ __forceinline__ void load(const float* p, float* v) {
        if constexpr (VEC == 4) {
            float4 x = *reinterpret_cast<const float4*>(p);
            v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        } else if constexpr (VEC == 2) {
            float2 x = *reinterpret_cast<const float2*>(p);
            v[0] = x.x; v[1] = x.y;
        } else {
            v[0] = *p;
        }
    }
    static __device__ __forceinline__ float load1(const float* p) { return *p; }
    static __device__ __forceinline__ void load_nt(const float* p, float* v) {
        typedef float f4 __attribute__((ext_vector_type(4)));
        typedef float f2 __attribute__((ext_vector_type(2)));
        if constexpr (VEC == 4) {
            f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
            v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
        } else if constexpr (VEC == 2) {
            f2 x = __builtin_nontemporal_load(reinterpret_cast<const f2*>(p));
            v[0] = x.x; v[1] = x.y;
        } else {
            v[0] = __builtin_nontemporal_load(p);
        }
    }
    static __device__ __forceinline__ float load1_nt(const float* p) { return __builtin_nontemporal_load(p); }
    static __device__ __forceinline__ void store(float* p, const float* v) {
        if constexpr (VEC == 4) {
            *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
        } else if constexpr (VEC == 2) {
            *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
        } else {
            *p = v[0];
        }
    }
    static __device__ __forceinline__ void store1(float* p, float v) { *p = v; }
    // nontemporal only for 16-byte vectors: narrower nontemporal stores are
    // partial-line writes that L2 does not merge (a g-SDDMM with one value
    // per edge ran twice as long with them); those stay plain
    static __device__ __forceinline__ void store_nt(float* p, const float* v) {
        typedef float f4 __attribute__((ext_vector_type(4)));
        if constexpr (VEC == 4) {
            f4 x = {v[0], v[1], v[2], v[3]};
            __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p));
        } else {
            store(p, v);
        }
    }
    // streaming store: scattered outputs that no later load of the kernel reads
    static __device__ __forceinline__ void store1_nt(float* p, float v) { __builtin_nontemporal_store(v, p); }
};

template <int VEC>
struct IO<bf16_t, VEC> {
    static __device__ __forceinline__ void load(const bf16_t* p, float* v) {
        if constexpr (VEC == 8) {
            uint4 x = *reinterpret_cast<const uint4*>(p);
            v[0] = bf_lo(x.x); v[1] = bf_hi(x.x); v[2] = bf_lo(x.y); v[3] = bf_hi(x.y);
            v[4] = bf_lo(x.z); v[5] = bf_hi(x.z); v[6] = bf_lo(x.w); v[7] = bf_hi(x.w);
        } else if constexpr (VEC == 4) {
            uint2 x = *reinterpret_cast<const uint2*>(p);
            v[0] = bf_lo(x.x); v[1] = bf_hi(x.x); v[2] = bf_lo(x.y); v[3] = bf_hi(x.y);
        } else if constexpr (VEC == 2) {
            uint32_t x = *reinterpret_cast<const uint32_t*>(p);
            v[0] = bf_lo(x); v[1] = bf_hi(x);
        } else {
            v[0] = bf_lo(*p);
        }
    }
    static __device__ __forceinline__ float load1(const bf16_t* p) { return bf_lo(*p); }
    static __device__ __forceinline__ void load_nt(const bf16_t* p, float* v) { load(p, v); }
    static __device__ __forceinline__ float load1_nt(const bf16_t* p) { return load1(p); }
    static __device__ __forceinline__ void store(bf16_t* p, const float* v) {
        if constexpr (VEC == 8) {
            uint4 x;
            x.x = f2bf(v[0]) | (f2bf(v[1]) << 16); x.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
            x.z = f2bf(v[4]) | (f2bf(v[5]) << 16); x.w = f2bf(v[6]) | (f2bf(v[7]) << 16);
            *reinterpret_cast<uint4*>(p) = x;
        } else if constexpr (VEC == 4) {
            uint2 x;
            x.x = f2bf(v[0]) | (f2bf(v[1]) << 16); x.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
            *reinterpret_cast<uint2*>(p) = x;
        } else if constexpr (VEC == 2) {
            *reinterpret_cast<uint32_t*>(p) = f2bf(v[0]) | (f2bf(v[1]) << 16);
        } else {
            *p = (bf16_t)f2bf(v[0]);
        }
    }
    static __device__ __forceinline__ void store1(bf16_t* p, float v) { *p = (bf16_t)f2bf(v); }
    static __device__ __forceinline__ void store_nt(bf16_t* p, const float* v) {
        typedef unsigned u4 __attribute__((ext_vector_type(4)));
        if constexpr (VEC == 8) {
            u4 x = {f2bf(v[0]) | (f2bf(v[1]) << 16), f2bf(v[2]) | (f2bf(v[3]) << 16), f2bf(v[4]) | (f2bf(v[5]) << 16),
                    f2bf(v[6]) | (f2bf(v[7]) << 16)};
            __builtin_nontemporal_store(x, reinterpret_cast<u4*>(p));
        } else {
            store(p, v);
        }
    }
    static __device__ __forceinline__ void store1_nt(bf16_t* p, float v) {
        __builtin_nontemporal_store((bf16_t)f2bf(v), p);
    }
};

template <int VEC>
__device__ __forceinline__ void load_i32(const int32_t* p, int32_t* v) {
    if constexpr (VEC >= 4 && VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            int4 x = reinterpret_cast<const int4*>(p)[q];
            v[4 * q] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
        }
    } else if constexpr (VEC == 2) {
        int2 x = *reinterpret_cast<const int2*>(p);
        v[0] = x.x; v[1] = x.y;
    } else {
        v[0] = *p;
    }
}

// the arg arrays of max/min are written once per call: nontemporal 16-byte
// vectors when NT (narrower ones stay plain, as in IO::store_nt)
template <int VEC, bool NT = true>
__device__ __forceinline__ void store_i32(int32_t* p, const int32_t* v) {
    typedef int i4 __attribute__((ext_vector_type(4)));
    if constexpr (NT && VEC >= 4 && VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            i4 x = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
            __builtin_nontemporal_store(x, reinterpret_cast<i4*>(p) + q);
        }
    } else if constexpr (VEC >= 4 && VEC % 4 == 0) {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q)
            reinterpret_cast<int4*>(p)[q] = make_int4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    } else if constexpr (VEC == 2) {
        *reinterpret_cast<int2*>(p) = make_int2(v[0], v[1]);
    } else {
        *p = v[0];
    }
}

// ---------------------------------------------------------------------------
// cross-lane helpers (64-bit values move as two 32-bit shuffles)

__device__ __forceinline__ double shfl_xor_d(double x, int m) {
    int2 v = *reinterpret_cast<int2*>(&x);
    v.x = __shfl_xor(v.x, m, WAVE);
    v.y = __shfl_xor(v.y, m, WAVE);
    return *reinterpret_cast<double*>(&v);
}

__device__ __forceinline__ double shfl_d(double x, int src) {
    int2 v = *reinterpret_cast<int2*>(&x);
    v.x = __shfl(v.x, src, WAVE);
    v.y = __shfl(v.y, src, WAVE);
    return *reinterpret_cast<double*>(&v);
}

// fp64 lane moves through DPP (two 32-bit halves); CTRL is a dpp_ctrl code
template <int CTRL>
__device__ __forceinline__ double dpp_d(double x) {
    int2 v = *reinterpret_cast<int2*>(&x);
    v.x = __builtin_amdgcn_mov_dpp(v.x, CTRL, 0xF, 0xF, false);
    v.y = __builtin_amdgcn_mov_dpp(v.y, CTRL, 0xF, 0xF, false);
    return *reinterpret_cast<double*>(&v);
}

// e^x for x <= 0 (or -inf) from the hardware base-2 exponential (v_exp_f32,
// 1 ulp).  Rounding x * log2(e) once adds |x| * 2^-24 relative error: 1e-6 at
// x = -16, where the term is already 1e-7 of a row's largest.
__device__ __forceinline__ float exp_le0(float x) { return __builtin_amdgcn_exp2f(x * 1.44269504088896341f); }

constexpr int DPP_QUAD_1032 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_2301 = 0x4E;  // quad_perm [2,3,0,1]
// row_ror:n hands lane i the value of lane (i - n) mod 16 of its 16-lane row
constexpr int DPP_ROR12 = 0x12C;     // row_ror:12: lane i reads lane (i + 4) mod 16
constexpr int DPP_ROR8 = 0x128;      // row_ror:8: lane i reads lane (i + 8) mod 16

// run_sum with the run length known at compile time (no per-step branches)
template <int RED>
__device__ __forceinline__ double run_sum_c(double v) {
    if constexpr (RED >= 2) v += dpp_d<DPP_QUAD_1032>(v);
    if constexpr (RED >= 4) v += dpp_d<DPP_QUAD_2301>(v);
    if constexpr (RED >= 8) v += dpp_d<DPP_ROR12>(v);
    if constexpr (RED >= 16) v += dpp_d<DPP_ROR8>(v);
    if constexpr (RED >= 32) v += shfl_xor_d(v, 16);
    if constexpr (RED >= 64) v += shfl_xor_d(v, 32);
    return v;
}

// Sum over aligned runs of `red` lanes (a power of two), correct in the first
// lane of each run: DPP within 16-lane rows, swizzles beyond.
__device__ __forceinline__ double run_sum(double v, int red) {
    if (red >= 2) v += dpp_d<DPP_QUAD_1032>(v);
    if (red >= 4) v += dpp_d<DPP_QUAD_2301>(v);
    if (red >= 8) v += dpp_d<DPP_ROR12>(v);  // lane i (i mod 8 < 4) adds the quad above it
    if (red >= 16) v += dpp_d<DPP_ROR8>(v);
    if (red >= 32) v += shfl_xor_d(v, 16);
    if (red >= 64) v += shfl_xor_d(v, 32);
    return v;
}

// Sum over aligned runs of `red` consecutive lanes starting at multiples of
// `red` within each lane group; the first lane of a run gets the total (the
// other lanes hold partial sums).  Every lane must call it.
__device__ __forceinline__ double seg_sum(double v, int lane_in_group, int red) {
    const int pos = lane_in_group % red;
    const int lane = __lane_id();
    for (int s = 1; s < red; s <<= 1) {
        double o = shfl_d(v, lane + s < WAVE ? lane + s : lane);
        v += ((pos & (2 * s - 1)) == 0 && pos + s < red) ? o : 0.0;
    }
    return v;
}

// ---------------------------------------------------------------------------
// operands and messages
//
// An operand's layout can be fixed at compile time (Spec): its target (the
// neighbour, the edge, or the row itself) and its kind (a full vector per
// lane, one value per head, one value per row).  DYN reads both from the
// runtime descriptor.  Fast specs address node operands with 32-bit byte
// offsets (the host checks that the table fits), which the compiler turns
// into scalar-base loads with one 32-bit vector offset.

enum : int { DYN = -1 };
enum : int { OK_FULL = 0, OK_HEAD = 1, OK_ROW = 2 };

template <int AT_, int AK_, int BT_, int BK_, int GC_, bool CB_, bool PRE_ = true>
struct Spec {
    static constexpr int AT = AT_, AK = AK_, BT = BT_, BK = BK_;
    static constexpr int GC = GC_;    // lane groups per wavefront, 0 = runtime (no scalar id batches)
    static constexpr bool CB = CB_;   // b is read with one coalesced load per batch (identity edge ids)
    static constexpr bool FAST = GC_ > 0;
    // an operand on the row itself is loaded once per row (false: per edge,
    // as in edge-parallel walks where consecutive edges change rows)
    static constexpr bool PRE = PRE_ && FAST;
};
using SpecDyn = Spec<DYN, DYN, DYN, DYN, 0, false>;

__device__ __forceinline__ int32_t row_of(int32_t target, int32_t nb, int32_t ed, int32_t self) {
    return target == T_NBR ? nb : (target == T_EDGE ? ed : self);
}

template <typename T, int VEC, int TGT, int KIND, bool FAST>
__device__ __forceinline__ void ld_opd(const OperandDev& o, int32_t nb, int32_t ed, int32_t self, int col0, int h,
                                       float* v, bool random_edges = false) {
    const int32_t row = row_of(TGT == DYN ? o.target : TGT, nb, ed, self);
    if constexpr (FAST && TGT != DYN && TGT != T_EDGE && KIND != DYN) {
        const uint32_t rb = (uint32_t)o.stride * (uint32_t)sizeof(T);
        const uint32_t c = KIND == OK_FULL ? (uint32_t)col0 : (KIND == OK_HEAD ? (uint32_t)h : 0u);
        const uint32_t off = __umul24((uint32_t)row, rb) + c * (uint32_t)sizeof(T);
        const T* p = reinterpret_cast<const T*>(reinterpret_cast<const char*>(o.data) + off);
        if constexpr (KIND == OK_FULL) {
            IO<T, VEC>::load(p, v);
        } else {
            const float x = IO<T, VEC>::load1(p);
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = x;
        }
    } else {
        const T* base = reinterpret_cast<const T*>(o.data) + (uint64_t)(uint32_t)row * (uint32_t)o.stride;
        const bool full = KIND == DYN ? (o.full != 0) : KIND == OK_FULL;
        // edge operands read through explicit edge ids (the reverse graph)
        // arrive in random order, one line per record: nontemporal loads
        // (c3's u_add_v backward 3.30 -> 3.09 ms, the dX pass of u_mul_e/sum
        // 7.57 -> 7.20 ms).  In edge-id order a lane group reads each line
        // several times in a row, so plain loads there (nontemporal ones
        // made u_mul_e/sum on a degree-32 graph up to 24% slower)
        const bool nt = random_edges && (TGT == DYN ? o.target == T_EDGE : TGT == T_EDGE);
        if (full) {
            if (nt) IO<T, VEC>::load_nt(base + col0, v);
            else IO<T, VEC>::load(base + col0, v);
        } else {
            const int hm = KIND == DYN ? o.hmul : (KIND == OK_HEAD ? 1 : 0);
            const float x = nt ? IO<T, VEC>::load1_nt(base + h * hm) : IO<T, VEC>::load1(base + h * hm);
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = x;
        }
    }
}

// the runtime-descriptor load (softmax and other generic callers)
template <typename T, int VEC>
__device__ __forceinline__ void load_operand(const OperandDev& o, int32_t row, int col0, int h, float* v) {
    ld_opd<T, VEC, DYN, DYN, false>(o, row, row, row, col0, h, v);
}

// Raw operand values of one edge for this lane's VEC columns (loaded first,
// combined after the loads of a whole batch are in flight).
template <int VEC>
struct Raw {
    float a[VEC];
    float b[VEC];
    float c[VEC];
    int32_t k[VEC];
    int32_t dg;
    uint32_t kb;  // EXT_BITS: the winner bits of this lane's VEC columns
};

// EXT_BITS: the winner bits of an edge (its CSR position) are read before
// the edge's operands, so a lane with no winning column skips its load of a.
template <int VEC, int EXT>
__device__ __forceinline__ void fetch_bits(const EngineArgs& A, int32_t pos, int col0, Raw<VEC>& r) {
    if constexpr (EXT == EXT_BITS) {
        const uint32_t* M = reinterpret_cast<const uint32_t*>(A.mask_arg);
        const uint32_t w = M[(uint64_t)(uint32_t)pos * (uint32_t)A.mask_ld + (uint32_t)(col0 >> 5)];
        r.kb = (w >> (col0 & 31)) & ((VEC == 32 ? 0u : (1u << VEC)) - 1u);
    }
}

// Values of an operand that targets the row itself, loaded once per row.
template <int VEC>
struct Pre {
    float a[VEC];
    float b[VEC];
};

// OPK: 0 message = a; 1 message = a * b; 2 any MsgOp (runtime).
// An operand that targets the row itself under a fast spec comes from `pre`;
// with S::CB the caller fills b from the batch's coalesced load.
template <typename T, int VEC, int OPK, int EXT, class S>
__device__ __forceinline__ void fetch(const EngineArgs& A, int32_t nb, int32_t ed, int32_t self, int col0, int h,
                                      const Pre<VEC>& pre, Raw<VEC>& r) {
    constexpr bool F = S::FAST;
    if constexpr (S::PRE && S::AT == T_SELF) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) r.a[i] = pre.a[i];
    } else if constexpr (EXT == EXT_BITS) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) r.a[i] = 0.0f;
        if (r.kb) ld_opd<T, VEC, S::AT, S::AK, F>(A.a, nb, ed, self, col0, h, r.a, A.csr.eid != nullptr);
    } else {
        ld_opd<T, VEC, S::AT, S::AK, F>(A.a, nb, ed, self, col0, h, r.a, A.csr.eid != nullptr);
    }
    if constexpr (OPK >= 1) {
        if constexpr (S::PRE && S::BT == T_SELF) {
#pragma unroll
            for (int i = 0; i < VEC; ++i) r.b[i] = pre.b[i];
        } else if constexpr (!S::CB) {
            ld_opd<T, VEC, S::BT, S::BK, F>(A.b, nb, ed, self, col0, h, r.b, A.csr.eid != nullptr);
        }
    }
    if constexpr (OPK == 2) {
        if (A.op == M_NEGDIV2)
            ld_opd<T, VEC, DYN, DYN, false>(A.c, nb, ed, self, col0, h, r.c, A.csr.eid != nullptr);
    }
    const int32_t ar = row_of(S::AT == DYN ? A.a.target : S::AT, nb, ed, self);
    if constexpr (EXT == EXT_SCALE) r.dg = A.deg[ar];
    if constexpr (EXT == EXT_MASK) {
        if constexpr (F) {
            const uint32_t off = __umul24((uint32_t)ar, (uint32_t)A.mask_ld * 4u) + (uint32_t)col0 * 4u;
            load_i32<VEC>(reinterpret_cast<const int32_t*>(reinterpret_cast<const char*>(A.mask_arg) + off), r.k);
        } else {
            load_i32<VEC>(A.mask_arg + (int64_t)ar * A.mask_ld + col0, r.k);
        }
    }
}

// the operands of a fast spec that target the row itself
template <typename T, int VEC, int OPK, class S>
__device__ __forceinline__ void load_pre(const EngineArgs& A, int32_t self, int col0, int h, Pre<VEC>& pre) {
    if constexpr (S::PRE && S::AT == T_SELF) ld_opd<T, VEC, T_SELF, S::AK, true>(A.a, 0, 0, self, col0, h, pre.a);
    if constexpr (S::PRE && OPK >= 1 && S::BT == T_SELF)
        ld_opd<T, VEC, T_SELF, S::BK, true>(A.b, 0, 0, self, col0, h, pre.b);
}

// message in fp64 (sums and g-SDDMM); single operations are exact in fp64
// before the final rounding
template <int VEC, int OPK, int EXT>
__device__ __forceinline__ void combine_f64(const EngineArgs& A, const Raw<VEC>& r, int32_t ed, double* m) {
    double ad[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
        // EXT_BITS: columns this edge did not win contribute zero (masked
        // before widening: one 32-bit select per column)
        if constexpr (EXT == EXT_BITS) ad[i] = (double)(((r.kb >> i) & 1u) ? r.a[i] : 0.0f);
        else ad[i] = r.a[i];
    }
    if constexpr (EXT == EXT_SCALE) {
        // one reciprocal per edge, not one division per column: the hardware
        // estimate refined by one Newton step (within an ulp of 1/deg in fp64)
        const double d = (double)r.dg;
        double inv = __builtin_amdgcn_rcp(d);
        inv = fma(inv, fma(-d, inv, 1.0), inv);
#pragma unroll
        for (int i = 0; i < VEC; ++i) ad[i] = ad[i] * inv;
    }
    if constexpr (EXT == EXT_MASK) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) ad[i] = (r.k[i] == ed) ? ad[i] : 0.0;
    }
    if constexpr (OPK == 0) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) m[i] = ad[i];
    } else if constexpr (OPK == 1) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) m[i] = ad[i] * (double)r.b[i];
    } else {
        switch (A.op) {
            case M_ADD:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = ad[i] + (double)r.b[i];
                break;
            case M_SUB:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = ad[i] - (double)r.b[i];
                break;
            case M_RSUB:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = (double)r.b[i] - ad[i];
                break;
            case M_MUL:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = ad[i] * (double)r.b[i];
                break;
            case M_DIV:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = ad[i] / (double)r.b[i];
                break;
            case M_NEGDIV2:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = -ad[i] * (double)r.b[i] / ((double)r.c[i] * (double)r.c[i]);
                break;
            default:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = ad[i];
        }
    }
}

// message for max/min: one fp32 operation, as a message tensor would hold it
template <int VEC, int OPK>
__device__ __forceinline__ void combine_f32(const EngineArgs& A, const Raw<VEC>& r, float* m) {
    if constexpr (OPK == 0) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) m[i] = r.a[i];
    } else {
        const int op = OPK == 1 ? (int)M_MUL : A.op;
        switch (op) {
            case M_ADD:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = r.a[i] + r.b[i];
                break;
            case M_SUB:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = r.a[i] - r.b[i];
                break;
            case M_MUL:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = r.a[i] * r.b[i];
                break;
            case M_DIV:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = r.a[i] / r.b[i];
                break;
            default:
#pragma unroll
                for (int i = 0; i < VEC; ++i) m[i] = r.a[i];
        }
    }
}

// ---------------------------------------------------------------------------
// max / min

// candidate (m, e) replaces (best, be): strictly better, or equal with a
// smaller edge id, or nothing recorded yet.  Bitwise operators keep it
// branch-free.
__device__ __forceinline__ bool better(float m, int32_t e, float best, int32_t be, bool is_min) {
    const bool strict = is_min ? (m < best) : (m > best);
    const bool tie = (m == best) & (e < be);
    return (be < 0) | strict | tie;
}

// ---------------------------------------------------------------------------
// output of one reduced row (sums)

// A reduced output of a row wider than one pass of the wavefront (nchunk > 1,
// so one lane group of 64 lanes, whole-row sums only) adds each pass's total
// into *carry (lane 0) and is written after the last pass; ch is the pass.
template <typename T, int VEC>
__device__ __forceinline__ void write_sum_row(const EngineArgs& A, int64_t row, bool active, int lig, int col0,
                                              int h, double* acc, int64_t deg, bool write_lane,
                                              bool may_reduce = true, int ch = 0, double* carry = nullptr) {
    if (A.flags & F_OWN_MEAN) {
        const double d = deg > 0 ? (double)deg : 1.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = acc[i] / d;
    }
    if (A.flags & F_NEGATE) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = -acc[i];
    }
    if (!may_reduce || !A.out.reduce) {
        if (active && write_lane && row >= 0) {
            float v[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) v[i] = (float)acc[i];
            IO<T, VEC>::store(reinterpret_cast<T*>(A.out.data) + row * A.out.stride + col0, v);
        }
    } else {
        double s = 0.0;
#pragma unroll
        for (int i = 0; i < VEC; ++i) s += acc[i];
        s = seg_sum(active ? s : 0.0, lig, A.out.red);
        if (A.geo.nchunk > 1 && carry) {
            *carry += s;
            if (ch + 1 < A.geo.nchunk) return;
            s = *carry;
        }
        if (active && write_lane && row >= 0 && (lig % A.out.red) == 0) {
            const int64_t o = A.out.per_head ? h : 0;
            IO<T, VEC>::store1(reinterpret_cast<T*>(A.out.data) + row * A.out.stride + o, (float)s);
        }
    }
}

// lane-group geometry of one wavefront
struct Lanes {
    int g;    // lane group
    int lig;  // lane in group
};

__device__ __forceinline__ Lanes lanes_of(const GeomDev& geo) {
    const int lane = threadIdx.x & (WAVE - 1);
    return Lanes{lane >> geo.log2L, lane & (geo.L - 1)};
}

// with the lane-group count fixed at compile time (GC > 0)
template <int GC>
__device__ __forceinline__ Lanes lanes_of(const GeomDev& geo) {
    if constexpr (GC > 0) {
        constexpr int L = WAVE / GC;
        const int lane = threadIdx.x & (WAVE - 1);
        return Lanes{lane / L, lane % L};
    } else {
        return lanes_of(geo);
    }
}

// sum over the lane groups of a wavefront (each lane keeps its columns)
template <int GC, int VEC>
__device__ __forceinline__ void sum_groups(const GeomDev& geo, double* acc) {
    const int L = GC > 0 ? WAVE / GC : geo.L;
    for (int s = L; s < WAVE; s <<= 1)
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] += shfl_xor_d(acc[i], s);
}

// a wave-uniform value, moved to scalar registers
__device__ __forceinline__ int64_t uniform64(int64_t x) {
    const int32_t lo = __builtin_amdgcn_readfirstlane((int32_t)(uint64_t)x);
    const int32_t hi = __builtin_amdgcn_readfirstlane((int32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// wave index within the grid, in a scalar register
__device__ __forceinline__ int wave_id() {
    return __builtin_amdgcn_readfirstlane((int)(blockIdx.x * WPB + (threadIdx.x >> 6)));
}

// ---------------------------------------------------------------------------
// template dispatch of the launchers

#define GNNK_VEC_DISPATCH_F32(VEC_, ...)                      \
    switch (VEC_) {                                           \
        case 4: { constexpr int V = 4; __VA_ARGS__; } break;  \
        case 2: { constexpr int V = 2; __VA_ARGS__; } break;  \
        default: { constexpr int V = 1; __VA_ARGS__; } break; \
    }

#define GNNK_VEC_DISPATCH_BF16(VEC_, ...)                     \
    switch (VEC_) {                                           \
        case 8: { constexpr int V = 8; __VA_ARGS__; } break;  \
        case 4: { constexpr int V = 4; __VA_ARGS__; } break;  \
        case 2: { constexpr int V = 2; __VA_ARGS__; } break;  \
        default: { constexpr int V = 1; __VA_ARGS__; } break; \
    }

// lane groups of a fast spec
#define GNNK_GC_DISPATCH(GC_, ...)                                \
    switch (GC_) {                                                \
        case 1: { constexpr int C = 1; __VA_ARGS__; } break;      \
        case 2: { constexpr int C = 2; __VA_ARGS__; } break;      \
        case 4: { constexpr int C = 4; __VA_ARGS__; } break;      \
        case 8: { constexpr int C = 8; __VA_ARGS__; } break;      \
        case 16: { constexpr int C = 16; __VA_ARGS__; } break;    \
        default: { constexpr int C = 32; __VA_ARGS__; } break;    \
    }

#define GNNK_OPK_DISPATCH(OPK_, ...)                          \
    switch (OPK_) {                                           \
        case 0: { constexpr int K = 0; __VA_ARGS__; } break;  \
        case 1: { constexpr int K = 1; __VA_ARGS__; } break;  \
        default: { constexpr int K = 2; __VA_ARGS__; } break; \
    }

// without EXT_BITS (g-SDDMM passes never read winner masks)
#define GNNK_EXT3_DISPATCH(EXT_, ...)                                 \
    switch (EXT_) {                                                   \
        case EXT_SCALE: { constexpr int X = EXT_SCALE; __VA_ARGS__; } break; \
        case EXT_MASK: { constexpr int X = EXT_MASK; __VA_ARGS__; } break;   \
        default: { constexpr int X = EXT_NONE; __VA_ARGS__; } break;         \
    }

#define GNNK_EXT_DISPATCH(EXT_, ...)                                  \
    switch (EXT_) {                                                   \
        case EXT_SCALE: { constexpr int X = EXT_SCALE; __VA_ARGS__; } break; \
        case EXT_MASK: { constexpr int X = EXT_MASK; __VA_ARGS__; } break;   \
        case EXT_BITS: { constexpr int X = EXT_BITS; __VA_ARGS__; } break;   \
        default: { constexpr int X = EXT_NONE; __VA_ARGS__; } break;         \
    }


inline unsigned blocks_for_waves(int64_t waves) { return (unsigned)((waves + WPB - 1) / WPB); }

}  // namespace gnnk
