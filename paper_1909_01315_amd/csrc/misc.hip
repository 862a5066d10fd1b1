// Elementwise and structural kernels: leaky ReLU and its backward, index
// validation, and small helpers of the graph handle.
#include "device.h"

namespace gnnk {

static inline unsigned grid_1d(int64_t n) {
    int64_t b = (n + 255) / 256;
    if (b > 65536) b = 65536;
    return (unsigned)(b > 0 ? b : 1);
}

template <typename T, bool BWD>
__global__ void leaky_kernel(const T* x, const T* dy, T* y, int64_t rows, int32_t cols, int64_t sx, int64_t sdy,
                             int64_t sy, float slope) {
    const int64_t n = rows * (int64_t)cols;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / cols, c = i - r * cols;
        float xv = IO<T, 1>::load1(x + r * sx + c);
        float out;
        if (BWD) {
            float d = IO<T, 1>::load1(dy + r * sdy + c);
            out = xv > 0.0f ? d : slope * d;
        } else {
            out = xv > 0.0f ? xv : slope * xv;
        }
        IO<T, 1>::store1(y + r * sy + c, out);
    }
}

// the same on a contiguous tensor: 16-byte vectors, grid-stride
template <typename T, int VEC, bool BWD>
__device__ __forceinline__ void leaky_vec(const float* xv, const float* d, float* out, float slope) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        const float v = BWD ? d[k] : xv[k];
        out[k] = xv[k] > 0.0f ? v : slope * v;
    }
}

template <typename T, int VEC, bool BWD>
__global__ __launch_bounds__(256) void leaky_flat_kernel(const T* x, const T* dy, T* y, int64_t n, float slope) {
    // a pure stream: nontemporal loads and stores (1.44 -> 1.40 ms on c3's
    // (E, 8) scores), several vectors in flight per thread (c3 backward
    // 2.03 -> 1.95 ms with 8, forward 1.41 -> 1.39 ms with 4; smaller grids
    // of longer-lived threads were slower)
    constexpr int U = BWD ? 8 : 4;
    const int64_t nv = n / VEC;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (; i + (U - 1) * stride < nv; i += U * stride) {
        float xv[U][VEC], d[U][VEC], out[VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            IO<T, VEC>::load_nt(x + (i + u * stride) * VEC, xv[u]);
            if (BWD) IO<T, VEC>::load_nt(dy + (i + u * stride) * VEC, d[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            leaky_vec<T, VEC, BWD>(xv[u], d[u], out, slope);
            IO<T, VEC>::store_nt(y + (i + u * stride) * VEC, out);
        }
    }
    for (; i < nv; i += stride) {
        float xv[VEC], d[VEC], out[VEC];
        IO<T, VEC>::load_nt(x + i * VEC, xv);
        if (BWD) IO<T, VEC>::load_nt(dy + i * VEC, d);
        leaky_vec<T, VEC, BWD>(xv, d, out, slope);
        IO<T, VEC>::store_nt(y + i * VEC, out);
    }
    // the tail (fewer than VEC elements), by the first threads
    const int64_t t = nv * VEC + blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t < n) {
        const float xv = IO<T, 1>::load1(x + t);
        const float out = BWD ? (xv > 0.0f ? IO<T, 1>::load1(dy + t) : slope * IO<T, 1>::load1(dy + t))
                              : (xv > 0.0f ? xv : slope * xv);
        IO<T, 1>::store1(y + t, out);
    }
}

__global__ void validate_kernel(const int32_t* idx, int64_t n, int64_t bound, int32_t* flag) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        int32_t v = idx[i];
        if (v < 0 || v >= bound) atomicOr(flag, 1);
    }
}

template <typename P>
__global__ void validate_ptr_kernel(const P* ptr, int64_t n_rows, int64_t n_edges, int32_t* flag) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i <= n_rows;
         i += (int64_t)gridDim.x * blockDim.x) {
        int64_t v = ptr[i];
        bool bad = v < 0 || v > n_edges || (i == 0 && v != 0) || (i == n_rows && v != n_edges) ||
                   (i < n_rows && ptr[i + 1] < v);
        if (bad) atomicOr(flag, 2);
    }
}

// row of every position of a CSR: the last row whose offset is <= p
template <typename P>
__global__ void fill_rows_kernel(const P* ptr, int64_t n_rows, int64_t n_edges, int32_t* row) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n_edges;
         p += (int64_t)gridDim.x * blockDim.x) {
        int64_t lo = 0, hi = n_rows;  // ptr[lo] <= p < ptr[hi]
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) / 2;
            if ((int64_t)ptr[mid] <= p) lo = mid;
            else hi = mid;
        }
        row[p] = (int32_t)lo;
    }
}

__global__ void inverse_kernel(const int32_t* perm, int64_t n, int32_t* pos) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n; q += (int64_t)gridDim.x * blockDim.x)
        pos[perm[q]] = (int32_t)q;
}

__global__ void zero_words_kernel(uint32_t* w, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        w[i] = 0u;
}

// Winner masks: half a wavefront per (row, 32-column word) of the arg array.
// Lanes whose columns have the same winning edge merge their bits, and the
// first of them stores the whole word.  The word of an edge belongs to the
// edge's one destination row, so no other lane writes it: plain stores, no
// atomics, and the result does not depend on any ordering.
__global__ __launch_bounds__(256) void winner_bits_kernel(const int32_t* arg_e, int64_t n_rows, int32_t D,
                                                          int64_t ld, const int32_t* pos_of_edge, uint32_t* bits,
                                                          int32_t words, int64_t n_edges) {
    const int lane = __lane_id();
    const int half = lane >> 5, b = lane & 31;
    const int64_t n_units = n_rows * words;
    const int64_t wave = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
    const int64_t stride = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t u0 = 2 * wave; u0 < n_units; u0 += 2 * stride) {
        const int64_t unit = u0 + half;
        const int64_t v = unit / words;
        const int32_t w = (int32_t)(unit - v * words);
        const int32_t c = w * 32 + b;
        int32_t e = -1;
        if (unit < n_units && c < D) e = arg_e[v * ld + c];
        const bool ok = e >= 0 && e < n_edges;  // empty rows (-1); ids outside the graph are ignored
        const int32_t pos = ok ? pos_of_edge[e] : 0;  // every lane's lookup in flight at once
        uint64_t todo = __ballot(ok);
        while (todo) {
            const int l0 = __builtin_ctzll(todo);
            const int32_t e0 = __builtin_amdgcn_readlane(e, l0);
            const int h0 = l0 >> 5;
            const uint64_t m = __ballot(ok && e == e0 && half == h0);
            if (lane == l0) bits[(int64_t)pos * words + w] = (uint32_t)(m >> (32 * h0));
            todo &= ~m;
        }
    }
}

// Winner masks by destination row, for identity edge ids (the in-CSR
// position of an edge is its id): one wavefront per unit of the in-CSR (a hub
// row's segment, or a whole smaller row), taking the unit's edges 64 at a
// time, one per lane, with the edge's reverse-CSR position loaded first.  The
// lanes scan the row's arg array, four 32-column words at a time: the winner
// of a column less the chunk's first position is the lane of the edge that
// won it, whose LDS word gets the column's bit.  Then every edge of the chunk
// that won a column stores its words at its reverse-CSR position; the rest
// stay as zeroed before.  An arg that names no edge of its own row matches
// nothing, as the gradient's definition has it.  An edge's words are written
// by the one wavefront that holds it and an OR does not depend on its order:
// no global atomics, and the result is fixed.  Against winner_bits_kernel it
// reads the positions of a row's edges in order and stores whole masks, where
// that one looks up a position and stores a word per winning column; it
// rescans the arg row for every 64 edges, so it suits rows short against D.
constexpr int WIN_WB = 4;

template <typename P>
__global__ __launch_bounds__(64) void winner_rows_kernel(WinnerRowsArgs a) {
    __shared__ uint4 lds[64];  // WIN_WB words per lane's edge
    uint32_t* ldw = reinterpret_cast<uint32_t*>(lds);
    const int lane = threadIdx.x;
    const int64_t n_units = a.n_seg + a.n_small;
    const P* ptr = static_cast<const P*>(a.ptr);
    for (int64_t u = blockIdx.x; u < n_units; u += gridDim.x) {
        int64_t v, b, e;
        if (u < a.n_seg) {
            const int4 sg = a.seg[u];
            v = sg.x, b = sg.y, e = sg.z;
        } else {
            v = a.perm[a.n_hub + (u - a.n_seg)];
            b = (int64_t)ptr[v], e = (int64_t)ptr[v + 1];
        }
        const int32_t* arow = a.arg + v * a.ld;
        for (int64_t c0 = b; c0 < e; c0 += 64) {
            const int nv = (int)(e - c0 < 64 ? e - c0 : 64);
            const int32_t p = lane < nv ? a.pos[c0 + lane] : 0;
            for (int w0 = 0; w0 < a.words; w0 += WIN_WB) {
                const int wb = a.words - w0 < WIN_WB ? a.words - w0 : WIN_WB;
                lds[lane] = make_uint4(0u, 0u, 0u, 0u);
                __syncthreads();
                const int cend = (w0 + wb) * 32 < a.D ? (w0 + wb) * 32 : a.D;
                for (int c = w0 * 32 + lane; c < cend; c += 64) {
                    const int64_t k = (int64_t)arow[c] - c0;
                    if (k >= 0 && k < nv) atomicOr(&ldw[k * WIN_WB + ((c >> 5) - w0)], 1u << (c & 31));
                }
                __syncthreads();
                const uint4 m = lds[lane];
                if (lane < nv && (m.x | m.y | m.z | m.w) != 0u) {
                    uint32_t* dst = a.bits + (int64_t)p * a.words + w0;
                    if (wb == WIN_WB && (a.words & (WIN_WB - 1)) == 0) {
                        *reinterpret_cast<uint4*>(dst) = m;
                    } else {
                        const uint32_t mw[WIN_WB] = {m.x, m.y, m.z, m.w};
                        for (int i = 0; i < wb; ++i) dst[i] = mw[i];
                    }
                }
                __syncthreads();
            }
        }
    }
}

__global__ void iota_kernel(int32_t* out, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        out[i] = (int32_t)i;
}

__global__ void copy_ptr_kernel(const void* src, int src64, void* dst, int dst64, int64_t n) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t v = src64 ? reinterpret_cast<const int64_t*>(src)[i] : reinterpret_cast<const int32_t*>(src)[i];
        if (dst64) reinterpret_cast<int64_t*>(dst)[i] = v;
        else reinterpret_cast<int32_t*>(dst)[i] = (int32_t)v;
    }
}


hipError_t launch_leaky(const void* x, const void* dy, void* y, int64_t rows, int32_t cols, int64_t sx,
                        int64_t sdy, int64_t sy, float slope, int dtype, bool backward, hipStream_t s) {
    int64_t n = rows * (int64_t)cols;
    if (n <= 0) return hipSuccess;
    const bool flat = (rows == 1 || (sx == cols && sy == cols && (!backward || sdy == cols)));
    const uintptr_t al = (uintptr_t)x | (uintptr_t)y | (backward ? (uintptr_t)dy : 0);
    if (flat && al % 16 == 0) {
        dim3 grid(grid_1d(n / (dtype == 0 ? 4 : 8) + 1)), block(256);
        if (dtype == 0) {
            if (backward)
                hipLaunchKernelGGL((leaky_flat_kernel<float, 4, true>), grid, block, 0, s, (const float*)x,
                                   (const float*)dy, (float*)y, n, slope);
            else
                hipLaunchKernelGGL((leaky_flat_kernel<float, 4, false>), grid, block, 0, s, (const float*)x,
                                   (const float*)dy, (float*)y, n, slope);
        } else {
            if (backward)
                hipLaunchKernelGGL((leaky_flat_kernel<bf16_t, 8, true>), grid, block, 0, s, (const bf16_t*)x,
                                   (const bf16_t*)dy, (bf16_t*)y, n, slope);
            else
                hipLaunchKernelGGL((leaky_flat_kernel<bf16_t, 8, false>), grid, block, 0, s, (const bf16_t*)x,
                                   (const bf16_t*)dy, (bf16_t*)y, n, slope);
        }
        return hipGetLastError();
    }
    dim3 grid(grid_1d(n)), block(256);
    if (dtype == 0) {
        if (backward)
            hipLaunchKernelGGL((leaky_kernel<float, true>), grid, block, 0, s, (const float*)x, (const float*)dy,
                               (float*)y, rows, cols, sx, sdy, sy, slope);
        else
            hipLaunchKernelGGL((leaky_kernel<float, false>), grid, block, 0, s, (const float*)x, (const float*)dy,
                               (float*)y, rows, cols, sx, sdy, sy, slope);
    } else {
        if (backward)
            hipLaunchKernelGGL((leaky_kernel<bf16_t, true>), grid, block, 0, s, (const bf16_t*)x,
                               (const bf16_t*)dy, (bf16_t*)y, rows, cols, sx, sdy, sy, slope);
        else
            hipLaunchKernelGGL((leaky_kernel<bf16_t, false>), grid, block, 0, s, (const bf16_t*)x,
                               (const bf16_t*)dy, (bf16_t*)y, rows, cols, sx, sdy, sy, slope);
    }
    return hipGetLastError();
}

hipError_t launch_validate(const int32_t* idx, int64_t n, int64_t bound, int32_t* flag, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(validate_kernel, dim3(grid_1d(n)), dim3(256), 0, s, idx, n, bound, flag);
    return hipGetLastError();
}

hipError_t launch_validate_ptr(const void* ptr, int ptr64, int64_t n_rows, int64_t n_edges, int32_t* flag,
                               hipStream_t s) {
    dim3 grid(grid_1d(n_rows + 1)), block(256);
    if (ptr64)
        hipLaunchKernelGGL((validate_ptr_kernel<int64_t>), grid, block, 0, s, (const int64_t*)ptr, n_rows, n_edges,
                           flag);
    else
        hipLaunchKernelGGL((validate_ptr_kernel<int32_t>), grid, block, 0, s, (const int32_t*)ptr, n_rows, n_edges,
                           flag);
    return hipGetLastError();
}

hipError_t launch_fill_rows(const void* ptr, int ptr64, int64_t n_rows, int64_t n_edges, int32_t* row,
                            hipStream_t s) {
    if (n_edges <= 0) return hipSuccess;
    if (ptr64)
        hipLaunchKernelGGL(fill_rows_kernel<int64_t>, dim3(grid_1d(n_edges)), dim3(256), 0, s,
                           reinterpret_cast<const int64_t*>(ptr), n_rows, n_edges, row);
    else
        hipLaunchKernelGGL(fill_rows_kernel<int32_t>, dim3(grid_1d(n_edges)), dim3(256), 0, s,
                           reinterpret_cast<const int32_t*>(ptr), n_rows, n_edges, row);
    return hipGetLastError();
}

hipError_t launch_inverse(const int32_t* perm, int64_t n, int32_t* pos, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(inverse_kernel, dim3(grid_1d(n)), dim3(256), 0, s, perm, n, pos);
    return hipGetLastError();
}

hipError_t launch_winner_bits(const int32_t* arg_e, int64_t n_rows, int32_t D, int64_t ld,
                              const int32_t* pos_of_edge, uint32_t* bits, int64_t n_edges, int32_t words,
                              hipStream_t s) {
    const int64_t nw = n_edges * words, n = n_rows * D;
    if (nw > 0) hipLaunchKernelGGL(zero_words_kernel, dim3(grid_1d(nw)), dim3(256), 0, s, bits, nw);
    if (n > 0)
        hipLaunchKernelGGL(winner_bits_kernel, dim3(grid_1d(n_rows * words * 32)), dim3(256), 0, s, arg_e, n_rows,
                           D, ld, pos_of_edge, bits, words, n_edges);
    return hipGetLastError();
}

hipError_t launch_winner_rows(const WinnerRowsArgs& a, int ptr64, int64_t n_edges, hipStream_t s) {
    const int64_t nw = n_edges * a.words, units = a.n_seg + a.n_small;
    if (nw > 0) hipLaunchKernelGGL(zero_words_kernel, dim3(grid_1d(nw)), dim3(256), 0, s, a.bits, nw);
    if (units <= 0 || a.D <= 0) return hipGetLastError();
    const dim3 grid((unsigned)(units < 65536 ? units : 65536));
    if (ptr64) hipLaunchKernelGGL(winner_rows_kernel<int64_t>, grid, dim3(64), 0, s, a);
    else hipLaunchKernelGGL(winner_rows_kernel<int32_t>, grid, dim3(64), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_iota(int32_t* out, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(iota_kernel, dim3(grid_1d(n)), dim3(256), 0, s, out, n);
    return hipGetLastError();
}

hipError_t launch_copy_ptr(const void* src, int src64, void* dst, int dst64, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(copy_ptr_kernel, dim3(grid_1d(n)), dim3(256), 0, s, src, src64, dst, dst64, n);
    return hipGetLastError();
}

}  // namespace gnnk
