// Graph formats built on the device (Section 4.1: the in-CSR for g-SpMM, the
// reverse graph's CSR for the backward pass; Appendix B: the reverse graph
// keeps the edge ids).
//
// A CSR is a stable sort of the edge list by row key: sorting the pairs
// (row of edge e, e) by row with a stable LSD radix sort leaves the edges of
// every row in ascending edge id, which is the order the kernels and the
// oracle reduce in.  Row offsets are then binary searches in the sorted keys
// (no atomics: every result is a pure function of the edge list), and a third
// stable sort, on (capacity - degree, row), gives the rows by descending
// degree with ties in ascending row id.
//
// Radix pass: 8-bit digits, 4,096 keys per workgroup.  Each wavefront ranks
// its 1,024 keys in 16 steps of 64: lanes with equal digits find each other
// with eight ballots, take their rank within the step from a popcount, and
// read the running count of their digit from the wavefront's LDS counters.
// Counts of all workgroups are scanned digit-major, so equal digits keep
// their input order across workgroups as well.
#include "device.h"

namespace gnnk {
namespace {

constexpr int RS_WAVES = 4;
constexpr int RS_STEPS = 16;                       // 64-key steps per wavefront
constexpr int RS_TILE = RS_WAVES * 64 * RS_STEPS;  // keys per workgroup
constexpr int SCAN_ITEMS = 16;
constexpr int SCAN_TILE = 256 * SCAN_ITEMS;

inline unsigned tiles_of(int64_t n, int64_t per) { return (unsigned)((n + per - 1) / per); }

inline unsigned grid_1d(int64_t n) {
    int64_t b = (n + 255) / 256;
    if (b > 65536) b = 65536;
    return (unsigned)(b > 0 ? b : 1);
}

// ---------------------------------------------------------------------------
// radix sort

__global__ __launch_bounds__(256) void rs_count_kernel(const uint32_t* keys, int64_t n, int shift, uint32_t* hist,
                                                       int64_t n_tiles) {
    __shared__ uint32_t c[256];
    c[threadIdx.x] = 0u;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * RS_TILE;
    for (int j = 0; j < RS_TILE / 256; ++j) {
        const int64_t i = base + j * 256 + threadIdx.x;
        if (i < n) atomicAdd(&c[(keys[i] >> shift) & 255u], 1u);
    }
    __syncthreads();
    hist[(int64_t)threadIdx.x * n_tiles + blockIdx.x] = c[threadIdx.x];
}

// hist holds the exclusive digit-major scan of the counts: the first output
// position of (digit, workgroup)
__global__ __launch_bounds__(256) void rs_scatter_kernel(const uint32_t* keys, const uint32_t* vals, int64_t n,
                                                         int shift, const uint32_t* hist, int64_t n_tiles,
                                                         uint32_t* keys_out, uint32_t* vals_out) {
    __shared__ uint32_t cnt[RS_WAVES][256];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int i = threadIdx.x; i < RS_WAVES * 256; i += 256) (&cnt[0][0])[i] = 0u;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * RS_TILE + (int64_t)w * (64 * RS_STEPS);
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    uint32_t k[RS_STEPS], v[RS_STEPS], rank[RS_STEPS];
#pragma unroll
    for (int j = 0; j < RS_STEPS; ++j) {
        const int64_t i = base + j * 64 + lane;
        const bool ok = i < n;
        k[j] = ok ? keys[i] : 0u;
        v[j] = ok ? (vals ? vals[i] : (uint32_t)i) : 0u;
        const uint32_t d = (k[j] >> shift) & 255u;
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const uint64_t m = __ballot((d >> b) & 1u);
            peers &= ((d >> b) & 1u) ? m : ~m;
        }
        // every lane reads its digit's count before the last lane of each
        // digit group advances it (one LDS read, then one LDS write, in the
        // wavefront's program order)
        const uint32_t start = cnt[w][d];
        rank[j] = start + (uint32_t)__popcll(peers & below);
        __builtin_amdgcn_wave_barrier();
        if (ok && (peers >> lane) == 1ull) cnt[w][d] = start + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    {
        const int d = threadIdx.x;
        uint32_t run = hist[(int64_t)d * n_tiles + blockIdx.x];
#pragma unroll
        for (int ww = 0; ww < RS_WAVES; ++ww) {
            const uint32_t c = cnt[ww][d];
            cnt[ww][d] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < RS_STEPS; ++j) {
        const int64_t i = base + j * 64 + lane;
        if (i < n) {
            const uint32_t p = cnt[w][(k[j] >> shift) & 255u] + rank[j];
            keys_out[p] = k[j];
            vals_out[p] = v[j];
        }
    }
}

__global__ void copy_pairs_kernel(const uint32_t* keys, const uint32_t* vals, int64_t n, uint32_t* keys_out,
                                  uint32_t* vals_out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        keys_out[i] = keys[i];
        vals_out[i] = vals ? vals[i] : (uint32_t)i;
    }
}

// ---------------------------------------------------------------------------
// exclusive scan of uint32 counts (in place)

__device__ uint32_t block_exclusive(uint32_t v, uint32_t* total) {
    __shared__ uint32_t wsum[4];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint32_t inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_up(inc, o, 64);
        if (lane >= o) inc += t;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    uint32_t off = 0u, tot = 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t t = wsum[i];
        if (i < w) off += t;
        tot += t;
    }
    __syncthreads();  // wsum is reused by the next call
    *total = tot;
    return off + inc - v;
}

__device__ uint32_t scan_tile(uint32_t* x, int64_t n, int64_t tile, uint32_t carry) {
    const int64_t b = tile + (int64_t)threadIdx.x * SCAN_ITEMS;
    uint32_t v[SCAN_ITEMS], s = 0u;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
        v[j] = b + j < n ? x[b + j] : 0u;
        s += v[j];
    }
    uint32_t total;
    uint32_t pre = block_exclusive(s, &total) + carry;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
        if (b + j < n) x[b + j] = pre;
        pre += v[j];
    }
    return total;
}

__global__ __launch_bounds__(256) void scan_reduce_kernel(const uint32_t* x, int64_t n, uint32_t* part) {
    const int64_t b = (int64_t)blockIdx.x * SCAN_TILE + (int64_t)threadIdx.x * SCAN_ITEMS;
    uint32_t s = 0u;
    for (int j = 0; j < SCAN_ITEMS; ++j)
        if (b + j < n) s += x[b + j];
    uint32_t total;
    (void)block_exclusive(s, &total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

// one workgroup: the tile sums, scanned tile by tile with a running carry
__global__ __launch_bounds__(256) void scan_carry_kernel(uint32_t* part, int64_t n) {
    uint32_t carry = 0u;
    for (int64_t t = 0; t < n; t += SCAN_TILE) carry += scan_tile(part, n, t, carry);
}

__global__ __launch_bounds__(256) void scan_apply_kernel(uint32_t* x, int64_t n, const uint32_t* part) {
    (void)scan_tile(x, n, (int64_t)blockIdx.x * SCAN_TILE, part[blockIdx.x]);
}

// ---------------------------------------------------------------------------
// structure from sorted keys

// offsets[r] = first position whose key is >= r, for r in [0, n_rows]
template <typename P>
__global__ void ptr_from_keys_kernel(const uint32_t* keys, int64_t n_keys, int64_t n_rows, P* ptr) {
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r <= n_rows;
         r += (int64_t)gridDim.x * blockDim.x) {
        int64_t lo = 0, hi = n_keys;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if ((int64_t)keys[mid] < r) lo = mid + 1;
            else hi = mid;
        }
        ptr[r] = (P)lo;
    }
}

template <typename P>
__global__ void degree_kernel(const P* ptr, int64_t n_rows, int32_t* deg, uint32_t* deg_key, uint32_t cap) {
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < n_rows;
         r += (int64_t)gridDim.x * blockDim.x) {
        const int32_t d = (int32_t)((int64_t)ptr[r + 1] - (int64_t)ptr[r]);
        deg[r] = d;
        deg_key[r] = cap - (uint32_t)d;
    }
}

__global__ void gather_kernel(const int32_t* table, const uint32_t* idx, int64_t n, int32_t* out) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x)
        out[p] = table[idx[p]];
}

__global__ void check_identity_kernel(const int32_t* eid, int64_t n, int32_t* flag, int32_t bit) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x)
        if (eid[p] != (int32_t)p) atomicOr(flag, bit);
}

__global__ void count_ids_kernel(const int32_t* eid, int64_t n, uint32_t* counts, int32_t* flag, int32_t bit) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x) {
        const int32_t e = eid[p];
        if (e < 0 || e >= n) atomicOr(flag, bit);
        else atomicAdd(counts + e, 1u);
    }
}

__global__ void check_once_kernel(const uint32_t* counts, int64_t n, int32_t* flag, int32_t bit) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        if (counts[i] != 1u) atomicOr(flag, bit);
}

__global__ void fill_u32_kernel(uint32_t* x, int64_t n, uint32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        x[i] = v;
}

// endpoints of every edge id from a CSR with explicit edge ids
__global__ void edge_ends_kernel(const int32_t* idx, const int32_t* eid, const int32_t* row, int64_t n,
                                 int32_t* src_of_e, int32_t* dst_of_e) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n; p += (int64_t)gridDim.x * blockDim.x) {
        const int32_t e = eid[p];
        src_of_e[e] = idx[p];
        dst_of_e[e] = row[p];
    }
}

template <typename P>
__global__ void hub_segments_kernel(const P* ptr, const int32_t* perm, const int32_t* hub_off, int64_t n_hub,
                                    int64_t seg_edges, int4* seg) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n_hub;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t r = perm[k];
        const int64_t b = (int64_t)ptr[r], e = (int64_t)ptr[r + 1];
        int32_t o = hub_off[k];
        for (int64_t s = b; s < e; s += seg_edges, ++o)
            seg[o] = make_int4(r, (int32_t)s, (int32_t)(s + seg_edges < e ? s + seg_edges : e), (int32_t)k);
    }
}

}  // namespace

// ---------------------------------------------------------------------------
// host launchers

int key_bits(uint64_t max_key) { return max_key == 0 ? 0 : 64 - __builtin_clzll(max_key); }

size_t radix_scratch_words(int64_t n) {
    const int64_t hist = 256 * (int64_t)tiles_of(n, RS_TILE);
    return (size_t)(hist + tiles_of(hist, SCAN_TILE) + 64);
}

hipError_t scan_exclusive_u32(uint32_t* x, int64_t n, uint32_t* part, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const unsigned tiles = tiles_of(n, SCAN_TILE);
    hipLaunchKernelGGL(scan_reduce_kernel, dim3(tiles), dim3(256), 0, s, x, n, part);
    hipLaunchKernelGGL(scan_carry_kernel, dim3(1), dim3(256), 0, s, part, (int64_t)tiles);
    hipLaunchKernelGGL(scan_apply_kernel, dim3(tiles), dim3(256), 0, s, x, n, part);
    return hipGetLastError();
}

hipError_t radix_sort_pairs(const uint32_t* keys_in, const uint32_t* vals_in, int64_t n, int bits,
                            uint32_t* keys_out, uint32_t* vals_out, uint32_t* tmp_keys, uint32_t* tmp_vals,
                            uint32_t* scratch, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int passes = (bits + 7) / 8;
    if (passes == 0) {
        hipLaunchKernelGGL(copy_pairs_kernel, dim3(grid_1d(n)), dim3(256), 0, s, keys_in, vals_in, n, keys_out,
                           vals_out);
        return hipGetLastError();
    }
    const int64_t n_tiles = tiles_of(n, RS_TILE);
    uint32_t* hist = scratch;
    uint32_t* part = scratch + 256 * n_tiles;
    const uint32_t* k_src = keys_in;
    const uint32_t* v_src = vals_in;
    for (int pass = 0; pass < passes; ++pass) {
        // the last pass lands in the output buffers
        const bool to_out = ((passes - 1 - pass) % 2) == 0;
        uint32_t* k_dst = to_out ? keys_out : tmp_keys;
        uint32_t* v_dst = to_out ? vals_out : tmp_vals;
        const int shift = 8 * pass;
        hipLaunchKernelGGL(rs_count_kernel, dim3((unsigned)n_tiles), dim3(256), 0, s, k_src, n, shift, hist, n_tiles);
        hipError_t e = scan_exclusive_u32(hist, 256 * n_tiles, part, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(rs_scatter_kernel, dim3((unsigned)n_tiles), dim3(256), 0, s, k_src, v_src, n, shift,
                           hist, n_tiles, k_dst, v_dst);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        k_src = k_dst;
        v_src = v_dst;
    }
    return hipSuccess;
}

hipError_t launch_ptr_from_keys(const uint32_t* keys, int64_t n_keys, int64_t n_rows, void* ptr, int ptr64,
                                hipStream_t s) {
    dim3 grid(grid_1d(n_rows + 1)), block(256);
    if (ptr64)
        hipLaunchKernelGGL(ptr_from_keys_kernel<int64_t>, grid, block, 0, s, keys, n_keys, n_rows, (int64_t*)ptr);
    else
        hipLaunchKernelGGL(ptr_from_keys_kernel<int32_t>, grid, block, 0, s, keys, n_keys, n_rows, (int32_t*)ptr);
    return hipGetLastError();
}

hipError_t launch_degrees(const void* ptr, int ptr64, int64_t n_rows, int32_t* deg, uint32_t* deg_key, uint32_t cap,
                          hipStream_t s) {
    if (n_rows <= 0) return hipSuccess;
    dim3 grid(grid_1d(n_rows)), block(256);
    if (ptr64)
        hipLaunchKernelGGL(degree_kernel<int64_t>, grid, block, 0, s, (const int64_t*)ptr, n_rows, deg, deg_key, cap);
    else
        hipLaunchKernelGGL(degree_kernel<int32_t>, grid, block, 0, s, (const int32_t*)ptr, n_rows, deg, deg_key, cap);
    return hipGetLastError();
}

hipError_t launch_gather(const int32_t* table, const uint32_t* idx, int64_t n, int32_t* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_kernel, dim3(grid_1d(n)), dim3(256), 0, s, table, idx, n, out);
    return hipGetLastError();
}

hipError_t launch_check_identity(const int32_t* eid, int64_t n, int32_t* flag, int32_t bit, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(check_identity_kernel, dim3(grid_1d(n)), dim3(256), 0, s, eid, n, flag, bit);
    return hipGetLastError();
}

hipError_t launch_check_permutation(const int32_t* eid, int64_t n, uint32_t* counts, int32_t* flag, int32_t bit,
                                    hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(grid_1d(n)), dim3(256), 0, s, counts, n, 0u);
    hipLaunchKernelGGL(count_ids_kernel, dim3(grid_1d(n)), dim3(256), 0, s, eid, n, counts, flag, bit);
    hipLaunchKernelGGL(check_once_kernel, dim3(grid_1d(n)), dim3(256), 0, s, counts, n, flag, bit);
    return hipGetLastError();
}

hipError_t launch_edge_ends(const int32_t* idx, const int32_t* eid, const int32_t* row, int64_t n, int32_t* src_of_e,
                            int32_t* dst_of_e, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(edge_ends_kernel, dim3(grid_1d(n)), dim3(256), 0, s, idx, eid, row, n, src_of_e, dst_of_e);
    return hipGetLastError();
}

// sort key of each hub segment: the halves of its first and last neighbour
// id, summed (below the neighbour count, so it fits the key's bits)
__global__ void seg_keys_kernel(const int4* seg, int64_t n_seg, const int32_t* idx, uint32_t* key) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n_seg; k += (int64_t)gridDim.x * blockDim.x) {
        const int4 s = seg[k];
        key[k] = ((uint32_t)idx[s.y] >> 1) + ((uint32_t)idx[s.z - 1] >> 1);
    }
}

hipError_t launch_seg_keys(const int4* seg, int64_t n_seg, const int32_t* idx, uint32_t* key, hipStream_t s) {
    if (n_seg <= 0) return hipSuccess;
    hipLaunchKernelGGL(seg_keys_kernel, dim3(grid_1d(n_seg)), dim3(256), 0, s, seg, n_seg, idx, key);
    return hipGetLastError();
}

namespace {

// the segment of each hub-segment wavefront, with its table index: the walk
// then finds its segment with one load instead of two dependent ones
__global__ void seg_wave_kernel(const int4* seg, const int32_t* order, int64_t n_seg, int4* segw) {
    for (int64_t w = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; w < n_seg; w += (int64_t)gridDim.x * blockDim.x) {
        const int32_t si = order[w];
        const int4 t = seg[si];
        segw[w] = make_int4(t.x, t.y, t.z, si);
    }
}

// {row, begin, end, 0} of every row in degree order
template <typename P>
__global__ void row_table_kernel(const P* ptr, const int32_t* perm, int64_t n_rows, int4* rowt) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n_rows; k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t r = perm[k];
        rowt[k] = make_int4(r, (int32_t)ptr[r], (int32_t)ptr[r + 1], 0);
    }
}

}  // namespace

hipError_t launch_seg_wave(const int4* seg, const int32_t* order, int64_t n_seg, int4* segw, hipStream_t s) {
    if (n_seg <= 0) return hipSuccess;
    hipLaunchKernelGGL(seg_wave_kernel, dim3(grid_1d(n_seg)), dim3(256), 0, s, seg, order, n_seg, segw);
    return hipGetLastError();
}

hipError_t launch_row_table(const void* ptr, int ptr64, const int32_t* perm, int64_t n_rows, int4* rowt,
                            hipStream_t s) {
    if (n_rows <= 0) return hipSuccess;
    dim3 grid(grid_1d(n_rows)), block(256);
    if (ptr64)
        hipLaunchKernelGGL(row_table_kernel<int64_t>, grid, block, 0, s, (const int64_t*)ptr, perm, n_rows, rowt);
    else
        hipLaunchKernelGGL(row_table_kernel<int32_t>, grid, block, 0, s, (const int32_t*)ptr, perm, n_rows, rowt);
    return hipGetLastError();
}

hipError_t launch_hub_segments(const void* ptr, int ptr64, const int32_t* perm, const int32_t* hub_off, int64_t n_hub,
                               int64_t seg_edges, int4* seg, hipStream_t s) {
    if (n_hub <= 0) return hipSuccess;
    dim3 grid(grid_1d(n_hub)), block(256);
    if (ptr64)
        hipLaunchKernelGGL(hub_segments_kernel<int64_t>, grid, block, 0, s, (const int64_t*)ptr, perm, hub_off, n_hub,
                           seg_edges, seg);
    else
        hipLaunchKernelGGL(hub_segments_kernel<int32_t>, grid, block, 0, s, (const int32_t*)ptr, perm, hub_off, n_hub,
                           seg_edges, seg);
    return hipGetLastError();
}

}  // namespace gnnk
