/*
 * Seeded synthetic inputs: graphs shaped like the paper's workloads and dense
 * feature tensors.  This module is shared by the oracle tests and by the GPU
 * path's tests and benchmark; it holds none of the message-passing
 * arithmetic (no gather, reduce, softmax or gradient): only random draws,
 * graph construction and sorting of edge lists.
 *
 * Random numbers come from a counter-based use of SplitMix64 (Steele, Lea and
 * Flood, "Fast splittable pseudorandom number generators", OOPSLA 2014): the
 * i-th value of stream s under seed k is the SplitMix64 finaliser applied to
 * key(k, s) + (i + 1) * gamma.  Every value depends only on (seed, stream,
 * index), so the OpenMP-parallel loops below give identical output for any
 * thread count.
 *
 * Edge order convention for every generated graph: edges are sorted by
 * (destination, source); the edge id is the position in that order.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define SM_GAMMA 0x9E3779B97F4A7C15ULL

static inline uint64_t sm_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t sm_key(uint64_t seed, uint64_t stream) {
    return sm_mix(sm_mix(seed * SM_GAMMA + 0x632BE59BD9B4E019ULL) ^ sm_mix(stream + SM_GAMMA));
}

static inline uint64_t sm_at(uint64_t key, uint64_t i) { return sm_mix(key + (i + 1) * SM_GAMMA); }

/* uniform integer in [0, n) by the 64x64->128 multiply-high method */
static inline uint64_t sm_below(uint64_t r, uint64_t n) {
    return (uint64_t)(((unsigned __int128)r * (unsigned __int128)n) >> 64);
}

static inline double sm_unit53(uint64_t r) { return (double)(r >> 11) * 0x1.0p-53; }

/* ------------------------------------------------------------------------ */
/* dense fills                                                               */

void synth_fill_normal_f32(uint64_t seed, uint64_t stream, int64_t n, float* out) {
    const uint64_t key = sm_key(seed, stream);
    const int64_t npair = (n + 1) / 2;
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < npair; ++j) {
        /* Box-Muller on two uniforms; u1 in (0,1] so the log is finite */
        double u1 = ((double)(sm_at(key, 2 * (uint64_t)j) >> 11) + 1.0) * 0x1.0p-53;
        double u2 = sm_unit53(sm_at(key, 2 * (uint64_t)j + 1));
        double r = sqrt(-2.0 * log(u1));
        double t = 6.283185307179586476925286766559 * u2;
        out[2 * j] = (float)(r * cos(t));
        if (2 * j + 1 < n) out[2 * j + 1] = (float)(r * sin(t));
    }
}

void synth_fill_uniform_f32(uint64_t seed, uint64_t stream, int64_t n, float lo, float hi, float* out) {
    const uint64_t key = sm_key(seed, stream);
    const double a = lo, w = (double)hi - (double)lo;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double u = (double)(sm_at(key, (uint64_t)i) >> 40) * 0x1.0p-24; /* [0,1) on a 2^-24 grid */
        out[i] = (float)(a + w * u);
    }
}

/* round-to-nearest-even fp32 -> bf16 (inputs only; NaN never generated) */
void synth_f32_to_bf16(int64_t n, const float* in, uint16_t* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b;
        memcpy(&b, &in[i], 4);
        uint32_t lsb = (b >> 16) & 1u;
        b += 0x7FFFu + lsb;
        out[i] = (uint16_t)(b >> 16);
    }
}

/* random permutation of [0, n) by Fisher-Yates driven by the counter stream */
void synth_permutation(uint64_t seed, uint64_t stream, int64_t n, int32_t* perm) {
    const uint64_t key = sm_key(seed, stream);
    for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
    for (int64_t i = n - 1; i > 0; --i) {
        int64_t j = (int64_t)sm_below(sm_at(key, (uint64_t)i), (uint64_t)(i + 1));
        int32_t t = perm[i];
        perm[i] = perm[j];
        perm[j] = t;
    }
}

/* ------------------------------------------------------------------------ */
/* stable parallel LSD radix sort of 64-bit keys (12-bit digits)            */

static int sort_keys(uint64_t* keys, int64_t n, int key_bits) {
    if (n <= 1 || key_bits <= 0) return 0;
    uint64_t* tmp = (uint64_t*)malloc((size_t)n * sizeof(uint64_t));
    if (!tmp) return -1;
    const int RB = 12, NB = 1 << RB;
    int nthreads = 1;
#ifdef _OPENMP
    nthreads = omp_get_max_threads();
#endif
    int64_t* hist = (int64_t*)malloc((size_t)nthreads * NB * sizeof(int64_t));
    if (!hist) { free(tmp); return -1; }
    uint64_t *src = keys, *dst = tmp;
    for (int shift = 0; shift < key_bits; shift += RB) {
        memset(hist, 0, (size_t)nthreads * NB * sizeof(int64_t));
#pragma omp parallel num_threads(nthreads)
        {
            int t = 0;
#ifdef _OPENMP
            t = omp_get_thread_num();
#endif
            int64_t lo = n * t / nthreads, hi = n * (t + 1) / nthreads;
            int64_t* h = hist + (size_t)t * NB;
            for (int64_t i = lo; i < hi; ++i) h[(src[i] >> shift) & (NB - 1)]++;
#pragma omp barrier
#pragma omp single
            {
                int64_t run = 0;
                for (int d = 0; d < NB; ++d)
                    for (int tt = 0; tt < nthreads; ++tt) {
                        int64_t c = hist[(size_t)tt * NB + d];
                        hist[(size_t)tt * NB + d] = run;
                        run += c;
                    }
            }
            for (int64_t i = lo; i < hi; ++i) {
                uint64_t k = src[i];
                dst[h[(k >> shift) & (NB - 1)]++] = k;
            }
        }
        uint64_t* s = src;
        src = dst;
        dst = s;
    }
    if (src != keys) memcpy(keys, src, (size_t)n * sizeof(uint64_t));
    free(hist);
    free(tmp);
    return 0;
}

static int bits_for(int64_t n) {
    int b = 0;
    while (b < 62 && ((int64_t)1 << b) < n) ++b;
    return b;
}

/* Sort an edge list by (dst, src); edges with equal (dst, src) are identical,
 * so the packed key alone carries the whole edge. */
int synth_sort_coo(int64_t n_edges, int32_t* src, int32_t* dst, int64_t n_src, int64_t n_dst) {
    int sb = bits_for(n_src), db = bits_for(n_dst);
    if (sb + db > 64) return -2;
    uint64_t* keys = (uint64_t*)malloc((size_t)(n_edges > 0 ? n_edges : 1) * sizeof(uint64_t));
    if (!keys) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_edges; ++i)
        keys[i] = ((uint64_t)(uint32_t)dst[i] << sb) | (uint64_t)(uint32_t)src[i];
    if (sort_keys(keys, n_edges, sb + db)) { free(keys); return -1; }
    const uint64_t smask = (sb == 0) ? 0 : ((1ULL << sb) - 1);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_edges; ++i) {
        src[i] = (int32_t)(keys[i] & smask);
        dst[i] = (int32_t)(keys[i] >> sb);
    }
    free(keys);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* uniform random multigraph                                                */

void synth_uniform_edges(uint64_t seed, uint64_t stream, int64_t n_edges, int64_t n_src, int64_t n_dst,
                         int32_t* src, int32_t* dst) {
    const uint64_t key = sm_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_edges; ++i) {
        src[i] = (int32_t)sm_below(sm_at(key, 2 * (uint64_t)i), (uint64_t)n_src);
        dst[i] = (int32_t)sm_below(sm_at(key, 2 * (uint64_t)i + 1), (uint64_t)n_dst);
    }
}

/* draws from a discrete distribution given by its cumulative weights (cdf[k] = sum of w[0..k]) */
static inline int64_t draw_cdf(const double* cdf, int64_t k, uint64_t r) {
    double u = sm_unit53(r) * cdf[k - 1];
    int64_t lo = 0, hi = k - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (cdf[mid] > u) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

/* truncated Zipf over {0..k-1}: P(r) proportional to (r+1)^-s */
void synth_zipf(uint64_t seed, uint64_t stream, int64_t n, int32_t k, double s, int32_t* out) {
    double* cdf = (double*)malloc((size_t)k * sizeof(double));
    double run = 0;
    for (int32_t r = 0; r < k; ++r) {
        run += pow((double)(r + 1), -s);
        cdf[r] = run;
    }
    const uint64_t key = sm_key(seed, stream);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (int32_t)draw_cdf(cdf, k, sm_at(key, (uint64_t)i));
    free(cdf);
}

/*
 * Chung-Lu graph: node of rank i (after a random relabelling) has weight
 * (i+1)^(-1/(gamma-1)); n_draws (src, dst) pairs are drawn independently in
 * proportion to the weights; self-loops and duplicate pairs are dropped, then
 * one self-loop per node is added.  Returns the edge count (<= n_draws + n) and
 * writes edges sorted by (dst, src).  src/dst must hold n_draws + n entries.
 */
int64_t synth_chung_lu(uint64_t seed, int64_t n, int64_t n_draws, double gamma, int32_t* src, int32_t* dst) {
    int32_t* perm = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    double* cdf = (double*)malloc((size_t)n * sizeof(double));
    synth_permutation(seed, 1, n, perm);
    double run = 0, ex = -1.0 / (gamma - 1.0);
    for (int64_t i = 0; i < n; ++i) {
        run += pow((double)(i + 1), ex);
        cdf[i] = run;
    }
    const uint64_t key = sm_key(seed, 2);
    uint64_t* keys = (uint64_t*)malloc((size_t)(n_draws + 1) * sizeof(uint64_t));
    int64_t m = 0;
    int nb = bits_for(n);
    for (int64_t i = 0; i < n_draws; ++i) {
        int32_t u = perm[draw_cdf(cdf, n, sm_at(key, 2 * (uint64_t)i))];
        int32_t v = perm[draw_cdf(cdf, n, sm_at(key, 2 * (uint64_t)i + 1))];
        if (u == v) continue;
        keys[m++] = ((uint64_t)(uint32_t)v << nb) | (uint64_t)(uint32_t)u;
    }
    sort_keys(keys, m, 2 * nb);
    int64_t w = 0;
    for (int64_t i = 0; i < m; ++i)
        if (i == 0 || keys[i] != keys[i - 1]) keys[w++] = keys[i];
    int64_t e = 0;
    for (int64_t i = 0; i < w; ++i) {
        src[e] = (int32_t)(keys[i] & ((1ULL << nb) - 1));
        dst[e] = (int32_t)(keys[i] >> nb);
        ++e;
    }
    for (int64_t i = 0; i < n; ++i) {
        src[e] = (int32_t)i;
        dst[e] = (int32_t)i;
        ++e;
    }
    free(keys);
    free(cdf);
    free(perm);
    synth_sort_coo(e, src, dst, n, n);
    return e;
}

/*
 * R-MAT graph (Chakrabarti, Zhan and Faloutsos, SDM 2004) on 2^scale ids with
 * quadrant probabilities (a, b, c, 1-a-b-c): quadrant a keeps both bits 0, b
 * sets the destination bit, c sets the source bit, d sets both; one level per
 * bit, most significant first, 16 random bits per level.  Draws with an id >=
 * n are rejected, (src, dst) pairs are deduplicated, exactly n_edges distinct
 * pairs are kept uniformly at random (the n_edges smallest of a per-pair
 * random priority), node ids are relabelled by a random permutation, and the
 * result is sorted by (dst, src).  Draws are taken in batches until enough
 * distinct pairs exist.  Returns n_edges, or a negative value on failure.
 */
int64_t synth_rmat(uint64_t seed, int scale, double a, double b, double c, int64_t n, int64_t n_edges,
                   int32_t* src, int32_t* dst) {
    if (scale < 1 || scale > 30 || n > ((int64_t)1 << scale) || n_edges <= 0) return -2;
    const uint32_t ta = (uint32_t)llround(a * 65536.0);
    const uint32_t tab = (uint32_t)llround((a + b) * 65536.0);
    const uint32_t tabc = (uint32_t)llround((a + b + c) * 65536.0);
    const int nb = scale;
    const int words = (scale + 3) / 4; /* 4 levels of 16 bits per 64-bit draw */
    const uint64_t key = sm_key(seed, 3);
    int nthreads = 1;
#ifdef _OPENMP
    nthreads = omp_get_max_threads();
#endif
    int64_t cap = n_edges + n_edges / 2 + 1024, count = 0, uniq = 0;
    uint64_t* keys = (uint64_t*)malloc((size_t)cap * sizeof(uint64_t));
    if (!keys) return -1;
    int64_t next_draw = 0;
    int64_t batch = n_edges + n_edges * 3 / 4; /* first batch: 1.75x oversample */
    int64_t* tcount = (int64_t*)malloc((size_t)nthreads * sizeof(int64_t));
    for (int round = 0; round < 64; ++round) {
        /* accepted draws of this batch, appended in draw order */
        uint64_t* bk = (uint64_t*)malloc((size_t)batch * sizeof(uint64_t));
        if (!bk) { free(keys); free(tcount); return -1; }
#pragma omp parallel num_threads(nthreads)
        {
            int t = 0;
#ifdef _OPENMP
            t = omp_get_thread_num();
#endif
            int64_t lo = batch * t / nthreads, hi = batch * (t + 1) / nthreads, w = lo;
            for (int64_t i = lo; i < hi; ++i) {
                uint64_t d = (uint64_t)(next_draw + i);
                uint32_t s = 0, v = 0;
                int lvl = 0;
                for (int wd = 0; wd < words && lvl < scale; ++wd) {
                    uint64_t r = sm_at(key, d * (uint64_t)words + (uint64_t)wd);
                    for (int q = 0; q < 4 && lvl < scale; ++q, ++lvl) {
                        uint32_t x = (uint32_t)(r >> (16 * q)) & 0xFFFFu;
                        uint32_t sb = x >= tab;                       /* quadrants c, d */
                        uint32_t db = (x >= ta && x < tab) || x >= tabc; /* quadrants b, d */
                        s = (s << 1) | sb;
                        v = (v << 1) | db;
                    }
                }
                if ((int64_t)s < n && (int64_t)v < n) bk[w++] = ((uint64_t)v << nb) | (uint64_t)s;
            }
            tcount[t] = w - lo;
#pragma omp barrier
#pragma omp single
            {
                int64_t need = uniq;
                for (int tt = 0; tt < nthreads; ++tt) need += tcount[tt];
                if (need > cap) {
                    cap = need;
                    keys = (uint64_t*)realloc(keys, (size_t)cap * sizeof(uint64_t));
                }
                int64_t off = uniq;
                for (int tt = 0; tt < nthreads; ++tt) {
                    memcpy(keys + off, bk + batch * tt / nthreads, (size_t)tcount[tt] * sizeof(uint64_t));
                    off += tcount[tt];
                }
                count = off;
            }
        }
        free(bk);
        if (!keys) { free(tcount); return -1; }
        next_draw += batch;
        sort_keys(keys, count, 2 * nb);
        int64_t w = 0;
        for (int64_t i = 0; i < count; ++i)
            if (i == 0 || keys[i] != keys[i - 1]) keys[w++] = keys[i];
        uniq = w;
        if (uniq >= n_edges) break;
        batch = n_edges / 4 + 1;
    }
    free(tcount);
    if (uniq < n_edges) { free(keys); return -3; }
    /* keep the n_edges pairs of smallest random priority: a histogram of the
     * priorities' top bits finds the bucket holding the cut, which is then
     * sorted on its own; equal priorities are taken in key order */
    if (uniq > n_edges) {
        const uint64_t pkey = sm_key(seed, 4);
        const int HB = 20;
        const int64_t NBK = (int64_t)1 << HB;
        int64_t* hcount = (int64_t*)calloc((size_t)NBK, sizeof(int64_t));
        for (int64_t i = 0; i < uniq; ++i) hcount[sm_mix(pkey ^ sm_mix(keys[i])) >> (64 - HB)]++;
        int64_t below = 0, cut = 0;
        while (below + hcount[cut] < n_edges) below += hcount[cut++];
        int64_t nin = hcount[cut];
        free(hcount);
        uint64_t* inb = (uint64_t*)malloc((size_t)(nin > 0 ? nin : 1) * sizeof(uint64_t));
        int64_t k = 0;
        for (int64_t i = 0; i < uniq; ++i) {
            uint64_t p = sm_mix(pkey ^ sm_mix(keys[i]));
            if ((int64_t)(p >> (64 - HB)) == cut) inb[k++] = p;
        }
        sort_keys(inb, nin, 64);
        uint64_t thr = inb[n_edges - below - 1];
        int64_t take_eq = 0;
        for (int64_t i = 0; i < n_edges - below; ++i) take_eq += inb[i] == thr;
        free(inb);
        int64_t w = 0;
        for (int64_t i = 0; i < uniq; ++i) {
            uint64_t p = sm_mix(pkey ^ sm_mix(keys[i]));
            if (p < thr || (p == thr && take_eq-- > 0)) keys[w++] = keys[i];
        }
        uniq = w;
    }
    int32_t* perm = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    synth_permutation(seed, 5, n, perm);
    const uint64_t m = (1ULL << nb) - 1;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_edges; ++i) {
        src[i] = perm[keys[i] & m];
        dst[i] = perm[keys[i] >> nb];
    }
    free(perm);
    free(keys);
    if (synth_sort_coo(n_edges, src, dst, n, n)) return -1;
    return n_edges;
}

/* number of edges sharing (dst, etype) with each edge, for the relational workload */
void synth_count_dst_type(int64_t n_edges, int64_t n_dst, int32_t n_types, const int32_t* dst,
                          const int32_t* etype, int32_t* count_out) {
    int64_t cells = n_dst * (int64_t)n_types;
    int32_t* cnt = (int32_t*)calloc((size_t)cells, sizeof(int32_t));
    for (int64_t e = 0; e < n_edges; ++e) cnt[(int64_t)dst[e] * n_types + etype[e]]++;
    for (int64_t e = 0; e < n_edges; ++e) count_out[e] = cnt[(int64_t)dst[e] * n_types + etype[e]];
    free(cnt);
}

/* count occurrences of each value of idx in [0, n) (graph statistics and GCN edge weights) */
void synth_bincount(int64_t m, const int32_t* idx, int64_t n, int64_t* out) {
    memset(out, 0, (size_t)n * sizeof(int64_t));
    for (int64_t i = 0; i < m; ++i) out[idx[i]]++;
}
