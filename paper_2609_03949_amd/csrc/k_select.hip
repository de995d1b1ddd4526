// k_select.hip -- exact per-sequence top-k and the certified two-tier admission.
//
// Selection (per sequence b, archive rows [0, A)), given fp32 keys key~ with a
// certified bound |key~ - key| <= E for every row (key = the fp64 index score,
// E from the per-sequence maxima of ||qt_h|| and ||x_u||).  Three launches:
//   1. bracket (one block per sequence): a strided sample of the keys places
//      [t_lo, t_hi] around the k-th largest key~ and fixes the early bounds
//      CLO = down(t_lo - E), CHI = up(t_hi + E);
//   2. count (one block per 4096 rows): rows with key~ - E > CHI are certainly
//      selected, rows with key~ + E < CLO certainly not; the others are
//      candidates, appended with their keys~ to the sequence's candidate list
//      at an offset taken with one atomic per block (the bracket launch of the
//      same call empties the list); per-block counts (selected, candidates,
//      keys~ above t_hi) are stored, not accumulated;
//   3. resolve (one block per sequence): a histogram of the candidates inside
//      [t_lo, t_hi] gives the fine bin of the k-th largest key~ (if the sample
//      missed, the block histograms the whole key range instead and classifies
//      every row itself); with v = key~ + E and w = key~ - E rounded outward
//      this gives HI >= k-th largest v and LO <= k-th largest w, so the k-th
//      largest exact key lies in [LO, HI].  The candidates with w > HI are
//      selected, with v < LO not; the rest are undecided.  Their exact keys:
//      each undecided row's heads are scored again in fp32 (the same bound E
//      holds) and only the heads within 2E of the row's maximum get the fp64
//      chain with d ascending, the exact definition.  The undecided rows are
//      ranked by (exact key desc, index asc) -- pairwise counting, or a radix
//      select on (key, ~index) when they are many -- and the first
//      k - n_selected join S; the last of them gives theta.  Finally an
//      ordered compaction of the flags writes S ascending.
// Every row certainly selected has exact key >= w > HI >= theta* and every
// row certainly excluded has exact key <= v < LO <= theta*, so S is the fp64
// definition bit for bit.
// Admission (Lemma (Index certificate)) applies the same band argument to the
// upper bound UB_u against theta: a classification launch per 4096 rows and a
// resolve block per sequence (exact bounds of the undecided rows, then the
// ordered compaction of the admitted rows).
#include "vkv_internal.h"

namespace vkv {

constexpr int SEL_THREADS = 256;             // counting / classification blocks
constexpr int CB_PER = CB_KEYS / SEL_THREADS;   // rows per thread of a counting block (16)
constexpr int RES_THREADS = 512;             // resolve blocks: one per sequence (8 waves)
constexpr int RES_WAVES = RES_THREADS / 64;
constexpr int RES_LDS = 144 * 1024;          // dynamic LDS of a resolve block
constexpr int SAMPLE_MAX = 2048;             // keys sampled per sequence to place the bracket
constexpr int SAMPLE_BINS = 2048;            // bins of the sample's histogram
constexpr int RANK_QUAD_MAX = RES_THREADS;   // undecided rows ranked pairwise; radix select above
constexpr int CPT = 16;                      // candidates per thread of a resolve block held in registers
constexpr int AMB_LDS = 2048;                // undecided rows kept in LDS by a resolve block (more: global list)
constexpr int XIN_LDS = 8192;                // counting blocks whose extra counts a resolve block sums in LDS
constexpr int EX_QT_MAX = 32768;             // qt elements staged in LDS (64 KB)

// order-preserving encoding of fp64 (for 64-bit compares); -0 maps as +0
__device__ __forceinline__ uint64_t f64_to_ord(double d) {
    const uint64_t u = d2u(d == 0.0 ? 0.0 : d);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}
__device__ __forceinline__ double ord_to_f64(uint64_t o) {
    return u2d((o >> 63) ? (o & 0x7FFFFFFFFFFFFFFFull) : ~o);
}

// ------------------------------------------------------------ error bounds

// nu_max >= max_u ||x_u|| from the scorer's fp32 sums of squares.
__device__ __forceinline__ double nu_max_of(const uint32_t* sq, int n) {
    const double nu2 = (double)__uint_as_float(sq[SQ_NU2MAX]);
    return sqrt(nu2 * (1.0 + (double)n * 0x1p-22)) * (1.0 + 0x1p-20);
}

// |fp32 MFMA key - fp64 key| <= E.  bf16 products are exact in fp32; the dot
// product of width n goes through at most n + n/32 fp32 additions (32-product
// MFMA steps plus the accumulator), each with relative error <= 2^-23 (so even
// truncation is covered) of a partial sum bounded by sum_d |q_d x_d| <=
// ||qt|| ||x|| (Cauchy-Schwarz): |error| <= (n + n/32) 2^-23 ||qt|| ||x|| to
// first order; factor 2 of slack, plus an absolute term for flushed
// subnormal products.
__device__ __forceinline__ double key_error_of(const uint32_t* sq, int n) {
    const double qmax = (double)__uint_as_float(sq[SQ_QMAX]);
    return 2.0 * (double)(n + n / 32) * 0x1p-23 * qmax * nu_max_of(sq, n) + (double)n * 0x1p-120;
}

// E rounded up to fp32, and the outward-rounded band of one key.
__device__ __forceinline__ float key_band_f32(const uint32_t* sq, int n) { return ru_f32(key_error_of(sq, n)); }
__device__ __forceinline__ float band_hi(float k, float E) { return next_up_f32(k + E); }
__device__ __forceinline__ float band_lo(float k, float E) { return next_down_f32(k - E); }

// fp32 evaluation of s^ + B in the scorer: |error| <= E + 2^-21 (smax + bmax); 2x slack.
__device__ __forceinline__ double ub_error_of(const uint32_t* sq, int n) {
    const double E = key_error_of(sq, n);
    const double smax = (double)__uint_as_float(sq[SQ_QMAX]) * nu_max_of(sq, n);
    const double bmax = (double)__uint_as_float(sq[SQ_BMAX]) * (1.0 + 0x1p-20);
    return E * (1.0 + 0x1p-20) + 0x1p-20 * (smax + bmax);
}

__device__ __forceinline__ float rd_f32(double x) {
    float f = (float)x;
    if ((double)f > x) f = next_down_f32(f);
    return f;
}

// --------------------------------------------------------- block helpers

// Workgroup barrier for exchanges through LDS only: this wave's LDS operations
// have completed, but its global stores may still be in flight (a full
// __syncthreads() would wait for them as well).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int NT>
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* s_red) {
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = v;
    lds_barrier();
    uint32_t t = 0;
    for (int w = 0; w < NT / 64; ++w) t += s_red[w];
    lds_barrier();
    return t;
}

// Exclusive prefix of v over the threads in index order; total = the sum.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_w, uint32_t& total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    uint32_t incl = v;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_up(incl, o);
        if (lane >= o) incl += t;
    }
    if (lane == 63) s_w[w] = incl;
    lds_barrier();
    uint32_t before = 0, tot = 0;
    for (int i = 0; i < NT / 64; ++i) {
        const uint32_t c = s_w[i];
        before += (i < w) ? c : 0u;
        tot += c;
    }
    lds_barrier();
    total = tot;
    return before + incl - v;
}

// Sum over threads t' >= tid of v.
template <int NT>
__device__ __forceinline__ uint32_t block_suffix_incl(uint32_t v, uint32_t* s_w) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_down(v, o);
        if (lane + o < 64) v += t;
    }
    lds_barrier();
    if (lane == 0) s_w[w] = v;
    lds_barrier();
    uint32_t add = 0;
    for (int w2 = w + 1; w2 < NT / 64; ++w2) add += s_w[w2];
    lds_barrier();
    return v + add;
}

// ---------------------------------------------------------- histogram bins

template <int NB = HIST_BINS>
__device__ __forceinline__ float bin_scale(float lo, float hi) {
    const float range = hi - lo;
    return (range > 0.f && range < INFINITY) ? (float)NB / range : 0.f;
}

template <int NB = HIST_BINS>
__device__ __forceinline__ int bin_of(float x, float lo, float scale) {
    const float t = (x - lo) * scale;
    const int bi = (t > 0.f) ? (int)t : 0;
    return bi < NB ? bi : NB - 1;
}

// In a block of NT threads holding a histogram s_h[NB]: the bin d where the
// count of keys in bins >= d first reaches `target` (1 <= target <= total).
// Returns -1 in threads that do not own it.
template <int NB, int NT>
__device__ __forceinline__ int find_rank_bin(const uint32_t* s_h, uint32_t target, uint32_t* s_w) {
    constexpr int PER = NB / NT;
    const int tid = threadIdx.x;
    uint32_t loc = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) loc += s_h[tid * PER + j];
    const uint32_t suf = block_suffix_incl<NT>(loc, s_w);
    int found = -1;
    if (suf - loc < target && target <= suf) {
        uint32_t run = suf - loc;
        for (int d = (tid + 1) * PER - 1; d >= tid * PER; --d) {
            run += s_h[d];
            if (run >= target) {
                found = d;
                break;
            }
        }
    }
    return found;
}

// Bin d of the linear bins of [lo, lo + HIST_BINS / scale): keys x with
// bin_of(x) = d satisfy edge_lo(d) <= x <= edge_hi(d) (the fp32 rounding of the
// binning is covered by the widening).
__device__ __forceinline__ double edge_hi_of(int d, float lo, float hi, float scale) {
    if (!(scale > 0.f)) return (double)hi;
    const double w = 1.0 / (double)scale;
    const double slack = fabs((double)lo) * 0x1p-22 + 0x1p-100;
    return fmin((double)hi, (double)lo + (double)(d + 1) * w * (1.0 + 0x1p-20) + slack);
}
__device__ __forceinline__ double edge_lo_of(int d, float lo, float scale) {
    if (!(scale > 0.f)) return (double)lo;
    const double w = 1.0 / (double)scale;
    const double slack = fabs((double)lo) * 0x1p-22 + 0x1p-100;
    return fmax((double)lo, (double)lo + (double)d * w * (1.0 - 0x1p-20) - slack);
}

// ---------------------------------------------------------- 1. the bracket

// The bracket of the k-th largest key~ placed from a sample of up to
// SAMPLE_MAX keys (runs of 32 consecutive keys at evenly spaced offsets; all
// keys if A <= SAMPLE_MAX): [t_lo, t_hi] with sample ranks k_s -/+ (4 sqrt(k_s)
// + 16), k_s = k m / A, from a histogram of the sample over its own range.
// Only a heuristic: the resolve block checks it.
__global__ __launch_bounds__(SEL_THREADS) void sel_bracket_kernel(SelectArgs a) {
    __shared__ uint32_t s_h[SAMPLE_BINS];
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ float s_mm[8];
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t A = a.A;
    const int m = (int)min(A, (int64_t)SAMPLE_MAX);
    const float* kt = a.kt + (int64_t)b * A;
    constexpr int PER = SAMPLE_MAX / SEL_THREADS;
    constexpr int RUN = 32;
    const int nrun = (m + RUN - 1) / RUN;
    const int64_t stride = (m < A && nrun > 1) ? (A - RUN) / (nrun - 1) : 0;
    const float kmax = ord_to_key(sq[SQ_KMAX]), kmin = ord_to_key(sq[SQ_KMIN]);
    float v[PER];
    float lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int i = tid + SEL_THREADS * j;
        const int64_t u = (i >= m) ? 0 : (m == A) ? i : min(A - 1, (int64_t)(i / RUN) * stride + (i % RUN));
        v[j] = kt[u];
        if (i < m) {
            lo = fminf(lo, v[j]);
            hi = fmaxf(hi, v[j]);
        }
    }
    for (int o = 32; o > 0; o >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, o));
        hi = fmaxf(hi, __shfl_xor(hi, o));
    }
    if ((tid & 63) == 0) {
        s_mm[tid >> 6] = lo;
        s_mm[4 + (tid >> 6)] = hi;
    }
    for (int i = tid; i < SAMPLE_BINS; i += SEL_THREADS) s_h[i] = 0u;
    __syncthreads();
    lo = fminf(fminf(s_mm[0], s_mm[1]), fminf(s_mm[2], s_mm[3]));
    hi = fmaxf(fmaxf(s_mm[4], s_mm[5]), fmaxf(s_mm[6], s_mm[7]));
    const float scale = bin_scale<SAMPLE_BINS>(lo, hi);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int i = tid + SEL_THREADS * j;
        if (i < m) atomicAdd(&s_h[bin_of<SAMPLE_BINS>(v[j], lo, scale)], 1u);
    }
    __syncthreads();
    const double ks = (double)a.k * (double)m / (double)A;
    const double dl = 4.0 * sqrt(ks) + 16.0;
    const int64_t c_hi = (int64_t)floor(ks - dl);   // fewer than c_hi samples above t_hi
    const int64_t c_lo = (int64_t)ceil(ks + dl);    // at least c_lo samples at or above t_lo
    const int d_hi = (c_hi >= 1) ? find_rank_bin<SAMPLE_BINS, SEL_THREADS>(s_h, (uint32_t)c_hi, s_w) : -1;
    const int d_lo = (c_lo <= m) ? find_rank_bin<SAMPLE_BINS, SEL_THREADS>(s_h, (uint32_t)c_lo, s_w) : -1;
    // no cut on a side the sample cannot place: the scorer's key extremes
    if (tid == 0) {
        s_mm[0] = kmax;
        s_mm[1] = kmin;
    }
    __syncthreads();
    if (d_hi >= 0) s_mm[0] = scale > 0.f ? lo + (float)(d_hi + 1) / scale : hi;
    if (d_lo >= 0) s_mm[1] = scale > 0.f ? lo + (float)d_lo / scale : lo;
    __syncthreads();
    if (tid == 0) {
        const float t_hi = s_mm[0], t_lo = s_mm[1];
        const float E = key_band_f32(sq, a.n);
        sq[SQ_BLO] = __float_as_uint(t_lo);
        sq[SQ_BHI] = __float_as_uint(t_hi);
        sq[SQ_CLO] = __float_as_uint(band_lo(t_lo, E));
        sq[SQ_CHI] = __float_as_uint(band_hi(t_hi, E));
        sq[SQ_NCAND] = 0u;     // the lists of this call start empty
        sq[SQ_NCAND2] = 0u;
    }
}

// ----------------------------------------------------------- 2. counting

// Rows of the block whose predicate held (bit j of mask: row ub0 + tid + 256 j)
// appended to the sequence's list, at an offset taken with one atomic per
// block; keys (may be NULL) receive the rows' keys.  Writes stay below `lim`.
__device__ __forceinline__ void block_append(uint32_t mask, int64_t ub0, uint32_t* counter, int32_t* list,
                                             float* keys, const float (&k)[CB_PER], int64_t lim, uint32_t* s_w,
                                             uint32_t* s_base) {
    uint32_t tot;
    uint32_t pos = block_excl_scan<SEL_THREADS>((uint32_t)__popc(mask), s_w, tot);
    if (threadIdx.x == 0) *s_base = tot ? atomicAdd(counter, tot) : 0u;
    lds_barrier();
    int64_t at = (int64_t)*s_base + pos;
#pragma unroll
    for (int j = 0; j < CB_PER; ++j)
        if (mask & (1u << j)) {
            if (at < lim) {
                list[at] = (int32_t)(ub0 + threadIdx.x + (int64_t)SEL_THREADS * j);
                if (keys) keys[at] = k[j];
            }
            ++at;
        }
}

__global__ __launch_bounds__(SEL_THREADS) void sel_count_kernel(SelectArgs a) {
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ uint32_t s_base;
    const int b = blockIdx.y, tid = threadIdx.x;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t ub0 = (int64_t)blockIdx.x * CB_KEYS;
    const int64_t ue = min(a.A, ub0 + CB_KEYS);
    const float* kt = a.kt + (int64_t)b * a.A;
    float k[CB_PER];
#pragma unroll
    for (int j = 0; j < CB_PER; ++j) {
        const int64_t u = ub0 + tid + (int64_t)SEL_THREADS * j;
        k[j] = kt[u < ue ? u : ub0];
    }
    const float CLO = __uint_as_float(sq[SQ_CLO]), CHI = __uint_as_float(sq[SQ_CHI]);
    const float thi = __uint_as_float(sq[SQ_BHI]);
    const float E = key_band_f32(sq, a.n);
    uint8_t* fb = a.flags + (int64_t)b * a.fstride;
    uint32_t nin = 0, nabove = 0, mask = 0;
#pragma unroll
    for (int j = 0; j < CB_PER; ++j) {
        const int64_t u = ub0 + tid + (int64_t)SEL_THREADS * j;
        if (u < ue) {
            const uint8_t f = (band_lo(k[j], E) > CHI) ? 1 : ((band_hi(k[j], E) < CLO) ? 0 : 2);
            fb[u] = f;
            nin += (f == 1);
            nabove += (k[j] > thi);
            mask |= (f == 2) ? (1u << j) : 0u;
        }
    }
    block_append(mask, ub0, a.seq + (int64_t)b * SQ_WORDS + SQ_NCAND, a.cand + (int64_t)b * a.A,
                 a.candkey + (int64_t)b * a.A, k, a.A, s_w, &s_base);
    const uint32_t packed = block_sum<SEL_THREADS>(nin | (nabove << 16), s_w);   // both <= 4096
    if (tid == 0) {
        uint32_t* w = a.blk + ((int64_t)b * a.nblk + blockIdx.x) * BLK_WORDS;
        w[BW_IN] = packed & 0xFFFFu;
        w[BW_XIN] = 0u;
        w[BW_ABOVE] = packed >> 16;
    }
}

// ------------------------------------------------------ exact re-scoring

// Carve of a resolve block's dynamic LDS for the exact-key phase.
struct ExLds {
    uint16_t* qt;                 // [H][n] (qlds) -- else qt is read from global memory
    float4* hs;                   // [128] head scalars (a', n, e) for bounds
    double* off;                  // [128] per-head thresholds subtracted (trigger)
    unsigned long long* best;     // [waves][16]
    uint32_t* list;               // [waves][64]
    uint16_t* x;                  // [waves][16 rows][n]
    int nwx;                      // waves that take row tiles
    bool qlds;
};

__device__ __forceinline__ ExLds ex_carve(uint8_t* lds, int H, int n) {
    ExLds e;
    size_t o = 0;
    e.qlds = H * n <= EX_QT_MAX;
    e.qt = reinterpret_cast<uint16_t*>(lds);
    o += e.qlds ? (size_t)H * n * 2 : 0;
    o = (o + 15) & ~(size_t)15;
    e.hs = reinterpret_cast<float4*>(lds + o);
    o += 128 * 16;
    e.off = reinterpret_cast<double*>(lds + o);
    o += 128 * 8;
    e.best = reinterpret_cast<unsigned long long*>(lds + o);
    o += RES_WAVES * 16 * 8;
    e.list = reinterpret_cast<uint32_t*>(lds + o);
    o += RES_WAVES * 64 * 4;
    e.x = reinterpret_cast<uint16_t*>(lds + o);
    const int avail = (int)(((size_t)RES_LDS - o) / ((size_t)32 * n));   // 16 rows of n bf16 per wave
    e.nwx = avail < RES_WAVES ? avail : RES_WAVES;
    return e;
}

template <bool UB>
__device__ __forceinline__ double exact_chain(const uint16_t* q, const uint16_t* x, int n, float4 hs, double et,
                                              double ep, double ga) {
    double acc = 0.0;
    const int n8 = n / 8;
#pragma unroll 1
    for (int p0 = 0; p0 < n8; p0 += 8) {
        u16x8_t qv[8], xv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool in = p0 + j < n8;
            qv[j] = in ? *reinterpret_cast<const u16x8_t*>(q + 8 * (p0 + j)) : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
            xv[j] = in ? *reinterpret_cast<const u16x8_t*>(x + 8 * (p0 + j)) : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (p0 + j >= n8) break;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc = fma((double)bf16_to_f32(qv[j][e]), (double)bf16_to_f32(xv[j][e]), acc);
        }
    }
    if (UB) acc = acc + fma((double)hs.x, et, fma((double)hs.y, ep, (double)hs.z * ga));
    return acc;
}

// a'_h of the bound: the smallest float >= cert_mult * a_h (exact product in fp64)
__device__ __forceinline__ float scaled_a(float cm, float ah) { return ru_f32((double)cm * (double)ah); }

// Exact keys (or, with UB, exact bounds) of the rows amb[0..namb) of sequence b
// into ak[i] (order-preserving encoding), in a resolve block.  A tile of 16
// rows per wave: the rows are gathered straight into the MFMA operand layout
// (lane 16 g + c: row c, dims 32 ks + 8 g ..) and scored against every head
// with fp32 accumulation -- the scorer's arithmetic, so the screened value is
// within E of the exact one for every (row, head).  Only heads within
// `margin` (2E) of their row's maximum can hold the exact maximum; each such
// (row, head) pair gets its fp64 chain (d ascending from +0) from one lane,
// and the row's exact value is the maximum over its pairs.  margin = +inf
// evaluates every head exactly.
// The sequence's query rows qt (H * n / 8 <= EX_QT_MAX / 8 pieces of 16 B),
// thread tid's pieces tid + RES_THREADS j: loads all in flight together.  A
// caller may issue them early and hand them to exact_keys_block.
constexpr int EX_QP = EX_QT_MAX / 8 / RES_THREADS;
__device__ __forceinline__ void qt_prefetch(const SelectArgs& a, int b, u16x8_t (&v)[EX_QP]) {
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const int np = a.H * a.n / 8;
    if (np > EX_QT_MAX / 8) return;
#pragma unroll
    for (int j = 0; j < EX_QP; ++j) {
        const int p = threadIdx.x + RES_THREADS * j;
        v[j] = *reinterpret_cast<const u16x8_t*>(qtb + 8 * (int64_t)(p < np ? p : 0));
    }
}

template <bool UB, bool OFF = false>
__device__ __forceinline__ void exact_keys_block(const SelectArgs& a, int b, int64_t namb, const int32_t* amb, uint64_t* ak,
                                 const ExLds& L, float margin, int blk = 0, int nblks = 1,
                                 const u16x8_t (*pre)[EX_QP] = nullptr, uint64_t* ak_lds = nullptr) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, c = lane & 15;
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const int n8 = a.n / 8;
    if (L.qlds) {
        const int np = a.H * n8;
        u16x8_t v[EX_QP];
        if (pre) {
#pragma unroll
            for (int j = 0; j < EX_QP; ++j) v[j] = (*pre)[j];
        } else {
            qt_prefetch(a, b, v);
        }
#pragma unroll
        for (int j = 0; j < EX_QP; ++j) {
            const int p = tid + RES_THREADS * j;
            if (p < np) *reinterpret_cast<u16x8_t*>(&L.qt[8 * p]) = v[j];
        }
    }
    if (UB && tid < a.H) {
        const float4 hs = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + tid];
        const float ax = scaled_a(a.cert_mult, hs.x);
        L.hs[tid] = make_float4(ax, hs.y, hs.z, hs.w);
    }
    if (OFF && tid < a.H) L.off[tid] = a.smax[(int64_t)b * a.H + tid];
    lds_barrier();
    if (wave < L.nwx && namb > 0) {
        const uint16_t* qsrc = L.qlds ? L.qt : qtb;
        const uint16_t* xb = a.x + (int64_t)b * a.xbs;
        uint16_t* sx = L.x + (size_t)wave * 16 * a.n;
        unsigned long long* best = L.best + wave * 16;
        const int KS = a.n / 32, HT = (a.H + 15) / 16;
        for (int64_t t0 = ((int64_t)blk * L.nwx + wave) * 16; t0 < namb; t0 += (int64_t)nblks * L.nwx * 16) {
            const int64_t i = min(t0 + c, namb - 1);
            const int64_t u = amb[i];
            const uint16_t* x = xb + u * a.xs;
            f32x4_t acc[8];
#pragma unroll
            for (int ht = 0; ht < 8; ++ht) acc[ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            float et = 0.f, ep = 0.f, ga = 0.f;
            if constexpr (UB) {
                // the row's pieces and its certificate scalars: all loads in
                // flight together (one memory round trip; pieces past the row
                // width re-read its last piece), then into the wave's LDS copy
                // of its rows, from which each lane reads back its own pieces
                constexpr int KSM = D_ROW / 32;
                bf16x8_t xr[KSM];
#pragma unroll
                for (int ks = 0; ks < KSM; ++ks)
                    xr[ks] = *reinterpret_cast<const bf16x8_t*>(x + 32 * min(ks, KS - 1) + 8 * g);
                const int64_t o = (int64_t)b * a.T + u;
                et = a.eta[o];
                ep = a.eps[o];
                ga = a.gam[o];
#pragma unroll
                for (int ks = 0; ks < KSM; ++ks)
                    if (ks < KS) *reinterpret_cast<bf16x8_t*>(&sx[c * a.n + 32 * ks + 8 * g]) = xr[ks];
            }
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8_t xf = UB ? *reinterpret_cast<const bf16x8_t*>(&sx[c * a.n + 32 * ks + 8 * g])
                                       : *reinterpret_cast<const bf16x8_t*>(x + 32 * ks + 8 * g);
                if (!UB) *reinterpret_cast<bf16x8_t*>(&sx[c * a.n + 32 * ks + 8 * g]) = xf;
#pragma unroll
                for (int ht = 0; ht < 8; ++ht) {
                    if (ht < HT) {
                        const int h = (16 * ht + c) % a.H;
                        const bf16x8_t qf = *reinterpret_cast<const bf16x8_t*>(qsrc + (int64_t)h * a.n + 32 * ks + 8 * g);
                        acc[ht] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf, xf, acc[ht], 0, 0, 0);
                    }
                }
            }
            // acc[ht][q] = screened value of head 16 ht + 4 g + q for row c
            float m = -INFINITY;
#pragma unroll
            for (int ht = 0; ht < 8; ++ht)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int h = 16 * ht + 4 * g + q;
                    float v = -INFINITY;
                    if (ht < HT && h < a.H) {
                        v = acc[ht][q];
                        if (UB) {
                            const float4 hs = L.hs[h];
                            v += fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga));
                        }
                        if (OFF) v -= (float)L.off[h];
                    }
                    acc[ht][q] = v;
                    m = fmaxf(m, v);
                }
            m = fmaxf(m, __shfl_xor(m, 16));
            m = fmaxf(m, __shfl_xor(m, 32));
            const float thr = next_down_f32(m - margin);
            if (lane < 16) best[lane] = (unsigned long long)f64_to_ord(-INFINITY);
            // the rows are in LDS for every lane of the wave (LDS operations of a
            // wave complete in order)
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_wave_barrier();
            // this lane's candidates: slot 4 ht + q (head 16 ht + 4 g + q of row c)
            uint32_t cm = 0;
#pragma unroll
            for (int ht = 0; ht < 8; ++ht)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    cm |= ((t0 + c < namb) && acc[ht][q] >= thr && acc[ht][q] > -INFINITY) ? (1u << (4 * ht + q)) : 0u;
            // one fp64 chain per lane and round until every lane's candidates are done
            // (a single copy of the chain's code)
            while (__ballot(cm != 0u)) {
                if (cm) {
                    const int sl = __ffs(cm) - 1;
                    cm &= cm - 1u;
                    const int h = 16 * (sl >> 2) + 4 * g + (sl & 3);
                    const float4 hs = UB ? L.hs[h] : make_float4(0.f, 0.f, 0.f, 0.f);
                    double v = exact_chain<UB>(qsrc + (int64_t)h * a.n, &sx[c * a.n], a.n, hs, (double)et,
                                               (double)ep, (double)ga);
                    if (OFF) v = v - L.off[h];
                    atomicMax(&best[c], (unsigned long long)f64_to_ord(v));
                }
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_wave_barrier();
            if (lane < 16 && t0 + lane < namb) {
                const uint64_t v = best[lane];
                ak[t0 + lane] = v;
                if (ak_lds && t0 + lane < RANK_QUAD_MAX) ak_lds[t0 + lane] = v;   // the ranking's copy
            }
            // the next tile's row stores must not overtake this tile's chain reads
            __builtin_amdgcn_wave_barrier();
        }
    }
    __syncthreads();
}



// Rank of the undecided rows by (exact key desc, index asc): the first
// `need` of them get flag 1; returns (in thread 0's view, via *theta_ord) the
// key of the last of them.  Pairwise counting with the list staged in LDS
// when it is short; otherwise a radix select on the 96-bit composite
// (order key, ~index), whose larger values come first.
// ak_lds (optional): the keys already in LDS (the first RANK_QUAD_MAX of them).
__device__ __forceinline__ void rank_winners(const int32_t* amb, const uint64_t* ak, int64_t namb, int64_t need, uint8_t* fb,
                             uint32_t* xin, uint8_t* lds, uint64_t* s_theta, uint8_t mark = 1,
                             const uint64_t* ak_lds = nullptr) {
    const int tid = threadIdx.x;
    if (namb <= RANK_QUAD_MAX) {
        uint64_t* s_kc = reinterpret_cast<uint64_t*>(lds);
        int32_t* s_u = reinterpret_cast<int32_t*>(lds + RANK_QUAD_MAX * 8);
        if (tid < namb) {
            if (!ak_lds) s_kc[tid] = ak[tid];
            s_u[tid] = amb[tid];
        }
        const uint64_t* s_k = ak_lds ? ak_lds : s_kc;
        lds_barrier();
        if (tid < namb) {
            const uint64_t ki = s_k[tid];
            const int32_t ui = s_u[tid];
            int64_t rank = 0;
            for (int64_t j = 0; j < namb; ++j) {
                const uint64_t kj = s_k[j];
                rank += (kj > ki) || (kj == ki && s_u[j] < ui);
            }
            if (rank < need) {
                fb[ui] = mark;
                atomicAdd(&xin[(int64_t)(ui / CB_KEYS) * BLK_WORDS], 1u);
                if (rank == need - 1) *s_theta = ki;
            }
        }
        lds_barrier();
        return;
    }
    uint32_t* s_h = reinterpret_cast<uint32_t*>(lds);            // 256 bins
    uint32_t* s_sel = s_h + 256;                                  // chosen digit, count above it
    uint64_t pre_hi = 0, mask_hi = 0;
    uint32_t pre_lo = 0, mask_lo = 0;
    uint32_t rem = (uint32_t)need;
#pragma unroll 1
    for (int p = 0; p < 12; ++p) {
        if (tid < 256) s_h[tid] = 0u;
        __syncthreads();
        for (int64_t i = tid; i < namb; i += RES_THREADS) {
            const uint64_t hi = ak[i];
            const uint32_t lo = ~(uint32_t)amb[i];
            if ((hi & mask_hi) == pre_hi && (lo & mask_lo) == pre_lo) {
                const uint32_t dg = p < 8 ? (uint32_t)(hi >> (56 - 8 * p)) & 255u : (lo >> (24 - 8 * (p - 8))) & 255u;
                atomicAdd(&s_h[dg], 1u);
            }
        }
        __syncthreads();
        if (tid < 64) {
            // lane l owns digits 4 l .. 4 l + 3; counts from the top digit down
            uint32_t loc = s_h[4 * tid] + s_h[4 * tid + 1] + s_h[4 * tid + 2] + s_h[4 * tid + 3];
            uint32_t suf = loc;
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t t = __shfl_down(suf, o);
                if (tid + o < 64) suf += t;
            }
            if (suf - loc < rem && rem <= suf) {
                uint32_t run = suf - loc;
                for (int d = 4 * tid + 3; d >= 4 * tid; --d) {
                    if (run + s_h[d] >= rem) {
                        s_sel[0] = (uint32_t)d;
                        s_sel[1] = run;
                        break;
                    }
                    run += s_h[d];
                }
            }
        }
        __syncthreads();
        const uint32_t d = s_sel[0];
        rem -= s_sel[1];
        if (p < 8) {
            pre_hi |= (uint64_t)d << (56 - 8 * p);
            mask_hi |= (uint64_t)255 << (56 - 8 * p);
        } else {
            pre_lo |= d << (24 - 8 * (p - 8));
            mask_lo |= 255u << (24 - 8 * (p - 8));
        }
        __syncthreads();
    }
    for (int64_t i = tid; i < namb; i += RES_THREADS) {
        const uint64_t hi = ak[i];
        const uint32_t lo = ~(uint32_t)amb[i];
        if (hi > pre_hi || (hi == pre_hi && lo >= pre_lo)) {
            fb[amb[i]] = mark;
            atomicAdd(&xin[(int64_t)(amb[i] / CB_KEYS) * BLK_WORDS], 1u);
        }
    }
    if (tid == 0) *s_theta = pre_hi;
    __syncthreads();
}

// ------------------------------------------------------------- 3. resolve

__global__ __launch_bounds__(RES_THREADS, 1) void sel_resolve_kernel(SelectArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    __shared__ uint32_t s_w[RES_WAVES];
    __shared__ uint32_t s_namb;
    __shared__ int s_bin;
    __shared__ uint64_t s_theta;
    __shared__ int32_t s_amb[AMB_LDS];         // the undecided rows (the global list holds them all)
    __shared__ uint64_t s_ak[RANK_QUAD_MAX];   // their exact keys when few (for the ranking)
    const int b = blockIdx.x, tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    uint8_t* fb = a.flags + (int64_t)b * a.fstride;
    const float* kt = a.kt + (int64_t)b * a.A;
    const int32_t* cr = a.cand + (int64_t)b * a.A;
    const float* ck = a.candkey + (int64_t)b * a.A;
    int32_t* amb = a.amb + (int64_t)b * a.A;
    uint64_t* ak = a.ambkey + (int64_t)b * a.A;
    const float tlo = __uint_as_float(sq[SQ_BLO]), thi = __uint_as_float(sq[SQ_BHI]);
    const int64_t ncand = min((int64_t)sq[SQ_NCAND], a.A);
    const float E = key_band_f32(sq, a.n);
    // the query rows of the exact re-scoring at the end, in flight from here on
    u16x8_t qpre[EX_QP];
    qt_prefetch(a, b, qpre);
    // the first NT * CPT candidates stay in registers for both passes below
    constexpr int64_t CH = (int64_t)RES_THREADS * CPT;
    int32_t cu[CPT];
    float cv[CPT];
    // (loads are unconditional, from a clamped index, so that they are all in
    // flight together and none is awaited inside a branch)
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
        const int64_t i = tid + (int64_t)RES_THREADS * j;
        const int64_t ic = min(i, max(ncand - 1, (int64_t)0));
        const int32_t u = cr[ic];
        const float kv = ck[ic];
        cu[j] = (i < ncand) ? u : -1;
        cv[j] = kv;
    }
    // counts of the counting blocks
    uint32_t nin = 0, nab = 0;
    for (int64_t i = tid; i < a.nblk; i += RES_THREADS) {
        const uint32_t* w = a.blk + ((int64_t)b * a.nblk + i) * BLK_WORDS;
        nin += w[BW_IN];
        nab += w[BW_ABOVE];
    }
    uint32_t* s_h = reinterpret_cast<uint32_t*>(lds);
    for (int i = tid; i < HIST_BINS; i += RES_THREADS) s_h[i] = 0u;
    if (tid == 0) {
        s_namb = 0u;
        s_bin = -1;
        s_theta = f64_to_ord(-INFINITY);
    }
    nin = block_sum<RES_THREADS>(nin, s_w);
    nab = block_sum<RES_THREADS>(nab, s_w);
    // fine histogram of the candidates inside [t_lo, t_hi]
    const float sc0 = bin_scale(tlo, thi);
    uint32_t nmid = 0;
    auto hist_one = [&](float kv) {
        if (kv >= tlo && kv <= thi) {
            atomicAdd(&s_h[bin_of(kv, tlo, sc0)], 1u);
            ++nmid;
        }
    };
#pragma unroll
    for (int j = 0; j < CPT; ++j)
        if (cu[j] >= 0) hist_one(cv[j]);
    for (int64_t c0 = CH; c0 < ncand; c0 += CH)
        for (int64_t i = c0 + tid; i < min(ncand, c0 + CH); i += RES_THREADS) hist_one(ck[i]);
    nmid = block_sum<RES_THREADS>(nmid, s_w);
    const int64_t need = a.k - (int64_t)nab;
    const bool ok = need >= 1 && need <= (int64_t)nmid;
    float lo = tlo, hi = thi, sc = sc0;
    if (!ok) {
        // the sample missed: histogram the whole key range here
        lo = ord_to_key(sq[SQ_KMIN]);
        hi = ord_to_key(sq[SQ_KMAX]);
        sc = bin_scale(lo, hi);
        for (int i = tid; i < HIST_BINS; i += RES_THREADS) s_h[i] = 0u;
        __syncthreads();
        for (int64_t u = tid; u < a.A; u += RES_THREADS) atomicAdd(&s_h[bin_of(kt[u], lo, sc)], 1u);
        __syncthreads();
    }
    const uint32_t target = (uint32_t)(ok ? need : a.k);
    const int d = find_rank_bin<HIST_BINS, RES_THREADS>(s_h, target, s_w);
    if (d >= 0) s_bin = d;
    __syncthreads();
    const int db = s_bin < 0 ? 0 : s_bin;
    const float HI = band_hi(ru_f32(edge_hi_of(db, lo, hi, sc)), E);
    const float LO = band_lo(rd_f32(edge_lo_of(db, lo, sc)), E);
    // classification: selected (w > HI), excluded (v < LO), undecided.  The
    // rows this block decides in are counted per counting block (in LDS after
    // the histogram, or with global atomics for very long archives), for the
    // ordered compaction that follows.
    auto classify = [&](float kv) -> uint8_t { return (band_lo(kv, E) > HI) ? 1 : ((band_hi(kv, E) < LO) ? 0 : 2); };
    uint32_t* blkb = a.blk + (int64_t)b * a.nblk * BLK_WORDS;
    const bool xlds = a.nblk <= XIN_LDS;
    uint32_t* s_x = reinterpret_cast<uint32_t*>(lds + HIST_BINS * 4);
    if (xlds)
        for (int64_t i = tid; i < a.nblk; i += RES_THREADS) s_x[i] = 0u;
    lds_barrier();
    auto count_in = [&](int64_t u) {
        if (xlds) atomicAdd(&s_x[u / CB_KEYS], 1u);
        else atomicAdd(&blkb[(u / CB_KEYS) * BLK_WORDS + BW_XIN], 1u);
    };
    auto append = [&](bool und, int32_t u) {
        const uint64_t bal = __ballot(und);
        if (bal == 0) return;
        const int lane = tid & 63;
        const int leader = __ffsll((unsigned long long)bal) - 1;
        uint32_t base = 0;
        if (lane == leader) base = atomicAdd(&s_namb, (uint32_t)__popcll(bal));
        base = __shfl(base, leader);
        if (und) {
            const uint32_t pos = base + __popcll(bal & ((1ull << lane) - 1ull));
            amb[pos] = u;
            if (pos < AMB_LDS) s_amb[pos] = u;
        }
    };
    if (ok) {
        // the candidates; every other row was decided by the counting pass.
        // A candidate's flag is 2 from that pass, and every reader takes any
        // flag but 1 as "not selected", so only the selected ones are written
        // (the undecided ones get theirs from the ranking below).
#pragma unroll
        for (int j = 0; j < CPT; ++j) {
            uint8_t f = 0;
            if (cu[j] >= 0) {
                f = classify(cv[j]);
                if (f == 1) {
                    fb[cu[j]] = 1;
                    count_in(cu[j]);
                }
            }
            append(f == 2, cu[j]);
        }
        for (int64_t c0 = CH; c0 < ncand; c0 += CH)
            for (int64_t i0 = c0; i0 < min(ncand, c0 + CH); i0 += RES_THREADS) {
                const int64_t i = i0 + tid;
                uint8_t f = 0;
                int32_t u = 0;
                if (i < ncand) {
                    u = cr[i];
                    f = classify(ck[i]);
                    if (f == 1) {
                        fb[u] = 1;
                        count_in(u);
                    }
                }
                append(f == 2, u);
            }
    } else {
        // every row again: the counting pass's early classification used the
        // missed bracket, so its counts of selected rows are void as well
        for (int64_t i = tid; i < a.nblk; i += RES_THREADS) blkb[i * BLK_WORDS + BW_IN] = 0u;
        for (int64_t u0 = 0; u0 < a.A; u0 += RES_THREADS) {
            const int64_t u = u0 + tid;
            const bool live = u < a.A;
            const uint8_t f = live ? classify(kt[u]) : 0;
            if (live) {
                fb[u] = f;
                if (f == 1) count_in(u);
            }
            append(live && f == 2, (int32_t)u);
        }
    }
    lds_barrier();
    if (xlds)
        for (int64_t i = tid; i < a.nblk; i += RES_THREADS) blkb[i * BLK_WORDS + BW_XIN] = s_x[i];
    uint32_t nin2 = 0;
    if (xlds)
        for (int64_t i = tid; i < a.nblk; i += RES_THREADS) nin2 += s_x[i];
    nin2 = block_sum<RES_THREADS>(nin2, s_w);
    if (!xlds) {
        __threadfence_block();
        __syncthreads();
        for (int64_t i = tid; i < a.nblk; i += RES_THREADS) nin2 += blkb[i * BLK_WORDS + BW_XIN];
        nin2 = block_sum<RES_THREADS>(nin2, s_w);
    }
    const int64_t namb = s_namb;
    const int64_t n_in = (ok ? (int64_t)nin : 0) + (int64_t)nin2;
    const int64_t need2 = a.k - n_in;   // >= 1 and <= namb by the band argument
    if (tid == 0) {
        sq[SQ_TLO] = __float_as_uint(LO);
        sq[SQ_THI] = __float_as_uint(HI);
        sq[SQ_NAMB] = (uint32_t)namb;
    }
    // exact keys of the undecided rows, then their ranking (the list from LDS
    // when it fits there, else from global memory once it is visible)
    const bool amb_lds = namb <= AMB_LDS;
    if (!amb_lds) __threadfence_block();
    __syncthreads();
    const int32_t* al = amb_lds ? s_amb : amb;
    const ExLds L = ex_carve(lds, a.H, a.n);
    exact_keys_block<false>(a, b, namb, al, ak, L, next_up_f32(2.0f * E), 0, 1, &qpre, s_ak);
    rank_winners(al, ak, namb, need2, fb, blkb + BW_XIN, lds, &s_theta, 1, s_ak);
    if (tid == 0) a.theta[b] = ord_to_f64(s_theta);
}

// ------------------------------------------------------ ordered compaction

// 0x80 in each byte of v that equals t (t replicated in each byte of tt)
__device__ __forceinline__ uint32_t bytes_equal(uint32_t v, uint32_t tt) {
    const uint32_t x = v ^ tt;
    return ~(((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x | 0x7F7F7F7Fu);
}

struct CompactArgs {
    const uint8_t* flags;  // [B, fstride]
    int64_t fstride;
    const uint32_t* blk;   // [B, nblk, BLK_WORDS]: rows decided in per counting block (BW_IN + BW_XIN)
    int64_t nblk, A;
    uint32_t target;
    int32_t* out;          // [B, out_stride]
    int64_t out_stride, cap;
    int32_t* total;        // [B] or null: the number of rows with the target flag
};

// One block per counting block (4096 rows) of a sequence: its offset is the
// sum of the decided-in counts of the blocks before it; thread t owns 16
// consecutive rows (one 16-byte load of flags), then one block scan orders
// the writes.
__global__ __launch_bounds__(SEL_THREADS) void compact_kernel(CompactArgs a) {
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    const int b = blockIdx.y, tid = threadIdx.x;
    const int64_t c = blockIdx.x;
    const uint32_t* w = a.blk + (int64_t)b * a.nblk * BLK_WORDS;
    uint32_t part = 0;
    for (int64_t j = tid; j < c; j += SEL_THREADS) part += w[j * BLK_WORDS + BW_IN] + w[j * BLK_WORDS + BW_XIN];
    const int64_t u0 = c * CB_KEYS + 16 * tid;
    const u32x4_t v = *reinterpret_cast<const u32x4_t*>(a.flags + (int64_t)b * a.fstride + (u0 < a.A ? u0 : 0));
    const uint32_t base = block_sum<SEL_THREADS>(part, s_w);
    const uint32_t tt = 0x01010101u * a.target;
    uint32_t m[4], cnt = 0;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const int64_t valid = min((int64_t)4, max((int64_t)0, a.A - (u0 + 4 * d)));
        const uint32_t keep = valid >= 4 ? 0xFFFFFFFFu : ((1u << (8 * valid)) - 1u);
        m[d] = bytes_equal(v[d], tt) & keep;
        cnt += (uint32_t)__popc(m[d]);
    }
    uint32_t tot;
    int64_t pos = (int64_t)base + block_excl_scan<SEL_THREADS>(cnt, s_w, tot);
    int32_t* ob = a.out ? a.out + (int64_t)b * a.out_stride : nullptr;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        uint32_t bits = m[d];
        while (bits) {
            const int e = (__ffs(bits) - 1) >> 3;
            if (pos < a.cap) ob[pos] = (int32_t)(u0 + 4 * d + e);
            ++pos;
            bits &= bits - 1u;
        }
    }
    if (a.total && c == a.nblk - 1 && tid == 0) a.total[b] = (int32_t)(base + tot);
}

static hipError_t run_compact(const SelectArgs& s, const uint8_t* flags, uint32_t target, int32_t* out, int64_t stride,
                              int64_t cap, int32_t* total, hipStream_t st) {
    const CompactArgs c{flags, s.fstride, s.blk, s.nblk, s.A, target, out, stride, cap, total};
    hipLaunchKernelGGL(compact_kernel, dim3((unsigned)s.nblk, s.B), dim3(SEL_THREADS), 0, st, c);
    return hipGetLastError();
}

__global__ __launch_bounds__(SEL_THREADS) void fill_u8_kernel(uint8_t* p, int64_t n, uint8_t v) {
    for (int64_t i = (int64_t)blockIdx.x * SEL_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * SEL_THREADS)
        p[i] = v;
}

__global__ __launch_bounds__(64) void theta_empty_kernel(double* theta, int B) {
    for (int b = threadIdx.x; b < B; b += 64) theta[b] = -INFINITY;
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    hipError_t e;
    if (a.k == 0) {
        // nothing selected: theta = -inf, every flag 0
        hipLaunchKernelGGL(theta_empty_kernel, dim3(1), dim3(64), 0, s, a.theta, a.B);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (a.A == 0) return hipSuccess;
        hipLaunchKernelGGL(fill_u8_kernel, dim3(256), dim3(SEL_THREADS), 0, s, a.flags, (int64_t)a.B * a.fstride,
                           (uint8_t)0);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(sel_bracket_kernel, dim3(a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sel_count_kernel, dim3((unsigned)a.nblk, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&sel_resolve_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, RES_LDS);
    hipLaunchKernelGGL(sel_resolve_kernel, dim3(a.B), dim3(RES_THREADS), RES_LDS, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags, 1, a.sel, a.k, a.k, nullptr, s);
}

// ---------------------------------------------------------------- admit

// Classification of UB~ against theta (rows outside S): admitted (3), not
// admitted (0) or undecided (4), listed in the block's candidate region.  If
// the scorer's bound used another certificate multiplier than this call, or
// none, every row outside S is undecided (its exact bound decides).
__global__ __launch_bounds__(SEL_THREADS) void adm_classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ uint32_t s_base;
    const int b = blockIdx.y, tid = threadIdx.x;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t ub0 = (int64_t)blockIdx.x * CB_KEYS;
    const int64_t ue = min(a.A, ub0 + CB_KEYS);
    const double th = a.theta[b];
    const bool same = sq[SQ_CMULT] == __float_as_uint(a.cert_mult);
    const double E = ub_error_of(sq, a.n) * (1.0 + 0x1p-20);
    const float* ubb = a.ub + (int64_t)b * a.A;
    const uint8_t* fb = a.flags + (int64_t)b * a.fstride;
    uint8_t* f2 = a.flags2 + (int64_t)b * a.fstride;
    float t[CB_PER];
    uint8_t fin[CB_PER];
#pragma unroll
    for (int j = 0; j < CB_PER; ++j) {
        const int64_t u = ub0 + tid + (int64_t)SEL_THREADS * j;
        const int64_t uc = u < ue ? u : ub0;
        t[j] = ubb[uc];
        fin[j] = (u < ue) ? fb[uc] : (uint8_t)1;
    }
    uint32_t mask = 0, nadm = 0;
#pragma unroll
    for (int j = 0; j < CB_PER; ++j) {
        const int64_t u = ub0 + tid + (int64_t)SEL_THREADS * j;
        if (u < ue) {
            uint8_t f = 0;
            if (fin[j] != 1) {
                if (th == -INFINITY) {
                    f = 3;
                } else if (!same) {
                    f = 4;
                } else {
                    const double tv = (double)t[j];
                    const double band = E + fabs(tv) * 0x1p-50 + fabs(th) * 0x1p-50;
                    f = (tv - band > th) ? 3 : ((tv + band <= th) ? 0 : 4);
                }
            }
            f2[u] = f;
            nadm += (f == 3);
            mask |= (f == 4) ? (1u << j) : 0u;
        }
    }
    block_append(mask, ub0, a.seq + (int64_t)b * SQ_WORDS + SQ_NCAND2, a.cand + (int64_t)b * a.A, nullptr, t,
                 a.A, s_w, &s_base);
    nadm = block_sum<SEL_THREADS>(nadm, s_w);
    if (tid == 0) {
        uint32_t* w = a.blk + ((int64_t)b * a.nblk + blockIdx.x) * BLK_WORDS;
        w[BW_IN] = nadm;
        w[BW_XIN] = 0u;
    }
}

// One block per sequence: exact bounds of the undecided rows (fp64), the
// decision UB > theta, then the ordered compaction of the admitted rows.
__global__ __launch_bounds__(RES_THREADS, 1) void adm_resolve_kernel(SelectArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    const int b = blockIdx.x, tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    uint8_t* f2 = a.flags2 + (int64_t)b * a.fstride;
    const int32_t* amb = a.cand + (int64_t)b * a.A;    // the undecided rows listed by the classification
    uint64_t* ak = a.ambkey + (int64_t)b * a.A;
    const double th = a.theta[b];
    const bool same = sq[SQ_CMULT] == __float_as_uint(a.cert_mult);
    const int64_t namb = min((int64_t)sq[SQ_NCAND2], a.A);
    __syncthreads();
    if (tid == 0) {
        sq[SQ_NAMB2] = (uint32_t)namb;
        sq[SQ_NCAND2] = 0u;    // consumed: a repeated admission starts an empty list
    }
    const ExLds L = ex_carve(lds, a.H, a.n);
    const float margin = same ? next_up_f32(2.0f * ru_f32(ub_error_of(sq, a.n) * (1.0 + 0x1p-20))) : INFINITY;
    exact_keys_block<true>(a, b, namb, amb, ak, L, margin);
    // the undecided rows admitted on their exact bound (the classification left them at 4)
    uint32_t* blkb = a.blk + (int64_t)b * a.nblk * BLK_WORDS;
    for (int64_t i = tid; i < namb; i += RES_THREADS)
        if (ord_to_f64(ak[i]) > th) {
            const int32_t u = amb[i];
            f2[u] = 3;
            atomicAdd(&blkb[(int64_t)(u / CB_KEYS) * BLK_WORDS + BW_XIN], 1u);
        }
}

__global__ __launch_bounds__(64) void zero_counts_kernel(int32_t* p, int n);

// ---------------------------------------------------------------- trigger
//
// The calibrated trigger (Sec. 4.2, Eq. (trigger) against the tier-1 maximum
// logit; the optional top-j cap of the deployment specification): a row u
// outside S fires iff some head has UB_h(u) > s*_h, UB_h with the certificate
// term scaled by cert_mult = z / sqrt(d_c - r).  Its margin is
// max_h (UB_h(u) - s*_h).  Three launches and the ordered compaction:
//   classify (one block per 4096 rows): a row whose UB~ (the maximum over
//     heads) stays below min_h s*_h by more than its band cannot fire; the
//     others are candidates;
//   exact (a few blocks per sequence): the exact margins of the candidates,
//     a per-head fp32 screen and fp64 chains for the heads near the row's
//     maximum (the exact-key machinery with the thresholds subtracted);
//   fire (one block per sequence): margin > 0, and with a cap the top j by
//     (margin desc, row asc).

// the smallest threshold of sequence b (wave 0 of the block; result in all its lanes)
__device__ __forceinline__ double min_threshold(const SelectArgs& a, int b) {
    double m = INFINITY;
    for (int h = threadIdx.x & 63; h < a.H; h += 64) m = fmin(m, a.smax[(int64_t)b * a.H + h]);
    for (int o = 32; o > 0; o >>= 1) m = fmin(m, __shfl_xor(m, o));
    return m;
}

__global__ __launch_bounds__(SEL_THREADS) void trig_classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ uint32_t s_base;
    __shared__ double s_min;
    const int b = blockIdx.y, tid = threadIdx.x;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t ub0 = (int64_t)blockIdx.x * CB_KEYS;
    const int64_t ue = min(a.A, ub0 + CB_KEYS);
    const float* ubb = a.ub + (int64_t)b * a.A;
    const uint8_t* fb = a.flags + (int64_t)b * a.fstride;
    uint8_t* f2 = a.flags2 + (int64_t)b * a.fstride;
    float t[CB_PER];
    uint8_t fin[CB_PER];
#pragma unroll
    for (int j = 0; j < CB_PER; ++j) {
        const int64_t u = ub0 + tid + (int64_t)SEL_THREADS * j;
        const int64_t uc = u < ue ? u : ub0;
        t[j] = ubb[uc];
        fin[j] = (u < ue) ? fb[uc] : (uint8_t)1;
    }
    // the scorer wrote either UB~ (max over heads of the bound) or, given the
    // thresholds, the trigger margins max_h (UB~_h - s*_h)
    const bool trgm = sq[SQ_TRGM] != 0u;
    __shared__ double s_absmax;
    if (tid < 64) {
        const double m = min_threshold(a, b);
        double am = 0.0;
        for (int h = tid; h < a.H; h += 64) {
            const double v = a.smax[(int64_t)b * a.H + h];
            am = fmax(am, isfinite(v) ? fabs(v) : 0.0);
        }
        for (int o = 32; o > 0; o >>= 1) am = fmax(am, __shfl_xor(am, o));
        if (tid == 0) {
            s_min = m;
            s_absmax = am;
        }
    }
    lds_barrier();
    const double smin = s_min;
    const bool same = sq[SQ_CMULT] == __float_as_uint(a.cert_mult);
    const double E = ub_error_of(sq, a.n) * (1.0 + 0x1p-20);
    // margins: the bound's fp32 error plus the fp32 rounding of s*_h and of the
    // difference (the screen of the exact pass uses the same band)
    const double ubmax = (double)__uint_as_float(sq[SQ_QMAX]) * nu_max_of(sq, a.n) +
                         (double)__uint_as_float(sq[SQ_BMAX]) * (1.0 + 0x1p-20);
    const double Em = E + 0x1p-21 * (s_absmax + ubmax);
    uint32_t mask = 0, nfire = 0;
#pragma unroll
    for (int j = 0; j < CB_PER; ++j) {
        const int64_t u = ub0 + tid + (int64_t)SEL_THREADS * j;
        if (u < ue) {
            uint8_t f = 0;
            if (fin[j] != 1) {
                if (!same || smin == -INFINITY) {
                    f = 5;
                } else if (trgm) {
                    // every head's margin is below zero: not fired; some head's
                    // above: fired (decided here unless the top-j cap ranks them)
                    const double m = (double)t[j];
                    f = (m + Em <= 0.0) ? 0 : ((a.topj == 0 && m - Em > 0.0) ? 6 : 5);
                } else {
                    const double tv = (double)t[j];
                    const double band = E + fabs(tv) * 0x1p-50 + fabs(smin) * 0x1p-50;
                    f = (tv + band <= smin) ? 0 : 5;
                }
            }
            f2[u] = f;
            mask |= (f == 5) ? (1u << j) : 0u;
            nfire += (f == 6);
        }
    }
    block_append(mask, ub0, a.seq + (int64_t)b * SQ_WORDS + SQ_NCAND3, a.cand + (int64_t)b * a.A, nullptr, t,
                 a.A, s_w, &s_base);
    nfire = block_sum<SEL_THREADS>(nfire, s_w);
    if (tid == 0) {
        uint32_t* w = a.blk + ((int64_t)b * a.nblk + blockIdx.x) * BLK_WORDS;
        w[BW_IN] = nfire;   // rows fired here; the exact pass adds its own to BW_XIN
        w[BW_XIN] = 0u;
    }
}

constexpr int TRIG_EX_BLOCKS = 4;   // blocks per sequence of the exact-margin pass

__global__ __launch_bounds__(RES_THREADS, 1) void trig_exact_kernel(SelectArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    __shared__ double s_absmax;
    const int b = blockIdx.y, tid = threadIdx.x;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t namb = min((int64_t)sq[SQ_NCAND3], a.A);
    if ((int64_t)blockIdx.x * 16 >= namb) return;
    if (tid < 64) {
        double m = 0.0;
        for (int h = tid; h < a.H; h += 64) {
            const double v = a.smax[(int64_t)b * a.H + h];
            m = fmax(m, isfinite(v) ? fabs(v) : 0.0);
        }
        for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
        if (tid == 0) s_absmax = m;
    }
    lds_barrier();
    const bool same = sq[SQ_CMULT] == __float_as_uint(a.cert_mult);
    // screen error: the bound's fp32 error plus the fp32 rounding of s*_h and of the difference
    const double ubmax = (double)__uint_as_float(sq[SQ_QMAX]) * nu_max_of(sq, a.n) +
                         (double)__uint_as_float(sq[SQ_BMAX]) * (1.0 + 0x1p-20);
    const double Et = ub_error_of(sq, a.n) * (1.0 + 0x1p-20) + 0x1p-21 * (s_absmax + ubmax);
    const float margin = same ? next_up_f32(2.0f * ru_f32(Et)) : INFINITY;
    const ExLds L = ex_carve(lds, a.H, a.n);
    exact_keys_block<true, true>(a, b, namb, a.cand + (int64_t)b * a.A, a.ambkey + (int64_t)b * a.A, L, margin,
                                 blockIdx.x, gridDim.x);
}

__global__ __launch_bounds__(RES_THREADS, 1) void trig_fire_kernel(SelectArgs a) {
    extern __shared__ __align__(16) uint8_t lds[];
    __shared__ uint32_t s_w[RES_WAVES];
    __shared__ uint64_t s_theta;
    const int b = blockIdx.x, tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    uint8_t* f2 = a.flags2 + (int64_t)b * a.fstride;
    const int32_t* cl = a.cand + (int64_t)b * a.A;
    const uint64_t* ak = a.ambkey + (int64_t)b * a.A;
    uint32_t* xin = a.blk + (int64_t)b * a.nblk * BLK_WORDS + BW_XIN;
    const int64_t namb = min((int64_t)sq[SQ_NCAND3], a.A);
    const uint64_t zero = f64_to_ord(0.0);
    uint32_t nf = 0;
    for (int64_t i = tid; i < namb; i += RES_THREADS) nf += ak[i] > zero;
    nf = block_sum<RES_THREADS>(nf, s_w);
    __syncthreads();
    if (tid == 0) {
        sq[SQ_NFIRED] = nf;
        sq[SQ_NCAND3] = 0u;   // consumed: a repeated trigger starts an empty list
        s_theta = 0;
    }
    if (a.topj > 0 && (int64_t)nf > a.topj) {
        // the top j margins among the candidates are all fired (margin > 0 >= the rest)
        rank_winners(cl, ak, namb, a.topj, f2, xin, lds, &s_theta, 6);
    } else {
        for (int64_t i = tid; i < namb; i += RES_THREADS)
            if (ak[i] > zero) {
                const int32_t u = cl[i];
                f2[u] = 6;
                atomicAdd(&xin[(int64_t)(u / CB_KEYS) * BLK_WORDS], 1u);
            }
    }
}

hipError_t launch_trigger(const SelectArgs& a, hipStream_t s) {
    hipError_t e;
    if (a.A == 0) {
        hipLaunchKernelGGL(zero_counts_kernel, dim3(1), dim3(64), 0, s, a.adm_count, a.B);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(trig_classify_kernel, dim3((unsigned)a.nblk, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&trig_exact_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, RES_LDS);
    hipLaunchKernelGGL(trig_exact_kernel, dim3(TRIG_EX_BLOCKS, a.B), dim3(RES_THREADS), RES_LDS, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&trig_fire_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, RES_LDS);
    hipLaunchKernelGGL(trig_fire_kernel, dim3(a.B), dim3(RES_THREADS), RES_LDS, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags2, 6, a.adm, a.cap, a.cap, a.adm_count, s);
}

__global__ __launch_bounds__(64) void zero_counts_kernel(int32_t* p, int n) {
    for (int i = threadIdx.x; i < n; i += 64) p[i] = 0;
}

hipError_t launch_admit(const SelectArgs& a, hipStream_t s) {
    hipError_t e;
    if (a.A == 0) {
        hipLaunchKernelGGL(zero_counts_kernel, dim3(1), dim3(64), 0, s, a.adm_count, a.B);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(adm_classify_kernel, dim3((unsigned)a.nblk, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&adm_resolve_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, RES_LDS);
    hipLaunchKernelGGL(adm_resolve_kernel, dim3(a.B), dim3(RES_THREADS), RES_LDS, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags2, 3, a.adm, a.cap, a.cap, a.adm_count, s);
}

}  // namespace vkv
