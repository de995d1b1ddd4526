// k_select.hip -- exact per-sequence top-k and the certified two-tier admission.
//
// Selection (per sequence b, archive rows [0, A)), given fp32 keys key~ with a
// certified bound |key~ - key| <= E for every row (key = the fp64 index score,
// E from the per-sequence maxima of ||qt_h|| and ||x_u||):
//   1. a strided sample of the keys places a bracket [t_lo, t_hi] around the
//      k-th largest key~; one counting pass counts the keys above t_hi and
//      lists the keys inside it; one block per sequence histograms the list
//      over 4096 fine bins and finds the bin of the k-th largest key~ (if the
//      sample missed, it histograms the whole key range instead).  With v = key~ + E and w = key~ - E
//      (rounded outward) this gives HI >= k-th largest v and LO <= k-th
//      largest w, so the k-th largest exact key lies in [LO, HI];
//   2. rows with w > HI are certainly selected and rows with v < LO certainly
//      not; the rows in between are appended to an ambiguous list;
//   3. each ambiguous row's heads are scored again in fp32 (any order: the
//      same bound E holds) and only the heads that can still hold the maximum
//      (within 2E of it) are re-scored in fp64 with d ascending -- the exact
//      definition -- as independent (row, head) chains;
//   4. the ambiguous rows are ranked among themselves by (exact key desc,
//      index asc); the first k - n_in join S, and rank k - n_in - 1 gives theta;
//   5. an ordered compaction writes S ascending.
// Admission (Lemma (Index certificate)) applies the same band argument to the
// upper bound UB_u against theta.
#include "vkv_internal.h"

namespace vkv {

constexpr int SEL_THREADS = 256;
constexpr int SAMPLE_MAX = 2048;             // keys sampled per sequence to place the bracket
constexpr int SAMPLE_BINS = 2048;            // bins of the sample's histogram
constexpr int COUNT_KEYS_PER_BLOCK = 4096;   // keys per block of the counting pass
constexpr int KEY_BATCH = 16;                // keys per thread in flight
constexpr int EX_BLOCKS = 4;                 // per sequence: blocks of the exact-key pass (one per CU: 140 KB of LDS)
constexpr int DECIDE_BLOCKS = 16;            // per sequence: blocks of the admission decision pass
constexpr int RANK_BLOCKS = 16;

// order-preserving encoding of fp64 (for 64-bit atomic max); -0 maps as +0
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

// ------------------------------------------------------------ small kernels

__global__ __launch_bounds__(SEL_THREADS) void fill_u8_kernel(uint8_t* p, int64_t n, uint8_t v) {
    for (int64_t i = (int64_t)blockIdx.x * SEL_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * SEL_THREADS)
        p[i] = v;
}

__global__ __launch_bounds__(64) void select_empty_kernel(SelectArgs a) {
    // k = 0: nothing selected, theta = -inf, chunk counters cleared
    const int b = blockIdx.x;
    if (threadIdx.x == 0) a.theta[b] = -INFINITY;
    if (threadIdx.x == 1) a.seq[(int64_t)b * SQ_WORDS + SQ_NAMB2] = 0u;
    for (int64_t i = threadIdx.x; i < a.nch * CC_WORDS; i += 64) a.ccount[(int64_t)b * a.nch * CC_WORDS + i] = 0u;
}

__device__ __forceinline__ uint32_t block_sum_u32(uint32_t v, uint32_t* s_red) {
    const int tid = threadIdx.x;
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((tid & 63) == 0) s_red[tid >> 6] = v;
    __syncthreads();
    uint32_t t = 0;
    for (int w = 0; w < SEL_THREADS / 64; ++w) t += s_red[w];
    __syncthreads();
    return t;
}

// ---------------------------------------------------------- histogram pass

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

// Sum over threads t' >= tid of v (block of SEL_THREADS threads).
__device__ __forceinline__ uint32_t block_suffix_incl(uint32_t v, uint32_t* s_w) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_down(v, o);
        if (lane + o < 64) v += t;
    }
    __syncthreads();
    if (lane == 0) s_w[w] = v;
    __syncthreads();
    uint32_t add = 0;
    for (int w2 = w + 1; w2 < SEL_THREADS / 64; ++w2) add += s_w[w2];
    return v + add;
}

// ------------------------------------------------------------ the bracket

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

// In a block of SEL_THREADS threads holding a histogram s_h[NB]: the bin d
// where the count of keys in bins >= d first reaches `target` (1 <= target <=
// total).  Returns -1 in threads that do not own it.
template <int NB = HIST_BINS>
__device__ __forceinline__ int find_rank_bin(const uint32_t* s_h, uint32_t target, uint32_t* s_w) {
    constexpr int PER = NB / SEL_THREADS;
    const int tid = threadIdx.x;
    uint32_t loc = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) loc += s_h[tid * PER + j];
    const uint32_t suf = block_suffix_incl(loc, s_w);
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

// The bracket of the k-th largest key~ placed from a sample of up to
// SAMPLE_MAX keys (runs of 32 consecutive keys at evenly spaced offsets; all
// keys if A <= SAMPLE_MAX): [t_lo, t_hi] with sample ranks k_s -/+ (4 sqrt(k_s)
// + 16), k_s = k m / A, from a histogram of the sample over its own range.  A
// deterministic function of the keys, so every block that evaluates it gets
// the same bracket.  Only a heuristic: the bracket pass checks it.
__device__ void sample_bracket(const SelectArgs& a, int b, const uint32_t* sq, uint32_t* s_h, uint32_t* s_w,
                               float* s_mm, float& t_lo, float& t_hi) {
    const int tid = threadIdx.x;
    const int64_t A = a.A;
    const int m = (int)min(A, (int64_t)SAMPLE_MAX);
    const float* kt = a.kt + (int64_t)b * A;
    constexpr int PER = SAMPLE_MAX / SEL_THREADS;
    constexpr int RUN = 32;
    const int nrun = (m + RUN - 1) / RUN;
    const int64_t stride = (m < A && nrun > 1) ? (A - RUN) / (nrun - 1) : 0;
    float v[PER];
    float lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int i = tid + SEL_THREADS * j;
        const int64_t u = (m == A) ? i : min(A - 1, (int64_t)(i / RUN) * stride + (i % RUN));
        v[j] = (i < m) ? kt[u] : 0.f;
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
    const int d_hi = (c_hi >= 1) ? find_rank_bin<SAMPLE_BINS>(s_h, (uint32_t)c_hi, s_w) : -1;
    const int d_lo = (c_lo <= m) ? find_rank_bin<SAMPLE_BINS>(s_h, (uint32_t)c_lo, s_w) : -1;
    __syncthreads();
    // no cut on a side the sample cannot place: the scorer's key extremes
    if (tid == 0) {
        s_mm[0] = ord_to_key(sq[SQ_KMAX]);
        s_mm[1] = ord_to_key(sq[SQ_KMIN]);
    }
    __syncthreads();
    if (d_hi >= 0) s_mm[0] = scale > 0.f ? lo + (float)(d_hi + 1) / scale : hi;
    if (d_lo >= 0) s_mm[1] = scale > 0.f ? lo + (float)d_lo / scale : lo;
    __syncthreads();
    t_hi = s_mm[0];
    t_lo = s_mm[1];
    __syncthreads();
}

// Counting pass: every block places the sampled bracket, counts its keys
// above t_hi and appends those in [t_lo, t_hi] (the bracket holds a few
// percent of the keys) to the sequence's list, one atomic per wave; the bulk
// of the keys, below t_lo, costs one compare.
__global__ __launch_bounds__(SEL_THREADS) void count_kernel(SelectArgs a) {
    __shared__ uint32_t s_h[SAMPLE_BINS];
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ float s_mm[8];
    const int b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    // this block's keys are loaded together with the sample (one round trip)
    static_assert(COUNT_KEYS_PER_BLOCK == KEY_BATCH * SEL_THREADS, "one batch of keys per thread");
    const float* kt = a.kt + (int64_t)b * a.A;
    const int64_t u0 = (int64_t)blockIdx.x * COUNT_KEYS_PER_BLOCK;
    const int64_t u1 = min(a.A, u0 + COUNT_KEYS_PER_BLOCK);
    float k[KEY_BATCH];
#pragma unroll
    for (int j = 0; j < KEY_BATCH; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        k[j] = (u < u1) ? kt[u] : 0.f;
    }
    float tlo, thi;
    sample_bracket(a, b, sq, s_h, s_w, s_mm, tlo, thi);
    if (blockIdx.x == 0 && tid == 0) {
        sq[SQ_BLO] = __float_as_uint(tlo);
        sq[SQ_BHI] = __float_as_uint(thi);
        sq[SQ_NAMB] = 0u;
        sq[SQ_NAMB2] = 0u;
    }
    uint32_t above = 0, nin = 0;
#pragma unroll
    for (int j = 0; j < KEY_BATCH; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        const bool live = u < u1;
        above += (live && k[j] > thi);
        nin += (live && k[j] <= thi && k[j] >= tlo);
    }
    // wave-inclusive scan of the in-bracket counts, one append slot range per wave
    uint32_t incl = nin;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = __shfl_up(incl, o);
        if (lane >= o) incl += t;
    }
    uint32_t base = 0;
    if (lane == 63 && incl) base = atomicAdd(&sq[SQ_NBR], incl);
    base = __shfl(base, 63) + (incl - nin);
    float* list = reinterpret_cast<float*>(a.amb) + (int64_t)b * a.A;
#pragma unroll
    for (int j = 0; j < KEY_BATCH; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        if (u < u1 && k[j] <= thi && k[j] >= tlo) list[base++] = k[j];
    }
    above = block_sum_u32(above, s_w);
    if (tid == 0 && above) atomicAdd(&sq[SQ_ABOVE], above);
}

// One block per sequence, after the counting pass: the bin of the k-th
// largest key~ (a histogram of the listed in-bracket keys) and the band
// around it,
//   THI = up(edge_hi + E) >= k-th largest v,  TLO = down(edge_lo - E) <= k-th largest w.
// If the sample missed (the k-th key~ lies outside [t_lo, t_hi]) the block
// histograms the sequence's whole key range itself.
__global__ __launch_bounds__(SEL_THREADS) void bracket_kernel(SelectArgs a) {
    __shared__ uint32_t s_h[HIST_BINS];
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ int s_bin;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const float tlo = __uint_as_float(sq[SQ_BLO]);
    const float thi = __uint_as_float(sq[SQ_BHI]);
    const uint32_t tot_above = sq[SQ_ABOVE];
    const uint32_t inr = sq[SQ_NBR];
    {
        // the keys inside the sampled bracket, listed by the counting pass
        const float sc0 = bin_scale(tlo, thi);
        for (int i = tid; i < HIST_BINS; i += SEL_THREADS) s_h[i] = 0u;
        __syncthreads();
        const float* list = reinterpret_cast<const float*>(a.amb) + (int64_t)b * a.A;
        for (uint32_t i0 = 0; i0 < inr; i0 += KEY_BATCH * SEL_THREADS) {   // loads of a batch in flight together
            float v[KEY_BATCH];
#pragma unroll
            for (int j = 0; j < KEY_BATCH; ++j) {
                const uint32_t i = i0 + tid + j * SEL_THREADS;
                v[j] = i < inr ? list[i] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < KEY_BATCH; ++j)
                if (i0 + tid + j * SEL_THREADS < inr) atomicAdd(&s_h[bin_of(v[j], tlo, sc0)], 1u);
        }
        __syncthreads();
    }
    const float E = key_band_f32(sq, a.n);
    const int64_t need = a.k - (int64_t)tot_above;
    const bool ok = need >= 1 && need <= (int64_t)inr;
    float lo = tlo, hi = thi, sc = bin_scale(tlo, thi);
    if (!ok) {
        // the sample missed: histogram the whole key range in this block
        lo = ord_to_key(sq[SQ_KMIN]);
        hi = ord_to_key(sq[SQ_KMAX]);
        sc = bin_scale(lo, hi);
        __syncthreads();
        for (int i = tid; i < HIST_BINS; i += SEL_THREADS) s_h[i] = 0u;
        __syncthreads();
        const float* kb = a.kt + (int64_t)b * a.A;
        for (int64_t ub = 0; ub < a.A; ub += KEY_BATCH * SEL_THREADS) {
            float k[KEY_BATCH];
#pragma unroll
            for (int j = 0; j < KEY_BATCH; ++j) {
                const int64_t u = ub + tid + (int64_t)j * SEL_THREADS;
                k[j] = (u < a.A) ? kb[u] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < KEY_BATCH; ++j) {
                const int64_t u = ub + tid + (int64_t)j * SEL_THREADS;
                if (u < a.A) atomicAdd(&s_h[bin_of(k[j], lo, sc)], 1u);
            }
        }
    }
    const uint32_t target = (uint32_t)(ok ? need : a.k);
    if (tid == 0) s_bin = -1;
    __syncthreads();
    const int d = find_rank_bin(s_h, target, s_w);
    if (d >= 0) s_bin = d;
    __syncthreads();
    if (tid == 0) {
        const int db = s_bin < 0 ? 0 : s_bin;
        sq[SQ_THI] = __float_as_uint(band_hi(ru_f32(edge_hi_of(db, lo, hi, sc)), E));
        sq[SQ_TLO] = __float_as_uint(band_lo(rd_f32(edge_lo_of(db, lo, sc)), E));
        a.theta[b] = -INFINITY;
    }
}

// ----------------------------------------------------------- classify

// Append the rows of a wave whose predicate holds to list[base..) (order
// within the list is irrelevant: the ranking below is by (key, index)).
__device__ __forceinline__ void wave_append(bool pred, int32_t value, uint32_t* counter, int32_t* list) {
    const uint64_t mask = __ballot(pred);
    if (mask == 0) return;
    const int lane = threadIdx.x & 63;
    const int leader = __ffsll((unsigned long long)mask) - 1;
    uint32_t base = 0;
    if (lane == leader) base = atomicAdd(counter, (uint32_t)__popcll(mask));
    base = __shfl(base, leader);
    if (pred) list[base + __popcll(mask & ((1ull << lane) - 1ull))] = value;
}

__global__ __launch_bounds__(SEL_THREADS) void classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_red[SEL_THREADS / 64];
    constexpr int PER = CHUNK / SEL_THREADS;
    const int b = blockIdx.y;
    const int c = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const float LO = __uint_as_float(sq[SQ_TLO]);
    const float HI = __uint_as_float(sq[SQ_THI]);
    const float E = key_band_f32(sq, a.n);
    const float* kt = a.kt + (int64_t)b * a.A;
    uint8_t* fb = a.flags + (int64_t)b * a.A;
    int32_t* amb = a.amb + (int64_t)b * a.A;
    const int64_t u0 = (int64_t)c * CHUNK;
    const int64_t u1 = min(a.A, u0 + CHUNK);
    float k[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        k[j] = (u < u1) ? kt[u] : 0.f;
    }
    uint32_t nin = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        uint8_t f = 0;
        if (u < u1) {
            // selected for sure: key >= w > HI >= theta*;  out for sure: key <= v < LO <= theta*
            f = (band_lo(k[j], E) > HI) ? 1 : ((band_hi(k[j], E) < LO) ? 0 : 2);
            fb[u] = f;
        }
        nin += (f == 1);
        wave_append(f == 2, (int32_t)u, &sq[SQ_NAMB], amb);
    }
    nin = block_sum_u32(nin, s_red);
    if (tid == 0) {
        uint32_t* cc = a.ccount + ((int64_t)b * a.nch + c) * CC_WORDS;
        cc[CC_IN] = nin;
        cc[CC_SELAMB] = 0u;
        cc[CC_ADM] = 0u;
        cc[CC_ADMAMB] = 0u;
    }
}

// ---------------------------------------------------- ordered compaction

struct CompactArgs {
    const uint8_t* flags;
    uint8_t target;
    const uint32_t* ccount;
    int w0, w1;            // count words of a chunk
    int32_t* out;
    int64_t out_stride;
    int64_t cap;
    int32_t* total;        // [B] or null
    int64_t A, nch;
};

__global__ __launch_bounds__(SEL_THREADS) void compact_kernel(CompactArgs a) {
    __shared__ uint32_t s_scan[SEL_THREADS];
    __shared__ uint32_t s_red[SEL_THREADS / 64];
    const int b = blockIdx.y;
    const int c = blockIdx.x;
    const int tid = threadIdx.x;
    const uint32_t* cc = a.ccount + (int64_t)b * a.nch * CC_WORDS;
    uint32_t part = 0;
    for (int64_t q = tid; q < c; q += SEL_THREADS) part += cc[q * CC_WORDS + a.w0] + cc[q * CC_WORDS + a.w1];
    const uint32_t base = block_sum_u32(part, s_red);
    const uint32_t mine = cc[(int64_t)c * CC_WORDS + a.w0] + cc[(int64_t)c * CC_WORDS + a.w1];
    if (a.total && c == a.nch - 1 && tid == 0) a.total[b] = (int32_t)(base + mine);
    if (mine == 0) return;
    // each thread owns 8 consecutive rows of the chunk
    const int64_t u0 = (int64_t)c * CHUNK + 8 * tid;
    const uint8_t* fb = a.flags + (int64_t)b * a.A;
    uint8_t f[8];
    uint32_t cnt = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int64_t u = u0 + e;
        f[e] = (u < a.A) ? fb[u] : (uint8_t)0xFF;
        cnt += (f[e] == a.target);
    }
    s_scan[tid] = cnt;
    __syncthreads();
    for (int o = 1; o < SEL_THREADS; o <<= 1) {
        uint32_t v = (tid >= o) ? s_scan[tid - o] : 0u;
        __syncthreads();
        s_scan[tid] += v;
        __syncthreads();
    }
    uint32_t pos = base + s_scan[tid] - cnt;
    int32_t* ob = a.out + (int64_t)b * a.out_stride;
#pragma unroll
    for (int e = 0; e < 8; ++e)
        if (f[e] == a.target) {
            if ((int64_t)pos < a.cap) ob[pos] = (int32_t)(u0 + e);
            ++pos;
        }
}

static hipError_t run_compact(const SelectArgs& s, const uint8_t* flags, uint8_t target, int w0, int w1,
                              int32_t* out, int64_t out_stride, int64_t cap, int32_t* total, hipStream_t st) {
    CompactArgs c{flags, target, s.ccount, w0, w1, out, out_stride, cap, total, s.A, s.nch};
    hipLaunchKernelGGL(compact_kernel, dim3((unsigned)s.nch, s.B), dim3(SEL_THREADS), 0, st, c);
    return hipGetLastError();
}

// --------------------------------------------------------- fp64 re-scoring

// Exact keys of the ambiguous rows, a tile of 16 rows per wave.  The rows are
// gathered straight into the MFMA operand layout (lane 16 g + c: row c, dims
// 32 ks + 8 g ..) and scored against every head with fp32 accumulation -- the
// scorer's arithmetic, so |s~ - s| <= E for every (row, head).  Only heads
// within 2E of their row's maximum can hold the exact maximum; each such
// (row, head) pair gets its fp64 chain (d ascending from +0: the exact
// definition) from one lane, and the row's exact key is the maximum over its
// pairs (LDS atomic max on the order-preserving encoding).  With UB the
// screened quantity is s^_h + B_h(u) (Lemma (Index certificate)) and the
// margin is that bound's own fp32 error.
constexpr int EX_QT_MAX = 32768;   // qt elements staged in LDS (64 KB)

template <bool UB>
__device__ __forceinline__ double exact_chain(const uint16_t* q, const uint16_t* x, int n, float4 hs, double et,
                                              double ep, double ga) {
    double acc = 0.0;
    const int n8 = n / 8;
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

template <bool UB, bool QLDS>
__global__ __launch_bounds__(SEL_THREADS) void exact_keys_kernel(SelectArgs a) {
    __shared__ __align__(16) uint16_t s_qt[QLDS ? EX_QT_MAX : 8];   // [H][n]
    __shared__ float4 s_hs[128];
    __shared__ unsigned long long s_best[4][16];
    __shared__ uint32_t s_list[4][64];
    __shared__ __align__(16) uint16_t s_x[4][16 * D_ROW];   // each wave's 16 gathered rows, for the fp64 chains
    const int b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, c = lane & 15;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t namb = sq[UB ? SQ_NAMB2 : SQ_NAMB];
    if ((int64_t)blockIdx.x * 64 >= namb) return;
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const int n8 = a.n / 8;
    if (QLDS) {
        constexpr int QP = EX_QT_MAX / 8 / SEL_THREADS;
        u16x8_t v[QP];
#pragma unroll
        for (int j = 0; j < QP; ++j) {
            const int p = tid + SEL_THREADS * j;
            v[j] = (p < a.H * n8) ? *reinterpret_cast<const u16x8_t*>(qtb + 8 * (int64_t)p)
                                  : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < QP; ++j) {
            const int p = tid + SEL_THREADS * j;
            if (p < a.H * n8) *reinterpret_cast<u16x8_t*>(&s_qt[8 * p]) = v[j];
        }
    }
    if (UB && tid < a.H) s_hs[tid] = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + tid];
    __syncthreads();
    const uint16_t* qsrc = QLDS ? s_qt : qtb;
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    const int32_t* amb = a.amb + (int64_t)b * a.A;
    uint64_t* ak = a.ambkey + (int64_t)b * a.A;
    const float E = ru_f32(UB ? ub_error_of(sq, a.n) * (1.0 + 0x1p-20) : key_error_of(sq, a.n));
    const float margin = next_up_f32(2.0f * E);
    const int KS = a.n / 32, HT = (a.H + 15) / 16;
    for (int64_t t0 = ((int64_t)blockIdx.x * 4 + wave) * 16; t0 < namb; t0 += (int64_t)gridDim.x * 64) {
        const int64_t i = min(t0 + c, namb - 1);
        const int64_t u = amb[i];
        const uint16_t* x = xb + u * a.xs;
        f32x4_t acc[8];
#pragma unroll
        for (int ht = 0; ht < 8; ++ht) acc[ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(x + 32 * ks + 8 * g);
            *reinterpret_cast<bf16x8_t*>(&s_x[wave][c * a.n + 32 * ks + 8 * g]) = xf;
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
        float et = 0.f, ep = 0.f, ga = 0.f;
        if (UB) {
            const int64_t o = (int64_t)b * a.T + u;
            et = a.eta[o];
            ep = a.eps[o];
            ga = a.gam[o];
        }
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
                        const float4 hs = s_hs[h];
                        v += fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga));
                    }
                }
                acc[ht][q] = v;
                m = fmaxf(m, v);
            }
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        const float thr = next_down_f32(m - margin);
        if (lane < 16) s_best[wave][lane] = (unsigned long long)f64_to_ord(-INFINITY);
        // the rows are in LDS for every lane of the wave (LDS operations of a
        // wave complete in order)
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_wave_barrier();
        // candidates in rounds of up to 64 pairs, one fp64 chain per lane
        int nl = 0;
        auto flush = [&]() {
            if (lane < nl) {
                const uint32_t e = s_list[wave][lane];
                const int cr = (int)(e >> 8), h = (int)(e & 255);
                const int64_t ir = t0 + cr;
                const int64_t ur = amb[ir];
                const int64_t o = (int64_t)b * a.T + ur;
                const float4 hs = UB ? s_hs[h] : make_float4(0.f, 0.f, 0.f, 0.f);
                const double v = exact_chain<UB>(qsrc + (int64_t)h * a.n, &s_x[wave][cr * a.n], a.n, hs,
                                                 UB ? (double)a.eta[o] : 0.0, UB ? (double)a.eps[o] : 0.0,
                                                 UB ? (double)a.gam[o] : 0.0);
                atomicMax(&s_best[wave][cr], (unsigned long long)f64_to_ord(v));
            }
            nl = 0;
        };
#pragma unroll
        for (int ht = 0; ht < 8; ++ht)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const bool cand = (t0 + c < namb) && acc[ht][q] >= thr && acc[ht][q] > -INFINITY;
                const uint64_t bal = __ballot(cand);
                const int cnt = __popcll(bal);
                if (cnt == 0) continue;
                if (nl + cnt > 64) flush();
                if (cand) {
                    const int pos = nl + __popcll(bal & ((1ull << lane) - 1ull));
                    s_list[wave][pos] = ((uint32_t)c << 8) | (uint32_t)(16 * ht + 4 * g + q);
                }
                nl += cnt;
            }
        flush();
        if (lane < 16 && t0 + lane < namb) ak[t0 + lane] = s_best[wave][lane];
    }
}

template <bool UB>
static hipError_t run_exact_keys(const SelectArgs& a, hipStream_t s) {
    dim3 g(EX_BLOCKS, a.B);
    if ((int64_t)a.H * a.n <= EX_QT_MAX)
        hipLaunchKernelGGL((exact_keys_kernel<UB, true>), g, dim3(SEL_THREADS), 0, s, a);
    else
        hipLaunchKernelGGL((exact_keys_kernel<UB, false>), g, dim3(SEL_THREADS), 0, s, a);
    return hipGetLastError();
}

// Rank of each ambiguous row among the ambiguous rows by (exact key desc,
// index asc); the first k - n_in are selected.  theta = the key at rank
// k - n_in - 1, which is the k-th largest exact key overall.  A block ranks
// RK_ROWS rows: thread (row r, quarter q) counts the rows ahead of r in the
// q-th quarter of each tile of the list (staged in LDS), then the four
// partial counts are summed.
constexpr int RK_ROWS = SEL_THREADS / 4;
constexpr int RK_TILE = 2048;

__global__ __launch_bounds__(SEL_THREADS) void rank_select_kernel(SelectArgs a) {
    __shared__ double s_k[RK_TILE];
    __shared__ int32_t s_u[RK_TILE];
    __shared__ uint32_t s_r[4][RK_ROWS];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int r = tid % RK_ROWS, q = tid / RK_ROWS;
    __shared__ uint32_t s_red[SEL_THREADS / 64];
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t namb = sq[SQ_NAMB];
    if ((int64_t)blockIdx.x * RK_ROWS >= namb) return;
    // rows certainly in S: the sum of the chunk counts of the classification
    uint32_t nin = 0;
    for (int64_t c = tid; c < a.nch; c += SEL_THREADS) nin += a.ccount[((int64_t)b * a.nch + c) * CC_WORDS + CC_IN];
    nin = block_sum_u32(nin, s_red);
    const int64_t need = a.k - (int64_t)nin;
    const uint64_t* kb = a.ambkey + (int64_t)b * a.A;
    const int32_t* ub = a.amb + (int64_t)b * a.A;
    for (int64_t base = (int64_t)blockIdx.x * RK_ROWS; base < namb; base += (int64_t)gridDim.x * RK_ROWS) {
        const int64_t i = base + r;
        const bool have = i < namb;
        const double ki = have ? ord_to_f64(kb[i]) : 0.0;
        const int32_t ui = have ? ub[i] : 0;
        uint32_t rank = 0;
        for (int64_t t0 = 0; t0 < namb; t0 += RK_TILE) {
            const int lim = (int)min((int64_t)RK_TILE, namb - t0);
            __syncthreads();
            constexpr int PER = RK_TILE / SEL_THREADS;
            double kv[PER];
            int32_t uv[PER];
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                const int e = tid + SEL_THREADS * j;
                kv[j] = (e < lim) ? ord_to_f64(kb[t0 + e]) : 0.0;
                uv[j] = (e < lim) ? ub[t0 + e] : 0;
            }
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                s_k[tid + SEL_THREADS * j] = kv[j];
                s_u[tid + SEL_THREADS * j] = uv[j];
            }
            __syncthreads();
            if (have) {
                const int qlen = (lim + 3) / 4;
                const int j0 = q * qlen, j1 = min(lim, j0 + qlen);
#pragma unroll 4
                for (int j = j0; j < j1; ++j) {
                    const double kj = s_k[j];
                    rank += (kj > ki) || (kj == ki && s_u[j] < ui);
                }
            }
        }
        s_r[q][r] = rank;
        __syncthreads();
        if (q == 0 && have) {
            const int64_t rk = (int64_t)s_r[0][r] + s_r[1][r] + s_r[2][r] + s_r[3][r];
            if (rk < need) {
                a.flags[(int64_t)b * a.A + ui] = 1;
                atomicAdd(&a.ccount[((int64_t)b * a.nch + ui / CHUNK) * CC_WORDS + CC_SELAMB], 1u);
                if (rk == need - 1) a.theta[b] = ki;
            }
        }
    }
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    hipError_t e;
    if (a.k == 0) {
        hipLaunchKernelGGL(select_empty_kernel, dim3(a.B), dim3(64), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (a.A == 0) return hipSuccess;
        hipLaunchKernelGGL(fill_u8_kernel, dim3(256), dim3(SEL_THREADS), 0, s, a.flags, (int64_t)a.B * a.A, (uint8_t)0);
        return hipGetLastError();
    }
    dim3 cg((unsigned)((a.A + COUNT_KEYS_PER_BLOCK - 1) / COUNT_KEYS_PER_BLOCK), a.B);
    hipLaunchKernelGGL(count_kernel, cg, dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(bracket_kernel, dim3(a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(classify_kernel, dim3((unsigned)a.nch, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = run_exact_keys<false>(a, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(rank_select_kernel, dim3(RANK_BLOCKS, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags, 1, CC_IN, CC_SELAMB, a.sel, a.k, a.k, nullptr, s);
}

// ---------------------------------------------------------------- admit

__global__ __launch_bounds__(SEL_THREADS) void admit_classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_red[SEL_THREADS / 64];
    constexpr int PER = CHUNK / SEL_THREADS;
    const int b = blockIdx.y;
    const int c = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const double th = a.theta[b];
    const double E = ub_error_of(sq, a.n) * (1.0 + 0x1p-20);
    const float* ubb = a.ub + (int64_t)b * a.A;
    const uint8_t* fb = a.flags + (int64_t)b * a.A;
    uint8_t* f2 = a.flags2 + (int64_t)b * a.A;
    int32_t* amb = a.amb + (int64_t)b * a.A;
    const int64_t u0 = (int64_t)c * CHUNK;
    const int64_t u1 = min(a.A, u0 + CHUNK);
    float t[PER];
    uint8_t fin[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        t[j] = (u < u1) ? ubb[u] : 0.f;
        fin[j] = (u < u1) ? fb[u] : (uint8_t)1;
    }
    uint32_t nadm = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int64_t u = u0 + tid + (int64_t)j * SEL_THREADS;
        uint8_t f = 0;
        if (u < u1) {
            if (fin[j] != 1) {
                if (th == -INFINITY) {
                    f = 3;
                } else {
                    const double tv = (double)t[j];
                    const double band = E + fabs(tv) * 0x1p-50 + fabs(th) * 0x1p-50;
                    f = (tv - band > th) ? 3 : ((tv + band <= th) ? 0 : 4);
                }
            }
            f2[u] = f;
        }
        nadm += (f == 3);
        wave_append(f == 4, (int32_t)u, &sq[SQ_NAMB2], amb);
    }
    nadm = block_sum_u32(nadm, s_red);
    if (tid == 0) a.ccount[((int64_t)b * a.nch + c) * CC_WORDS + CC_ADM] = nadm;
}

// Ambiguous rows of the admission, decided on their exact bound.
__global__ __launch_bounds__(SEL_THREADS) void admit_decide_kernel(SelectArgs a) {
    const int b = blockIdx.y;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t namb = sq[SQ_NAMB2];
    const double th = a.theta[b];
    const uint64_t* ak = a.ambkey + (int64_t)b * a.A;
    const int32_t* amb = a.amb + (int64_t)b * a.A;
    for (int64_t i = (int64_t)blockIdx.x * SEL_THREADS + threadIdx.x; i < namb; i += (int64_t)gridDim.x * SEL_THREADS) {
        if (ord_to_f64(ak[i]) > th) {
            const int32_t u = amb[i];
            a.flags2[(int64_t)b * a.A + u] = 3;
            atomicAdd(&a.ccount[((int64_t)b * a.nch + u / CHUNK) * CC_WORDS + CC_ADMAMB], 1u);
        }
    }
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
    hipLaunchKernelGGL(admit_classify_kernel, dim3((unsigned)a.nch, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = run_exact_keys<true>(a, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(admit_decide_kernel, dim3(DECIDE_BLOCKS, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags2, 3, CC_ADM, CC_ADMAMB, a.adm, a.cap, a.cap, a.adm_count, s);
}

}  // namespace vkv
