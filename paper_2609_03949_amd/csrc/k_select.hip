// k_select.hip -- exact per-sequence top-k and the certified two-tier admission.
//
// Selection (per sequence b, archive rows [0, A)), given fp32 keys key~ with a
// certified bound |key~ - key| <= E for every row (key = the fp64 index score,
// E from the per-sequence maxima of ||qt_h|| and ||x_u||):
//   1. one histogram pass over 4096 linear bins of [min key~ - E, max key~ + E]
//      of v = key~ + E and w = key~ - E (rounded outward) brackets the k-th
//      largest exact key: HI >= k-th largest v and LO <= k-th largest w;
//   2. rows with w > HI are certainly selected and rows with v < LO certainly
//      not; the rows in between are appended to an ambiguous list;
//   3. the ambiguous rows are re-scored in fp64 (d ascending: the exact
//      definition) and ranked among themselves by (score desc, index asc); the
//      first k - n_in join S, and the one of rank k - n_in - 1 gives theta;
//   4. an ordered compaction writes S ascending.
// Admission (Lemma (Index certificate)) applies the same band argument to the
// upper bound UB_u against theta.
#include "vkv_internal.h"

namespace vkv {

constexpr int SEL_THREADS = 256;
constexpr int HIST_KEYS_PER_BLOCK = 16384;
constexpr int REFINE_BLOCKS = 32;
constexpr int RANK_BLOCKS = 16;

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

__device__ __forceinline__ float bin_scale(float lo, float hi) {
    const float range = hi - lo;
    return (range > 0.f && range < INFINITY) ? (float)HIST_BINS / range : 0.f;
}

__device__ __forceinline__ int bin_of(float x, float lo, float scale) {
    const float t = (x - lo) * scale;
    const int bi = (t > 0.f) ? (int)t : 0;
    return bi < HIST_BINS ? bi : HIST_BINS - 1;
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

// Histograms of v_u = key~_u + E and w_u = key~_u - E over linear bins of
// [min v, max v].  The last block to finish finds the bins holding the k-th
// largest v and the k-th largest w and stores
//   HI >= k-th largest v  and  LO <= k-th largest w
// (bin edges widened past the fp32 rounding of the binning).  Since
// w_u <= key_u <= v_u, the k-th largest exact key lies in [LO, HI].
constexpr int HIST_BATCH = 16;   // keys per thread in flight

__global__ __launch_bounds__(SEL_THREADS) void hist_kernel(SelectArgs a) {
    __shared__ uint32_t s_hv[HIST_BINS];
    __shared__ uint32_t s_hw[HIST_BINS];
    __shared__ uint32_t s_w[SEL_THREADS / 64];
    __shared__ int s_last;
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    uint32_t* gv = a.hist + (int64_t)b * 2 * HIST_BINS;
    uint32_t* gw = gv + HIST_BINS;
    if (blockIdx.x == 0 && tid == 0) {
        sq[SQ_NIN] = 0u;
        sq[SQ_NAMB] = 0u;
        sq[SQ_NAMB2] = 0u;
        a.theta[b] = -INFINITY;
    }
    const float E = key_band_f32(sq, a.n);
    const float lo = band_lo(ord_to_key(sq[SQ_KMIN]), E);
    const float hi = band_hi(ord_to_key(sq[SQ_KMAX]), E);
    const float scale = bin_scale(lo, hi);
    for (int i = tid; i < HIST_BINS; i += SEL_THREADS) {
        s_hv[i] = 0u;
        s_hw[i] = 0u;
    }
    __syncthreads();
    const float* kt = a.kt + (int64_t)b * a.A;
    const int64_t u0 = (int64_t)blockIdx.x * HIST_KEYS_PER_BLOCK;
    const int64_t u1 = min(a.A, u0 + HIST_KEYS_PER_BLOCK);
    for (int64_t ub = u0; ub < u1; ub += HIST_BATCH * SEL_THREADS) {
        float k[HIST_BATCH];
#pragma unroll
        for (int j = 0; j < HIST_BATCH; ++j) {
            const int64_t u = ub + tid + (int64_t)j * SEL_THREADS;
            k[j] = (u < u1) ? kt[u] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < HIST_BATCH; ++j) {
            const int64_t u = ub + tid + (int64_t)j * SEL_THREADS;
            if (u < u1) {
                atomicAdd(&s_hv[bin_of(band_hi(k[j], E), lo, scale)], 1u);
                atomicAdd(&s_hw[bin_of(band_lo(k[j], E), lo, scale)], 1u);
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < HIST_BINS; i += SEL_THREADS) {
        if (s_hv[i]) atomicAdd(&gv[i], s_hv[i]);
        if (s_hw[i]) atomicAdd(&gw[i], s_hw[i]);
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&sq[SQ_DONE], 1u) == gridDim.x - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    constexpr int PER = HIST_BINS / SEL_THREADS;
    uint32_t lv = 0, lw = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int d = tid * PER + j;
        const uint32_t hv = __hip_atomic_load(&gv[d], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t hw = __hip_atomic_load(&gw[d], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_hv[d] = hv;
        s_hw[d] = hw;
        lv += hv;
        lw += hw;
    }
    const uint32_t sv = block_suffix_incl(lv, s_w);
    const uint32_t sw = block_suffix_incl(lw, s_w);
    const uint32_t k = (uint32_t)a.k;
    const double w_bin = (scale > 0.f) ? 1.0 / (double)scale : 0.0;
    const double slack = fabs((double)lo) * 0x1p-22 + 0x1p-100;
    if (sv - lv < k && k <= sv) {
        uint32_t run = sv - lv;
        for (int d = (tid + 1) * PER - 1; d >= tid * PER; --d) {
            if (run + s_hv[d] >= k) {
                double edge = (double)hi;
                if (scale > 0.f) edge = fmin(edge, (double)lo + (double)(d + 1) * w_bin * (1.0 + 0x1p-20) + slack);
                sq[SQ_THI] = __float_as_uint(ru_f32(edge));
                break;
            }
            run += s_hv[d];
        }
    }
    if (sw - lw < k && k <= sw) {
        uint32_t run = sw - lw;
        for (int d = (tid + 1) * PER - 1; d >= tid * PER; --d) {
            if (run + s_hw[d] >= k) {
                double edge = (double)lo;
                if (scale > 0.f) edge = fmax(edge, (double)lo + (double)d * w_bin * (1.0 - 0x1p-20) - slack);
                sq[SQ_TLO] = __float_as_uint(rd_f32(edge));
                break;
            }
            run += s_hw[d];
        }
    }
    __syncthreads();
    for (int i = tid; i < 2 * HIST_BINS; i += SEL_THREADS) gv[i] = 0u;
    if (tid == 0) sq[SQ_DONE] = 0u;
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
        atomicAdd(&sq[SQ_NIN], nin);
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

// Exact index scores of the ambiguous rows, RF_ROWS rows per block iteration:
// thread (slot, hq) runs the fp64 dot products (d ascending, from +0; bf16
// products are exact in fp64) of heads hq, hq+32, hq+64, hq+96 for row slot
// `slot`, with qt held transposed in LDS (head-contiguous, conflict-free) when
// it fits.  The rows of the next iteration are loaded while the current ones
// are scored (double-buffered LDS).
constexpr int RF_ROWS = 8;
constexpr int RF_QT_MAX = 32768;   // elements of qt staged in LDS (64 KB)
constexpr int RF_PIECES = (RF_ROWS * D_ROW / 8 + SEL_THREADS - 1) / SEL_THREADS;   // 16-byte row pieces per thread (max)

template <bool UB, bool QLDS>
__global__ __launch_bounds__(SEL_THREADS) void refine_kernel(SelectArgs a) {
    constexpr int XW = QLDS ? RF_QT_MAX / 128 : D_ROW;                // row width held (n <= XW)
    __shared__ __align__(16) uint16_t s_qt[QLDS ? RF_QT_MAX : 8];     // [n][128]
    __shared__ __align__(16) uint16_t s_x[2][RF_ROWS][XW];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int slot = tid >> 5, hq = tid & 31;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const uint32_t namb = sq[UB ? SQ_NAMB2 : SQ_NAMB];
    if ((uint32_t)(blockIdx.x * RF_ROWS) >= namb) return;
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const int n8 = a.n / 8;
    if (QLDS) {
        // 16-byte pieces of qt, all loads in flight, then transposed writes
        constexpr int QP = RF_QT_MAX / 8 / SEL_THREADS;
        u16x8_t v[QP];
#pragma unroll
        for (int j = 0; j < QP; ++j) {
            const int p = tid + SEL_THREADS * j;
            const int h = p & 127, d8 = p >> 7;
            v[j] = (d8 < n8 && h < a.H) ? *reinterpret_cast<const u16x8_t*>(qtb + (int64_t)h * a.n + 8 * d8)
                                        : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < QP; ++j) {
            const int p = tid + SEL_THREADS * j;
            const int h = p & 127, d8 = p >> 7;
            if (d8 < n8)
#pragma unroll
                for (int e = 0; e < 8; ++e) s_qt[(8 * d8 + e) * 128 + h] = v[j][e];
        }
    }
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    const int32_t* amb = a.amb + (int64_t)b * a.A;
    const double th = UB ? a.theta[b] : 0.0;
    const float4* hs = reinterpret_cast<const float4*>(a.hsc) + (int64_t)b * a.H;
    const uint32_t step = gridDim.x * RF_ROWS;
    // row pieces of iteration i0 into registers
    u16x8_t pf[RF_PIECES];
    auto fetch = [&](uint32_t i0) {
#pragma unroll
        for (int j = 0; j < RF_PIECES; ++j) {
            const int idx = tid + SEL_THREADS * j;
            const int rl = idx / n8, p = idx % n8;
            pf[j] = u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
            if (rl < RF_ROWS && i0 + rl < namb)
                pf[j] = *reinterpret_cast<const u16x8_t*>(xb + (int64_t)amb[i0 + rl] * a.xs + 8 * p);
        }
    };
    auto park = [&](int buf) {
#pragma unroll
        for (int j = 0; j < RF_PIECES; ++j) {
            const int idx = tid + SEL_THREADS * j;
            const int rl = idx / n8, p = idx % n8;
            if (rl < RF_ROWS) *reinterpret_cast<u16x8_t*>(&s_x[buf][rl][8 * p]) = pf[j];
        }
    };
    uint32_t i0 = blockIdx.x * RF_ROWS;
    fetch(i0);
    park(0);
    __syncthreads();
    for (int buf = 0; i0 < namb; i0 += step, buf ^= 1) {
        const bool more = i0 + step < namb;
        if (more) fetch(i0 + step);
        const uint32_t i = i0 + slot;
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 8
        for (int d = 0; d < a.n; ++d) {
            const double xv = (double)bf16_to_f32(s_x[buf][slot][d]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int h = hq + 32 * j;
                const uint16_t qb = QLDS ? s_qt[d * 128 + h] : ((h < a.H) ? qtb[(int64_t)h * a.n + d] : (uint16_t)0);
                acc[j] = fma((double)bf16_to_f32(qb), xv, acc[j]);
            }
        }
        double best = -INFINITY;
        const int64_t u = (i < namb) ? (int64_t)amb[i] : 0;
        double et = 0.0, ep = 0.0, ga = 0.0;
        if (UB && i < namb) {
            const int64_t o = (int64_t)b * a.T + u;
            et = (double)a.eta[o];
            ep = (double)a.eps[o];
            ga = (double)a.gam[o];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int h = hq + 32 * j;
            if (h < a.H) {
                double v = acc[j];
                if (UB) {
                    const float4 q = hs[h];
                    v = v + fma((double)q.x, et, fma((double)q.y, ep, (double)q.z * ga));
                }
                best = fmax(best, v);
            }
        }
        for (int o = 16; o > 0; o >>= 1) best = fmax(best, __shfl_xor(best, o));
        if (hq == 0 && i < namb) {
            if (!UB) {
                a.ambkey[(int64_t)b * a.A + i] = best;
            } else if (best > th) {
                a.flags2[(int64_t)b * a.A + u] = 3;
                atomicAdd(&a.ccount[((int64_t)b * a.nch + u / CHUNK) * CC_WORDS + CC_ADMAMB], 1u);
            }
        }
        if (more) park(buf ^ 1);
        __syncthreads();
    }
}

template <bool UB>
static hipError_t run_refine(const SelectArgs& a, hipStream_t s) {
    dim3 g(REFINE_BLOCKS, a.B);
    if ((int64_t)a.n * 128 <= RF_QT_MAX)
        hipLaunchKernelGGL((refine_kernel<UB, true>), g, dim3(SEL_THREADS), 0, s, a);
    else
        hipLaunchKernelGGL((refine_kernel<UB, false>), g, dim3(SEL_THREADS), 0, s, a);
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
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t namb = sq[SQ_NAMB];
    const int64_t need = a.k - (int64_t)sq[SQ_NIN];
    const double* kb = a.ambkey + (int64_t)b * a.A;
    const int32_t* ub = a.amb + (int64_t)b * a.A;
    for (int64_t base = (int64_t)blockIdx.x * RK_ROWS; base < namb; base += (int64_t)gridDim.x * RK_ROWS) {
        const int64_t i = base + r;
        const bool have = i < namb;
        const double ki = have ? kb[i] : 0.0;
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
                kv[j] = (e < lim) ? kb[t0 + e] : 0.0;
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
    if (a.A == 0 || a.k == 0) {
        hipLaunchKernelGGL(select_empty_kernel, dim3(a.B), dim3(64), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (a.A == 0) return hipSuccess;
        hipLaunchKernelGGL(fill_u8_kernel, dim3(256), dim3(SEL_THREADS), 0, s, a.flags, (int64_t)a.B * a.A, (uint8_t)0);
        return hipGetLastError();
    }
    dim3 hg((unsigned)((a.A + HIST_KEYS_PER_BLOCK - 1) / HIST_KEYS_PER_BLOCK), a.B);
    hipLaunchKernelGGL(hist_kernel, hg, dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(classify_kernel, dim3((unsigned)a.nch, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = run_refine<false>(a, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(rank_select_kernel, dim3(RANK_BLOCKS, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags, 1, CC_IN, CC_SELAMB, a.sel, a.k, a.k, nullptr, s);
}

// ---------------------------------------------------------------- admit

__global__ __launch_bounds__(SEL_THREADS) void admit_classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_red[SEL_THREADS / 64];
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
    uint32_t nadm = 0;
    const int64_t u0 = (int64_t)c * CHUNK;
    const int64_t u1 = min(a.A, u0 + CHUNK);
    for (int64_t base = u0; base < u1; base += SEL_THREADS) {
        const int64_t u = base + tid;
        uint8_t f = 0;
        if (u < u1) {
            if (fb[u] != 1) {
                if (th == -INFINITY) {
                    f = 3;
                } else {
                    const double t = (double)ubb[u];
                    const double band = E + fabs(t) * 0x1p-50 + fabs(th) * 0x1p-50;
                    f = (t - band > th) ? 3 : ((t + band <= th) ? 0 : 4);
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
    if ((e = run_refine<true>(a, s)) != hipSuccess) return e;
    return run_compact(a, a.flags2, 3, CC_ADM, CC_ADMAMB, a.adm, a.cap, a.cap, a.adm_count, s);
}

}  // namespace vkv
