// k_sigma.hip -- the query-independent tier-1 selector sigma_u (Sec. 4.1, the
// sigma equation; App. H, block close) and the tier it keeps.
//
// Per closed block of 4096 rows and per channel of the 64-dim branch r_u as
// the cache row stores it (its last 64 elements), sigma keeps the
// frequency bins [0, kappa) of the sequence-axis DFT (and their mirrors),
// inverts, and takes the norm over the channels of what that low-pass
// reconstruction misses at each row.
//
// sigma_fft_kernel: one workgroup per (8-channel group, block, sequence).  Two
// real channels travel as one complex sequence z = x + i y (the mask keeps
// f and N - f together, so masking z masks x and y alike).  The 4096-point
// transform runs in LDS in place as six radix-4 decimation-in-frequency
// stages (natural order in, base-4 digit-reversed order out); the mask is
// applied in that order; the inverse is the adjoint of the same stages taken
// in reverse (digit-reversed in, natural out), which gives N times the
// inverse transform with no permutation pass.  fp64 throughout; twiddles
// come from a quarter-wave cosine table.  The squared residuals of the
// group's 8 channels are summed per row and stored; sigma_reduce_kernel adds
// the 8 groups in order and takes the square root.
//
// sigma_select_kernel: one workgroup per sequence.  The tier is the first
// nsink rows plus the top-m of the other closed rows by (sigma desc, row asc):
// an MSB-first radix select over the fp64 bit patterns (sigma >= 0, so the
// bits order like the values) finds the m-th key, then one ordered pass
// writes the rows above it and the first rows equal to it, ascending.
//
// Also here: the flags of a caller's tier (for the step on a given kept set)
// and the all-layer CSR pack of row lists (offsets by one block's prefix sum,
// then one copy per list).
#include "vkv_internal.h"

namespace vkv {

constexpr int SG_N = 4096;                 // rows per closed block
constexpr int SG_Q4 = SG_N / 4;            // quarter wave
constexpr int SG_THREADS = 256;
constexpr int SG_ROWS = SG_N / SG_THREADS; // rows per thread in the residual pass
constexpr int SG_GROUPS = 8;               // 8-channel groups of the 64-dim branch
constexpr size_t SG_LDS = (size_t)SG_N * sizeof(double2) + (size_t)(SG_Q4 + 1) * sizeof(double);

// exp(-2 pi i k / N) for k in [0, N), from ct[j] = cos(2 pi j / N), j in [0, N/4]
__device__ __forceinline__ double2 sg_twiddle(const double* ct, int k) {
    const int q = k >> 10, r = k & (SG_Q4 - 1);
    double c, s;
    if (q == 0) {
        c = ct[r];
        s = ct[SG_Q4 - r];
    } else if (q == 1) {
        c = -ct[SG_Q4 - r];
        s = ct[r];
    } else if (q == 2) {
        c = -ct[r];
        s = -ct[SG_Q4 - r];
    } else {
        c = ct[SG_Q4 - r];
        s = -ct[r];
    }
    return make_double2(c, -s);
}

__device__ __forceinline__ double2 cmul(double2 a, double2 b) {
    return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 cmulc(double2 a, double2 b) {   // a * conj(b)
    return make_double2(a.x * b.x + a.y * b.y, a.y * b.x - a.x * b.y);
}
__device__ __forceinline__ double2 cadd(double2 a, double2 b) { return make_double2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ double2 csub(double2 a, double2 b) { return make_double2(a.x - b.x, a.y - b.y); }

// base-4 digit reversal of a 12-bit index (six digits)
__device__ __forceinline__ int rev4(int p) {
    int f = 0;
#pragma unroll
    for (int d = 0; d < 6; ++d) f = (f << 2) | ((p >> (2 * d)) & 3);
    return f;
}

// Stage st of the forward transform (in place): groups of 4Q = N / 4^st, the
// butterfly (a, b, c, d) at quarter offsets, twiddles w^i, w^2i, w^3i with
// w = exp(-2 pi i / 4Q).
__device__ __forceinline__ void dif_stage(double2* X, const double* ct, int st, int tid) {
    const int lq = 10 - 2 * st;            // log2 Q
    const int Q = 1 << lq;
#pragma unroll
    for (int m = 0; m < SG_N / 4 / SG_THREADS; ++m) {
        const int j = tid + SG_THREADS * m;
        const int i = j & (Q - 1);
        const int i0 = ((j >> lq) << (lq + 2)) + i;
        const double2 a = X[i0], b = X[i0 + Q], c = X[i0 + 2 * Q], d = X[i0 + 3 * Q];
        const double2 apc = cadd(a, c), amc = csub(a, c), bpd = cadd(b, d), bmd = csub(b, d);
        const int k = i << (2 * st);
        X[i0] = cadd(apc, bpd);
        X[i0 + Q] = cmul(make_double2(amc.x + bmd.y, amc.y - bmd.x), sg_twiddle(ct, k));
        X[i0 + 2 * Q] = cmul(csub(apc, bpd), sg_twiddle(ct, 2 * k));
        X[i0 + 3 * Q] = cmul(make_double2(amc.x - bmd.y, amc.y + bmd.x), sg_twiddle(ct, 3 * k));
    }
}

// The adjoint of dif_stage: conjugate twiddles first, then the conjugate butterfly.
__device__ __forceinline__ void dit_adjoint_stage(double2* X, const double* ct, int st, int tid) {
    const int lq = 10 - 2 * st;
    const int Q = 1 << lq;
#pragma unroll
    for (int m = 0; m < SG_N / 4 / SG_THREADS; ++m) {
        const int j = tid + SG_THREADS * m;
        const int i = j & (Q - 1);
        const int i0 = ((j >> lq) << (lq + 2)) + i;
        const int k = i << (2 * st);
        const double2 A = X[i0];
        const double2 B = cmulc(X[i0 + Q], sg_twiddle(ct, k));
        const double2 C = cmulc(X[i0 + 2 * Q], sg_twiddle(ct, 2 * k));
        const double2 D = cmulc(X[i0 + 3 * Q], sg_twiddle(ct, 3 * k));
        const double2 apc = cadd(A, C), amc = csub(A, C), bpd = cadd(B, D), bmd = csub(B, D);
        X[i0] = cadd(apc, bpd);
        X[i0 + Q] = make_double2(amc.x - bmd.y, amc.y + bmd.x);
        X[i0 + 2 * Q] = csub(apc, bpd);
        X[i0 + 3 * Q] = make_double2(amc.x + bmd.y, amc.y - bmd.x);
    }
}

__global__ __launch_bounds__(SG_THREADS) void sigma_fft_kernel(SigmaArgs a) {
    extern __shared__ __align__(16) uint8_t sg_lds[];
    double2* X = reinterpret_cast<double2*>(sg_lds);
    double* ct = reinterpret_cast<double*>(sg_lds + (size_t)SG_N * sizeof(double2));
    const int grp = blockIdx.x, blk = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
    for (int j = tid; j <= SG_Q4; j += SG_THREADS)
        ct[j] = (j == 0) ? 1.0 : (j == SG_Q4 ? 0.0 : cospi((double)j / (double)(SG_N / 2)));
    const uint16_t* base = a.cache + (int64_t)b * a.cbs + (a.t0 + (int64_t)blk * SG_N) * a.crs + D_LAT + 8 * grp;
    double acc[SG_ROWS];
#pragma unroll
    for (int m = 0; m < SG_ROWS; ++m) acc[m] = 0.0;
    for (int pair = 0; pair < 4; ++pair) {
        float xv[SG_ROWS], yv[SG_ROWS];
#pragma unroll
        for (int m = 0; m < SG_ROWS; ++m) {
            const int t = tid + SG_THREADS * m;
            const uint32_t w = *reinterpret_cast<const uint32_t*>(base + (int64_t)t * a.crs + 2 * pair);
            xv[m] = __uint_as_float(w << 16);
            yv[m] = __uint_as_float(w & 0xFFFF0000u);
            X[t] = make_double2((double)xv[m], (double)yv[m]);
        }
        __syncthreads();
        for (int st = 0; st < 6; ++st) {
            dif_stage(X, ct, st, tid);
            __syncthreads();
        }
        // keep bins f < kappa and f > N - kappa (position p holds bin rev4(p))
        for (int p = tid; p < SG_N; p += SG_THREADS) {
            const int f = rev4(p);
            if (f >= a.kappa && f <= SG_N - a.kappa) X[p] = make_double2(0.0, 0.0);
        }
        __syncthreads();
        for (int st = 5; st >= 0; --st) {
            dit_adjoint_stage(X, ct, st, tid);
            __syncthreads();
        }
        constexpr double inv_n = 1.0 / SG_N;
#pragma unroll
        for (int m = 0; m < SG_ROWS; ++m) {
            const int t = tid + SG_THREADS * m;
            const double2 l = X[t];
            const double dx = (double)xv[m] - l.x * inv_n, dy = (double)yv[m] - l.y * inv_n;
            acc[m] += dx * dx + dy * dy;
        }
        __syncthreads();
    }
    double* out = a.part + (((int64_t)b * a.nblk + blk) * SG_GROUPS + grp) * SG_N;
#pragma unroll
    for (int m = 0; m < SG_ROWS; ++m) out[tid + SG_THREADS * m] = acc[m];
}

__global__ __launch_bounds__(256) void sigma_reduce_kernel(SigmaArgs a) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;   // row within the closed range
    const int b = blockIdx.y;
    if (e >= (int64_t)a.nblk * SG_N) return;
    const int64_t blk = e / SG_N, t = e % SG_N;
    const double* p = a.part + ((int64_t)b * a.nblk + blk) * SG_GROUPS * SG_N + t;
    double s = 0.0;
#pragma unroll
    for (int g = 0; g < SG_GROUPS; ++g) s += p[(int64_t)g * SG_N];
    a.sigma[(int64_t)b * a.sstride + a.t0 + e] = sqrt(s);
}

size_t sigma_workspace_bytes(int64_t B, int64_t nblk) { return (size_t)(B * nblk) * SG_GROUPS * SG_N * sizeof(double); }

hipError_t launch_sigma(const SigmaArgs& a, hipStream_t s) {
    if (a.nblk == 0 || a.B == 0) return hipSuccess;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&sigma_fft_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)SG_LDS);
    hipLaunchKernelGGL(sigma_fft_kernel, dim3(SG_GROUPS, (unsigned)a.nblk, (unsigned)a.B), dim3(SG_THREADS), SG_LDS,
                       s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t rows = (int64_t)a.nblk * SG_N;
    hipLaunchKernelGGL(sigma_reduce_kernel, dim3((unsigned)((rows + 255) / 256), (unsigned)a.B), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------------------ the sigma tier

constexpr int SS_THREADS = 1024;
constexpr int SS_WAVES = SS_THREADS / 64;

// exclusive count of set flags below this lane in the block, and the block total
__device__ __forceinline__ int block_rank(bool f, int* s_w, int tid, int* total) {
    const uint64_t bal = __ballot(f);
    const int lane = tid & 63, w = tid >> 6;
    const int below = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) s_w[w] = __popcll(bal);
    __syncthreads();
    int off = 0, tot = 0;
    for (int i = 0; i < SS_WAVES; ++i) {
        const int c = s_w[i];
        off += (i < w) ? c : 0;
        tot += c;
    }
    __syncthreads();
    *total = tot;
    return off + below;
}

__global__ __launch_bounds__(SS_THREADS) void sigma_select_kernel(SigmaSelArgs a) {
    __shared__ uint32_t hist[256];
    __shared__ int s_w[SS_WAVES];
    __shared__ uint64_t s_prefix;
    __shared__ int64_t s_need;
    const int b = blockIdx.x, tid = threadIdx.x;
    const uint64_t* key = reinterpret_cast<const uint64_t*>(a.sigma + (int64_t)b * a.sstride);
    int32_t* out = a.kept + (int64_t)b * a.kstride;
    const int64_t lo = a.n < a.nsink ? a.n : a.nsink;
    const int64_t navail = a.n - lo;
    const int64_t take = a.m < navail ? a.m : navail;
    // the take-th largest key among rows [lo, n): MSB-first, 8 bits per pass
    uint64_t prefix = 0, mask = 0;
    int64_t need = take;
    if (take > 0 && take < navail) {
        for (int pass = 0; pass < 8; ++pass) {
            const int shift = 56 - 8 * pass;
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
            for (int64_t u = lo + tid; u < a.n; u += SS_THREADS) {
                const uint64_t k = key[u];
                if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (tid == 0) {
                int64_t cum = 0;
                int d = 255;
                for (; d > 0; --d) {
                    if (cum + hist[d] >= need) break;
                    cum += hist[d];
                }
                s_prefix = prefix | ((uint64_t)d << shift);
                s_need = need - cum;
            }
            __syncthreads();
            prefix = s_prefix;
            need = s_need;
            mask |= 255ull << shift;
            __syncthreads();
        }
    }
    // ordered pass: sinks, keys above the threshold, and the first `need` rows equal to it
    const bool all = take == navail;
    int64_t base = 0, eq_seen = 0;
    for (int64_t u0 = 0; u0 < a.n; u0 += SS_THREADS) {
        const int64_t u = u0 + tid;
        bool in = false, eq = false;
        if (u < a.n) {
            if (u < lo) {
                in = true;
            } else if (all) {
                in = true;
            } else if (take > 0) {
                const uint64_t k = key[u];
                in = k > prefix;
                eq = k == prefix;
            }
        }
        int neq = 0;
        const int er = block_rank(eq, s_w, tid, &neq);
        if (eq && eq_seen + er < need) in = true;
        eq_seen += neq;
        int nin = 0;
        const int r = block_rank(in, s_w, tid, &nin);
        if (in) out[base + r] = (int32_t)u;
        base += nin;
    }
}

hipError_t launch_sigma_select(const SigmaSelArgs& a, hipStream_t s) {
    if (a.B == 0) return hipSuccess;
    hipLaunchKernelGGL(sigma_select_kernel, dim3((unsigned)a.B), dim3(SS_THREADS), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------ a caller's tier into the flags

// flags[b][u] = 1 for the k rows of sel[b] inside [0, A), 0 for the other rows
// The per-row tier flags of a kept table (ascending rows in [0, A)), in one
// pass: block (c, b) owns rows [4096 c, 4096 (c + 1)) of sequence b, clears
// their flags, finds the table's entries inside its range by two searches of
// the ascending list, and marks them.  No block depends on another's writes.
constexpr int TF_ROWS = 4096;

// first position i of the ascending list ks[0, k) with ks[i] >= v (k if none),
// by one wave: each round probes 64 evenly spaced positions and keeps the
// interval between the last probe below v and the first one at or above it
__device__ __forceinline__ int64_t wave_lower_bound(const int32_t* ks, int64_t k, int64_t v, int lane) {
    int64_t lo = 0, hi = k;   // the answer lies in [lo, hi]
    while (hi - lo > 64) {
        const int64_t step = (hi - lo + 63) / 64;
        const int64_t p = lo + (int64_t)lane * step;
        const bool below = p < hi && (int64_t)ks[p] < v;
        const int cnt = __popcll(__ballot(below));   // the probes below v are a prefix of the lanes
        const int64_t nlo = cnt == 0 ? lo : lo + (int64_t)(cnt - 1) * step + 1;
        hi = min(hi, lo + (int64_t)cnt * step);
        lo = nlo;
    }
    const int64_t p = lo + lane;
    const bool below = p < hi && (int64_t)ks[p] < v;
    return lo + __popcll(__ballot(below));
}

__global__ __launch_bounds__(256) void tier_flags_kernel(uint8_t* flags, int64_t fstride, int64_t A, const int32_t* sel,
                                                         int64_t k) {
    __shared__ int64_t s_range[2];
    const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t u0 = (int64_t)blockIdx.x * TF_ROWS, u1 = min(A, u0 + TF_ROWS);
    uint8_t* fb = flags + (int64_t)b * fstride;
    const int32_t* ks = sel + (int64_t)b * k;
    for (int64_t u = u0 + tid; u < u1; u += 256) fb[u] = 0;
    if (wave < 2) {   // wave 0: the first entry >= u0, wave 1: the first entry >= u1
        const int64_t pos = wave_lower_bound(ks, k, wave == 0 ? u0 : u1, lane);
        if (lane == 0) s_range[wave] = pos;
    }
    __syncthreads();   // the clears are done before any mark, and the range is known
    for (int64_t i = s_range[0] + tid; i < s_range[1]; i += 256) {
        const int32_t u = ks[i];
        if (u >= u0 && u < u1) fb[u] = 1;
    }
}

hipError_t launch_mark_tier(uint8_t* flags, int64_t fstride, int64_t A, int B, const int32_t* sel, int64_t k,
                            hipStream_t s) {
    if (B == 0 || A == 0) return hipSuccess;
    const unsigned g = (unsigned)((A + TF_ROWS - 1) / TF_ROWS);
    hipLaunchKernelGGL(tier_flags_kernel, dim3(g, (unsigned)B), dim3(256), 0, s, flags, fstride, A, sel, k);
    return hipGetLastError();
}

}  // namespace vkv

namespace vkv {

// ------------------------------------------------ all-layer CSR pack of row lists

// offsets[i] = sum_{j < i} min(max(counts[j], 0), cap), i in [0, n]; one block, 1024 threads
__global__ __launch_bounds__(1024) void pack_offsets_kernel(const int32_t* counts, int64_t n, int64_t cap,
                                                            int32_t* offsets) {
    __shared__ int64_t s_part[1024];
    const int tid = threadIdx.x;
    const int64_t per = (n + 1023) / 1024;
    const int64_t i0 = tid * per, i1 = min(n, i0 + per);
    int64_t s = 0;
    for (int64_t i = i0; i < i1; ++i) {
        const int64_t c = counts[i];
        s += c < 0 ? 0 : (c < cap ? c : cap);
    }
    s_part[tid] = s;
    __syncthreads();
    int64_t base = 0;
    for (int j = 0; j < tid; ++j) base += s_part[j];
    for (int64_t i = i0; i < i1; ++i) {
        offsets[i] = (int32_t)base;
        const int64_t c = counts[i];
        base += c < 0 ? 0 : (c < cap ? c : cap);
    }
    if (tid == 1023) offsets[n] = (int32_t)base;
}

__global__ __launch_bounds__(256) void pack_copy_kernel(const int32_t* lists, const int32_t* offsets, int64_t cap,
                                                        int32_t* packed) {
    const int64_t i = blockIdx.y;
    const int64_t len = offsets[i + 1] - offsets[i];
    for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < len; t += (int64_t)gridDim.x * 256)
        packed[offsets[i] + t] = lists[i * cap + t];
}

hipError_t launch_pack_rows(const int32_t* lists, const int32_t* counts, int64_t n, int64_t cap, int32_t* offsets,
                            int32_t* packed, hipStream_t s) {
    hipLaunchKernelGGL(pack_offsets_kernel, dim3(1), dim3(1024), 0, s, counts, n, cap, offsets);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n == 0 || cap == 0) return e;
    const unsigned gx = (unsigned)((cap + 255) / 256 < 64 ? (cap + 255) / 256 : 64);
    hipLaunchKernelGGL(pack_copy_kernel, dim3(gx, (unsigned)n), dim3(256), 0, s, lists, offsets, cap, packed);
    return hipGetLastError();
}

}  // namespace vkv
