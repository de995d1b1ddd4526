// k_select.hip -- exact per-sequence top-k and the certified two-tier admission.
//
// Selection (per sequence b, archive rows [0, A)):
//   1. radix select (11 + 11 + 10 bits of the order-preserving key encoding)
//      finds the k-th largest fp32 key t~; per-pass histograms live in LDS and
//      are merged in global memory; the last block of a pass picks the digit.
//   2. with the certified bound E on |key~ - key| (key = the fp64 index score),
//      rows with key~ > t~ + 2E are certainly selected and rows with
//      key~ < t~ - 2E certainly not (order statistics are 1-Lipschitz);
//   3. the rows in between are re-scored in fp64 (d ascending, the exact
//      definition) and ranked by (score desc, index asc) among themselves;
//   4. an ordered compaction writes S ascending.
// Admission (Lemma (Index certificate)): the same band argument on the upper
// bound UB_u against theta = min over S of the exact score.
#include "vkv_internal.h"

namespace vkv {

constexpr int SEL_THREADS = 256;

// ------------------------------------------------------------ error bounds

// nu_max >= max_u ||x_u|| from the scorer's fp32 sum of squares.
__device__ __forceinline__ double nu_max_of(const uint32_t* sq, int n) {
    const double nu2 = (double)__uint_as_float(sq[SQ_NU2MAX]);
    return sqrt(nu2 * (1.0 + (double)n * 0x1p-22)) * (1.0 + 0x1p-20);
}

// |fp32 MFMA key - fp64 key| <= E: products of bf16 are exact in fp32; each
// of the <= n + n/32 fp32 roundings of a partial sum is at most 2^-23 of
// sum|q_d x_d| <= ||qt|| ||x|| (Cauchy-Schwarz); factor 8 of slack, plus an
// absolute term for flushed subnormal products.
__device__ __forceinline__ double key_error_of(const uint32_t* sq, int n) {
    const double qmax = (double)__uint_as_float(sq[SQ_QMAX]);
    return 8.0 * (double)n * 0x1p-23 * qmax * nu_max_of(sq, n) + (double)n * 0x1p-120;
}

// ------------------------------------------------------------------ init

__global__ __launch_bounds__(SEL_THREADS) void select_init_kernel(SelectArgs a) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    if (tid == 0) {
        sq[SQ_EKEY] = __float_as_uint(ru_f32(key_error_of(sq, a.n)));
        sq[SQ_PREFIX] = 0u;
        sq[SQ_KREM] = (uint32_t)a.k;
        sq[SQ_DONE] = 0u;
        sq[SQ_NIN] = 0u;
        sq[SQ_NAMB] = 0u;
        a.theta[b] = -INFINITY;
    }
    for (int i = tid; i < RADIX_BINS; i += SEL_THREADS) a.hist[(int64_t)b * RADIX_BINS + i] = 0u;
    for (int64_t i = tid; i < a.nch * CC_WORDS; i += SEL_THREADS) a.ccount[(int64_t)b * a.nch * CC_WORDS + i] = 0u;
}

__global__ __launch_bounds__(SEL_THREADS) void fill_flags_kernel(uint8_t* flags, int64_t n, uint8_t v) {
    for (int64_t i = (int64_t)blockIdx.x * SEL_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * SEL_THREADS)
        flags[i] = v;
}

// ------------------------------------------------------------ radix select

constexpr int RADIX_KEYS_PER_BLOCK = 8192;

__global__ __launch_bounds__(SEL_THREADS) void radix_pass_kernel(SelectArgs a, int pass) {
    __shared__ uint32_t s_hist[RADIX_BINS];
    __shared__ uint32_t s_part[SEL_THREADS];
    __shared__ int s_last;
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    uint32_t* gh = a.hist + (int64_t)b * RADIX_BINS;
    const uint32_t prefix = sq[SQ_PREFIX];
    const int pshift = (pass == 0) ? 32 : (pass == 1 ? 21 : 10);   // bits of the prefix position
    const int dshift = (pass == 0) ? 21 : (pass == 1 ? 10 : 0);
    const uint32_t dmask = (pass == 2) ? 0x3FFu : 0x7FFu;
    for (int i = tid; i < RADIX_BINS; i += SEL_THREADS) s_hist[i] = 0u;
    __syncthreads();
    const float* kb = a.key + (int64_t)b * a.A;
    const int64_t u0 = (int64_t)blockIdx.x * RADIX_KEYS_PER_BLOCK;
    const int64_t u1 = min(a.A, u0 + RADIX_KEYS_PER_BLOCK);
    for (int64_t u = u0 + tid; u < u1; u += SEL_THREADS) {
        const uint32_t o = key_to_ord(kb[u]);
        if (pass == 0 || (o >> pshift) == prefix) atomicAdd(&s_hist[(o >> dshift) & dmask], 1u);
    }
    __syncthreads();
    for (int i = tid; i < RADIX_BINS; i += SEL_THREADS)
        if (s_hist[i]) atomicAdd(&gh[i], s_hist[i]);
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&sq[SQ_DONE], 1u) == gridDim.x - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    // last block: choose the digit holding the krem-th largest key
    const uint32_t krem = sq[SQ_KREM];
    const int nb = (int)dmask + 1;
    const int per = (nb + SEL_THREADS - 1) / SEL_THREADS;
    uint32_t local = 0;
    for (int d = tid * per; d < min(nb, (tid + 1) * per); ++d) {
        const uint32_t h = __hip_atomic_load(&gh[d], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        s_hist[d] = h;
        local += h;
    }
    s_part[tid] = local;
    __syncthreads();
    // exclusive suffix sum over threads (count of keys in higher bins)
    uint32_t above = 0;
    for (int t = tid + 1; t < SEL_THREADS; ++t) above += s_part[t];
    if (above < krem && krem <= above + local) {
        uint32_t run = above;
        for (int d = min(nb, (tid + 1) * per) - 1; d >= tid * per; --d) {
            if (run + s_hist[d] >= krem) {
                sq[SQ_PREFIX] = (pass == 0 ? 0u : (prefix << (pass == 2 ? 10 : 11))) | (uint32_t)d;
                sq[SQ_KREM] = krem - run;
                break;
            }
            run += s_hist[d];
        }
    }
    __syncthreads();
    for (int i = tid; i < RADIX_BINS; i += SEL_THREADS) gh[i] = 0u;
    if (tid == 0) sq[SQ_DONE] = 0u;
}

// ----------------------------------------------------------- classify

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

__global__ __launch_bounds__(SEL_THREADS) void classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_red[SEL_THREADS / 64];
    const int b = blockIdx.y;
    const int c = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const double th = (double)ord_to_key(sq[SQ_PREFIX]);
    const double E = (double)__uint_as_float(sq[SQ_EKEY]);
    const double band = 2.0 * E * (1.0 + 0x1p-20) + fabs(th) * 0x1p-50;
    const double hi = th + band, lo = th - band;
    const float* kb = a.key + (int64_t)b * a.A;
    uint8_t* fb = a.flags + (int64_t)b * a.A;
    uint32_t nin = 0, namb = 0;
    const int64_t u0 = (int64_t)c * CHUNK;
    const int64_t u1 = min(a.A, u0 + CHUNK);
    for (int64_t u = u0 + tid; u < u1; u += SEL_THREADS) {
        const double kv = (double)kb[u];
        uint8_t f = (kv > hi) ? 1 : ((kv < lo) ? 0 : 2);
        fb[u] = f;
        nin += (f == 1);
        namb += (f == 2);
    }
    nin = block_sum_u32(nin, s_red);
    namb = block_sum_u32(namb, s_red);
    if (tid == 0) {
        uint32_t* cc = a.ccount + ((int64_t)b * a.nch + c) * CC_WORDS;
        cc[CC_IN] = nin;
        cc[CC_AMB] = namb;
        atomicAdd(&sq[SQ_NIN], nin);
        atomicAdd(&sq[SQ_NAMB], namb);
    }
}

// ---------------------------------------------------- ordered compaction

struct CompactArgs {
    const uint8_t* flags;
    uint8_t target;
    const uint32_t* ccount;
    int w0, w1;            // count words of a chunk (w1 < 0: none)
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
    for (int64_t q = tid; q < c; q += SEL_THREADS)
        part += cc[q * CC_WORDS + a.w0] + (a.w1 >= 0 ? cc[q * CC_WORDS + a.w1] : 0u);
    const uint32_t base = block_sum_u32(part, s_red);
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
    if (a.total && c == a.nch - 1 && tid == SEL_THREADS - 1) a.total[b] = (int32_t)(base + s_scan[tid]);
}

static hipError_t run_compact(const SelectArgs& s, const uint8_t* flags, uint8_t target, int w0, int w1,
                              int32_t* out, int64_t out_stride, int64_t cap, int32_t* total,
                              hipStream_t st) {
    CompactArgs c{flags, target, s.ccount, w0, w1, out, out_stride, cap, total, s.A, s.nch};
    hipLaunchKernelGGL(compact_kernel, dim3((unsigned)s.nch, s.B), dim3(SEL_THREADS), 0, st, c);
    return hipGetLastError();
}

// --------------------------------------------------------- fp64 re-scoring

// Exact index score of row u for head h: fp64, d ascending, from +0 (the
// definition; bf16 products are exact in fp64, so fma == mul + add).
__device__ __forceinline__ double exact_score(const uint16_t* qrow, const uint16_t* xrow, int n) {
    double acc = 0.0;
    for (int d = 0; d < n; ++d) acc = fma((double)bf16_to_f32(qrow[d]), (double)bf16_to_f32(xrow[d]), acc);
    return acc;
}

__device__ __forceinline__ double wave_max_f64(double v) {
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
    return v;
}

constexpr int REFINE_BLOCKS = 16;

__global__ __launch_bounds__(SEL_THREADS) void refine_keys_kernel(SelectArgs a) {
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int wave = blockIdx.x * (SEL_THREADS / 64) + (threadIdx.x >> 6);
    const int nwaves = gridDim.x * (SEL_THREADS / 64);
    const uint32_t namb = a.seq[(int64_t)b * SQ_WORDS + SQ_NAMB];
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    for (int64_t i = wave; i < namb; i += nwaves) {
        const int32_t u = a.amb[(int64_t)b * a.A + i];
        const uint16_t* xr = xb + (int64_t)u * a.xs;
        double best = -INFINITY;
        for (int h = lane; h < a.H; h += 64) best = fmax(best, exact_score(qtb + (int64_t)h * a.n, xr, a.n));
        best = wave_max_f64(best);
        if (lane == 0) a.ambkey[(int64_t)b * a.A + i] = best;
    }
}

// Rank of each ambiguous row among the ambiguous rows by (exact key desc,
// index asc); the first k - n_in are selected.  theta = the key at rank
// k - n_in - 1, which is the k-th largest exact key overall.
__global__ __launch_bounds__(SEL_THREADS) void rank_select_kernel(SelectArgs a) {
    __shared__ double s_k[SEL_THREADS];
    __shared__ int32_t s_u[SEL_THREADS];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const int64_t namb = sq[SQ_NAMB];
    const int64_t need = a.k - (int64_t)sq[SQ_NIN];
    const double* kb = a.ambkey + (int64_t)b * a.A;
    const int32_t* ub = a.amb + (int64_t)b * a.A;
    for (int64_t base = (int64_t)blockIdx.x * SEL_THREADS; base < namb; base += (int64_t)gridDim.x * SEL_THREADS) {
        const int64_t i = base + tid;
        const bool have = i < namb;
        const double ki = have ? kb[i] : 0.0;
        const int32_t ui = have ? ub[i] : 0;
        int64_t rank = 0;
        for (int64_t t0 = 0; t0 < namb; t0 += SEL_THREADS) {
            __syncthreads();
            if (t0 + tid < namb) {
                s_k[tid] = kb[t0 + tid];
                s_u[tid] = ub[t0 + tid];
            }
            __syncthreads();
            const int lim = (int)min((int64_t)SEL_THREADS, namb - t0);
            if (have)
                for (int j = 0; j < lim; ++j) {
                    const double kj = s_k[j];
                    rank += (kj > ki) || (kj == ki && s_u[j] < ui);
                }
        }
        if (have && rank < need) {
            a.flags[(int64_t)b * a.A + ui] = 1;
            atomicAdd(&a.ccount[((int64_t)b * a.nch + ui / CHUNK) * CC_WORDS + CC_SELAMB], 1u);
            if (rank == need - 1) a.theta[b] = ki;
        }
    }
}

hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(select_init_kernel, dim3(a.B), dim3(SEL_THREADS), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.A == 0) return hipSuccess;
    if (a.k == 0) {
        hipLaunchKernelGGL(fill_flags_kernel, dim3(256), dim3(SEL_THREADS), 0, s, a.flags, (int64_t)a.B * a.A,
                           (uint8_t)0);
        return hipGetLastError();
    }
    dim3 rg((unsigned)((a.A + RADIX_KEYS_PER_BLOCK - 1) / RADIX_KEYS_PER_BLOCK), a.B);
    for (int p = 0; p < 3; ++p) {
        hipLaunchKernelGGL(radix_pass_kernel, rg, dim3(SEL_THREADS), 0, s, a, p);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    dim3 cg((unsigned)a.nch, a.B);
    hipLaunchKernelGGL(classify_kernel, cg, dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = run_compact(a, a.flags, 2, CC_AMB, -1, a.amb, a.A, a.A, nullptr, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(refine_keys_kernel, dim3(REFINE_BLOCKS, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(rank_select_kernel, dim3(REFINE_BLOCKS, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags, 1, CC_IN, CC_SELAMB, a.sel, a.k, a.k, nullptr, s);
}

// ---------------------------------------------------------------- admit

__global__ __launch_bounds__(SEL_THREADS) void admit_init_kernel(SelectArgs a) {
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    if (tid == 0) {
        const double E = key_error_of(sq, a.n);
        const double smax = (double)__uint_as_float(sq[SQ_QMAX]) * nu_max_of(sq, a.n);
        const double bmax = (double)__uint_as_float(sq[SQ_BMAX]) * (1.0 + 0x1p-20);
        // fp32 evaluation of s^ + B: |error| <= E + 2^-21 (smax + bmax); 2x slack
        sq[SQ_EUB] = __float_as_uint(ru_f32(E * (1.0 + 0x1p-20) + 0x1p-20 * (smax + bmax)));
        sq[SQ_NAMB] = 0u;
        sq[SQ_NADM] = 0u;
    }
    uint32_t* cc = a.ccount + (int64_t)b * a.nch * CC_WORDS;
    for (int64_t q = tid; q < a.nch; q += SEL_THREADS) {
        cc[q * CC_WORDS + CC_ADM] = 0u;
        cc[q * CC_WORDS + CC_AAMB] = 0u;
        cc[q * CC_WORDS + CC_ADMAMB] = 0u;
    }
}

__global__ __launch_bounds__(SEL_THREADS) void admit_classify_kernel(SelectArgs a) {
    __shared__ uint32_t s_red[SEL_THREADS / 64];
    const int b = blockIdx.y;
    const int c = blockIdx.x;
    const int tid = threadIdx.x;
    uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const double th = a.theta[b];
    const double E = (double)__uint_as_float(sq[SQ_EUB]);
    const float* ubb = a.ub + (int64_t)b * a.A;
    const uint8_t* fb = a.flags + (int64_t)b * a.A;
    uint8_t* f2 = a.flags2 + (int64_t)b * a.A;
    uint32_t nadm = 0, namb = 0;
    const int64_t u0 = (int64_t)c * CHUNK;
    const int64_t u1 = min(a.A, u0 + CHUNK);
    for (int64_t u = u0 + tid; u < u1; u += SEL_THREADS) {
        uint8_t f = 0;
        if (fb[u] != 1) {
            if (th == -INFINITY) {
                f = 3;
            } else {
                const double t = (double)ubb[u];
                const double band = E * (1.0 + 0x1p-20) + fabs(t) * 0x1p-50 + fabs(th) * 0x1p-50;
                f = (t - band > th) ? 3 : ((t + band <= th) ? 0 : 4);
            }
        }
        f2[u] = f;
        nadm += (f == 3);
        namb += (f == 4);
    }
    nadm = block_sum_u32(nadm, s_red);
    namb = block_sum_u32(namb, s_red);
    if (tid == 0) {
        uint32_t* cc = a.ccount + ((int64_t)b * a.nch + c) * CC_WORDS;
        cc[CC_ADM] = nadm;
        cc[CC_AAMB] = namb;
        atomicAdd(&sq[SQ_NAMB], namb);
    }
}

__global__ __launch_bounds__(SEL_THREADS) void admit_refine_kernel(SelectArgs a) {
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int wave = blockIdx.x * (SEL_THREADS / 64) + (threadIdx.x >> 6);
    const int nwaves = gridDim.x * (SEL_THREADS / 64);
    const uint32_t namb = a.seq[(int64_t)b * SQ_WORDS + SQ_NAMB];
    const double th = a.theta[b];
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    const float4* hs = reinterpret_cast<const float4*>(a.hsc) + (int64_t)b * a.H;
    for (int64_t i = wave; i < namb; i += nwaves) {
        const int32_t u = a.amb[(int64_t)b * a.A + i];
        const uint16_t* xr = xb + (int64_t)u * a.xs;
        const int64_t o = (int64_t)b * a.T + u;
        const double et = (double)a.eta[o], ep = (double)a.eps[o], ga = (double)a.gam[o];
        double best = -INFINITY;
        for (int h = lane; h < a.H; h += 64) {
            const double s = exact_score(qtb + (int64_t)h * a.n, xr, a.n);
            const float4 q = hs[h];
            const double bh = fma((double)q.x, et, fma((double)q.y, ep, (double)q.z * ga));
            best = fmax(best, s + bh);
        }
        best = wave_max_f64(best);
        if (lane == 0 && best > th) {
            a.flags2[(int64_t)b * a.A + u] = 3;
            atomicAdd(&a.ccount[((int64_t)b * a.nch + u / CHUNK) * CC_WORDS + CC_ADMAMB], 1u);
        }
    }
}

hipError_t launch_admit(const SelectArgs& a, hipStream_t s) {
    hipError_t e;
    if (a.A == 0) {
        hipLaunchKernelGGL(fill_flags_kernel, dim3(1), dim3(SEL_THREADS), 0, s, reinterpret_cast<uint8_t*>(a.adm_count),
                           (int64_t)a.B * 4, (uint8_t)0);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(admit_init_kernel, dim3(a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    dim3 cg((unsigned)a.nch, a.B);
    hipLaunchKernelGGL(admit_classify_kernel, cg, dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = run_compact(a, a.flags2, 4, CC_AAMB, -1, a.amb, a.A, a.A, nullptr, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(admit_refine_kernel, dim3(REFINE_BLOCKS, a.B), dim3(SEL_THREADS), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return run_compact(a, a.flags2, 3, CC_ADM, CC_ADMAMB, a.adm, a.cap, a.cap, a.adm_count, s);
}

}  // namespace vkv
