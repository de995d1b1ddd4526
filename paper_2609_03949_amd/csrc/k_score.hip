// k_score.hip -- query preparation and the streaming index scorer (gfx950).
//
// Index score of archived row u for head h (Eq. (trigger), the exact-branch
// and sketch terms; Sec. 4.2):
//     s^_h(u) = qt_h . x_u,   qt_h = [q_rope_h ; RNE_bf16(P q_lat_h)],   x_u = index row
// key_u = max_h s^_h(u).  The scorer streams only the narrow index slice
// (64 + r bf16 per row) from HBM and runs the heads x rows contraction on the
// matrix cores (v_mfma_f32_16x16x32_bf16): A = qt (16 heads x 32 dims per
// fragment, resident in VGPRs for the whole wave), B = 16 index rows x 32 dims
// loaded straight from global memory in MFMA operand layout, so each lane
// issues 16-byte loads of one row.  The heads maximum is taken in registers
// (4 heads per lane per tile, then two cross-lane steps).
#include "vkv_internal.h"

namespace vkv {

// ----------------------------------------------------------- query prep

// Stage 1: w[b,h,j] = sum_i P[j,i] q_lat[b,h,i] (fp64, i ascending) and the
// query digest qt[b,h,off+j] = RNE_bf16(w).  A block owns 64 basis rows (held
// transposed in LDS) and 4 heads.  Block (0,0,b) also clears the step state.
__global__ __launch_bounds__(256) void qprep_project_kernel(QprepArgs a) {
    __shared__ uint16_t s_pt[D_LAT][66];   // P^T tile, padded against bank conflicts
    __shared__ double s_q[4][D_LAT];
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    if (blockIdx.x == 0 && blockIdx.y == 0 && tid < SQ_WORDS) a.seq[b * SQ_WORDS + tid] = 0u;
    if (a.r == 0 || !(a.mode & 2)) return;
    const int j0 = 64 * blockIdx.x;
    const int jn = min(64, a.r - j0);
    const int h0 = 4 * blockIdx.y;
    for (int idx = tid; idx < jn * D_LAT; idx += 256) {
        int jl = idx / D_LAT, i = idx % D_LAT;
        s_pt[i][jl] = a.P[(int64_t)(j0 + jl) * D_LAT + i];
    }
    for (int idx = tid; idx < 4 * D_LAT; idx += 256) {
        int hl = idx / D_LAT, i = idx % D_LAT;
        int h = h0 + hl;
        s_q[hl][i] = (h < a.H) ? (double)bf16_to_f32(a.q_lat[((int64_t)b * a.H + h) * D_LAT + i]) : 0.0;
    }
    __syncthreads();
    const int hl = tid >> 6, jl = tid & 63;
    const int h = h0 + hl, j = j0 + jl;
    if (h >= a.H || jl >= jn) return;
    double acc = 0.0;
    for (int i = 0; i < D_LAT; ++i) acc = fma((double)bf16_to_f32(s_pt[i][jl]), s_q[hl][i], acc);
    const int64_t bh = (int64_t)b * a.H + h;
    a.wproj[bh * a.r + j] = acc;
    const int off = (a.mode & 1) ? D_ROPE : 0;
    a.qt[bh * a.n + off + j] = f64_to_bf16_rne(acc);
}

// Stage 2 (one wave per head): certificate scalars of the head, each an fp32
// upper bound (Lemma (Index certificate) plus the bf16 rounding of the stored
// sketch; fixed fp64 evaluation order):
//   a_h >= sqrt(q^T (I - P^T P) q),  n_h >= ||qd_h||,  e_h >= ||qd_h - P q||
// plus ||qt_h|| for the scorer's error bound, and the rope half of qt.
__global__ __launch_bounds__(64) void qprep_finish_kernel(QprepArgs a) {
    const int bh = blockIdx.x;
    const int b = bh / a.H;
    const int lane = threadIdx.x;
    const uint16_t* q = a.q_lat + (int64_t)bh * D_LAT;
    const double* w = a.wproj + (int64_t)bh * a.r;
    uint16_t* qt = a.qt + (int64_t)bh * a.n;
    const int off = (a.mode & 1) ? D_ROPE : 0;
    const int rd = (a.mode & 2) ? a.r : 0;
    if (a.mode & 1) qt[lane] = a.q_rope[(int64_t)bh * D_ROPE + lane];
    // four sequential fp64 sums, one per lane, in the oracle's order
    double acc = 0.0;
    if (lane == 0) {
        for (int i = 0; i < D_LAT; ++i) {
            double v = (double)bf16_to_f32(q[i]);
            acc = fma(v, v, acc);
        }
    } else if (lane == 1) {
        for (int j = 0; j < rd; ++j) acc = fma(w[j], w[j], acc);
    } else if (lane == 2) {
        for (int j = 0; j < rd; ++j) {
            double t = (double)bf16_to_f32(qt[off + j]) - w[j];
            acc = fma(t, t, acc);
        }
    } else if (lane == 3) {
        for (int j = 0; j < rd; ++j) {
            double d = (double)bf16_to_f32(qt[off + j]);
            acc = fma(d, d, acc);
        }
    }
    const double Nq = __shfl(acc, 0), Nw = __shfl(acc, 1), Ne = __shfl(acc, 2), Nd = __shfl(acc, 3);
    // ||qt_h||^2 over all n columns (an upper bound only; order irrelevant)
    double s2 = 0.0;
    for (int d = lane; d < a.n; d += 64) {
        double v = (double)bf16_to_f32(qt[d]);
        s2 += v * v;
    }
    for (int o = 32; o > 0; o >>= 1) s2 += __shfl_xor(s2, o);
    if (lane == 0) {
        const double G = CERT_G;
        double Dm = G * (double)ru_sqrt_f32((double)rd * Nq);
        double sw = (double)ru_sqrt_f32(Nw);
        double X = ((Nq - Nw) + G * (Nq + Nw)) + (2.0 * Dm) * sw;
        float ah = ru_sqrt_f32((X > 0.0 ? X : 0.0) * (1.0 + G));
        float eh = ru_f32((double)ru_sqrt_f32(Ne) * (1.0 + G) + Dm);
        float nh = ru_sqrt_f32(Nd * (1.0 + G));
        float qn = ru_sqrt_f32(s2 * (1.0 + 0x1p-30));
        float4 hs = make_float4(ah, nh, eh, qn);
        reinterpret_cast<float4*>(a.hsc)[bh] = hs;
        uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        atomicMax(sq + SQ_QMAX, __float_as_uint(qn));
        atomicMax(sq + SQ_AMAX, __float_as_uint(ah));
        atomicMax(sq + SQ_NMAX, __float_as_uint(nh));
        atomicMax(sq + SQ_EMAX, __float_as_uint(eh));
    }
}

hipError_t launch_qprep(const QprepArgs& a, hipStream_t s) {
    int jt = (a.r > 0 && (a.mode & 2)) ? (a.r + 63) / 64 : 1;
    dim3 g1(jt, (a.H + 3) / 4, a.B);
    hipLaunchKernelGGL(qprep_project_kernel, g1, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(qprep_finish_kernel, dim3(a.B * a.H), dim3(64), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------------------- the scorer

constexpr int SCORE_TPW = 32;                       // 16-row tiles per wave
constexpr int SCORE_ROWS_PER_BLOCK = 4 * 16 * SCORE_TPW;

__device__ __forceinline__ float wave_max16(float m) {
    m = fmaxf(m, __shfl_xor(m, 16));
    m = fmaxf(m, __shfl_xor(m, 32));
    return m;
}

__device__ __forceinline__ float wave_max_all(float m) {
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    return m;
}

// HT head tiles of 16 and KS dim steps of 32 held in VGPRs (HT*KS <= 32).
template <int HT, int KS, bool UB>
__global__ __launch_bounds__(256, 2) void score_kernel(ScoreArgs a) {
    __shared__ float4 s_hs[UB ? 128 : 1];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    if (UB) {
        for (int h = tid; h < a.H; h += 256)
            s_hs[h] = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + h];
        __syncthreads();
    }
    const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * SCORE_TPW);
    if (r0 >= a.A) return;
    const int64_t rend = min(a.A, r0 + (int64_t)(16 * SCORE_TPW));

    bf16x8_t qf[HT][KS];
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
        const int h = 16 * ht + c;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (h < a.H)
                qf[ht][ks] = *reinterpret_cast<const bf16x8_t*>(qtb + (int64_t)h * a.n + 32 * ks + 8 * g);
            else
                qf[ht][ks] = bf16x8_t{};
        }
    }
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    float amax = 0.f, nmax = 0.f, emax = 0.f;
    if (UB) {
        const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        amax = __uint_as_float(sq[SQ_AMAX]);
        nmax = __uint_as_float(sq[SQ_NMAX]);
        emax = __uint_as_float(sq[SQ_EMAX]);
    }
    float nu2m = 0.f, bmm = 0.f;

    bf16x8_t xf[KS];
    {
        const int64_t row = r0 + c;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            xf[ks] = (row < rend) ? *reinterpret_cast<const bf16x8_t*>(xb + row * a.xs + 32 * ks + 8 * g)
                                  : bf16x8_t{};
    }
    for (int64_t t0 = r0; t0 < rend; t0 += 16) {
        const int64_t row = t0 + c;
        const bool valid = row < rend;
        // prefetch the next tile while this one runs on the matrix cores
        bf16x8_t xn[KS];
        const int64_t nrow = row + 16;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            xn[ks] = (nrow < rend) ? *reinterpret_cast<const bf16x8_t*>(xb + nrow * a.xs + 32 * ks + 8 * g)
                                   : bf16x8_t{};
        float et = 0.f, ep = 0.f, ga = 0.f;
        if (UB && valid) {
            const int64_t o = (int64_t)b * a.T + row;
            et = a.eta[o];
            ep = a.eps[o];
            ga = a.gam[o];
        }
        f32x4_t acc[HT];
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) acc[ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
                acc[ht] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[ht][ks], xf[ks], acc[ht], 0, 0, 0);
        // acc[ht][i] = score of head 16*ht + 4*g + i for row t0 + c
        float m = -INFINITY;
        float ubv = -INFINITY;
#pragma unroll
        for (int ht = 0; ht < HT; ++ht)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int h = 16 * ht + 4 * g + i;
                if (h < a.H) {
                    m = fmaxf(m, acc[ht][i]);
                    if (UB) {
                        const float4 hs = s_hs[h];
                        const float bh = fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga));
                        ubv = fmaxf(ubv, acc[ht][i] + bh);
                    }
                }
            }
        m = wave_max16(m);
        float s2 = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float v = (float)xf[ks][e];
                s2 = fmaf(v, v, s2);
            }
        s2 += __shfl_xor(s2, 16);
        s2 += __shfl_xor(s2, 32);
        if (valid) nu2m = fmaxf(nu2m, s2);
        if (UB) {
            ubv = wave_max16(ubv);
            if (valid) bmm = fmaxf(bmm, fmaf(amax, et, fmaf(nmax, ep, emax * ga)));
            if (g == 0 && valid) a.ub[(int64_t)b * a.A + row] = ubv;
        }
        if (g == 0 && valid) a.key[(int64_t)b * a.A + row] = m;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) xf[ks] = xn[ks];
    }
    nu2m = wave_max_all(nu2m);
    if (UB) bmm = wave_max_all(bmm);
    if (lane == 0) {
        uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        atomicMax(sq + SQ_NU2MAX, __float_as_uint(nu2m));
        if (UB) atomicMax(sq + SQ_BMAX, __float_as_uint(bmm));
    }
}

// Any head count / width within the limits: heads and dims in runtime loops,
// query fragments re-read from the (cache-resident) qt buffer per tile.
template <bool UB>
__global__ __launch_bounds__(256, 2) void score_generic_kernel(ScoreArgs a) {
    constexpr int KSMAX = D_ROW / 32;
    __shared__ float4 s_hs[UB ? 128 : 1];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    if (UB) {
        for (int h = tid; h < a.H; h += 256)
            s_hs[h] = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + h];
        __syncthreads();
    }
    const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * SCORE_TPW);
    if (r0 >= a.A) return;
    const int64_t rend = min(a.A, r0 + (int64_t)(16 * SCORE_TPW));
    const int KS = a.n / 32;
    const int HT = (a.H + 15) / 16;
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    float amax = 0.f, nmax = 0.f, emax = 0.f;
    if (UB) {
        const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        amax = __uint_as_float(sq[SQ_AMAX]);
        nmax = __uint_as_float(sq[SQ_NMAX]);
        emax = __uint_as_float(sq[SQ_EMAX]);
    }
    float nu2m = 0.f, bmm = 0.f;
    for (int64_t t0 = r0; t0 < rend; t0 += 16) {
        const int64_t row = t0 + c;
        const bool valid = row < rend;
        bf16x8_t xf[KSMAX];
#pragma unroll
        for (int ks = 0; ks < KSMAX; ++ks)
            xf[ks] = (valid && ks < KS) ? *reinterpret_cast<const bf16x8_t*>(xb + row * a.xs + 32 * ks + 8 * g)
                                        : bf16x8_t{};
        float et = 0.f, ep = 0.f, ga = 0.f;
        if (UB && valid) {
            const int64_t o = (int64_t)b * a.T + row;
            et = a.eta[o];
            ep = a.eps[o];
            ga = a.gam[o];
        }
        float m = -INFINITY, ubv = -INFINITY;
        for (int ht = 0; ht < HT; ++ht) {
            const int hq = 16 * ht + c;
            f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KSMAX; ++ks) {
                if (ks < KS) {
                    bf16x8_t q = (hq < a.H) ? *reinterpret_cast<const bf16x8_t*>(qtb + (int64_t)hq * a.n + 32 * ks + 8 * g)
                                            : bf16x8_t{};
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q, xf[ks], acc, 0, 0, 0);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int h = 16 * ht + 4 * g + i;
                if (h < a.H) {
                    m = fmaxf(m, acc[i]);
                    if (UB) {
                        const float4 hs = s_hs[h];
                        ubv = fmaxf(ubv, acc[i] + fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga)));
                    }
                }
            }
        }
        m = wave_max16(m);
        float s2 = 0.f;
#pragma unroll
        for (int ks = 0; ks < KSMAX; ++ks)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float v = (float)xf[ks][e];
                s2 = fmaf(v, v, s2);
            }
        s2 += __shfl_xor(s2, 16);
        s2 += __shfl_xor(s2, 32);
        if (valid) nu2m = fmaxf(nu2m, s2);
        if (UB) {
            ubv = wave_max16(ubv);
            if (valid) bmm = fmaxf(bmm, fmaf(amax, et, fmaf(nmax, ep, emax * ga)));
            if (g == 0 && valid) a.ub[(int64_t)b * a.A + row] = ubv;
        }
        if (g == 0 && valid) a.key[(int64_t)b * a.A + row] = m;
    }
    nu2m = wave_max_all(nu2m);
    if (UB) bmm = wave_max_all(bmm);
    if (lane == 0) {
        uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        atomicMax(sq + SQ_NU2MAX, __float_as_uint(nu2m));
        if (UB) atomicMax(sq + SQ_BMAX, __float_as_uint(bmm));
    }
}

template <int HT, int KS>
static void launch_fast(const ScoreArgs& a, dim3 grid, hipStream_t s) {
    if (a.ub)
        hipLaunchKernelGGL((score_kernel<HT, KS, true>), grid, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((score_kernel<HT, KS, false>), grid, dim3(256), 0, s, a);
}

template <int HT>
static bool dispatch_ks(const ScoreArgs& a, dim3 grid, hipStream_t s, int KS) {
    switch (KS) {
        case 1: launch_fast<HT, 1>(a, grid, s); return true;
        case 2: launch_fast<HT, 2>(a, grid, s); return true;
        case 3: launch_fast<HT, 3>(a, grid, s); return true;
        case 4: launch_fast<HT, 4>(a, grid, s); return true;
        case 5: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 5>(a, grid, s); return true; } return false;
        case 6: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 6>(a, grid, s); return true; } return false;
        case 7: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 7>(a, grid, s); return true; } return false;
        case 8: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 8>(a, grid, s); return true; } return false;
        default: return false;
    }
}

hipError_t launch_score(const ScoreArgs& a, hipStream_t s) {
    if (a.A <= 0) return hipSuccess;
    dim3 grid((unsigned)((a.A + SCORE_ROWS_PER_BLOCK - 1) / SCORE_ROWS_PER_BLOCK), a.B);
    const int KS = a.n / 32;
    const int HT = (a.H + 15) / 16;
    bool done = false;
    if (HT == 1) done = dispatch_ks<1>(a, grid, s, KS);
    else if (HT == 2) done = dispatch_ks<2>(a, grid, s, KS);
    else if (HT <= 4) done = dispatch_ks<4>(a, grid, s, KS);
    else if (HT <= 8) done = dispatch_ks<8>(a, grid, s, KS);
    if (!done) {
        if (a.ub)
            hipLaunchKernelGGL((score_generic_kernel<true>), grid, dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((score_generic_kernel<false>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace vkv
