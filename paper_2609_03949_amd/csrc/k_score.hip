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
// query digest qt[b,h,off+j] = RNE_bf16(w).  A block owns 32 basis rows and
// 16 heads; each thread runs two independent fp64 chains (two heads of one
// basis row).  The i axis is walked in chunks of 128 held in LDS as fp64 (P^T
// and the queries, converted once), and the next chunk is fetched into
// registers while the current one is consumed.  Block (0,0,b) also clears the
// step state of sequence b.
constexpr int QP_HEADS = 16;
constexpr int QP_ROWS = 32;
constexpr int QP_IC = 128;

__global__ __launch_bounds__(256) void qprep_project_kernel(QprepArgs a) {
    __shared__ __align__(16) double s_p[QP_IC][QP_ROWS];     // P^T chunk: [i][j]
    __shared__ __align__(16) double s_q[QP_IC][QP_HEADS];    // query chunk: [i][head]
    const int b = blockIdx.z;
    const int tid = threadIdx.x;
    if (blockIdx.x == 0 && blockIdx.y == 0) {
        if (tid < SQ_WORDS) a.seq[b * SQ_WORDS + tid] = (tid == SQ_KMIN) ? 0xFFFFFFFFu : 0u;
        for (int i = tid; i < 2 * HIST_BINS; i += 256) a.hist[(int64_t)b * 2 * HIST_BINS + i] = 0u;
    }
    if (a.r == 0 || !(a.mode & 2)) return;
    const int j0 = QP_ROWS * blockIdx.x;
    const int jn = min(QP_ROWS, a.r - j0);
    const int h0 = QP_HEADS * blockIdx.y;
    // chunk c: P rows j0.. (lane row = p & 31, piece p >> 5) and query rows
    // h0.. (head = p & 15, piece p >> 4), 16-byte pieces of 8 i each
    u16x8_t pv[2], qv;
    auto fetch = [&](int c) {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int p = tid + 256 * jj;
            const int row = p & 31, pc = p >> 5;
            pv[jj] = (row < jn) ? *reinterpret_cast<const u16x8_t*>(a.P + (int64_t)(j0 + row) * D_LAT + QP_IC * c + 8 * pc)
                                : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
        }
        const int hh = tid & 15, pc = tid >> 4;
        qv = (h0 + hh < a.H) ? *reinterpret_cast<const u16x8_t*>(a.q_lat + ((int64_t)b * a.H + h0 + hh) * D_LAT + QP_IC * c + 8 * pc)
                             : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    };
    auto park = [&]() {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int p = tid + 256 * jj;
            const int row = p & 31, pc = p >> 5;
#pragma unroll
            for (int e = 0; e < 8; ++e) s_p[8 * pc + e][row] = (double)bf16_to_f32(pv[jj][e]);
        }
        const int hh = tid & 15, pc = tid >> 4;
#pragma unroll
        for (int e = 0; e < 8; ++e) s_q[8 * pc + e][hh] = (double)bf16_to_f32(qv[e]);
    };
    const int jl = tid & 31, hg = tid >> 5;    // heads 2 hg, 2 hg + 1
    double acc0 = 0.0, acc1 = 0.0;
    fetch(0);
    park();
    __syncthreads();
    for (int c = 0; c < D_LAT / QP_IC; ++c) {
        const bool more = c + 1 < D_LAT / QP_IC;
        if (more) fetch(c + 1);
#pragma unroll 8
        for (int i = 0; i < QP_IC; ++i) {
            const double p = s_p[i][jl];
            const double2 q2 = *reinterpret_cast<const double2*>(&s_q[i][2 * hg]);
            acc0 = fma(p, q2.x, acc0);
            acc1 = fma(p, q2.y, acc1);
        }
        __syncthreads();
        if (more) {
            park();
            __syncthreads();
        }
    }
    if (jl >= jn) return;
    const int off = (a.mode & 1) ? D_ROPE : 0;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int h = h0 + 2 * hg + t;
        if (h >= a.H) continue;
        const int64_t bh = (int64_t)b * a.H + h;
        const double v = t ? acc1 : acc0;
        a.wproj[bh * a.r + j0 + jl] = v;
        a.qt[bh * a.n + off + j0 + jl] = f64_to_bf16_rne(v);
    }
}

// Stage 2 (16 heads per wave): certificate scalars of each head, each an fp32
// upper bound (Lemma (Index certificate) plus the bf16 rounding of the stored
// sketch; fixed fp64 evaluation order, the same as the oracle's):
//   a_h >= sqrt(q^T (I - P^T P) q),  n_h >= ||qd_h||,  e_h >= ||qd_h - P q||
// plus ||qt_h|| for the scorer's error bound, and the rope half of qt.  The
// wave first stages its heads' q_lat, projections and digests in LDS (all
// loads in flight); then lane 4*hl + t runs sum t of head hl sequentially:
// t=0 ||q||^2, t=1 ||w||^2, t=2 ||qd - w||^2, t=3 ||qd||^2.
constexpr int QF_HEADS = 16;
constexpr int QF_RMAX = 512;

__global__ __launch_bounds__(64) void qprep_finish_kernel(QprepArgs a) {
    __shared__ __align__(16) uint16_t s_ql[QF_HEADS][D_LAT];   // 16 KB
    __shared__ __align__(16) uint16_t s_qd[QF_HEADS][QF_RMAX]; // 16 KB
    __shared__ __align__(16) double s_w[QF_HEADS][QF_RMAX];    // 64 KB
    const int lane = threadIdx.x;
    const int hl = lane >> 2, t = lane & 3;
    const int64_t bh0 = (int64_t)blockIdx.x * QF_HEADS;
    const int64_t nbh = (int64_t)a.B * a.H;
    const int off = (a.mode & 1) ? D_ROPE : 0;
    const int rd = (a.mode & 2) ? a.r : 0;
    {
        // q_lat rows: 16 heads x 64 pieces; digests: 16 heads x rd/8 pieces
        constexpr int PER = QF_HEADS * (D_LAT / 8) / 64;
        u16x8_t v[PER];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int p = lane + 64 * j;
            const int h = p >> 6, pc = p & 63;
            v[j] = (bh0 + h < nbh) ? *reinterpret_cast<const u16x8_t*>(a.q_lat + (bh0 + h) * D_LAT + 8 * pc)
                                   : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int p = lane + 64 * j;
            *reinterpret_cast<u16x8_t*>(&s_ql[p >> 6][8 * (p & 63)]) = v[j];
        }
        // digests (16 B = 8 values) and projections (16 B = 2 values), 4 of
        // each per lane per round, loads in flight together
        const int r8 = rd / 8, r2 = rd / 2;
        for (int p0 = 0; p0 < QF_HEADS * r8; p0 += 256) {
            u16x8_t d[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int p = p0 + lane + 64 * j;
                const int h = p / max(r8, 1), pc = p % max(r8, 1);
                d[j] = (p < QF_HEADS * r8 && bh0 + h < nbh)
                           ? *reinterpret_cast<const u16x8_t*>(a.qt + (bh0 + h) * a.n + off + 8 * pc)
                           : u16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int p = p0 + lane + 64 * j;
                if (p < QF_HEADS * r8) *reinterpret_cast<u16x8_t*>(&s_qd[p / r8][8 * (p % r8)]) = d[j];
            }
        }
        for (int p0 = 0; p0 < QF_HEADS * r2; p0 += 512) {
            double2 wv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int p = p0 + lane + 64 * j;
                const int h = p / max(r2, 1), pc = p % max(r2, 1);
                wv[j] = (p < QF_HEADS * r2 && bh0 + h < nbh)
                            ? *reinterpret_cast<const double2*>(a.wproj + (bh0 + h) * a.r + 2 * pc)
                            : make_double2(0.0, 0.0);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int p = p0 + lane + 64 * j;
                if (p < QF_HEADS * r2) *reinterpret_cast<double2*>(&s_w[p / r2][2 * (p % r2)]) = wv[j];
            }
        }
    }
    __syncthreads();
    const int64_t bh = bh0 + hl;
    const bool have = bh < nbh;
    const int64_t bhc = have ? bh : 0;
    const int b = (int)(bhc / a.H);
    uint16_t* qt = a.qt + bhc * a.n;
    const double* w = &s_w[hl][0];
    // rope half of qt: 8 pieces of 16 B per head, 4 lanes per head
    if ((a.mode & 1) && have) {
        const u16x8_t* src = reinterpret_cast<const u16x8_t*>(a.q_rope + bhc * D_ROPE);
        u16x8_t* dst = reinterpret_cast<u16x8_t*>(qt);
        dst[t] = src[t];
        dst[t + 4] = src[t + 4];
    }
    double acc = 0.0;
    if (have) {
        if (t == 0) {
#pragma unroll 4
            for (int p = 0; p < D_LAT / 8; ++p) {
                const u16x8_t v = *reinterpret_cast<const u16x8_t*>(&s_ql[hl][8 * p]);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const double x = (double)bf16_to_f32(v[e]);
                    acc = fma(x, x, acc);
                }
            }
        } else if (t == 1) {
            for (int j0 = 0; j0 < rd; j0 += 8) {
                double wv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) wv[e] = w[j0 + e];
#pragma unroll
                for (int e = 0; e < 8; ++e) acc = fma(wv[e], wv[e], acc);
            }
        } else {
            for (int j0 = 0; j0 < rd; j0 += 8) {
                double wv[8];
                if (t == 2) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) wv[e] = w[j0 + e];
                }
                const u16x8_t dv = *reinterpret_cast<const u16x8_t*>(&s_qd[hl][j0]);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const double d = (double)bf16_to_f32(dv[e]);
                    if (t == 2) {
                        const double ee = d - wv[e];
                        acc = fma(ee, ee, acc);
                    } else {
                        acc = fma(d, d, acc);
                    }
                }
            }
        }
    }
    const int base = lane & ~3;
    const double Nq = __shfl(acc, base + 0), Nw = __shfl(acc, base + 1);
    const double Ne = __shfl(acc, base + 2), Nd = __shfl(acc, base + 3);
    // ||q_rope||^2 (an upper-bound input only; order irrelevant)
    double r2 = 0.0;
    if ((a.mode & 1) && have) {
        for (int i = t; i < D_ROPE; i += 4) {
            const double v = (double)bf16_to_f32(a.q_rope[bhc * D_ROPE + i]);
            r2 += v * v;
        }
    }
    r2 += __shfl_xor(r2, 1);
    r2 += __shfl_xor(r2, 2);
    float ah = 0.f, eh = 0.f, nh = 0.f, qn = 0.f;
    if (t == 0 && have) {
        const double G = CERT_G;
        const double Dm = G * (double)ru_sqrt_f32((double)rd * Nq);
        const double sw = (double)ru_sqrt_f32(Nw);
        const double X = ((Nq - Nw) + G * (Nq + Nw)) + (2.0 * Dm) * sw;
        ah = ru_sqrt_f32((X > 0.0 ? X : 0.0) * (1.0 + G));
        eh = ru_f32((double)ru_sqrt_f32(Ne) * (1.0 + G) + Dm);
        nh = ru_sqrt_f32(Nd * (1.0 + G));
        qn = ru_sqrt_f32((r2 + Nd) * (1.0 + 0x1p-30));
        reinterpret_cast<float4*>(a.hsc)[bhc] = make_float4(ah, nh, eh, qn);
    }
    // per-sequence maxima (all values are >= 0, so float order = bit order):
    // reduced over the wave's heads first when they all belong to one sequence
    const int64_t bl = min(bh0 + QF_HEADS, nbh) - 1;
    const bool one_seq = (bh0 / a.H) == (bl / a.H);
    if (one_seq) {
        for (int o = 4; o < 64; o <<= 1) {
            ah = fmaxf(ah, __shfl_xor(ah, o));
            eh = fmaxf(eh, __shfl_xor(eh, o));
            nh = fmaxf(nh, __shfl_xor(nh, o));
            qn = fmaxf(qn, __shfl_xor(qn, o));
        }
    }
    if (t == 0 && have && (!one_seq || hl == 0)) {
        uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        atomicMax(sq + SQ_QMAX, __float_as_uint(qn));
        atomicMax(sq + SQ_AMAX, __float_as_uint(ah));
        atomicMax(sq + SQ_NMAX, __float_as_uint(nh));
        atomicMax(sq + SQ_EMAX, __float_as_uint(eh));
    }
}

hipError_t launch_qprep(const QprepArgs& a, hipStream_t s) {
    int jt = (a.r > 0 && (a.mode & 2)) ? (a.r + QP_ROWS - 1) / QP_ROWS : 1;
    dim3 g1(jt, (a.H + QP_HEADS - 1) / QP_HEADS, a.B);
    hipLaunchKernelGGL(qprep_project_kernel, g1, dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(qprep_finish_kernel, dim3((a.B * a.H + QF_HEADS - 1) / QF_HEADS), dim3(64), 0, s, a);
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

// ||x||^2 of this lane's 8*KS index dims (exact bf16 products, fp32 sums)
template <int KS>
__device__ __forceinline__ float row_sq(const bf16x8_t (&xf)[KS]) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    float s2 = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bf16x2_t p = {xf[ks][2 * e], xf[ks][2 * e + 1]};
            s2 = __builtin_amdgcn_fdot2_f32_bf16(p, p, s2, false);
        }
    return s2;
}

// Epilogue of one 16-row tile for the lane holding row `row`: key~ (max over
// heads, already reduced) and the lane's partial of ||x||^2.  The scorer
// keeps the per-sequence extremes of key~ and of ||x||^2; the selection
// derives the certified band of every key from them.
struct TileOut {
    float kmax, kmin, nu2m, bmm;
};

__device__ __forceinline__ void tile_epilogue(const ScoreArgs& a, int b, int g, int64_t row, bool valid, float m,
                                              float s2, TileOut& t) {
    s2 += __shfl_xor(s2, 16);
    s2 += __shfl_xor(s2, 32);
    if (valid) {
        t.nu2m = fmaxf(t.nu2m, s2);
        t.kmax = fmaxf(t.kmax, m);
        t.kmin = fminf(t.kmin, m);
        if (g == 0) {
            const int64_t o = (int64_t)b * a.A + row;
            a.kt[o] = m;
            if (a.key) a.key[o] = m;
        }
    }
}

__device__ __forceinline__ void score_finish(const ScoreArgs& a, int b, int lane, TileOut t, bool ub) {
    t.nu2m = wave_max_all(t.nu2m);
    t.kmax = wave_max_all(t.kmax);
    t.kmin = -wave_max_all(-t.kmin);
    if (ub) t.bmm = wave_max_all(t.bmm);
    if (lane == 0) {
        uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        atomicMax(sq + SQ_NU2MAX, __float_as_uint(t.nu2m));
        atomicMin(sq + SQ_KMIN, key_to_ord(t.kmin));
        atomicMax(sq + SQ_KMAX, key_to_ord(t.kmax));
        if (ub) atomicMax(sq + SQ_BMAX, __float_as_uint(t.bmm));
    }
}

// HT head tiles of 16 and KS dim steps of 32 held in VGPRs (HT*KS <= 32).
// Head slots beyond H repeat a real head (h mod H), which leaves the maximum
// over heads unchanged and needs no masking in the loop.
template <int HT, int KS, bool UB>
__global__ __launch_bounds__(256, 2) void score_kernel(ScoreArgs a) {
    __shared__ float4 s_hs[UB ? 128 : 1];
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    if (UB) {
        for (int h = tid; h < 16 * HT; h += 256)
            s_hs[h] = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + (h % a.H)];
        __syncthreads();
    }
    const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * SCORE_TPW);
    if (r0 >= a.A) return;
    const int64_t rend = min(a.A, r0 + (int64_t)(16 * SCORE_TPW));
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;

    bf16x8_t qf[HT][KS];
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
        const int h = (16 * ht + c) % a.H;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            qf[ht][ks] = *reinterpret_cast<const bf16x8_t*>(qtb + (int64_t)h * a.n + 32 * ks + 8 * g);
    }
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    float amax = 0.f, nmax = 0.f, emax = 0.f;
    if (UB) {
        amax = __uint_as_float(sq[SQ_AMAX]);
        nmax = __uint_as_float(sq[SQ_NMAX]);
        emax = __uint_as_float(sq[SQ_EMAX]);
    }
    TileOut to{-INFINITY, INFINITY, 0.f, 0.f};
    const int64_t rlast = rend - 1;

    // PF tiles in flight ahead of the one on the matrix cores (one when the
    // bound is also evaluated, for registers); rows past the end are clamped
    // to the last row (loaded, never stored)
    constexpr int PF = UB ? 1 : 2;
    bf16x8_t xf[KS], x1[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const int64_t row0 = min(r0 + c, rlast), row1 = min(r0 + 16 + c, rlast);
        xf[ks] = *reinterpret_cast<const bf16x8_t*>(xb + row0 * a.xs + 32 * ks + 8 * g);
        if (PF == 2) x1[ks] = *reinterpret_cast<const bf16x8_t*>(xb + row1 * a.xs + 32 * ks + 8 * g);
    }
    for (int64_t t0 = r0; t0 < rend; t0 += 16) {
        const int64_t row = t0 + c;
        const bool valid = row < rend;
        bf16x8_t x2[KS];
        const int64_t nrow = min(row + 16 * PF, rlast);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            x2[ks] = *reinterpret_cast<const bf16x8_t*>(xb + nrow * a.xs + 32 * ks + 8 * g);
        float et = 0.f, ep = 0.f, ga = 0.f;
        if (UB) {
            const int64_t o = (int64_t)b * a.T + min(row, rlast);
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
        // keep the per-head bound scalars in LDS (re-read per tile) instead of
        // letting them be hoisted into 4 * 16 * HT registers
        if (UB) asm volatile("" ::: "memory");
        // acc[ht][i] = score of head slot 16*ht + 4*g + i for row t0 + c
        float m = -INFINITY;
        float ubv = -INFINITY;
#pragma unroll
        for (int ht = 0; ht < HT; ++ht)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                m = fmaxf(m, acc[ht][i]);
                if (UB) {
                    const float4 hs = s_hs[16 * ht + 4 * g + i];
                    ubv = fmaxf(ubv, acc[ht][i] + fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga)));
                }
            }
        m = wave_max16(m);
        tile_epilogue(a, b, g, row, valid, m, row_sq<KS>(xf), to);
        if (UB) {
            ubv = wave_max16(ubv);
            if (valid) to.bmm = fmaxf(to.bmm, fmaf(amax, et, fmaf(nmax, ep, emax * ga)));
            if (g == 0 && valid) a.ub[(int64_t)b * a.A + row] = ubv;
        }
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (PF == 2) {
                xf[ks] = x1[ks];
                x1[ks] = x2[ks];
            } else {
                xf[ks] = x2[ks];
            }
        }
    }
    score_finish(a, b, lane, to, UB);
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
    const int KS = a.n / 32;
    const int HT = (a.H + 15) / 16;
    if (UB) {
        for (int h = tid; h < 16 * HT; h += 256)
            s_hs[h] = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + (h % a.H)];
        __syncthreads();
    }
    const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * SCORE_TPW);
    if (r0 >= a.A) return;
    const int64_t rend = min(a.A, r0 + (int64_t)(16 * SCORE_TPW));
    const int64_t rlast = rend - 1;
    const uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    float amax = 0.f, nmax = 0.f, emax = 0.f;
    if (UB) {
        amax = __uint_as_float(sq[SQ_AMAX]);
        nmax = __uint_as_float(sq[SQ_NMAX]);
        emax = __uint_as_float(sq[SQ_EMAX]);
    }
    TileOut to{-INFINITY, INFINITY, 0.f, 0.f};
    for (int64_t t0 = r0; t0 < rend; t0 += 16) {
        const int64_t row = t0 + c;
        const bool valid = row < rend;
        const int64_t lrow = min(row, rlast);
        bf16x8_t xf[KSMAX];
#pragma unroll
        for (int ks = 0; ks < KSMAX; ++ks)
            xf[ks] = (ks < KS) ? *reinterpret_cast<const bf16x8_t*>(xb + lrow * a.xs + 32 * ks + 8 * g) : bf16x8_t{};
        float et = 0.f, ep = 0.f, ga = 0.f;
        if (UB) {
            const int64_t o = (int64_t)b * a.T + lrow;
            et = a.eta[o];
            ep = a.eps[o];
            ga = a.gam[o];
        }
        float m = -INFINITY, ubv = -INFINITY;
        for (int ht = 0; ht < HT; ++ht) {
            const int hq = (16 * ht + c) % a.H;
            f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KSMAX; ++ks) {
                if (ks < KS) {
                    const bf16x8_t q = *reinterpret_cast<const bf16x8_t*>(qtb + (int64_t)hq * a.n + 32 * ks + 8 * g);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(q, xf[ks], acc, 0, 0, 0);
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                m = fmaxf(m, acc[i]);
                if (UB) {
                    const float4 hs = s_hs[16 * ht + 4 * g + i];
                    ubv = fmaxf(ubv, acc[i] + fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga)));
                }
            }
        }
        m = wave_max16(m);
        tile_epilogue(a, b, g, row, valid, m, row_sq<KSMAX>(xf), to);
        if (UB) {
            ubv = wave_max16(ubv);
            if (valid) to.bmm = fmaxf(to.bmm, fmaf(amax, et, fmaf(nmax, ep, emax * ga)));
            if (g == 0 && valid) a.ub[(int64_t)b * a.A + row] = ubv;
        }
    }
    score_finish(a, b, lane, to, UB);
}

// ------------------------------------------------------ streaming scorer
//
// The form used when the bound is not evaluated.  A block owns a contiguous
// span of one sequence's archive; its four waves take alternate 16-row tiles
// of it (so the block streams one region of HBM), each through a private LDS
// ring of NST stages filled by direct global->LDS loads
// (global_load_lds_dwordx4, 1 KB per instruction, KS instructions per tile,
// non-temporal: the index is read once per step).  Slot S of row R in a stage
// holds the row's 16-byte chunk (S + R) mod N8, so the MFMA operand reads (16
// rows, one chunk each) hit distinct banks; the per-lane source offsets are
// the same for every tile, only the wave-uniform tile base moves.
//
// Per tile: the heads x rows contraction on the matrix cores (queries resident
// in VGPRs) overlaps the read-out of the next tile from the ring; the per-lane
// maximum over head slots and sum of squares are kept for four tiles, then a
// reduce-scatter over the four 16-lane groups (permlane swaps) leaves row c of
// tile t4+j in lane 16j+c.  Row keys collect in LDS and are written every
// RES_GROUPS groups: stores share vmcnt with the ring loads, so they are kept
// rare, and every wait counts ring loads only -- safe whether or not stores
// complete in order with loads (loads complete in order among themselves).
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt immediate");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// wait until at most `rem` tiles (KS loads each) younger than the current one
// are still in flight (rem is wave-uniform, 0 <= rem < NST)
template <int KS, int NST>
__device__ __forceinline__ void wait_tiles(int rem) {
    switch (rem) {
        case 0: wait_vmcnt<0>(); break;
        case 1: if (NST > 1) wait_vmcnt<(NST > 1 ? 1 : 0) * KS>(); break;
        case 2: if (NST > 2) wait_vmcnt<(NST > 2 ? 2 : 0) * KS>(); break;
        case 3: if (NST > 3) wait_vmcnt<(NST > 3 ? 3 : 0) * KS>(); break;
        case 4: if (NST > 4) wait_vmcnt<(NST > 4 ? 4 : 0) * KS>(); break;
        case 5: if (NST > 5) wait_vmcnt<(NST > 5 ? 5 : 0) * KS>(); break;
        case 6: if (NST > 6) wait_vmcnt<(NST > 6 ? 6 : 0) * KS>(); break;
        default: if (NST > 7) wait_vmcnt<(NST > 7 ? 7 : 0) * KS>(); break;
    }
}

constexpr int STAGE_BUDGET = 16384;   // bytes of tile ring per wave
constexpr int STREAM_WAVES = 4;       // waves per block
constexpr int RES_GROUPS = 16;        // 4-tile groups of row keys buffered per wave

template <int KS>
struct StreamGeom {
    static constexpr int N = 32 * KS;          // index dims per row
    static constexpr int N8 = N / 8;           // 16-byte slots per row
    static constexpr int STAGE = 16 * N * 2;   // one 16-row tile; KS loads of 1 KB
    static constexpr int NST = (STAGE_BUDGET / STAGE) > 8 ? 8 : ((STAGE_BUDGET / STAGE) < 2 ? 2 : (STAGE_BUDGET / STAGE));
    static constexpr int RES = RES_GROUPS * 64 * 4;
    static constexpr int WAVE = NST * STAGE + RES;
};

template <int HT, int KS>
__global__ __launch_bounds__(256, 2) void score_stream_kernel(ScoreArgs a, int tpw) {
    using Gm = StreamGeom<KS>;
    constexpr int N8 = Gm::N8, STAGE = Gm::STAGE, NST = Gm::NST;
    constexpr int TST = STREAM_WAVES;   // block tiles between consecutive tiles of a wave
    extern __shared__ __align__(16) uint8_t smem[];
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    uint8_t* wbase = smem + wave * Gm::WAVE;
    float* s_res = reinterpret_cast<float*>(wbase + NST * STAGE);
    // block span [bs0, bs1); this wave's tile j covers rows r0 + 16 TST j + [0, 16)
    const int64_t bs0 = (int64_t)blockIdx.x * STREAM_WAVES * 16 * tpw;
    if (bs0 >= a.A) return;
    const int64_t bs1 = min(a.A, bs0 + (int64_t)STREAM_WAVES * 16 * tpw);
    const int64_t nbt = (bs1 - bs0 + 15) / 16;
    if (wave >= nbt) return;
    const int ntl = (int)((nbt - 1 - wave) / TST + 1);
    const int64_t r0 = bs0 + 16 * wave;

    bf16x8_t qf[HT][KS];
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
        const int h = (16 * ht + c) % a.H;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            qf[ht][ks] = *reinterpret_cast<const bf16x8_t*>(qtb + (int64_t)h * a.n + 32 * ks + 8 * g);
    }
    wait_vmcnt<0>();   // query fragments resident before the ring's count starts

    const uint32_t rowb = (uint32_t)(a.xs * 2);   // row stride in bytes
    const uint8_t* span = reinterpret_cast<const uint8_t*>(a.x + (int64_t)b * a.xbs + r0 * a.xs);
    uint32_t voff[KS];
    int vrow[KS];
#pragma unroll
    for (int j = 0; j < KS; ++j) {
        const int q = 64 * j + lane;
        const int R = q / N8, S = q % N8;
        vrow[j] = R;
        voff[j] = (uint32_t)R * rowb + 16u * (uint32_t)((S + R) % N8);
    }
    auto issue = [&](int t, int stage) {
        const uint8_t* tb = span + (int64_t)t * (TST * 16) * rowb;
        const int nv = (int)min((int64_t)16, bs1 - (r0 + (int64_t)(TST * 16) * t));   // rows of this tile
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            uint32_t o = voff[j];
            if (nv < 16 && vrow[j] >= nv) o -= (uint32_t)(vrow[j] - (nv - 1)) * rowb;   // past-the-end rows re-read the last
            __builtin_amdgcn_global_load_lds((gbl_void_t*)(tb + o), (lds_void_t*)(wbase + stage * STAGE + 1024 * j),
                                             16, 0, 2 /* nt */);
        }
    };
    for (int t = 0; t < NST && t < ntl; ++t) issue(t, t);

    // operand fragments of tile t from its ring stage
    auto read_tile = [&](int t, bf16x8_t (&x)[KS]) {
        const uint8_t* st = wbase + (t % NST) * STAGE;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int S = (4 * ks + g - c + 16 * N8) % N8;
            x[ks] = *reinterpret_cast<const bf16x8_t*>(st + c * (2 * Gm::N) + 16 * S);
        }
    };
    bf16x8_t xf[KS];
    wait_tiles<KS, NST>(min(NST - 1, ntl - 1));
    read_tile(0, xf);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // stage read out before it is refilled
    if (NST < ntl) issue(NST, 0);

    TileOut to{-INFINITY, INFINITY, 0.f, 0.f};
    float* kto = a.kt + (int64_t)b * a.A;
    // the row held by this lane in 4-tile group q of the wave
    auto group_row = [&](int q) { return r0 + (int64_t)(TST * 16) * (4 * q + g) + c; };
    auto flush = [&](int q0, int nq) {
        for (int q = 0; q < nq; ++q) {
            const int64_t row = group_row(q0 + q);
            const float k = s_res[64 * q + lane];
            if (row < bs1) {
                kto[row] = k;
                if (a.key) a.key[(int64_t)b * a.A + row] = k;
            }
        }
    };
    // Per-lane partials of the four tiles of a group: pm = max over this
    // lane's head slots, ps = sum of squares over this lane's dims.
    float pm0 = -INFINITY, pm1 = -INFINITY, pm2 = -INFINITY, pm3 = -INFINITY;
    float ps0 = 0.f, ps1 = 0.f, ps2 = 0.f, ps3 = 0.f;

    for (int t = 0; t < ntl; ++t) {
        // the matrix-core contraction of tile t (operands in xf) while tile
        // t+1 is read out of the ring, then the per-lane partials of tile t
        f32x4_t acc[HT];
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) acc[ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
                acc[ht] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[ht][ks], xf[ks], acc[ht], 0, 0, 0);
        const float ps = row_sq<KS>(xf);
        bf16x8_t xn[KS];
        const bool more = t + 1 < ntl;
        if (more) {
            wait_tiles<KS, NST>(min(NST - 1, ntl - 2 - t));
            read_tile(t + 1, xn);
        }
        // acc[ht][i] = score of head slot 16*ht + 4*g + i for row c of tile t
        float pm = -INFINITY;
#pragma unroll
        for (int ht = 0; ht < HT; ++ht)
#pragma unroll
            for (int i = 0; i < 4; ++i) pm = fmaxf(pm, acc[ht][i]);
        const int j = t & 3;
        if (j == 0) {
            pm1 = pm2 = pm3 = -INFINITY;
            ps1 = ps2 = ps3 = 0.f;
        }
        pm0 = (j == 0) ? pm : pm0;
        pm1 = (j == 1) ? pm : pm1;
        pm2 = (j == 2) ? pm : pm2;
        pm3 = (j == 3) ? pm : pm3;
        ps0 = (j == 0) ? ps : ps0;
        ps1 = (j == 1) ? ps : ps1;
        ps2 = (j == 2) ? ps : ps2;
        ps3 = (j == 3) ? ps : ps3;
        if (more) {
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // stage read out before it is refilled
            if (t + 1 + NST < ntl) issue(t + 1 + NST, (t + 1) % NST);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) xf[ks] = xn[ks];
        }
        if (j != 3 && more) continue;
        // reduce-scatter over the four 16-lane groups: afterwards lane 16j + c
        // holds the maximum and the sum of squares of row c of tile 4q + j
        const int q = t >> 2;
        float m, s2;
        {
            auto sw32 = [](float x, float y) {
                const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
                return f32x2_t{__uint_as_float(r[0]), __uint_as_float(r[1])};
            };
            auto sw16 = [](float x, float y) {
                const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
                return f32x2_t{__uint_as_float(r[0]), __uint_as_float(r[1])};
            };
            f32x2_t u = sw32(pm0, pm2), v = sw32(pm1, pm3);
            const float m02 = fmaxf(u[0], u[1]), m13 = fmaxf(v[0], v[1]);
            u = sw16(m02, m13);
            m = fmaxf(u[0], u[1]);
            u = sw32(ps0, ps2);
            v = sw32(ps1, ps3);
            const float s02 = u[0] + u[1], s13 = v[0] + v[1];
            u = sw16(s02, s13);
            s2 = u[0] + u[1];
        }
        if (group_row(q) < bs1) {
            to.nu2m = fmaxf(to.nu2m, s2);
            to.kmax = fmaxf(to.kmax, m);
            to.kmin = fminf(to.kmin, m);
        }
        const int qb = q % RES_GROUPS;
        s_res[64 * qb + lane] = m;
        if (qb == RES_GROUPS - 1 || !more) flush(q - qb, qb + 1);
    }
    score_finish(a, b, lane, to, false);
}

// tiles per wave: enough waves for two blocks per CU, spans of 8..512 tiles
static int stream_tpw(const ScoreArgs& a) {
    const int64_t tiles = (int64_t)a.B * ((a.A + 15) / 16);
    const int64_t waves = 2LL * 256 * STREAM_WAVES;
    int64_t tpw = (tiles + waves - 1) / waves;
    tpw = tpw < 8 ? 8 : (tpw > 512 ? 512 : tpw);
    return (int)tpw;
}

template <int HT, int KS>
static void launch_fast(const ScoreArgs& a, hipStream_t s) {
    if (a.ub) {
        dim3 grid((unsigned)((a.A + SCORE_ROWS_PER_BLOCK - 1) / SCORE_ROWS_PER_BLOCK), a.B);
        hipLaunchKernelGGL((score_kernel<HT, KS, true>), grid, dim3(256), 0, s, a);
    } else {
        const int tpw = stream_tpw(a);
        const int64_t rows_per_block = (int64_t)STREAM_WAVES * 16 * tpw;   // block span
        dim3 grid((unsigned)((a.A + rows_per_block - 1) / rows_per_block), a.B);
        const size_t sm = STREAM_WAVES * (size_t)StreamGeom<KS>::WAVE;
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&score_stream_kernel<HT, KS>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
        hipLaunchKernelGGL((score_stream_kernel<HT, KS>), grid, dim3(256), sm, s, a, tpw);
    }
}

template <int HT>
static bool dispatch_ks(const ScoreArgs& a, hipStream_t s, int KS) {
    switch (KS) {
        case 1: launch_fast<HT, 1>(a, s); return true;
        case 2: launch_fast<HT, 2>(a, s); return true;
        case 3: launch_fast<HT, 3>(a, s); return true;
        case 4: launch_fast<HT, 4>(a, s); return true;
        case 5: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 5>(a, s); return true; } return false;
        case 6: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 6>(a, s); return true; } return false;
        case 7: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 7>(a, s); return true; } return false;
        case 8: if (HT <= 4) { launch_fast<(HT <= 4 ? HT : 4), 8>(a, s); return true; } return false;
        default: return false;
    }
}

hipError_t launch_score(const ScoreArgs& a, hipStream_t s) {
    if (a.A <= 0) return hipSuccess;
    const int KS = a.n / 32;
    const int HT = (a.H + 15) / 16;
    bool done = false;
    if (HT == 1) done = dispatch_ks<1>(a, s, KS);
    else if (HT == 2) done = dispatch_ks<2>(a, s, KS);
    else if (HT <= 4) done = dispatch_ks<4>(a, s, KS);
    else if (HT <= 8) done = dispatch_ks<8>(a, s, KS);
    if (!done) {
        dim3 grid((unsigned)((a.A + SCORE_ROWS_PER_BLOCK - 1) / SCORE_ROWS_PER_BLOCK), a.B);
        if (a.ub)
            hipLaunchKernelGGL((score_generic_kernel<true>), grid, dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((score_generic_kernel<false>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace vkv
