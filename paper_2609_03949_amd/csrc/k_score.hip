// k_score.hip -- query preparation and the streaming index scorer (gfx950).
//
// Index score of archived row u for head h (Eq. (trigger), the exact-branch
// and sketch terms; Sec. 4.2):
//     s^_h(u) = qt_h . x_u,   qt_h = [q_rope_h ; RNE_bf16(P q_lat_h)],   x_u = index row
// key_u = max_h s^_h(u).  The scorer streams only the narrow index slice
// (64 + r bf16 per row) from HBM and runs the heads x rows contraction on the
// matrix cores (v_mfma_f32_16x16x32_bf16): A = qt (16 heads x 32 dims per
// fragment, resident in VGPRs for the whole wave), B = 16 index rows x 32 dims
// read from an LDS ring that direct global->LDS loads fill.  The heads maximum
// is taken in registers (4 heads per lane per tile, then cross-lane steps).
#include <type_traits>

#include "vkv_internal.h"

namespace vkv {

// ----------------------------------------------------------- query prep

// Query prep, one kernel: w[b,h,j] = sum_i P[j,i] q_lat[b,h,i] (fp64, i
// ascending, one rounding per term), the query digest qt[b,h,off+j] =
// RNE_bf16(w) and the rope half of qt, Nq[b,h] = ||q_lat||^2 (fp64, i
// ascending), and the head's certificate scalars.  A block owns 16 heads of
// one sequence.  The projection runs on the fp64 matrix cores: one
// v_mfma_f64_16x16x4f64 per 4 consecutive i adds the 4 products to the
// accumulator one after another in k order, each with a single rounding (the
// same bits as the sequential FMA chain; the GPU tests compare the digest with
// the fp64 oracle on inputs spread over 2^60, where other summation orders
// give other bits), so a chain of 128 of them, i ascending, is the fp64
// definition.  Wave w computes basis tile w
// (16 heads x 16 basis rows) of the current chunk of 128 basis rows; one more
// wave runs the Nq chains on the vector unit meanwhile (a chain of 512 fp64
// steps on its own, so it overlaps the matrix chains instead of lengthening
// one of them).  The query rows and the chunk of P are staged as bf16 by
// direct loads into rows padded to QP_ROW bytes, so the operand reads (16
// rows, one 16-bit element each) fall into distinct banks; they are widened
// in registers.  The rope half of qt is loaded at the start and written at
// the end.  Block (0,b) also clears the step state of sequence b.
constexpr int QP_ROW = 1040;          // LDS bytes per staged row of 512 bf16
constexpr int QP_CHUNK_ROWS = 128;    // basis rows staged at a time: one 16-row tile per wave
constexpr int QP_MAX_WAVES = QP_CHUNK_ROWS / 16;
constexpr int QP_WSTRIDE = QP_CHUNK_ROWS + 1;   // doubles per head of the staged w values (heads in distinct banks)
constexpr int QP_TAIL_BATCH = 16;              // staged values per LDS batch of the tail sums

// waves with a basis tile (0 without a digest); one more wave takes the Nq chains
__host__ __device__ inline int qp_tile_waves(int r) {
    const int t = r / 16;
    return t < 0 ? 0 : (t > QP_MAX_WAVES ? QP_MAX_WAVES : t);
}

__global__ __launch_bounds__(64 * (QP_MAX_WAVES + 1)) void qprep_project_kernel(QprepArgs a) {
    __shared__ __align__(16) uint8_t s_q[16 * QP_ROW];              // the block's 16 query rows, [h][i]
    __shared__ __align__(16) uint8_t s_p[QP_CHUNK_ROWS * QP_ROW];   // a chunk of P rows, then its w values
    __shared__ double s_nq[16];
    const int b = blockIdx.y, hb0 = 16 * blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nw = blockDim.x >> 6;
    if (blockIdx.x == 0) {
        if (tid < SQ_WORDS) a.seq[b * SQ_WORDS + tid] = (tid == SQ_KMIN) ? 0xFFFFFFFFu : 0u;
    }
    const int r = (a.mode & 2) ? a.r : 0;
    const int off = (a.mode & 1) ? D_ROPE : 0;
    const int nq_wave = qp_tile_waves(r);
    // wave 0, lane 4 hl + t: rope pieces t and t + 4 of head hb0 + hl (loaded now, stored at the end)
    const int hl = lane >> 2, t = lane & 3;
    const int h = hb0 + hl;
    const bool have = h < a.H;
    const int64_t bhc = (int64_t)b * a.H + (have ? h : 0);
    u16x8_t rope0 = u16x8_t{}, rope1 = u16x8_t{};
    if (wave == 0 && (a.mode & 1) && have) {
        const u16x8_t* src = reinterpret_cast<const u16x8_t*>(a.q_rope + bhc * D_ROPE);
        rope0 = src[t];
        rope1 = src[t + 4];
    }
    typedef __attribute__((address_space(3))) void lds_t;
    typedef __attribute__((address_space(1))) void gbl_t;
    // query rows: one 1 KB direct load per row; rows past H are zero
    for (int row = wave; row < 16; row += nw) {
        const int h = hb0 + row;
        if (h < a.H)
            __builtin_amdgcn_global_load_lds((gbl_t*)(a.q_lat + ((int64_t)b * a.H + h) * D_LAT + 8 * lane),
                                             (lds_t*)(s_q + row * QP_ROW), 16, 0, 0);
        else
            *reinterpret_cast<u32x4_t*>(s_q + row * QP_ROW + 16 * lane) = u32x4_t{0u, 0u, 0u, 0u};
    }
    // operand rows of this lane: A = query row (lane mod 16), B = basis row
    // 16 wave + (lane mod 16) of the chunk; element k = lane / 16 of each step
    const uint16_t* qa = reinterpret_cast<const uint16_t*>(s_q + (lane & 15) * QP_ROW) + (lane >> 4);
    const uint16_t* pb = reinterpret_cast<const uint16_t*>(s_p + (16 * wave + (lane & 15)) * QP_ROW) + (lane >> 4);
    const uint16_t* qn = reinterpret_cast<const uint16_t*>(s_q + (lane & 15) * QP_ROW);   // Nq: head lane mod 16
    double* s_w = reinterpret_cast<double*>(s_p);   // [16][QP_WSTRIDE] w, then RNE(w), once the chunk is used
    double* s_d = s_w + 16 * QP_WSTRIDE;
    double anq = 0.0;
    // tail sums of lane 4 hl + t of wave 0, j ascending over all chunks:
    // t=1 ||w||^2, t=2 ||qd - w||^2, t=3 ||qd||^2 (t=0 takes Nq at the end)
    double tsum = 0.0;
    const int nchunk = (r + QP_CHUNK_ROWS - 1) / QP_CHUNK_ROWS;
    for (int ch = 0; ch < (nchunk > 0 ? nchunk : 1); ++ch) {
        const int j0 = ch * QP_CHUNK_ROWS;
        const int nj = min(QP_CHUNK_ROWS, r - j0);   // basis rows of this chunk (<= 0 without a digest)
        for (int row = wave; row < nj; row += nw)
            __builtin_amdgcn_global_load_lds((gbl_t*)(a.P + (int64_t)(j0 + row) * D_LAT + 8 * lane),
                                             (lds_t*)(s_p + row * QP_ROW), 16, 0, 0);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        const bool tile = wave < nq_wave && 16 * wave < nj;
        const bool nq = ch == 0 && wave == nq_wave;
        f64x4_t acc = f64x4_t{0.0, 0.0, 0.0, 0.0};
        if (tile) {
            acc = mfma_f64_rowdot512<false>(qa, pb, qn, anq);
        } else if (nq) {
            // Nq of head lane mod 16, i ascending (eight elements per LDS read)
            const u16x8_t* qv = reinterpret_cast<const u16x8_t*>(qn);
#pragma unroll 4
            for (int i8 = 0; i8 < D_LAT / 8; ++i8) {
                const u16x8_t v = qv[i8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const double x = bf16_bits_f64(v[e]);
                    anq = fma(x, x, anq);
                }
            }
        }
        __syncthreads();   // the chunk's rows are read out; its LDS takes the w values
        if (tile) {
            // acc[i] = w of head 4 i + lane / 16, basis row j0 + 16 wave + lane mod 16
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int hh = 4 * i + (lane >> 4), jl = 16 * wave + (lane & 15);
                const double v = acc[i];
                const uint16_t d = f64_to_bf16_rne(v);
                s_w[hh * QP_WSTRIDE + jl] = v;
                s_d[hh * QP_WSTRIDE + jl] = (double)bf16_to_f32(d);
                if (hb0 + hh < a.H) a.qt[((int64_t)b * a.H + hb0 + hh) * a.n + off + j0 + jl] = d;
            }
        }
        if (nq && lane < 16) s_nq[lane] = anq;
        __syncthreads();
        if (wave == 0 && t > 0 && nj > 0) {
            const double* w = s_w + hl * QP_WSTRIDE;
            const double* dq = s_d + hl * QP_WSTRIDE;
            // the three sums share one loop: x = w, qd - w or qd by lane (qd - 0
            // is qd exactly), chosen by selects.  The staged values are read in
            // batches, all reads of a batch in flight before its chain starts.
            for (int j0 = 0; j0 < nj; j0 += QP_TAIL_BATCH) {
                double wv[QP_TAIL_BATCH], dv[QP_TAIL_BATCH];
#pragma unroll
                for (int e = 0; e < QP_TAIL_BATCH; ++e) {
                    const int j = min(j0 + e, nj - 1);
                    wv[e] = w[j];
                    dv[e] = dq[j];
                }
#pragma unroll
                for (int e = 0; e < QP_TAIL_BATCH; ++e) asm volatile("" : "+v"(wv[e]), "+v"(dv[e]));
#pragma unroll
                for (int e = 0; e < QP_TAIL_BATCH; ++e) {
                    const double sub = (t == 2) ? wv[e] : 0.0;
                    const double x = (j0 + e >= nj) ? 0.0 : ((t == 1) ? wv[e] : dv[e] - sub);
                    tsum = fma(x, x, tsum);   // + 0 past the end: tsum >= 0 is unchanged
                }
            }
        }
        __syncthreads();   // before the next chunk's rows overwrite the w values
    }
    if (wave != 0) return;
    // certificate scalars of each head (fp32 upper bounds; Lemma (Index
    // certificate) plus the bf16 rounding of the stored sketch; fixed fp64
    // evaluation order, the same as the oracle's):
    //   a_h >= sqrt(q^T (I - P^T P) q),  n_h >= ||qd_h||,  e_h >= ||qd_h - P q||
    // plus ||qt_h|| for the scorer's error bound.
    // rope half of qt (8 pieces of 16 B per head, 4 lanes per head) and
    // ||q_rope||^2 (an upper-bound input only; order irrelevant)
    double r2 = 0.0;
    if ((a.mode & 1) && have) {
        u16x8_t* dst = reinterpret_cast<u16x8_t*>(a.qt + bhc * a.n);
        const u16x8_t v0 = rope0, v1 = rope1;
        dst[t] = v0;
        dst[t + 4] = v1;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const double x0 = (double)bf16_to_f32(v0[e]), x1 = (double)bf16_to_f32(v1[e]);
            r2 += x0 * x0 + x1 * x1;
        }
    }
    r2 += __shfl_xor(r2, 1);
    r2 += __shfl_xor(r2, 2);
    const double acc_t = t == 0 ? s_nq[hl] : tsum;
    const int base = lane & ~3;
    const double Nq = __shfl(acc_t, base + 0), Nw = __shfl(acc_t, base + 1);
    const double Ne = __shfl(acc_t, base + 2), Nd = __shfl(acc_t, base + 3);
    if (t == 0 && have) {
        const double G = CERT_G;
        const double Dm = G * (double)ru_sqrt_f32((double)r * Nq);
        const double sw = (double)ru_sqrt_f32(Nw);
        const double X = ((Nq - Nw) + G * (Nq + Nw)) + (2.0 * Dm) * sw;
        const float ah = ru_sqrt_f32((X > 0.0 ? X : 0.0) * (1.0 + G));
        const float eh = ru_f32((double)ru_sqrt_f32(Ne) * (1.0 + G) + Dm);
        const float nh = ru_sqrt_f32(Nd * (1.0 + G));
        const float qn2 = ru_sqrt_f32((r2 + Nd) * (1.0 + 0x1p-30));
        reinterpret_cast<float4*>(a.hsc)[bhc] = make_float4(ah, nh, eh, qn2);
    }
}

// Per-sequence maxima of the head scalars (a, n, e, ||qt||), for the error
// bounds of the scorer and the selection: computed by wave 0 of the first
// block of each sequence in the scorer launch (the query prep of the step has
// finished and cleared the words); all values are >= 0.
// a'_h of the bound: the smallest float >= cert_mult * a_h (exact product in fp64)
__device__ __forceinline__ float scaled_a(float cm, float ah) { return ru_f32((double)cm * (double)ah); }

__device__ __forceinline__ void store_head_maxima(const ScoreArgs& a, int b, int lane) {
    float4 m = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int h = lane; h < a.H; h += 64) {
        const float4 v = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + h];
        const float ax = a.ub ? scaled_a(a.cert_mult, v.x) : v.x;
        m = make_float4(fmaxf(m.x, ax), fmaxf(m.y, v.y), fmaxf(m.z, v.z), fmaxf(m.w, v.w));
    }
    for (int o = 32; o > 0; o >>= 1) {
        m.x = fmaxf(m.x, __shfl_xor(m.x, o));
        m.y = fmaxf(m.y, __shfl_xor(m.y, o));
        m.z = fmaxf(m.z, __shfl_xor(m.z, o));
        m.w = fmaxf(m.w, __shfl_xor(m.w, o));
    }
    if (lane == 0) {
        uint32_t* sq = a.seq + (int64_t)b * SQ_WORDS;
        sq[SQ_AMAX] = __float_as_uint(m.x);
        sq[SQ_NMAX] = __float_as_uint(m.y);
        sq[SQ_EMAX] = __float_as_uint(m.z);
        sq[SQ_QMAX] = __float_as_uint(m.w);
        // the multiplier the bound below used (an impossible float pattern without one)
        sq[SQ_CMULT] = a.ub ? __float_as_uint(a.cert_mult) : 0xFFFFFFFFu;
        sq[SQ_TRGM] = (a.ub && a.thr) ? 1u : 0u;
    }
}

// maxima of (a, n, e) over the head scalars staged in LDS
__device__ __forceinline__ void staged_head_maxima(const float4* s_hs, int n, float& amax, float& nmax, float& emax) {
    amax = nmax = emax = 0.f;
    for (int i = 0; i < n; ++i) {
        const float4 v = s_hs[i];
        amax = fmaxf(amax, v.x);
        nmax = fmaxf(nmax, v.y);
        emax = fmaxf(emax, v.z);
    }
}

hipError_t launch_qprep(const QprepArgs& a, hipStream_t s) {
    const int r = (a.mode & 2) ? a.r : 0;
    dim3 g1((a.H + 15) / 16, a.B);
    hipLaunchKernelGGL(qprep_project_kernel, g1, dim3(64 * (qp_tile_waves(r) + 1)), 0, s, a);
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

// __shfl_xor whose lane arithmetic the compiler cannot share between call
// sites: shared lane addresses would stay live across the scan loops and
// crowd out the registers the loops need
__device__ __forceinline__ float shfl_xor_local(float v, int o) {
    int ln = __lane_id();
    asm volatile("" : "+v"(ln));
    return __int_as_float(__builtin_amdgcn_ds_bpermute((ln ^ o) << 2, __float_as_int(v)));
}
__device__ __forceinline__ float shfl_local(float v, int src) {
    int ln = src;
    asm volatile("" : "+v"(ln));
    return __int_as_float(__builtin_amdgcn_ds_bpermute(ln << 2, __float_as_int(v)));
}

__device__ __forceinline__ float wave_max_all(float m) {
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, shfl_xor_local(m, o));
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

// Any head count / width within the limits: heads and dims in runtime loops,
// query fragments re-read from the (cache-resident) qt buffer per tile.
template <bool UB>
__global__ __launch_bounds__(256, 2) void score_generic_kernel(ScoreArgs a) {
    constexpr int KSMAX = D_ROW / 32;
    __shared__ float4 s_hs[UB ? 128 : 1];
    __shared__ float s_thr[UB ? 128 : 1];   // -s*_h (trigger margins) or 0
    const int b = blockIdx.y;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, c = lane & 15;
    const int KS = a.n / 32;
    const int HT = (a.H + 15) / 16;
    if (UB) {
        for (int h = tid; h < 16 * HT; h += 256) {
            const float4 v = reinterpret_cast<const float4*>(a.hsc)[(int64_t)b * a.H + (h % a.H)];
            s_hs[h] = make_float4(scaled_a(a.cert_mult, v.x), v.y, v.z, v.w);
            s_thr[h] = a.thr ? -(float)a.thr[(int64_t)b * a.H + (h % a.H)] : 0.f;
        }
        __syncthreads();
    }
    if (blockIdx.x == 0 && threadIdx.x < 64) store_head_maxima(a, b, threadIdx.x);
    const int64_t r0 = ((int64_t)blockIdx.x * 4 + wave) * (16 * SCORE_TPW);
    if (r0 >= a.A) return;
    const int64_t rend = min(a.A, r0 + (int64_t)(16 * SCORE_TPW));
    const int64_t rlast = rend - 1;
    const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
    const uint16_t* xb = a.x + (int64_t)b * a.xbs;
    float amax = 0.f, nmax = 0.f, emax = 0.f, tabs = 0.f;
    if (UB) {
        staged_head_maxima(s_hs, 16 * HT, amax, nmax, emax);
        for (int i = 0; i < 16 * HT; ++i) tabs = fmaxf(tabs, fabsf(s_thr[i]));
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
                    ubv = fmaxf(ubv, (acc[i] + fmaf(hs.x, et, fmaf(hs.y, ep, hs.z * ga))) + s_thr[16 * ht + 4 * g + i]);
                }
            }
        }
        m = wave_max16(m);
        tile_epilogue(a, b, g, row, valid, m, row_sq<KSMAX>(xf), to);
        if (UB) {
            ubv = wave_max16(ubv);
            if (valid) to.bmm = fmaxf(to.bmm, fmaf(amax, et, fmaf(nmax, ep, emax * ga)) + tabs);
            if (g == 0 && valid) a.ub[(int64_t)b * a.A + row] = ubv;
        }
    }
    score_finish(a, b, lane, to, UB);
}

// ------------------------------------------------------ streaming scorer
//
// A block owns a contiguous
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
// in VGPRs), then the read-out of the next tile from the ring and the refill
// of its stage; the per-lane maximum over head slots and sum of squares are
// kept for four tiles, then a reduce-scatter over the four 16-lane groups
// (permlane swaps) leaves row c of tile 4q+j in lane 16j+c.  The keys of the
// whole span collect in LDS and are stored after the last tile: key stores
// mixed into the stream of index reads cost more than a tenth of the scan's
// time on MI355X, one burst at the end costs a few microseconds.  The bulk of
// the span runs in a loop of four tiles with fixed stages and fixed wait
// counts; the last tiles, whose look-ahead loads would run past the span,
// take a loop with run-time counts.  Every wait counts the ring loads issued
// after the awaited tile (loads complete in order among themselves).
//
// With the admission bound (UB): the tile's row scalars eta, eps, gam come
// with the tile, one more direct load of 64 dwords per tile (lanes 16j + c:
// scalar j of row c; the fourth group repeats eta), so lane 16j + c reads its
// own dword of the stage, which is the B operand of a v_mfma_f32_16x16x4_f32
// with A = the head scalars (lane 16j + c: a, n, e, 0 of head slot c): one
// such step per head tile adds B_h(u) = a_h eta_u + n_h eps_u + e_h gam_u to
// the finished scores, UB_u = max_h (s^_h(u) + B_h(u)).  Four fp32 products
// and sums of non-negative terms (all scalars are >= 0) on top of the score:
// the selection's band for UB covers that error.  With trigger thresholds
// s*_h (the kept-tier step: the tier's maximum logit is known before the
// scan), the fourth group carries -s*_h against a row scalar of 1, so the same
// step yields the trigger margin max_h (s^_h(u) + B_h(u) - s*_h) (Eq. (trigger)
// per head, fused into the scan); the band then also covers |s*_h|.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void gbl_void_t;

// the row scalar of head slot g = 3 when the bound carries the trigger threshold
__device__ float k_one = 1.0f;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt immediate");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}

// wait until at most `rem` tiles (LPT loads each) younger than the current one
// are still in flight (rem is wave-uniform, 0 <= rem < NST)
template <int LPT, int NST>
__device__ __forceinline__ void wait_tiles(int rem) {
    switch (rem) {
        case 0: wait_vmcnt<0>(); break;
        case 1: if (NST > 1) wait_vmcnt<(NST > 1 ? 1 : 0) * LPT>(); break;
        case 2: if (NST > 2) wait_vmcnt<(NST > 2 ? 2 : 0) * LPT>(); break;
        case 3: if (NST > 3) wait_vmcnt<(NST > 3 ? 3 : 0) * LPT>(); break;
        case 4: if (NST > 4) wait_vmcnt<(NST > 4 ? 4 : 0) * LPT>(); break;
        case 5: if (NST > 5) wait_vmcnt<(NST > 5 ? 5 : 0) * LPT>(); break;
        case 6: if (NST > 6) wait_vmcnt<(NST > 6 ? 6 : 0) * LPT>(); break;
        default: if (NST > 7) wait_vmcnt<(NST > 7 ? 7 : 0) * LPT>(); break;
    }
}

constexpr int STAGE_BUDGET = 12288;   // bytes of tile ring per wave
constexpr int STREAM_WAVES = 4;       // waves per block
constexpr int STREAM_TPW_MAX = 128;   // tiles per wave, bounded by the LDS key buffer
constexpr int WAVE_LDS = 20480;       // LDS per wave for two blocks of four waves per CU (160 KB)

template <int KS, bool UB>
struct StreamGeom {
    static constexpr int N = 32 * KS;          // index dims per row
    static constexpr int N8 = N / 8;           // 16-byte slots per row
    static constexpr int STAGE = 16 * N * 2;   // one 16-row tile; KS loads of 1 KB
    // ring depth 4 or 2, so that a run of four tiles maps to fixed stages
    static constexpr int NST = STAGE_BUDGET / STAGE >= 4 ? 4 : 2;
    static constexpr int RUN = 4;                       // tiles per fixed-stage run
    static constexpr int LPT = KS + (UB ? 1 : 0);       // ring loads per tile
    static constexpr int RV = UB ? 256 : 0;             // per stage: the tile's row scalars
    // the span's keys (fp32) for KT tiles: STREAM_TPW_MAX, or fewer where the
    // ring is so wide that two blocks per CU would not fit otherwise (rows of
    // 224 and 256 dims); with UB the first half holds the keys and the second
    // half the bounds of at most KT / 2 tiles
    static constexpr int RING = NST * (STAGE + RV);
    static constexpr int KT = RING + 64 * STREAM_TPW_MAX <= WAVE_LDS       ? STREAM_TPW_MAX
                              : RING + 64 * (STREAM_TPW_MAX / 2) <= WAVE_LDS ? STREAM_TPW_MAX / 2
                                                                            : STREAM_TPW_MAX / 4;
    static constexpr int KEYS = 16 * KT * 4;
    static constexpr int WAVE = RING + KEYS;   // 16 KB per wave at 128 dims
    static constexpr int TPW_MAX = UB ? KT / 2 : KT;   // tiles one wave may own
};

__device__ __forceinline__ f32x2_t swap32(float x, float y) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return f32x2_t{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ f32x2_t swap16(float x, float y) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
    return f32x2_t{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
// reduce-scatter of four per-lane partials over the four 16-lane groups:
// lane 16j + c receives the reduction over the groups of v_j at position c
__device__ __forceinline__ float group_max(float v0, float v1, float v2, float v3) {
    f32x2_t u = swap32(v0, v2), w = swap32(v1, v3);
    u = swap16(fmaxf(u[0], u[1]), fmaxf(w[0], w[1]));
    return fmaxf(u[0], u[1]);
}
__device__ __forceinline__ float group_sum(float v0, float v1, float v2, float v3) {
    f32x2_t u = swap32(v0, v2), w = swap32(v1, v3);
    u = swap16(u[0] + u[1], w[0] + w[1]);
    return u[0] + u[1];
}

// v_j = x for j == i, the others unchanged (i wave-uniform, v in registers)
__device__ __forceinline__ void put4(float& v0, float& v1, float& v2, float& v3, int i, float x) {
    v0 = (i == 0) ? x : v0;
    v1 = (i == 1) ? x : v1;
    v2 = (i == 2) ? x : v2;
    v3 = (i == 3) ? x : v3;
}

template <int HT, int KS, bool UB>
__global__ __launch_bounds__(256, 2) void score_stream_kernel(ScoreArgs a, int tpw) {
    using Gm = StreamGeom<KS, UB>;
    constexpr int N8 = Gm::N8, STAGE = Gm::STAGE, NST = Gm::NST, RUN = Gm::RUN, LPT = Gm::LPT;
    constexpr int TST = STREAM_WAVES;   // block tiles between consecutive tiles of a wave
    extern __shared__ __align__(16) uint8_t smem[];
    const int b = blockIdx.y;
    const int lane = threadIdx.x & 63, g = lane >> 4, c = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    uint8_t* wbase = smem + wave * Gm::WAVE;
    uint8_t* rvbase = wbase + NST * STAGE;                                   // [NST][64] row scalars
    float* s_key = reinterpret_cast<float*>(wbase + NST * (STAGE + Gm::RV));   // [64 q + lane]
    // (UB) [64 q + lane]: the second half of the buffer, or all of it without keys
    const bool keys = !UB || !a.no_keys;
    float* s_ub = keys ? s_key + 16 * Gm::KT / 2 : s_key;
    // block span [bs0, bs1); this wave's tile j covers rows r0 + 16 TST j + [0, 16)
    if (blockIdx.x == 0 && threadIdx.x < 64) store_head_maxima(a, b, threadIdx.x);
    const int64_t bs0 = (int64_t)blockIdx.x * STREAM_WAVES * 16 * tpw;
    if (bs0 >= a.A) return;
    const int64_t bs1 = min(a.A, bs0 + (int64_t)STREAM_WAVES * 16 * tpw);
    const int64_t nbt = (bs1 - bs0 + 15) / 16;

    // the sequence's query rows qt[b] (H x N bf16), staged once per block in
    // LDS (rows padded by 16 bytes), then read into registers by every wave;
    // head slots beyond H repeat a real head (h mod H), which leaves the
    // maximum over heads unchanged and needs no masking in the tile loop
    bf16x8_t qf[HT][KS];
    {
        constexpr int QROW = 2 * Gm::N + 16;
        static_assert(16 * HT * QROW <= STREAM_WAVES * Gm::WAVE, "query rows fit the block's LDS");
        const uint16_t* qtb = a.qt + (int64_t)b * a.H * a.n;
        for (int p = threadIdx.x; p < a.H * N8; p += 64 * STREAM_WAVES) {
            const int h = p / N8, j = p % N8;
            *reinterpret_cast<bf16x8_t*>(smem + h * QROW + 16 * j) =
                *reinterpret_cast<const bf16x8_t*>(qtb + (int64_t)h * a.n + 8 * j);
        }
        __syncthreads();
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) {
            const int h = (16 * ht + c) % a.H;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                qf[ht][ks] = *reinterpret_cast<const bf16x8_t*>(smem + h * QROW + 64 * ks + 16 * g);
        }
        __syncthreads();   // read out before the rings overwrite it
    }
    if (wave >= nbt) return;
    const int ntl = (int)((nbt - 1 - wave) / TST + 1);
    const int64_t r0 = bs0 + 16 * wave;

    // (UB) A operand of the bound step: scalar g of head slot 16 ht + c (for
    // g = 3: -s*_h or zero), and in lane 16 g + c the maximum over heads of
    // its magnitude
    float hsf[UB ? HT : 1];
    float coef = 0.f;

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
    // (UB) source of this lane's row scalar: scalar g of row c of tile 0
    const float* rvsrc = nullptr;
    if (UB) {
        const float* base = (g == 1) ? a.eps : (g == 2) ? a.gam : a.eta;
        rvsrc = base + (int64_t)b * a.T + r0 + c;
    }
    const bool ones = UB && g == 3 && a.thr;   // this lane's row scalar is the constant 1
    auto issue_rv = [&](int t, int stage, int nv) {
        if (UB) {
            const int cc = c < nv ? 0 : c - (nv - 1);
            const float* src = ones ? &k_one : rvsrc + (int64_t)t * (TST * 16) - cc;
            __builtin_amdgcn_global_load_lds((gbl_void_t*)src, (lds_void_t*)(rvbase + 256 * stage), 4, 0, 2 /* nt */);
        }
    };
    // loads of tile t into `stage`; rows past the span re-read its last row
    auto issue = [&](int t, int stage) {
        const uint8_t* tb = span + (int64_t)t * (TST * 16) * rowb;
        const int nv = (int)min((int64_t)16, bs1 - (r0 + (int64_t)(TST * 16) * t));   // rows of this tile
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            uint32_t o = voff[j];
            if (nv < 16 && vrow[j] >= nv) o -= (uint32_t)(vrow[j] - (nv - 1)) * rowb;
            __builtin_amdgcn_global_load_lds((gbl_void_t*)(tb + o), (lds_void_t*)(wbase + stage * STAGE + 1024 * j),
                                             16, 0, 2 /* nt */);
        }
        issue_rv(t, stage, nv);
    };
    // loads of a tile that lies wholly inside the span
    auto issue_full = [&](int t, int stage) {
        const uint8_t* tb = span + (int64_t)t * (TST * 16) * rowb;
#pragma unroll
        for (int j = 0; j < KS; ++j)
            __builtin_amdgcn_global_load_lds((gbl_void_t*)(tb + voff[j]),
                                             (lds_void_t*)(wbase + stage * STAGE + 1024 * j), 16, 0, 2 /* nt */);
        issue_rv(t, stage, 16);
    };
    // operand fragments (and the row scalar) of the tile in `stage`
    auto read_stage = [&](int stage, bf16x8_t (&x)[KS], float& rv) {
        const uint8_t* st = wbase + stage * STAGE;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int S = (4 * ks + g - c + 16 * N8) % N8;
            x[ks] = *reinterpret_cast<const bf16x8_t*>(st + c * (2 * Gm::N) + 16 * S);
        }
        if (UB) rv = reinterpret_cast<const float*>(rvbase + 256 * stage)[lane];
    };
    // scores of this lane's head slots for the tile whose fragments are in x
    auto contract = [&](const bf16x8_t (&x)[KS], f32x4_t (&acc)[HT]) {
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) acc[ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int ht = 0; ht < HT; ++ht)
                acc[ht] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[ht][ks], x[ks], acc[ht], 0, 0, 0);
    };
    auto head_max = [&](const f32x4_t (&acc)[HT]) {
        float pm = -INFINITY;
#pragma unroll
        for (int ht = 0; ht < HT; ++ht)
#pragma unroll
            for (int i = 0; i < 4; ++i) pm = fmaxf(pm, acc[ht][i]);
        return pm;
    };
    // (UB) the scores plus the per-head bound term of the tile's rows
    auto add_bound = [&](f32x4_t (&acc)[HT], float rv) {
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) acc[ht] = __builtin_amdgcn_mfma_f32_16x16x4f32(hsf[ht], rv, acc[ht], 0, 0, 0);
    };
    for (int t = 0; t < NST && t < ntl; ++t) issue(t, t);
    if (UB) {
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) {
            const int h = (16 * ht + c) % a.H;
            // slot g = 3: -s*_h against a row scalar of 1 (trigger margins), else 0
            const float v = g < 3 ? a.hsc[((int64_t)b * a.H + h) * 4 + g]
                                  : (a.thr ? -(float)a.thr[(int64_t)b * a.H + h] : 0.f);
            hsf[ht] = g == 0 ? scaled_a(a.cert_mult, v) : v;
            coef = fmaxf(coef, fabsf(hsf[ht]));
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) coef = fmaxf(coef, shfl_xor_local(coef, o));
    }
    wait_vmcnt<0>();   // the first tiles (and the head scalars) resident

    TileOut to{-INFINITY, INFINITY, 0.f, 0.f};
    // row of group q (tiles 4q..4q+3) held by this lane: row c of tile 4q + g
    auto group_row = [&](int q) { return r0 + (int64_t)(TST * 16) * (4 * q + g) + c; };
    auto group_out = [&](int q, float m, float s2, float u) {
        if (group_row(q) < bs1) {
            to.nu2m = fmaxf(to.nu2m, s2);
            to.kmax = fmaxf(to.kmax, m);
            to.kmin = fminf(to.kmin, m);
        }
        if (keys) s_key[64 * q + lane] = m;
        if (UB) s_ub[64 * q + lane] = u;
    };

    bf16x8_t xf[KS];
    float rvc = 0.f;
    // (UB) the largest row scalar this lane has seen (scalar g of the rows c):
    // the bound term's maximum is taken as sum_g (max over heads of scalar g of
    // the heads) x (max over rows of scalar g of the rows), no smaller than the
    // largest B_h(u) and cheaper to keep than per-row sums
    float rvmax = 0.f;
    read_stage(0, xf, rvc);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // stage read out before it is refilled
    if (NST < ntl) issue(NST, 0);

    // runs of RUN tiles whose look-ahead loads (up to tile RUN (s+1) + NST)
    // stay inside the span: fixed stages, fixed wait counts
    // (rows wider than 192 dims leave no registers for the unrolled run;
    // those shapes take the run-time loop throughout)
    const int nrun = (KS <= 6 && ntl > NST) ? (ntl - NST - 1) / RUN : 0;
    for (int s = 0; s < nrun; ++s) {
        float pmv[RUN], psv[RUN], puv[RUN];
#pragma unroll
        for (int j = 0; j < RUN; ++j) {
            f32x4_t acc[HT];
            contract(xf, acc);
            psv[j] = row_sq<KS>(xf);
            if (UB) rvmax = fmaxf(rvmax, rvc);
            __builtin_amdgcn_sched_barrier(0);
            wait_vmcnt<(NST - 1) * LPT>();
            // the next tile's fragments overwrite this tile's, whose matrix
            // steps have been issued
            float rvn = 0.f;
            read_stage((j + 1) % NST, xf, rvn);
            pmv[j] = head_max(acc);
            if (UB) {
                add_bound(acc, rvc);
                puv[j] = head_max(acc);
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // stage read out before it is refilled
            issue_full(RUN * s + j + 1 + NST, (j + 1) % NST);
            rvc = rvn;
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int j4 = 0; j4 < RUN; j4 += 4)
            group_out((RUN * s + j4) / 4, group_max(pmv[j4], pmv[j4 + 1], pmv[j4 + 2], pmv[j4 + 3]),
                      group_sum(psv[j4], psv[j4 + 1], psv[j4 + 2], psv[j4 + 3]),
                      UB ? group_max(puv[j4], puv[j4 + 1], puv[j4 + 2], puv[j4 + 3]) : 0.f);
    }

    // the remaining tiles, with run-time stages and wait counts
    float pm0 = -INFINITY, pm1 = -INFINITY, pm2 = -INFINITY, pm3 = -INFINITY;
    float ps0 = 0.f, ps1 = 0.f, ps2 = 0.f, ps3 = 0.f;
    float pu0 = -INFINITY, pu1 = -INFINITY, pu2 = -INFINITY, pu3 = -INFINITY;
    for (int t = RUN * nrun; t < ntl; ++t) {
        f32x4_t acc[HT];
        contract(xf, acc);
        const float ps = row_sq<KS>(xf);
        if (UB) rvmax = fmaxf(rvmax, rvc);
        float rvn = 0.f;
        const bool more = t + 1 < ntl;
        __builtin_amdgcn_sched_barrier(0);
        if (more) {
            wait_tiles<LPT, NST>(min(NST - 1, ntl - 2 - t));
            read_stage((t + 1) % NST, xf, rvn);   // over this tile's fragments (matrix steps issued)
        }
        const float pm = head_max(acc);
        float pu = -INFINITY;
        if (UB) {
            add_bound(acc, rvc);
            pu = head_max(acc);
        }
        const int j = t & 3;
        if (j == 0) {
            pm1 = pm2 = pm3 = -INFINITY;
            ps1 = ps2 = ps3 = 0.f;
            pu1 = pu2 = pu3 = -INFINITY;
        }
        put4(pm0, pm1, pm2, pm3, j, pm);
        put4(ps0, ps1, ps2, ps3, j, ps);
        if (UB) {
            put4(pu0, pu1, pu2, pu3, j, pu);
        }
        if (more) {
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // stage read out before it is refilled
            if (t + 1 + NST < ntl) issue(t + 1 + NST, (t + 1) % NST);
            rvc = rvn;
        }
        if (j != 3 && more) continue;
        group_out(t >> 2, group_max(pm0, pm1, pm2, pm3), group_sum(ps0, ps1, ps2, ps3),
                  UB ? group_max(pu0, pu1, pu2, pu3) : 0.f);
    }
    // the span's keys (and bounds), each lane its own LDS words
    float* kto = a.kt + (int64_t)b * a.A;
    float* kuo = a.key ? a.key + (int64_t)b * a.A : nullptr;
    float* ubo = UB ? a.ub + (int64_t)b * a.A : nullptr;
    for (int q = 0; q < (ntl + 3) / 4; ++q) {
        const int64_t row = group_row(q);
        if (row < bs1) {
            if (keys) {
                const float m = s_key[64 * q + lane];
                kto[row] = m;
                if (kuo) kuo[row] = m;
            }
            if (UB) ubo[row] = s_ub[64 * q + lane];
        }
    }
    if (UB) {
        float m = rvmax;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, shfl_xor_local(m, o));
        const float v = coef * m;   // lane 16 g + c; for g = 3: max |s*_h| x 1, or 0
        to.bmm = ((shfl_local(v, 0) + shfl_local(v, 16)) + shfl_local(v, 32)) + shfl_local(v, 48);
    }
    score_finish(a, b, lane, to, UB);
}

// tiles per wave: enough waves for two blocks per CU, spans of 8..tmax tiles
// (tmax: the tiles whose keys, or keys and bounds, the wave's LDS buffer holds)
static int stream_tpw(const ScoreArgs& a, int tmax) {
    const int64_t tiles = (int64_t)a.B * ((a.A + 15) / 16);
    const int64_t waves = 2LL * 256 * STREAM_WAVES;
    int64_t tpw = (tiles + waves - 1) / waves;
    tpw = tpw < 8 ? 8 : (tpw > tmax ? tmax : tpw);
    return (int)tpw;
}

template <int HT, int KS, bool UB>
static void launch_stream(const ScoreArgs& a, hipStream_t s) {
    // without keys the bounds take the whole key buffer (twice the tiles per wave)
    const int tpw = stream_tpw(a, (UB && a.no_keys) ? StreamGeom<KS, UB>::KT : StreamGeom<KS, UB>::TPW_MAX);
    const int64_t rows_per_block = (int64_t)STREAM_WAVES * 16 * tpw;   // block span
    dim3 grid((unsigned)((a.A + rows_per_block - 1) / rows_per_block), a.B);
    const size_t sm = STREAM_WAVES * (size_t)StreamGeom<KS, UB>::WAVE;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&score_stream_kernel<HT, KS, UB>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
    hipLaunchKernelGGL((score_stream_kernel<HT, KS, UB>), grid, dim3(256), sm, s, a, tpw);
}

template <int HT, int KS>
static void launch_fast(const ScoreArgs& a, hipStream_t s) {
    if (a.ub)
        launch_stream<HT, KS, true>(a, s);
    else
        launch_stream<HT, KS, false>(a, s);
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
